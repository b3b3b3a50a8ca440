// k_stage1_gemm.hip -- stage 1 for large batches: bf16 MFMA GEMM with the top-1 fused into its epilogue.
//
// Stage 1 of the lookup (Algorithm 1: search the cache with the query key) is
// an exact top-1 over all stored keys by the dot product of normalised
// vectors.  With hundreds to thousands of queries per call each key byte feeds
// that many multiply-adds, so the search is a dense bf16 contraction Q K^T
// that belongs on the matrix cores -- but only its row maxima are needed, so
// the B x N score matrix never leaves registers.
//
// Tiling.  A workgroup is four waves, one per SIMD, each with the whole
// register file of its SIMD (256 accumulators + 256 vector registers).  It
// owns a tile of 128 queries and walks a contiguous range of 512-key tiles;
// wave w multiplies keys w*128 .. w*128+127 of each tile against all 128
// queries, as 8 x 8 blocks of v_mfma_f32_16x16x32_bf16 (keys as the row
// operand).  The store's tiled layout makes every 1 KiB chunk (16 rows x 32
// columns) exactly one operand fragment of that instruction, so:
//   * keys go straight from memory into registers -- one coalesced 1 KiB
//     buffer load per fragment, each fragment loaded by exactly one wave,
//     three 32-column steps ahead, the 8 loads of a step spread one per 8
//     MFMAs (bursts of loads fill the memory pipeline's command queue and
//     stall the wave's MFMA issue);
//   * the 128 queries, shared by the four waves, pass through LDS: a ring of
//     four stages of 64 columns, each staged with plain loads and LDS stores
//     two steps before use, published by a barrier that waits on LDS traffic
//     only (the key loads stay in flight across it).
// Only the query operand is read from LDS (8 KiB per 64 MFMAs of a wave), so
// LDS bandwidth is far from a bound; each key byte read from L2 feeds 128
// queries.
//
// Epilogue.  After the last step of a key tile each lane holds, for each of
// its 8 queries, 4 rows of each of the 8 16-row key blocks of its wave.  Per
// query it takes the maximum of each block, the overall maximum, and the first
// block reaching it; a strictly larger maximum replaces the running best, so
// ties keep the lowest block.  The exact lowest row is recovered afterwards by
// replaying the winning 16-row group with the same instruction sequence
// (verify.hpp), which keeps this epilogue branch-free.  Rows past the entry
// count (zero padding, which must never win) occur only in the last tile of
// the last range and are masked there.  At the end each workgroup writes one
// packed candidate per query.
#include <type_traits>

#include "common.hpp"
#include "launch.hpp"

namespace lacache {

namespace {

constexpr int kWK = 4;                 // waves per workgroup, one 128-key slice each
constexpr int kKB = 8;                 // 16-row key blocks per wave
constexpr int kQB = 8;                 // 16-query blocks per wave (all waves share them)
constexpr int kTK = kWK * kKB * 16;    // keys per workgroup tile
constexpr int kTQ = kQB * 16;          // queries per workgroup tile
constexpr int kS = 2;                  // 32-column steps per LDS stage of the query tile
constexpr int kR = 4;                  // LDS stage slots
constexpr int kU = 4;                  // steps per unrolled body (a multiple of kS and kNK)
constexpr int kNK = 4;                 // key fragment sets in registers: the current step and 3 ahead
constexpr int kPD = kNK - 1;           // key prefetch distance in steps
constexpr int kSC = kS * kQB;          // 1 KiB chunks per stage
constexpr int kCPW = kSC / kWK;        // chunks each wave stages per stage
constexpr int kSlot = kSC * 1024;      // bytes per stage slot
constexpr int kRing = kR * kSlot;      // bytes of the ring
constexpr int kBest = kWK * kQB * 64 * 8;  // running best of every lane and query block (after the ring)
constexpr int kLds = kRing + kBest;
static_assert(kTK == kGemmKeyTile && kTQ == kGemmQueryTile, "tile sizes the host pads to");
static_assert(kU % kS == 0 && kU % kNK == 0 && kSC % kWK == 0, "");
static_assert((kRing & (kRing - 1)) == 0, "ring size is a power of two");

// Buffer resource over `base`: loads through it read offsets up to 2^31.
__device__ inline __amdgpu_buffer_rsrc_t make_rsrc(const void* base) {
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), 0, 0x7FFFFFFF, 0x00020000);
}

// The lane index computed afresh (not kept live across the main loop, whose registers are all in use).
__device__ inline int fresh_lane() {
    int r;
    __asm__ volatile("v_mbcnt_lo_u32_b32 %0, -1, 0\n\tv_mbcnt_hi_u32_b32 %0, -1, %0" : "=v"(r));
    return r;
}

// Workgroup barrier that orders LDS accesses only: outstanding global loads are not waited for.
__device__ inline void lds_barrier() {
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup", "local");
    __builtin_amdgcn_s_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup", "local");
}

}  // namespace

// Workgroup -> (query tile, key range): with xq > 0 the 8 XCDs (dispatch is round-robin over them) form xq
// query groups x (8 / xq) key parts; XCD x serves the query tiles of group x % xq against key part x / xq,
// so each key range is fetched into as few L2s as possible while the query tiles an XCD re-reads stay
// resident there.  Requires n_qtiles % xq == 0 and n_ranges % (8 / xq) == 0.
__global__ __launch_bounds__(kWK * 64, 1) void k_stage1_gemm(const u32x4* __restrict__ keys,
                                                             const u32x4* __restrict__ qt, int kc, int n_rows,
                                                             int n_ktiles, int n_qtiles, int n_ranges, int xq, int B,
                                                             int P, uint64_t* __restrict__ part) {
    extern __shared__ __attribute__((aligned(16))) unsigned char lds[];
    const int lane = threadIdx.x & 63;
    const int wk = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);

    int qtile, range;
    if (xq > 0) {
        const int xcd = (int)blockIdx.x % 8, j = (int)blockIdx.x / 8;
        const int qpg = n_qtiles / xq, rpp = n_ranges / (8 / xq);
        qtile = (xcd % xq) * qpg + j % qpg;
        range = (xcd / xq) * rpp + j / qpg;
    } else {
        qtile = (int)blockIdx.x % n_qtiles;
        range = (int)blockIdx.x / n_qtiles;
    }
    const int kt0 = (int)((int64_t)range * n_ktiles / n_ranges);
    const int kt1 = (int)((int64_t)(range + 1) * n_ktiles / n_ranges);
    const int T = kt1 - kt0;

    // ---- query staging: stage u holds steps (u % (kc / kS)) * kS .. + kS - 1 of the query tile; chunk
    // c = s * kQB + qb of a stage is query block qb at step s; wave wk stages chunks wk, wk + kWK, ...
    // (the lane's byte offset is the one vector offset of every buffer load; the rest is uniform and travels
    // in the scalar offset)
    const uint32_t lane16 = (uint32_t)lane * 16;
    const __amdgpu_buffer_rsrc_t qrs = make_rsrc(qt + (int64_t)qtile * kQB * kc * 64);
    auto qchunk = [&](int i) {  // byte offset of the i-th chunk this wave stages, at step 0
        const int c = wk + kWK * i;
        return ((c % kQB) * kc + c / kQB) * 1024;
    };
    u32x4 sr[kCPW];
    int ld_step = 0;   // first step of the next stage to load
    int st_base = 0;   // ring offset of the next stage to store
    auto stage_load = [&]() {
#pragma unroll
        for (int i = 0; i < kCPW; ++i)
            sr[i] = __builtin_amdgcn_raw_buffer_load_b128(qrs, lane16, qchunk(i) + ld_step * 1024, 0);
        ld_step += kS;
        if (ld_step == kc) ld_step = 0;
    };
    auto stage_store = [&]() {
        unsigned char* dst = lds + st_base + lane * 16;
#pragma unroll
        for (int i = 0; i < kCPW; ++i) *(u32x4*)(dst + (wk + kWK * i) * 1024) = sr[i];
        st_base = (st_base + kSlot) & (kRing - 1);
    };
    int rd_base = 0;   // ring offset of the stage being multiplied
    auto read_q = [&](int base, int s, u32x4 (&dst)[kQB]) {
        const unsigned char* src = lds + base + s * kQB * 1024 + lane * 16;
#pragma unroll
        for (int qb = 0; qb < kQB; ++qb) dst[qb] = *(const u32x4*)(src + qb * 1024);
    };

    // ---- keys: chunk (block kb, step j of tile t of the range) at byte ((t * kTK / 16 + kb) * kc + j) * 1024
    // from the wave's first block.  The loads run kPD steps ahead without bounds checks: the store keeps one
    // spare tile of zero rows past its last tile, so the prefetches beyond a range stay inside it.
    const __amdgpu_buffer_rsrc_t krs = make_rsrc(keys + ((int64_t)kt0 * (kTK / 16) + wk * kKB) * kc * 64);
    int kstep = 0, ksoff = 0;  // step inside its tile of the next key load, its byte offset in the range
    auto key_next = [&]() {
        ksoff += 1024;
        if (++kstep == kc) {
            kstep = 0;
            ksoff += (kTK / 16 - 1) * kc * 1024;
        }
    };
    u32x4 kf[kNK][kKB];
    auto key_load = [&](u32x4 (&dst)[kKB]) {
#pragma unroll
        for (int kb = 0; kb < kKB; ++kb)
            dst[kb] = __builtin_amdgcn_raw_buffer_load_b128(krs, lane16, ksoff + kb * kc * 1024, 0);
        key_next();
    };

    // running best of each lane per query block, packed (orderable score, ~16-row group): the unsigned
    // maximum keeps the higher score and, on equal scores, the lower group.  Kept in LDS between epilogues
    // (it changes once per key tile), which leaves the vector registers to the operand pipeline.
    auto best_slot = [&]() {  // this lane's running best of query block qb at [qb * 64]
        return (uint64_t*)(lds + kRing) + (wk * kQB) * 64 + fresh_lane();
    };
    {
        uint64_t* bp = best_slot();
#pragma unroll
        for (int q = 0; q < kQB; ++q) bp[q * 64] = 0ull;
    }
    f32x4 acc[kKB][kQB];
    u32x4 qf[2][kQB];

    if (T > 0) {
#pragma unroll
        for (int p = 0; p < kPD; ++p) key_load(kf[p]);
        stage_load();
        stage_store();
        stage_load();
        stage_store();
        stage_load();
        lds_barrier();
        read_q(0, 0, qf[0]);
    }

    auto mm = [&](int kb0, int kb1, const u32x4 (&a)[kKB], const u32x4 (&b)[kQB], bool zero) {
#pragma unroll
        for (int kb = kb0; kb < kb1; ++kb)
#pragma unroll
            for (int qb = 0; qb < kQB; ++qb) acc[kb][qb] = mfma16x16x32(a[kb], b[qb], zero ? f32x4{} : acc[kb][qb]);
    };
    // one MFMA-issue pattern: one key load, then n MFMAs, repeated for the 8 loads of a step
    auto spread_loads = [&](auto n_tag) {
        constexpr int N = decltype(n_tag)::value;
#pragma unroll
        for (int i = 0; i < kKB; ++i) {
            __builtin_amdgcn_sched_group_barrier(0x020, 1, 0);  // VMEM read
            __builtin_amdgcn_sched_group_barrier(0x008, N, 0);  // MFMA
        }
    };
    // kU steps; FIRST: the body opens a key tile, its first MFMAs start from a zero accumulator.  In the last
    // step of a stage the next stage's ring slot is published: the stage two ahead is stored, the workgroup
    // synchronises, the stage three ahead is loaded and the next stage's first fragments are read.
    auto body = [&](auto first_tag) {
        constexpr bool FIRST = decltype(first_tag)::value;
#pragma unroll
        for (int u = 0; u < kU; ++u) {
            const bool zero = FIRST && u == 0;
            if (u % kS == kS - 1) {
                key_load(kf[(u + kPD) % kNK]);
                mm(0, kKB / 2, kf[u % kNK], qf[u & 1], zero);
                spread_loads(std::integral_constant<int, kQB / 2>{});
                __builtin_amdgcn_sched_barrier(0);
                stage_store();
                lds_barrier();
                stage_load();
                rd_base = (rd_base + kSlot) & (kRing - 1);
                read_q(rd_base, 0, qf[(u + 1) & 1]);
                mm(kKB / 2, kKB, kf[u % kNK], qf[u & 1], zero);
            } else {
                key_load(kf[(u + kPD) % kNK]);
                read_q(rd_base, u % kS + 1, qf[(u + 1) & 1]);
                mm(0, kKB, kf[u % kNK], qf[u & 1], zero);
                spread_loads(std::integral_constant<int, kQB>{});
            }
            __builtin_amdgcn_sched_barrier(0);
        }
    };

    for (int t = 0; t < T; ++t) {
        body(std::true_type{});
        for (int j = kU; j < kc; j += kU) body(std::false_type{});
        // epilogue of tile kt0 + t: lane holds rows 4 * (lane / 16) + i of block kb for query lane % 16 of
        // block qb
        const int tg = kt0 + t;
        const int grp0 = tg * (kTK / 16) + wk * kKB;
        const int vw = n_rows - (tg * kTK + wk * kKB * 16);  // valid rows of the wave's slice (uniform)
        auto epi = [&](auto masked_tag) {
            constexpr bool MASKED = decltype(masked_tag)::value;
            const int valid = vw - 4 * (fresh_lane() >> 4);
            uint64_t* bp = best_slot();
#pragma unroll
            for (int qb = 0; qb < kQB; ++qb) {
                float mk[kKB];
#pragma unroll
                for (int kb = 0; kb < kKB; ++kb) {
                    float a[4];
#pragma unroll
                    for (int i = 0; i < 4; ++i)
                        a[i] = (!MASKED || kb * 16 + i < valid) ? acc[kb][qb][i] : -__builtin_inff();
                    mk[kb] = fmaxf(fmaxf(a[0], a[1]), fmaxf(a[2], a[3]));
                }
                float m = mk[0];
#pragma unroll
                for (int kb = 1; kb < kKB; ++kb) m = fmaxf(m, mk[kb]);
                int gk = kKB - 1;
#pragma unroll
                for (int kb = kKB - 2; kb >= 0; --kb) gk = (mk[kb] == m) ? kb : gk;
                // m = -inf only for a fully masked slice: no candidate
                if (m != -__builtin_inff()) bp[qb * 64] = umax64(bp[qb * 64], pack_top1(m, grp0 + gk));
                __builtin_amdgcn_sched_barrier(0);
            }
        };
        if (vw >= kKB * 16)
            epi(std::false_type{});
        else
            epi(std::true_type{});
    }
    __syncthreads();
    const int ln = fresh_lane();
    const uint64_t* bp = best_slot();

    // merge the four lanes of each query (lanes l, l^16, l^32, l^48), then the four waves, and write one
    // candidate per query
    uint64_t* red = (uint64_t*)lds;  // [kWK][kTQ]; the ring is no longer read
#pragma unroll
    for (int qb = 0; qb < kQB; ++qb) {
        uint64_t p = bp[qb * 64];
        p = umax64(p, (uint64_t)__shfl_xor((unsigned long long)p, 16, kWave));
        p = umax64(p, (uint64_t)__shfl_xor((unsigned long long)p, 32, kWave));
        if (ln < 16) red[wk * kTQ + qb * 16 + ln] = p;
    }
    __syncthreads();
    for (int q = wk * 64 + ln; q < kTQ; q += kWK * 64) {
        uint64_t m = 0;
#pragma unroll
        for (int w = 0; w < kWK; ++w) m = umax64(m, red[w * kTQ + q]);
        const int gq = qtile * kTQ + q;
        if (gq < B) part[(int64_t)gq * P + range] = m;
    }
}

hipError_t launch_stage1_gemm(const uint16_t* keys, const uint16_t* qt, int B, int n_rows, int d_pad, uint64_t* part,
                              int num_cu, int* P_out, hipStream_t s, hipEvent_t e0, hipEvent_t e1) {
    const int kc = d_pad / 32;
    if (n_rows <= 0 || B <= 0 || kc % kU != 0) return hipErrorInvalidValue;
    const int n_qtiles = (B + kTQ - 1) / kTQ;
    const int n_ktiles = (n_rows + kTK - 1) / kTK;
    // one workgroup per CU (each wave holds a SIMD's whole register file): as many key ranges per query tile
    // as fill the CUs once
    int n_ranges = (num_cu + n_qtiles - 1) / n_qtiles;
    if (n_ranges > n_ktiles) n_ranges = n_ktiles;
    if (n_ranges > kMaxPartials) n_ranges = kMaxPartials;
    // the key offsets of a range stay below 2^31 bytes (its tiles plus the prefetch overrun)
    const int64_t tile_bytes = (int64_t)kTK * d_pad * 2;
    const int64_t max_tiles = ((int64_t(1) << 31) - 1) / tile_bytes - 1;
    if (max_tiles < 1) return hipErrorInvalidValue;
    if ((n_ktiles + n_ranges - 1) / n_ranges > max_tiles) n_ranges = (int)((n_ktiles + max_tiles - 1) / max_tiles);
    if (n_ranges > kMaxPartials) return hipErrorInvalidValue;
    *P_out = n_ranges;
    // XCD placement: the fewest query groups (1, 2, 4 or 8) whose query tiles fit one XCD's L2 beside the key
    // stream, at most 3 MiB per XCD; plain round-robin when the counts do not divide evenly
    int xq = 0;
    for (int x = 1; x <= 8; x *= 2) {
        if (n_qtiles % x != 0 || n_ranges % (8 / x) != 0) continue;
        if ((int64_t)(n_qtiles / x) * kTQ * d_pad * 2 <= (int64_t(3) << 20)) {
            xq = x;
            break;
        }
    }
    static std::atomic<uint64_t> lds_done{0};
    hipError_t e = allow_dynamic_lds((const void*)k_stage1_gemm, kLds, lds_done);
    if (e != hipSuccess) return e;
    return launch_timed(k_stage1_gemm, dim3(n_qtiles * n_ranges), dim3(kWK * 64), kLds, s, e0, e1, (const u32x4*)keys,
                        (const u32x4*)qt, kc, n_rows, n_ktiles, n_qtiles, n_ranges, xq, B, n_ranges, part);
}

}  // namespace lacache
