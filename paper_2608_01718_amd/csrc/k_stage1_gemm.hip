// k_stage1_gemm.hip -- stage 1 for large batches: bf16 MFMA GEMM with the top-1 fused into its epilogue.
//
// Stage 1 of the lookup (Algorithm 1: search the cache with the query key) is
// an exact top-1 over all stored keys by the dot product of normalised
// vectors.  With hundreds to thousands of queries per call each key byte feeds
// that many multiply-adds, so the search is a dense bf16 contraction Q K^T
// that belongs on the matrix cores -- but only its row maxima are needed, so
// the B x N score matrix never leaves registers.
//
// Tiling: a workgroup of 8 waves owns a tile of 256 queries and walks a
// contiguous range of 256-key tiles.  Each key tile is consumed in stages of
// kBK columns of d: a stage (256 x kBK keys + 256 x kBK queries, 1 KiB chunks
// of the tiled store layout) is copied by buffer loads straight into one of
// two LDS buffers (no staging registers), one stage ahead of the one being
// multiplied.  Waves are arranged 2 (key halves of 128) x 4 (query quarters
// of 64), two per SIMD; a wave multiplies its 128 x 64 block with
// v_mfma_f32_32x32x16_bf16, keys as the row operand, so a lane's 16
// accumulators per fragment are 16 keys of one query.  Within a stage the
// MFMAs of one 16-column substep run while the next substep's fragments are
// read; the workgroup synchronises before the last substep's MFMAs, so the
// copy of the stage after next and the first fragment reads of the next stage
// are issued under matrix-core work rather than behind a drained pipeline.
// The first MFMAs of a key tile start from a zero accumulator.  After the last
// stage of a key tile each lane takes, per query, the maximum of each of its
// four 32-row groups and keeps a running (best score, 32-row group); only a
// strictly larger score replaces the best and the lowest group wins within a
// tile, so ties keep the lowest group.  The exact lowest row is recovered
// afterwards by replaying the winning group (verify.hpp), which keeps this
// epilogue branch-free.  The one partial key tile (rows beyond the entry
// count are zero padding and must not win) is handled by separate, masked
// workgroups of the same launch, dispatched first so that they overlap the
// full tiles (a masked epilogue inside the main loop measured 3 % slower: it
// adds scalar-register pressure to every stage).  At the end each workgroup
// writes one packed candidate per query.
#include <type_traits>

#include "common.hpp"
#include "launch.hpp"

namespace lacache {

namespace {

constexpr int kTile = 256;                           // queries and keys per workgroup tile
constexpr int kWaves = 8;                            // 2 key halves x 4 query quarters
constexpr int QF = 2;                                // 32-query MFMA fragments per wave
constexpr int kBK = 64;                              // columns of d per LDS stage (32 measured slower)
constexpr int kNBuf = 2;                             // LDS stage buffers
constexpr int kBlk = kBK / 32;                       // 32-column blocks of the tiled layout per stage
constexpr int kSub = kBK / 16;                       // MFMA k-steps (16 columns) per stage
constexpr int kChunks = 16 * kBlk;                   // 1 KiB chunks per operand per stage
constexpr int kStageBytes = 2 * kChunks * 1024;      // keys + queries
constexpr int kPerWave = kChunks / kWaves;           // chunks of each operand a wave copies per stage
static_assert(kNBuf * kStageBytes <= 160 * 1024, "two LDS stage buffers");

// byte offset, inside one operand's stage, of the 32x32x16 fragment read by lane l:
// rows [row0, row0 + 32), columns 16 s .. 16 s + 15 of the stage (chunk j of a stage = 16-row group
// j / kBlk, 32-column block j % kBlk)
__device__ inline int frag_offset(int row0, int s, int lane) {
    const int g = (row0 >> 4) + ((lane & 31) >> 4);  // 16-row group inside the 256-row tile
    const int c = ((s & 1) << 1) + (lane >> 5);      // 8-column chunk inside the 32-column block
    return ((g * kBlk + (s >> 1)) * 64 + c * 16 + (lane & 15)) * 16;
}

// Buffer resource over `bytes` bytes at `base`: loads through it outside [0, bytes) return zeros
// instead of touching memory.
__device__ inline __amdgpu_buffer_rsrc_t make_rsrc(const void* base, uint32_t bytes) {
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), 0, (int)bytes, 0x00020000);
}

// 16 bytes per lane from buffer offset soff + voff straight into LDS: lane l writes lds_wave_base + 16 l.
__device__ inline void buffer_to_lds16(__amdgpu_buffer_rsrc_t r, uint32_t voff, uint32_t soff,
                                       unsigned char* lds_wave_base) {
    __builtin_amdgcn_raw_ptr_buffer_load_lds(r, (__attribute__((address_space(3))) void*)lds_wave_base, 16, voff,
                                             soff, 0, 0);
}

}  // namespace

// One workgroup's work: query tile qtile against key tiles [kt0, kt1), its candidates written to partial
// slot `slot` (P is the partial stride of a query).  MASKED = false: every tile is full.  MASKED = true: the
// single partial tile (rows beyond n_rows are zero padding and must not win).
template <bool MASKED>
__device__ __forceinline__ void gemm_tiles(const u32x4* __restrict__ keys, const u32x4* __restrict__ qt, int kc,
                                           int n_rows, int B, int qtile, int kt0, int kt1, int slot, int P,
                                           uint64_t* __restrict__ part) {
    extern __shared__ __attribute__((aligned(16))) unsigned char lds[];
    const int tid = threadIdx.x, lane = tid & 63;
    const int wid = __builtin_amdgcn_readfirstlane(tid >> 6);  // wave-uniform, kept in scalar registers
    const int wk = wid & 1, wq = wid >> 1;                     // key half (128 keys), query quarter (64)
    const int spt = kc / kBlk;                // stages per key tile
    const int T = (kt1 - kt0) * spt;          // stages of the whole range

    // running best of each lane per 32-query fragment b: the score, and the 32-row group (global row / 32)
    // holding it -- the exact row is recovered later by replaying that group (verify.hpp)
    float best[QF];
    int bgrp[QF];
#pragma unroll
    for (int q = 0; q < QF; ++q) {
        best[q] = -__builtin_inff();
        bgrp[q] = 0x7FFFFFFF;
    }

    // copies: stage u covers columns kBK (u % spt) .. of key tile kt0 + u / spt and goes to LDS buffer u % 2.
    // Wave w copies chunks j = w, w + 8, ... of both operands; the buffer offset of chunk j in stage column
    // block i_st is jb[p] + i_st * kBlk * 1024.
    const uint32_t tile_bytes = (uint32_t)kTile * kc * 64;
    const __amdgpu_buffer_rsrc_t qr = make_rsrc(qt + (int64_t)qtile * 16 * kc * 64, tile_bytes);
    const uint32_t voff = (uint32_t)lane * 16;
    uint32_t jb[kPerWave];
#pragma unroll
    for (int p = 0; p < kPerWave; ++p) {
        const int j = p * kWaves + wid;
        jb[p] = (uint32_t)(((j / kBlk) * kc + (j % kBlk)) * 1024);
    }
    const u32x4* kbase = keys + (int64_t)kt0 * 16 * kc * 64;  // key tile of the next copy
    int i_st = 0, i_buf = 0;
    auto issue = [&]() {
        const __amdgpu_buffer_rsrc_t kr = make_rsrc(kbase, tile_bytes);
        unsigned char* dk = lds + i_buf * kStageBytes;
        unsigned char* dq = dk + kChunks * 1024;
        const uint32_t so = (uint32_t)i_st * (kBlk * 1024);
#pragma unroll
        for (int p = 0; p < kPerWave; ++p) {
            const int j = p * kWaves + wid;
            buffer_to_lds16(kr, voff, jb[p] + so, dk + j * 1024);
            buffer_to_lds16(qr, voff, jb[p] + so, dq + j * 1024);
        }
        i_buf ^= 1;
        if (++i_st == spt) {
            i_st = 0;
            kbase += 16 * kc * 64;
        }
    };
    // fragments of substep s of the stage in LDS buffer `buf`
    auto read_frags = [&](int buf, int s, u32x4* fa, u32x4* fb) {
        const unsigned char* sk = lds + buf * kStageBytes;
        const unsigned char* sq = sk + kChunks * 1024;
#pragma unroll
        for (int i = 0; i < 4; ++i) fa[i] = *(const u32x4*)(sk + frag_offset(wk * 128 + i * 32, s, lane));
#pragma unroll
        for (int i = 0; i < QF; ++i) fb[i] = *(const u32x4*)(sq + frag_offset(wq * 64 + i * 32, s, lane));
    };

    f32x16 acc[4][QF];
    u32x4 fa[kSub][4], fb[kSub][QF];
    int kt = kt0, st = 0;

    // Stage t (buffer t % 2), fragments of its substep 0 already in fa[0] / fb[0].  Substeps 0 .. kSub-2 are
    // multiplied while the fragments of the next substep are read; then the workgroup synchronises (stage
    // t + 1 has landed, every wave is done reading buffer t % 2), the copy of stage t + 2 into buffer t % 2
    // and the reads of stage t + 1's first fragments are issued, and the last substep's MFMAs run over
    // their latency.  FIRST: stage t opens a key tile, its first MFMAs start from a zero accumulator.
    auto step = [&](int t, auto first_tag) {
        constexpr bool FIRST = decltype(first_tag)::value;
        const int buf = t & 1;
#pragma unroll
        for (int s = 0; s + 1 < kSub; ++s) {
            read_frags(buf, s + 1, fa[s + 1], fb[s + 1]);
#pragma unroll
            for (int a = 0; a < 4; ++a)
#pragma unroll
                for (int b = 0; b < QF; ++b)
                    acc[a][b] = mfma32x32x16(fa[s][a], fb[s][b], (FIRST && s == 0) ? f32x16{} : acc[a][b]);
            constexpr int kReads = 4 + QF, kMfma = 4 * QF;
#pragma unroll
            for (int i = 0; i < kReads; ++i) {
                __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);  // MFMA
                __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);  // DS read
            }
            __builtin_amdgcn_sched_group_barrier(0x008, kMfma - kReads, 0);
        }
        // every fragment read of buffer t % 2 has returned before any wave may overwrite that buffer
        __builtin_amdgcn_s_waitcnt(0xC07F);  // lgkmcnt(0)
        __syncthreads();
        if (t + 2 < T) issue();
        u32x4 na[4], nb[QF];
        if (t + 1 < T) read_frags(buf ^ 1, 0, na, nb);
        constexpr int L = kSub - 1;
#pragma unroll
        for (int a = 0; a < 4; ++a)
#pragma unroll
            for (int b = 0; b < QF; ++b)
                acc[a][b] = mfma32x32x16(fa[L][a], fb[L][b], (FIRST && L == 0) ? f32x16{} : acc[a][b]);
#pragma unroll
        for (int i = 0; i < 4; ++i) fa[0][i] = na[i];
#pragma unroll
        for (int i = 0; i < QF; ++i) fb[0][i] = nb[i];

        if (++st == spt) {
            // end of key tile kt: lane holds, for query column wq*64 + b*32 + lane%32, the keys
            // kt*256 + wk*128 + a*32 + 8*(r/4) + 4*(lane/32) + r%4 (a = 0..3, r = 0..15).  Per 32-row group a
            // take the maximum; the first group reaching the overall maximum is the lowest-index candidate.
            const int grp0 = (kt * kTile + wk * 128) >> 5;
            const int valid = n_rows - (kt * kTile + wk * 128 + 4 * (lane >> 5));
#pragma unroll
            for (int b = 0; b < QF; ++b) {
                float ma[4];
#pragma unroll
                for (int a = 0; a < 4; ++a) {
                    float m = -__builtin_inff();
#pragma unroll
                    for (int r = 0; r < 16; ++r) {
                        const int off = a * 32 + 8 * (r >> 2) + (r & 3);
                        m = fmaxf(m, (!MASKED || off < valid) ? acc[a][b][r] : -__builtin_inff());
                    }
                    ma[a] = m;
                }
                const float m = fmaxf(fmaxf(ma[0], ma[1]), fmaxf(ma[2], ma[3]));
                const int ga = ma[0] == m ? 0 : ma[1] == m ? 1 : ma[2] == m ? 2 : 3;
                if (m > best[b]) {
                    best[b] = m;
                    bgrp[b] = grp0 + ga;
                }
            }
            st = 0;
            ++kt;
        }
    };

    if (T > 0) {
        issue();
        __syncthreads();
        if (T > 1) issue();
        read_frags(0, 0, fa[0], fb[0]);
    }
    for (int t = 0; t < T; ++t) {
        if (st == 0)
            step(t, std::true_type{});
        else
            step(t, std::false_type{});
    }
    __syncthreads();

    // merge lanes l and l^32 (same query), then the two key-half waves, and write one candidate per query
    uint64_t* red = (uint64_t*)lds;  // [2 key halves][256 queries]; the stage buffers are no longer read
#pragma unroll
    for (int b = 0; b < QF; ++b) {
        uint64_t p = (bgrp[b] == 0x7FFFFFFF) ? 0ull : pack_top1(best[b], bgrp[b]);
        p = umax64(p, (uint64_t)__shfl_xor((unsigned long long)p, 32, kWave));
        if (lane < 32) red[wk * kTile + wq * 64 + b * 32 + lane] = p;
    }
    __syncthreads();
    if (tid < kTile) {
        const uint64_t m = umax64(red[tid], red[kTile + tid]);
        const int gq = qtile * kTile + tid;
        if (gq < B) part[(int64_t)gq * P + slot] = m;
    }
}

// The partial key tile n_ktiles for query tile qtile, into partial slot P - 1.  Kept out of line: its masked
// epilogue needs more scalar registers than the hardware has (the spills stay in this function), and inlined
// into the kernel it would take the full tiles' loop down with it.
__device__ __attribute__((noinline)) void gemm_tail(const u32x4* __restrict__ keys, const u32x4* __restrict__ qt,
                                                    int kc, int n_rows, int B, int qtile, int n_ktiles, int P,
                                                    uint64_t* __restrict__ part) {
    gemm_tiles<true>(keys, qt, kc, n_rows, B, qtile, n_ktiles, n_ktiles + 1, P - 1, P, part);
}

// The first tail_blocks workgroups (n_qtiles of them, padded to a multiple of 8 so that the others keep their
// XCD) take the single partial key tile n_ktiles, one query tile each, into partial slot P - 1; they are
// dispatched first and overlap the full tiles.  The other workgroups split the full key tiles [0, n_ktiles)
// into n_ranges contiguous ranges, range r into partial slot r.  xq selects the XCD placement of those
// (below); it requires n_qtiles % xq == 0 and n_ranges % (8 / xq) == 0.
__global__ __launch_bounds__(512, 1) void k_stage1_gemm(const u32x4* __restrict__ keys, const u32x4* __restrict__ qt,
                                                        int kc, int n_rows, int B, int n_qtiles, int n_ktiles,
                                                        int n_ranges, int tail_blocks, int P, int xq,
                                                        uint64_t* __restrict__ part) {
    if ((int)blockIdx.x < tail_blocks) {
        if ((int)blockIdx.x < n_qtiles) gemm_tail(keys, qt, kc, n_rows, B, blockIdx.x, n_ktiles, P, part);
        return;
    }
    const int bid = (int)blockIdx.x - tail_blocks;
    // workgroup -> (query tile, key range).  Dispatch is round-robin over the 8 XCDs (one L2 each).  With
    // xq > 0 the XCDs form xq query groups x (8 / xq) key parts: XCD x serves the query tiles of group
    // x % xq (small enough to stay in its L2) against key part x / xq, and consecutive workgroups of an XCD
    // take consecutive query tiles of one key range, so that range's keys come into that L2 once.
    int qtile, range;
    if (xq > 0) {
        const int xcd = bid % 8, j = bid / 8;
        const int qpg = n_qtiles / xq, rpp = n_ranges / (8 / xq);
        qtile = (xcd % xq) * qpg + j % qpg;
        range = (xcd / xq) * rpp + j / qpg;
    } else {
        qtile = bid % n_qtiles;
        range = bid / n_qtiles;
    }
    const int kt0 = (int)((int64_t)range * n_ktiles / n_ranges);
    const int kt1 = (int)((int64_t)(range + 1) * n_ktiles / n_ranges);
    gemm_tiles<false>(keys, qt, kc, n_rows, B, qtile, kt0, kt1, range, P, part);
}

hipError_t launch_stage1_gemm(const uint16_t* keys, const uint16_t* qt, int B, int n_rows, int d_pad, uint64_t* part,
                              int num_cu, int* P_out, hipStream_t s) {
    const int kc = d_pad / 32;
    if (n_rows <= 0 || B <= 0) return hipErrorInvalidValue;
    const int n_qtiles = (B + kTile - 1) / kTile;
    const int n_full = n_rows / kTile;      // key tiles without padded rows
    const bool tail = n_rows % kTile != 0;  // one more, partial, tile
    // enough workgroups to fill every CU a few times over, each with a run of key tiles
    int n_ranges = (4 * num_cu + n_qtiles - 1) / n_qtiles;
    if (n_ranges > n_full) n_ranges = n_full;
    if (n_ranges > kMaxPartials - 1) n_ranges = kMaxPartials - 1;
    const int P = n_ranges + (tail ? 1 : 0);
    *P_out = P;
    // XCD placement: the fewest query groups (1, 2, 4 or 8) whose query tiles fit one XCD's L2 beside the key
    // stream, at most 3 MiB per XCD, so that each key range is fetched by as few XCDs as possible (measured:
    // 4096 x 768 queries run best as 2 groups of 3 MiB, 1024 x 1024 as 1 group of 2 MiB, 3 % faster than 2);
    // plain round-robin when the tile counts do not divide evenly
    const int grid = n_qtiles * n_ranges;
    int xq = 0;
    for (int x = 1; x <= 8; x *= 2) {
        if (n_qtiles % x != 0 || n_ranges % (8 / x) != 0) continue;
        if ((int64_t)(n_qtiles / x) * kTile * d_pad * 2 <= (int64_t(3) << 20)) {
            xq = x;
            break;
        }
    }
    const size_t lds = (size_t)kNBuf * kStageBytes;
    static std::atomic<uint64_t> lds_done{0};
    hipError_t e = allow_dynamic_lds((const void*)k_stage1_gemm, (int)lds, lds_done);
    if (e != hipSuccess) return e;
    // the partial tile's workgroups first (a separate launch after the full tiles measured 23 us on its own)
    const int tail_blocks = tail ? (n_qtiles + 7) / 8 * 8 : 0;
    k_stage1_gemm<<<dim3(tail_blocks + grid), dim3(kWaves * 64), lds, s>>>(
        (const u32x4*)keys, (const u32x4*)qt, kc, n_rows, B, n_qtiles, n_full, n_ranges, tail_blocks, P, xq, part);
    return hipGetLastError();
}

}  // namespace lacache
