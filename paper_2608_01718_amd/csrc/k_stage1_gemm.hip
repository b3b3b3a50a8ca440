// k_stage1_gemm.hip -- stage 1 for large batches: bf16 MFMA GEMM with the top-1 fused into its epilogue.
//
// Stage 1 of the lookup (Algorithm 1: search the cache with the query key) is
// an exact top-1 over all stored keys by the dot product of normalised
// vectors.  With hundreds to thousands of queries per call each key byte feeds
// that many multiply-adds, so the search is a dense bf16 contraction Q K^T
// that belongs on the matrix cores -- but only its row maxima are needed, so
// the B x N score matrix never leaves registers.
//
// Tiling: a workgroup (4 waves, 2 x 2) owns a tile of 256 queries and walks a
// contiguous range of 256-key tiles.  For each key tile it streams d in steps
// of 64 through double-buffered LDS (keys and queries arrive as 1 KiB chunks of
// the tiled layout, one coalesced wave access each); every wave computes a
// 128-key x 128-query block with v_mfma_f32_32x32x16_bf16 (keys are the row
// operand, so a lane's 16 accumulators are 16 keys of one query).  At the end
// of a key tile each lane reduces its 64 keys per query in registers and
// updates a running (best score, index); a scan for the index runs only when
// some lane improved.  Key rows are visited in increasing order and only a
// strictly larger score replaces the best, so ties keep the lowest index.
// Rows past the stored entry count are masked in the last tile.  At the end
// the workgroup writes one packed candidate per query for its key range.
#include "common.hpp"
#include "launch.hpp"

namespace lacache {

namespace {

constexpr int kTile = 256;     // queries and keys per workgroup tile
constexpr int kChunks = 32;    // 1 KiB chunks per operand per stage: (256 / 16 rows) x (64 / 32 cols)
constexpr int kStageBytes = 2 * kChunks * 1024;  // keys + queries
constexpr int kWaves = 8;      // 2 key halves x 4 query quarters
constexpr int QF = 2;          // 32-query MFMA fragments per wave

// byte offset in an operand's LDS stage of the 32x32x16 fragment for lane l:
// rows [row0, row0 + 32), the 16 columns of substep s (0..3) of the 64-column stage
__device__ inline int frag_offset(int row0, int s, int lane) {
    const int g = (row0 >> 4) + ((lane & 31) >> 4);  // 16-row group inside the 256-row tile
    const int c = ((s & 1) << 1) + (lane >> 5);      // 8-column chunk inside the 32-column block
    return ((g * 2 + (s >> 1)) * 64 + c * 16 + (lane & 15)) * 16;
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

__device__ inline void wait_vm_all() { asm volatile("s_waitcnt vmcnt(0)" ::: "memory"); }

}  // namespace

// MASKED = false: key tiles [0, n_ktiles) are all full; they are split into n_ranges contiguous ranges and
// range r writes partial slot r.  MASKED = true: the single partial tile n_ktiles (rows n_ktiles*256 ..
// n_rows-1), written to partial slot `slot`.  P is the partial stride of a query.
template <bool MASKED>
__global__ __launch_bounds__(512, 1) void k_stage1_gemm(const u32x4* __restrict__ keys, const u32x4* __restrict__ qt,
                                                        int kc, int n_rows, int B, int n_qtiles, int n_ktiles,
                                                        int n_ranges, int slot, int P, uint64_t* __restrict__ part) {
    extern __shared__ __attribute__((aligned(16))) unsigned char lds[];
    const int tid = threadIdx.x, lane = tid & 63;
    const int wid = __builtin_amdgcn_readfirstlane(tid >> 6);  // wave-uniform, kept in scalar registers
    const int wk = wid & 1, wq = wid >> 1;  // key half (128 keys), query quarter (64 queries)

    // workgroup -> (query tile, key range); consecutive workgroups take consecutive query tiles of one key
    // range, so the key tiles they share are fetched from HBM once and then served by L2.
    const int wg = blockIdx.x;
    const int qtile = wg % n_qtiles;
    const int range = wg / n_qtiles;
    const int kt0 = MASKED ? n_ktiles : (int)((int64_t)range * n_ktiles / n_ranges);
    const int kt1 = MASKED ? n_ktiles + 1 : (int)((int64_t)(range + 1) * n_ktiles / n_ranges);
    const int ksteps = kc / 2;  // 64-column stages per key tile

    float best[QF];
    int bidx[QF];
#pragma unroll
    for (int q = 0; q < QF; ++q) {
        best[q] = -__builtin_inff();
        bidx[q] = 0x7FFFFFFF;
    }

    f32x16 acc[4][QF];

    // global -> LDS without registers: each wave copies whole 1 KiB chunks (lane l moves bytes 16l..16l+15)
    // global -> LDS without registers: wave w copies chunks w, w+4, ..., lane l moving bytes 16l .. 16l+15
    const uint32_t tile_bytes = (uint32_t)kTile * kc * 64;  // one 256-row tile of the tiled layout
    const __amdgpu_buffer_rsrc_t qr = make_rsrc(qt + (int64_t)qtile * 16 * kc * 64, tile_bytes);
    const uint32_t voff = (uint32_t)lane * 16;
    auto load_stage = [&](int kt, int st, int buf) {
        const __amdgpu_buffer_rsrc_t kr = make_rsrc(keys + (int64_t)kt * 16 * kc * 64, tile_bytes);
        unsigned char* dk = lds + buf * kStageBytes;
        unsigned char* dq = dk + kChunks * 1024;
#pragma unroll
        for (int p = 0; p < kChunks / kWaves; ++p) {
            const int j = p * kWaves + wid;  // chunk 0..31 of the stage
            const uint32_t soff = (uint32_t)(((j >> 1) * kc + st * 2 + (j & 1)) * 1024);
            buffer_to_lds16(kr, voff, soff, dk + j * 1024);
            buffer_to_lds16(qr, voff, soff, dq + j * 1024);
        }
    };

    // one flat loop over (key tile, 64-column stage); the next stage streams into the other buffer
    const int T = (kt1 - kt0) * ksteps;
    if (T > 0) load_stage(kt0, 0, 0);
    wait_vm_all();
    __syncthreads();
#pragma unroll
    for (int a = 0; a < 4; ++a)
#pragma unroll
        for (int b = 0; b < QF; ++b) acc[a][b] = f32x16{};

    int kt = kt0, st = 0, buf = 0;
    for (int t = 0; t < T; ++t) {
        if (t + 1 < T) {
            // buffer buf^1 was last read before the barrier that ended the previous stage
            if (st + 1 < ksteps)
                load_stage(kt, st + 1, buf ^ 1);
            else
                load_stage(kt + 1, 0, buf ^ 1);
        }
        const unsigned char* sk = lds + buf * kStageBytes;
        const unsigned char* sq = sk + kChunks * 1024;
        // fragments of substep s+1 are read from LDS while the 16 MFMAs of substep s run
        u32x4 fa[2][4], fb[2][QF];
#pragma unroll
        for (int i = 0; i < 4; ++i) fa[0][i] = *(const u32x4*)(sk + frag_offset(wk * 128 + i * 32, 0, lane));
#pragma unroll
        for (int i = 0; i < QF; ++i) fb[0][i] = *(const u32x4*)(sq + frag_offset(wq * 32 * QF + i * 32, 0, lane));
#pragma unroll
        for (int s = 0; s < 4; ++s) {
            const int cur = s & 1;
            if (s < 3) {
#pragma unroll
                for (int i = 0; i < 4; ++i)
                    fa[cur ^ 1][i] = *(const u32x4*)(sk + frag_offset(wk * 128 + i * 32, s + 1, lane));
#pragma unroll
                for (int i = 0; i < QF; ++i)
                    fb[cur ^ 1][i] = *(const u32x4*)(sq + frag_offset(wq * 32 * QF + i * 32, s + 1, lane));
            }
#pragma unroll
            for (int a = 0; a < 4; ++a)
#pragma unroll
                for (int b = 0; b < QF; ++b) acc[a][b] = mfma32x32x16(fa[cur][a], fb[cur][b], acc[a][b]);
            __builtin_amdgcn_sched_barrier(0);
        }
        wait_vm_all();
        __syncthreads();
        buf ^= 1;

        if (++st == ksteps) {
            // epilogue of key tile kt: lane holds, for query column wq*64 + b*32 + lane%32, the keys
            // kt*256 + wk*128 + a*32 + 8*(r/4) + 4*(lane/32) + r%4, a = 0..3, r = 0..15 (increasing in (a, r))
            const int rowbase = kt * kTile + wk * 128 + 4 * (lane >> 5);
            const int valid = n_rows - rowbase;  // row rowbase + off is a stored entry iff off < valid
#pragma unroll
            for (int b = 0; b < QF; ++b) {
                float m = -__builtin_inff();
#pragma unroll
                for (int a = 0; a < 4; ++a)
#pragma unroll
                    for (int r = 0; r < 16; ++r) {
                        const int off = a * 32 + 8 * (r >> 2) + (r & 3);
                        m = fmaxf(m, (!MASKED || off < valid) ? acc[a][b][r] : -__builtin_inff());
                    }
                const bool up = m > best[b];
                if (__ballot(up) != 0ull) {
                    int found = 0;
#pragma unroll
                    for (int a = 3; a >= 0; --a)
#pragma unroll
                        for (int r = 15; r >= 0; --r) {
                            const int off = a * 32 + 8 * (r >> 2) + (r & 3);
                            if ((!MASKED || off < valid) && acc[a][b][r] == m) found = off;
                        }
                    if (up) {
                        best[b] = m;
                        bidx[b] = rowbase + found;
                    }
                }
                __builtin_amdgcn_sched_barrier(0);
            }
#pragma unroll
            for (int a = 0; a < 4; ++a)
#pragma unroll
                for (int b = 0; b < QF; ++b) acc[a][b] = f32x16{};
            st = 0;
            ++kt;
        }
    }

    // merge lanes l and l^32 (same query), then the two key-half waves, and write one candidate per query
    uint64_t* red = (uint64_t*)lds;  // [2 key halves][256 queries]; the LDS stages are no longer read
#pragma unroll
    for (int b = 0; b < QF; ++b) {
        uint64_t p = (bidx[b] == 0x7FFFFFFF) ? 0ull : pack_top1(best[b], bidx[b]);
        p = umax64(p, (uint64_t)__shfl_xor((unsigned long long)p, 32, kWave));
        if (lane < 32) red[wk * kTile + wq * 32 * QF + b * 32 + lane] = p;
    }
    __syncthreads();
    if (tid < kTile) {
        const int q = tid;  // 0..255
        const uint64_t m = umax64(red[q], red[kTile + q]);
        const int gq = qtile * kTile + q;
        if (gq < B) part[(int64_t)gq * P + (MASKED ? slot : range)] = m;
    }
}

hipError_t launch_stage1_gemm(const uint16_t* keys, const uint16_t* qt, int B, int n_rows, int d_pad, uint64_t* part,
                              int num_cu, int* P_out, hipStream_t s) {
    const int kc = d_pad / 32;
    if (kc % 2 != 0 || n_rows <= 0 || B <= 0) return hipErrorInvalidValue;
    const int n_qtiles = (B + kTile - 1) / kTile;
    const int n_full = n_rows / kTile;              // key tiles without padded rows
    const bool tail = n_rows % kTile != 0;          // one more, partial, tile
    // enough workgroups to fill every CU a few times over, each with a run of key tiles
    int n_ranges = (4 * num_cu + n_qtiles - 1) / n_qtiles;
    if (n_ranges > n_full) n_ranges = n_full;
    if (n_ranges > kMaxPartials - 1) n_ranges = kMaxPartials - 1;
    const int P = n_ranges + (tail ? 1 : 0);
    *P_out = P;
    const size_t lds = 2 * (size_t)kStageBytes;
    static bool attr = false;
    if (!attr) {
        (void)hipFuncSetAttribute((const void*)k_stage1_gemm<false>, hipFuncAttributeMaxDynamicSharedMemorySize,
                                  (int)lds);
        (void)hipFuncSetAttribute((const void*)k_stage1_gemm<true>, hipFuncAttributeMaxDynamicSharedMemorySize,
                                  (int)lds);
        attr = true;
    }
    if (n_ranges > 0)
        k_stage1_gemm<false><<<dim3(n_qtiles * n_ranges), dim3(kWaves * 64), lds, s>>>(
            (const u32x4*)keys, (const u32x4*)qt, kc, n_rows, B, n_qtiles, n_full, n_ranges, 0, P, part);
    if (tail)
        k_stage1_gemm<true><<<dim3(n_qtiles), dim3(kWaves * 64), lds, s>>>(
            (const u32x4*)keys, (const u32x4*)qt, kc, n_rows, B, n_qtiles, n_full, 1, P - 1, P, part);
    return hipGetLastError();
}

}  // namespace lacache
