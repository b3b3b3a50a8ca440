// k_stage1_stream.hip -- stage 1 for small batches: one pass over the keys at HBM speed.
//
// Stage 1 of the lookup (Algorithm 1: search the cache with the query key) is
// an exact top-1 over every stored key by the dot product of normalised
// vectors.  With B <= 64 queries a key byte feeds at most 64 multiply-adds,
// far below the matrix-core/HBM balance point, so the kernel is bound by
// reading the keys once: every wave streams a contiguous run of 16-key groups
// (d_pad*32 contiguous bytes each) with 1 KiB coalesced non-temporal loads
// (read once, they are not kept in the caches: ~13 % more read bandwidth than
// plain loads; plain loads when several query groups share the range), double
// buffered, while the queries sit in LDS for the whole launch.  Larger
// batches run as up to four 64-query groups: the workgroups of one key range
// sit on the same XCD and start together, so the range comes from HBM once
// and the other readers find it in that XCD's L2 (or the infinity cache).
// Dot products run on v_mfma_f32_16x16x32_bf16 with the keys as the row
// operand, so each lane accumulates 4 keys x 1 query and keeps a running
// (best score, index) per query in registers; rows are visited in increasing
// order and only a strictly larger score replaces the best, so the lowest
// index wins ties.
#include "common.hpp"
#include "launch.hpp"

namespace lacache {

constexpr int kStreamWaves = 16;     // waves per workgroup; one workgroup per CU
constexpr int kStreamMaxGroups = 4;  // query groups of one launch, each reading every key range

// NT: the keys are loaded non-temporally (one query group: each key range has a single reader); with several
// query groups plain loads keep a range in L2 for the other groups' workgroups.
// NCQ = 0: the queries come normalised and tiled in qt (staged by the query normaliser).  NCQ = 1, 2, 4: every
// workgroup normalises its own query rows from the caller's input qraw ([B][d], dtype 0 f32 / 1 bf16; rows of up
// to 512 * NCQ columns) straight into its LDS fragments, with the row normaliser's own steps (a wave per row,
// the same sums and roundings), so the values are bit for bit the staged ones and the staging launch is saved.
template <int QG, bool NT, int NCQ>
__global__ __launch_bounds__(1024) void k_stage1_stream(const u32x4* __restrict__ keys, const u32x4* __restrict__ qt,
                                                        const void* __restrict__ qraw, int dtype, int d, int kc,
                                                        int groups, int n_rows, int n_ranges, int n_qgroups, int B,
                                                        uint64_t* __restrict__ part) {
    extern __shared__ u32x4 smem[];
    u32x4* qs = smem;                                        // [QG][kc][64] query fragments
    uint64_t* red = (uint64_t*)(smem + QG * kc * 64);        // [kStreamWaves][QG * 16]
    const int tid = threadIdx.x, lane = tid & 63, wid = tid >> 6;
    // workgroup -> (query group h of 16 * QG queries, key range r).  Dispatch is round-robin over the 8 XCDs:
    // with n_ranges % 8 == 0 the n_qgroups workgroups of a range are consecutive on one XCD.
    int h, r;
    if (n_qgroups > 1 && n_ranges % 8 == 0) {
        const int xcd = blockIdx.x % 8, j = blockIdx.x / 8;
        h = j % n_qgroups;
        r = (j / n_qgroups) * 8 + xcd;
    } else {
        h = blockIdx.x % n_qgroups;
        r = blockIdx.x / n_qgroups;
    }
    // contiguous, balanced split of the 16-key groups over all waves of the grid; the first key loads are issued
    // before the queries are staged, so that their latency overlaps the staging
    const int64_t waves_total = (int64_t)n_ranges * kStreamWaves;
    const int64_t w = (int64_t)r * kStreamWaves + wid;
    const int g0 = (int)(w * groups / waves_total);
    const int g1 = (int)((w + 1) * groups / waves_total);
    const int nchunks = (g1 - g0) * kc;
    const u32x4* kp = keys + (int64_t)g0 * kc * 64 + lane;
    u32x4 cur[4], nxt[4];
    if (nchunks > 0) {
#pragma unroll
        for (int u = 0; u < 4; ++u) cur[u] = NT ? __builtin_nontemporal_load(kp + u * 64) : kp[u * 64];
    }

    if constexpr (NCQ == 0) {
        const u32x4* qg = qt + (int64_t)h * QG * kc * 64;   // 16 * QG query rows of the tiled scratch
        for (int i = tid; i < QG * kc * 64; i += kStreamWaves * 64) qs[i] = qg[i];
    } else {
        // wave wid normalises row wid of each 16-row query block; piece J (columns 8J .. 8J+7) of that row is
        // lane 16 (J % 4) + wid of fragment J / 4 (rows past B are zero, as in the staged scratch).  When they
        // fit in 32 registers all of the wave's rows are loaded before any is reduced, so their loads overlap.
        const size_t esz = dtype == 0 ? 4 : 2;
        constexpr int kAhead = QG * NCQ <= 4 ? QG : 1;      // rows held in registers at once
#pragma unroll
        for (int q0 = 0; q0 < QG; q0 += kAhead) {
            float x[kAhead][NCQ][8];
#pragma unroll
            for (int t = 0; t < kAhead; ++t) {
                const int64_t rq = ((int64_t)h * QG + q0 + t) * 16 + wid;
                const bool live = rq < B;
                row_to_regs<NCQ>((const char*)qraw + (live ? rq * (int64_t)d * esz : 0), dtype, d, live, lane, x[t]);
            }
#pragma unroll
            for (int t = 0; t < kAhead; ++t) {
                const int q = q0 + t;
                const bool live = ((int64_t)h * QG + q) * 16 + wid < B;
                const double n = regs_norm<NCQ>(x[t]);
                const float rnf = quotient_rcp_f32(n);
#pragma unroll
                for (int c = 0; c < NCQ; ++c) {
                    const int j0 = lane * 8 + 512 * c, J = j0 >> 3;
                    if (j0 < kc * 32)
                        qs[(q * kc + (J >> 2)) * 64 + (J & 3) * 16 + wid] =
                            regs_quantise8(x[t][c], j0, d, n, rnf, live);
                }
            }
        }
    }
    __syncthreads();

    float best[QG];
    int bidx[QG];
#pragma unroll
    for (int q = 0; q < QG; ++q) {
        best[q] = -__builtin_inff();
        bidx[q] = 0x7FFFFFFF;
    }
    f32x4 acc[QG];
#pragma unroll
    for (int q = 0; q < QG; ++q) acc[q] = f32x4{0.f, 0.f, 0.f, 0.f};
    int ks = 0, g = g0;
    for (int c = 0; c < nchunks; c += 4) {
        if (c + 4 < nchunks) {
#pragma unroll
            for (int u = 0; u < 4; ++u) {
                const u32x4* a = kp + (int64_t)(c + 4 + u) * 64;
                nxt[u] = NT ? __builtin_nontemporal_load(a) : *a;
            }
        }
#pragma unroll
        for (int u = 0; u < 4; ++u) {
#pragma unroll
            for (int q = 0; q < QG; ++q) acc[q] = mfma16x16x32(cur[u], qs[(q * kc + ks + u) * 64 + lane], acc[q]);
        }
        ks += 4;
        if (ks == kc) {
            // lane holds rows 4*(lane/16)+j of the group, query column lane%16
            const int row0 = g * 16 + 4 * (lane >> 4);
#pragma unroll
            for (int q = 0; q < QG; ++q) {
#pragma unroll
                for (int j = 0; j < 4; ++j) {
                    const float s = acc[q][j];
                    if (row0 + j < n_rows && s > best[q]) {
                        best[q] = s;
                        bidx[q] = row0 + j;
                    }
                }
                acc[q] = f32x4{0.f, 0.f, 0.f, 0.f};
            }
            ks = 0;
            ++g;
        }
#pragma unroll
        for (int u = 0; u < 4; ++u) cur[u] = nxt[u];
    }

    // lanes l, l^16, l^32, l^48 hold the same query: merge, then merge the waves
#pragma unroll
    for (int q = 0; q < QG; ++q) {
        uint64_t p = (bidx[q] == 0x7FFFFFFF) ? 0ull : pack_top1(best[q], bidx[q]);
        p = umax64(p, (uint64_t)__shfl_xor((unsigned long long)p, 16, kWave));
        p = umax64(p, (uint64_t)__shfl_xor((unsigned long long)p, 32, kWave));
        if (lane < 16) red[wid * (QG * 16) + q * 16 + lane] = p;
    }
    __syncthreads();
    const int q = h * QG * 16 + tid;  // query of the batch
    if (tid < QG * 16 && q < B) {
        uint64_t m = 0;
        for (int v = 0; v < kStreamWaves; ++v) m = umax64(m, red[v * (QG * 16) + tid]);
        part[(int64_t)q * n_ranges + r] = m;
    }
}

// Arguments of one streaming launch.
struct StreamLaunch {
    const u32x4* keys;
    const u32x4* qt;
    const void* qraw;
    int dtype, d, ncq, kc, groups, n_rows, n_ranges, n_qgroups, B;
    uint64_t* part;
    hipStream_t s;
    hipEvent_t e0, e1;
};

template <int QG, bool NT, int NCQ>
static hipError_t launch_qgn(const StreamLaunch& a) {
    const size_t lds = (size_t)QG * a.kc * 1024 + (size_t)kStreamWaves * QG * 16 * 8;
    static std::atomic<uint64_t> lds_allowed{0};
    const hipError_t e = allow_dynamic_lds((const void*)k_stage1_stream<QG, NT, NCQ>, 160 * 1024, lds_allowed);
    if (e != hipSuccess) return e;
    return launch_timed(k_stage1_stream<QG, NT, NCQ>, dim3(a.n_ranges * a.n_qgroups), dim3(kStreamWaves * 64), lds,
                        a.s, a.e0, a.e1, a.keys, a.qt, a.qraw, a.dtype, a.d, a.kc, a.groups, a.n_rows, a.n_ranges,
                        a.n_qgroups, a.B, a.part);
}

// ncq: 0 reads the staged queries, 1 / 2 / 4 normalises the caller's rows in the kernel (d_pad <= 512 * ncq)
template <int QG, bool NT>
static hipError_t launch_qg(const StreamLaunch& a) {
    switch (a.ncq) {
        case 0: return launch_qgn<QG, NT, 0>(a);
        case 1: return launch_qgn<QG, NT, 1>(a);
        case 2: return launch_qgn<QG, NT, 2>(a);
        case 4: return launch_qgn<QG, NT, 4>(a);
        default: return hipErrorInvalidValue;
    }
}

// Largest query-group count QG (16 queries each, at most 4) whose query
// fragments fit in LDS next to the reduction area, for d_pad columns.
int stream_max_qg(int d_pad) {
    const int kc = d_pad / 32;
    for (int qg = 4; qg >= 1; --qg)
        if ((size_t)qg * kc * 1024 + (size_t)kStreamWaves * qg * 16 * 8 <= 160 * 1024) return qg;
    return 0;
}

hipError_t launch_stage1_stream(const uint16_t* keys, const uint16_t* qt, int B, int n_rows, int d_pad,
                                uint64_t* part, int num_cu, int* P_out, hipStream_t s, hipEvent_t e0, hipEvent_t e1,
                                const void* qraw, int dtype, int d) {
    const int kc = d_pad / 32;
    const int ncq = qraw == nullptr ? 0 : stream_fused_ncq(d_pad);
    if (qraw != nullptr && (ncq == 0 || d < 1 || d > d_pad || (dtype != 0 && dtype != 1)))
        return hipErrorInvalidValue;
    const int groups = (n_rows + 15) / 16;
    const int maxqg = stream_max_qg(d_pad);
    if (maxqg < 1 || kc % 4 != 0 || n_rows <= 0 || B < 1) return hipErrorInvalidValue;
    // up to 16 * maxqg queries in one group; more as up to kStreamMaxGroups full groups (query rows
    // zero-padded to a multiple of 16 * maxqg by the caller)
    const int grp = 16 * maxqg;
    const int n_qgroups = (B + grp - 1) / grp;
    if (n_qgroups > kStreamMaxGroups) return hipErrorInvalidValue;
    const int qg = n_qgroups == 1 ? (B + 15) / 16 : maxqg;
    // one workgroup per CU, fewer when there is too little work to give every wave a 16-key group (small
    // caches spread over as many CUs as they can: their time is the chain of loads each wave walks); with
    // several query groups a multiple of 8 ranges keeps each range's workgroups on one XCD
    int cap = num_cu / n_qgroups;
    if (n_qgroups > 1 && cap >= 8) cap = cap / 8 * 8;
    int n_ranges = (groups + kStreamWaves - 1) / kStreamWaves;
    if (n_ranges > cap) n_ranges = cap;
    if (n_ranges > kMaxPartials) n_ranges = kMaxPartials;
    if (n_ranges < 1) n_ranges = 1;
    *P_out = n_ranges;
    const StreamLaunch a{(const u32x4*)keys, (const u32x4*)qt, qraw, dtype, d, ncq, kc, groups, n_rows,
                         n_ranges, n_qgroups, B, part, s, e0, e1};
    const bool single = n_qgroups == 1;
    switch (qg) {
        case 1: return single ? launch_qg<1, true>(a) : launch_qg<1, false>(a);
        case 2: return single ? launch_qg<2, true>(a) : launch_qg<2, false>(a);
        case 3: return single ? launch_qg<3, true>(a) : launch_qg<3, false>(a);
        default: return single ? launch_qg<4, true>(a) : launch_qg<4, false>(a);
    }
}

// Row width class for normalising the queries inside the kernel: 1, 2 or 4 pieces of 512 columns per lane; 0
// when the rows are wider (they are staged by the query normaliser first).
int stream_fused_ncq(int d_pad) { return d_pad <= 512 ? 1 : d_pad <= 1024 ? 2 : d_pad <= 2048 ? 4 : 0; }

// Largest batch the streaming kernel takes for d_pad columns.
int stream_max_batch(int d_pad) { return kStreamMaxGroups * 16 * stream_max_qg(d_pad); }

}  // namespace lacache
