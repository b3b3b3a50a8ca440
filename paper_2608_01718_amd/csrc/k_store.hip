// k_store.hip -- normalise-and-store kernels (insert, query staging) and the store export.
//
// Cosine similarity (Section 3: the distance of embeddings is e.g. the cosine
// distance; Section 5.1: hits are decided on cosine similarities) is computed
// as the dot product of L2-normalised vectors.  Each vector is normalised in
// double and rounded once, to nearest-even, to bfloat16 as it is written, so a
// query equal to a stored key quantises bit-identically to it.
#include "common.hpp"
#include "launch.hpp"

namespace lacache {

// The row-major layout (prefix embeddings), one wave per row (grid-stride over the rows).  Rows >= rows (up to
// rows_pad) are written as zeros, as are the columns d .. d_pad-1.  NC > 0 (d_pad <= 512 NC): the row is
// read once into registers; the stored bits are those of normalise_row.  NC = 0: any d, through normalise_row
// (the row read twice).
template <int NC>
__global__ __launch_bounds__(256) void k_normalise_rows(const void* __restrict__ in, int dtype, int64_t rows,
                                                        int64_t rows_pad, int d, int d_pad,
                                                        uint16_t* __restrict__ out, int64_t row0) {
    const int lane = threadIdx.x & 63;
    for (int64_t r = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6); r < rows_pad; r += (int64_t)gridDim.x * 4) {
        const bool live = r < rows;
        const char* src = (const char*)in + (live ? r * (int64_t)d * (dtype == 0 ? 4 : 2) : 0);
        uint16_t* dst = out + (row0 + r) * (int64_t)d_pad;
        if constexpr (NC > 0) {
            float x[NC][8];
            row_to_regs<NC>(src, dtype, d, live, lane, x);
            const double n = regs_norm<NC>(x);
            const float rnf = quotient_rcp_f32(n);
#pragma unroll
            for (int c = 0; c < NC; ++c) {
                const int j0 = lane * 8 + 512 * c;
                if (j0 < d_pad) *(u32x4*)(dst + j0) = regs_quantise8(x[c], j0, d, n, rnf, live);
            }
        } else {
            normalise_row(src, dtype, d, d_pad, live, lane, [&](int j0, u32x4 w) { *(u32x4*)(dst + j0) = w; });
        }
    }
}

// The tiled layout for any d (inserts of more than kTiledRowsMax keys, and every call past d_pad = 2048), one
// workgroup of 4 waves per 16-row group of the destination
// (grid-stride over the groups): the waves first take the norms of the group's rows (row_norm, as above),
// then each wave writes whole 1 KiB chunks -- lane l holds row l % 16, columns 8 (l / 16) .. +7 of the chunk --
// so every store is one contiguous wave access.  Destination rows outside [row0, row0 + rows_pad) belong
// to other calls and are not written; rows >= rows are written as zeros.
__global__ __launch_bounds__(256) void k_normalise_tiled(const void* __restrict__ in, int dtype, int64_t rows,
                                                         int64_t rows_pad, int d, int d_pad,
                                                         uint16_t* __restrict__ out, int64_t row0) {
    __shared__ double norms[16];
    const int lane = threadIdx.x & 63, wid = threadIdx.x >> 6;
    const int kc = d_pad >> 5;
    const size_t esz = dtype == 0 ? 4 : 2;
    const int64_t g0 = row0 >> 4, g1 = (row0 + rows_pad + 15) >> 4;
    for (int64_t g = g0 + blockIdx.x; g < g1; g += gridDim.x) {
        const int64_t r_first = g * 16 - row0;  // call row of the group's row 0
#pragma unroll
        for (int k = 0; k < 4; ++k) {
            const int i = wid * 4 + k;
            const int64_t r = r_first + i;
            const bool live = r >= 0 && r < rows;
            const double n = row_norm((const char*)in + (live ? r * (int64_t)d * esz : 0), dtype, d, live, lane);
            if (lane == 0) norms[i] = n;
        }
        __syncthreads();
        const int i = lane & 15;
        const int64_t r = r_first + i;
        const bool live = r >= 0 && r < rows;
        const bool mine = r >= 0 && r < rows_pad;
        const char* src = (const char*)in + (live ? r * (int64_t)d * esz : 0);
        for (int c = wid; c < kc; c += 4) {
            const u32x4 w = quantise8(src, dtype, d, c * 32 + 8 * (lane >> 4), norms[i], live);
            if (mine) *(u32x4*)(out + ((g * kc + c) * 64 + lane) * 8) = w;
        }
        __syncthreads();  // norms[] is rewritten by the next group
    }
}

// The tiled layout for d_pad <= 512 NC and calls of up to kTiledRowsMax rows (query staging, small inserts):
// one workgroup of 16 waves per 16-row group (grid-stride over the groups), wave i on row i of the group.  Each wave reads its row once into registers, rounds it as above and
// puts the 16-byte pieces into LDS, piece J (columns 8 J .. 8 J + 7) of row i at slot 16 J + (i ^ (J % 16)):
// the XOR keeps both the row-wise writes and the chunk-wise reads on distinct banks.  Then the waves write
// whole 1 KiB chunks as above.  With a wave per row, a group costs one read of each row and a few
// round trips: 16 queries are staged in ~5 us.
template <int NC>
__global__ __launch_bounds__(1024) void k_normalise_tiled_rows(const void* __restrict__ in, int dtype, int64_t rows,
                                                               int64_t rows_pad, int d, int d_pad,
                                                               uint16_t* __restrict__ out, int64_t row0) {
    __shared__ u32x4 stage[16 * 64 * NC];
    const int lane = threadIdx.x & 63, i = threadIdx.x >> 6;
    const int kc = d_pad >> 5;
    const size_t esz = dtype == 0 ? 4 : 2;
    const int64_t g0 = row0 >> 4, g1 = (row0 + rows_pad + 15) >> 4;
    for (int64_t g = g0 + blockIdx.x; g < g1; g += gridDim.x) {
        const int64_t r_first = g * 16 - row0;  // call row of the group's row 0
        {
            const int64_t r = r_first + i;
            const bool live = r >= 0 && r < rows;
            float x[NC][8];
            row_to_regs<NC>((const char*)in + (live ? r * (int64_t)d * esz : 0), dtype, d, live, lane, x);
            const double n = regs_norm<NC>(x);
            const float rnf = quotient_rcp_f32(n);
#pragma unroll
            for (int c = 0; c < NC; ++c) {
                const int j0 = lane * 8 + 512 * c, J = j0 >> 3;
                if (j0 < d_pad) stage[J * 16 + (i ^ (J & 15))] = regs_quantise8(x[c], j0, d, n, rnf, live);
            }
        }
        __syncthreads();
        const int row = lane & 15;
        const int64_t r = r_first + row;
        const bool mine = r >= 0 && r < rows_pad;
        for (int c = i; c < kc; c += 16) {
            const int J = c * 4 + (lane >> 4);
            const u32x4 w = stage[J * 16 + (row ^ (J & 15))];
            if (mine) *(u32x4*)(out + ((g * kc + c) * 64 + lane) * 8) = w;
        }
        __syncthreads();  // stage[] is rewritten by the next group
    }
}

// Copy rows first .. first+n-1 of a bfloat16 matrix (tiled or row-major with
// d_pad columns) into a dense [n][d] array.
template <bool TILED>
__global__ __launch_bounds__(256) void k_export_rows(const uint16_t* __restrict__ src, int64_t first, int n, int d,
                                                     int d_pad, uint16_t* __restrict__ dst) {
    const int64_t total = (int64_t)n * d;
    for (int64_t t = (int64_t)blockIdx.x * 256 + threadIdx.x; t < total; t += (int64_t)gridDim.x * 256) {
        const int64_t r = t / d;
        const int j = (int)(t - r * d);
        const int64_t off = TILED ? tiled_offset(first + r, j, d_pad >> 5) : (first + r) * (int64_t)d_pad + j;
        dst[t] = src[off];
    }
}

constexpr int64_t kTiledRowsMax = 8192;  // rows per call up to which the tiled layout takes a wave per row

hipError_t launch_normalise(const void* in, int dtype, int64_t rows, int64_t rows_pad, int d, int d_pad,
                            uint16_t* out, int64_t row0, bool tiled, hipStream_t s) {
    if (rows_pad <= 0) return hipSuccess;
    if (tiled) {
        const int64_t groups = ((row0 + rows_pad + 15) >> 4) - (row0 >> 4);
        const dim3 grid((unsigned)grid_blocks(groups)), wide(1024);
        // a wave per row for query staging and small inserts (latency: 16 queries staged in ~5 us instead of
        // ~13); bulk inserts keep the two-pass kernel, whose smaller workgroups overlap more groups per CU
        // (1M x 768 rows 13 % faster)
        if (rows_pad > kTiledRowsMax)
            k_normalise_tiled<<<grid, dim3(256), 0, s>>>(in, dtype, rows, rows_pad, d, d_pad, out, row0);
        else if (d_pad <= 512)
            k_normalise_tiled_rows<1><<<grid, wide, 0, s>>>(in, dtype, rows, rows_pad, d, d_pad, out, row0);
        else if (d_pad <= 1024)
            k_normalise_tiled_rows<2><<<grid, wide, 0, s>>>(in, dtype, rows, rows_pad, d, d_pad, out, row0);
        else if (d_pad <= 2048)
            k_normalise_tiled_rows<4><<<grid, wide, 0, s>>>(in, dtype, rows, rows_pad, d, d_pad, out, row0);
        else
            k_normalise_tiled<<<grid, dim3(256), 0, s>>>(in, dtype, rows, rows_pad, d, d_pad, out, row0);
    } else {
        const dim3 grid((unsigned)grid_blocks((rows_pad + 3) / 4)), block(256);
        if (d_pad <= 512)
            k_normalise_rows<1><<<grid, block, 0, s>>>(in, dtype, rows, rows_pad, d, d_pad, out, row0);
        else if (d_pad <= 1024)
            k_normalise_rows<2><<<grid, block, 0, s>>>(in, dtype, rows, rows_pad, d, d_pad, out, row0);
        else if (d_pad <= 2048)
            k_normalise_rows<4><<<grid, block, 0, s>>>(in, dtype, rows, rows_pad, d, d_pad, out, row0);
        else
            k_normalise_rows<0><<<grid, block, 0, s>>>(in, dtype, rows, rows_pad, d, d_pad, out, row0);
    }
    return hipGetLastError();
}

hipError_t launch_export(const uint16_t* src, int64_t first, int n, int d, int d_pad, uint16_t* dst, bool tiled,
                         hipStream_t s) {
    const int64_t total = (int64_t)n * d;
    if (total <= 0) return hipSuccess;
    const dim3 grid((unsigned)grid_blocks((total + 255) / 256)), block(256);
    if (tiled)
        k_export_rows<true><<<grid, block, 0, s>>>(src, first, n, d, d_pad, dst);
    else
        k_export_rows<false><<<grid, block, 0, s>>>(src, first, n, d, d_pad, dst);
    return hipGetLastError();
}

}  // namespace lacache
