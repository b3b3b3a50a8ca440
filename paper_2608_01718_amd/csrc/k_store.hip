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

// One wave per row (grid-stride over the rows).  Rows >= rows (up to rows_pad) are written as zeros, as are the
// columns d .. d_pad-1.
template <bool TILED>
__global__ __launch_bounds__(256) void k_normalise_rows(const void* __restrict__ in, int dtype, int64_t rows,
                                                        int64_t rows_pad, int d, int d_pad,
                                                        uint16_t* __restrict__ out, int64_t row0) {
    const int lane = threadIdx.x & 63;
    const int kc = d_pad >> 5;
    for (int64_t r = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6); r < rows_pad; r += (int64_t)gridDim.x * 4) {
        const bool live = r < rows;
        const char* src = (const char*)in + (live ? r * (int64_t)d * (dtype == 0 ? 4 : 2) : 0);
        normalise_row(src, dtype, d, d_pad, live, lane, [&](int j0, u32x4 w) {
            const int64_t off = TILED ? tiled_offset(row0 + r, j0, kc) : (row0 + r) * (int64_t)d_pad + j0;
            *(u32x4*)(out + off) = w;
        });
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

hipError_t launch_normalise(const void* in, int dtype, int64_t rows, int64_t rows_pad, int d, int d_pad,
                            uint16_t* out, int64_t row0, bool tiled, hipStream_t s) {
    if (rows_pad <= 0) return hipSuccess;
    const dim3 grid((unsigned)grid_blocks((rows_pad + 3) / 4)), block(256);
    if (tiled)
        k_normalise_rows<true><<<grid, block, 0, s>>>(in, dtype, rows, rows_pad, d, d_pad, out, row0);
    else
        k_normalise_rows<false><<<grid, block, 0, s>>>(in, dtype, rows, rows_pad, d, d_pad, out, row0);
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
