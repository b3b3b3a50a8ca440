// common.hpp -- types, store layout and device helpers shared by the gfx950 kernels.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace lacache {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));

constexpr int kWave = 64;

// ---------------------------------------------------------------------------
// Store layout of the normalised bfloat16 keys ("tiled"):
//   a 16-row x 32-column block of the key matrix is one contiguous 1 KiB
//   "chunk", ordered [c = col/8 % 4][r = row % 16][e = col % 8];
//   chunks are ordered [row/16][col/32].
// Lane l of a wave reading the chunk as 64 x 16 bytes gets row l%16 and
// columns 8*(l/16) .. 8*(l/16)+7 -- exactly the A/B operand fragment of
// v_mfma_f32_16x16x32_bf16 -- so every operand load is one fully coalesced
// 1 KiB wave access, and a run of 16 keys is d_pad*32 contiguous bytes.
// The same layout holds the normalised queries in scratch.
// ---------------------------------------------------------------------------
__host__ __device__ inline int64_t tiled_offset(int64_t row, int32_t col, int32_t kc /* d_pad / 32 */) {
    return ((row >> 4) * kc + (col >> 5)) * 512 + (((col >> 3) & 3) * 16 + (row & 15)) * 8 + (col & 7);
}

// ---------------------------------------------------------------------------
// Rounding of a double to bfloat16, once, to nearest with ties to even.
// Normal range (|v| >= 2^-126): round the 52-bit double significand to 7
// stored bits by adding just under half an ulp plus the kept lsb and
// truncating; a carry moves into the exponent by itself.  Below 2^-126 the
// bfloat16 grid is uniform with spacing 2^-133 (subnormals): round v*2^133 to
// an integer.  Overflow gives infinity.
// ---------------------------------------------------------------------------
__host__ __device__ inline uint64_t f64_bits(double v) {
    uint64_t b;
    __builtin_memcpy(&b, &v, sizeof b);
    return b;
}

__host__ __device__ inline uint16_t bf16_rne_from_f64(double v) {
    const uint64_t b = f64_bits(v);
    const uint16_t sign = (uint16_t)((b >> 48) & 0x8000u);
    const uint64_t mag = b & 0x7FFFFFFFFFFFFFFFull;
    const int e = (int)(mag >> 52) - 1023;
    if (e >= -126) {
        uint64_t m = mag + ((1ull << 44) - 1) + ((mag >> 45) & 1);
        const int e2 = (int)(m >> 52) - 1023;
        if (e2 > 127) return (uint16_t)(sign | 0x7F80u);
        return (uint16_t)(sign | ((uint32_t)(e2 + 127) << 7) | (uint32_t)((m >> 45) & 0x7F));
    }
    const double s = __builtin_rint(__builtin_ldexp(__builtin_fabs(v), 133));
    return (uint16_t)(sign | (uint16_t)s);
}

// bfloat16 rounding of the quotient v / n of a float32 v, identical to bf16_rne_from_f64(v / n) with the
// division correctly rounded (call that double q), computed as f = v * rnf in float32, where rnf is 1 / n
// rounded to double and then to float32 (quotient_rcp_f32).  The roundings of rn, rnf, f and q (at most
// 2^-53, 2^-24, 2^-24 and 2^-53 relative) put f within 2^-23 (1 + 2^-28) |v / n| of q: at most 2 float32 units
// in the last place of f's binade, plus a sliver.  Every bfloat16 rounding midpoint is a float32 with low 16
// bits 0x8000, and the only one closer to f than 2^14 such units is the one inside f's own bfloat16 interval;
// so unless f's low 16 bits are within 2 of 0x8000, no midpoint lies between f and q and both round to the
// same bfloat16.  The fallback window is twice that (within 4).  Those rare cases, zero,
// values below 2^-125 (where the float32 product loses relative precision) and rows whose reciprocal is not
// a normal float32 (rnf = 0, so every product is zero) divide instead.
// The reciprocal for bf16_rne_quotient_fast: 1 / n rounded to double, then to float32, or 0 where that double
// is not a normal float32.
__host__ __device__ inline float quotient_rcp_f32(double n) {
    const double rn = 1.0 / n;
    return (rn >= 0x1p-126 && rn < 0x1p127) ? (float)rn : 0.0f;
}

// The rounding without the division: the result as the float32 of the same value (its low 16 bits zero), and
// whether it may be wrong, when the caller must take bf16_rne_quotient_f32 instead.
__host__ __device__ inline float bf16_rne_quotient_fast(float v, float rnf, bool& exact_needed) {
    const float f = v * rnf;
    uint32_t u;
    __builtin_memcpy(&u, &f, 4);
    exact_needed = (u & 0x7FFFFFFFu) < 0x01000000u || (u & 0xFFFFu) - 0x7FFCu <= 8u;
    u = (u + 0x7FFFu + ((u >> 16) & 1u)) & 0xFFFF0000u;
    float r;
    __builtin_memcpy(&r, &u, 4);
    return r;
}

// The result as the float32 of the same value (its low 16 bits zero); rnf = quotient_rcp_f32(n).
__host__ __device__ inline float bf16_rne_quotient_f32(float v, double n, float rnf) {
    bool exact_needed;
    const float r = bf16_rne_quotient_fast(v, rnf, exact_needed);
    if (!exact_needed) return r;
    float vv = v;
#if defined(__HIP_DEVICE_COMPILE__)
    // convert here, on the rare path, rather than keep a double of every element live across the caller's loop
    __asm__ volatile("" : "+v"(vv));
#endif
    const uint32_t u = (uint32_t)bf16_rne_from_f64((double)vv / n) << 16;
    float e;
    __builtin_memcpy(&e, &u, 4);
    return e;
}
__host__ __device__ inline uint16_t bf16_rne_quotient(float v, double n, float rnf) {
    const float r = bf16_rne_quotient_f32(v, n, rnf);
    uint32_t u;
    __builtin_memcpy(&u, &r, 4);
    return (uint16_t)(u >> 16);
}

__device__ inline float bf16_to_f32(uint16_t h) { return __uint_as_float((uint32_t)h << 16); }

// Elements j0 .. j0+7 of a row as floats (0 beyond d; bfloat16 widens exactly): one or two 16-byte loads when
// the chunk is whole and 16-byte aligned, element loads otherwise.  The values are the same either way.
__device__ inline void load8f(const void* row, int dtype, int d, int j0, float v[8]) {
    const size_t esz = dtype == 0 ? 4 : 2;
    const char* p = (const char*)row + (size_t)j0 * esz;
    if (j0 + 8 <= d && ((uintptr_t)p & 15) == 0) {
        if (dtype == 0) {
            const float4 x = ((const float4*)p)[0], y = ((const float4*)p)[1];
            v[0] = x.x, v[1] = x.y, v[2] = x.z, v[3] = x.w, v[4] = y.x, v[5] = y.y, v[6] = y.z, v[7] = y.w;
        } else {
            const uint4 x = *(const uint4*)p;
            const uint32_t w[4] = {x.x, x.y, x.z, x.w};
#pragma unroll
            for (int t = 0; t < 4; ++t) {
                v[2 * t] = __uint_as_float(w[t] << 16);
                v[2 * t + 1] = __uint_as_float(w[t] & 0xFFFF0000u);
            }
        }
        return;
    }
#pragma unroll
    for (int e = 0; e < 8; ++e)
        v[e] = (j0 + e < d) ? (dtype == 0 ? ((const float*)row)[j0 + e] : bf16_to_f32(((const uint16_t*)row)[j0 + e]))
                            : 0.0f;
}

// The same elements as doubles.
__device__ inline void load8(const void* row, int dtype, int d, int j0, double v[8]) {
    float f[8];
    load8f(row, dtype, d, j0, f);
#pragma unroll
    for (int e = 0; e < 8; ++e) v[e] = (double)f[e];
}

// ---------------------------------------------------------------------------
// Wave-wide butterfly reductions: every lane ends with the same value, and
// the combination order is fixed, so results are run-to-run identical.
// ---------------------------------------------------------------------------
__device__ inline double wave_sum_f64(double x) {
#pragma unroll
    for (int m = 32; m >= 1; m >>= 1) x += __shfl_xor(x, m, kWave);
    return x;
}
__device__ inline float wave_sum_f32(float x) {
#pragma unroll
    for (int m = 32; m >= 1; m >>= 1) x += __shfl_xor(x, m, kWave);
    return x;
}
__device__ inline uint64_t umax64(uint64_t a, uint64_t b) { return a > b ? a : b; }
__device__ inline uint64_t wave_max_u64(uint64_t x) {
#pragma unroll
    for (int m = 32; m >= 1; m >>= 1) x = umax64(x, (uint64_t)__shfl_xor((unsigned long long)x, m, kWave));
    return x;
}

// ---------------------------------------------------------------------------
// One wave L2-normalises one input row and rounds it to bfloat16: the sum of
// squares is taken in double (lane-local in column order, then the butterfly
// above), n = sqrt in double, and each component v / n is rounded once to
// bfloat16.  A zero row (or live == false) gives zeros, as do the columns
// d .. d_pad-1.  Lane l produces columns 8l + 512t .. 8l + 512t + 7 and hands
// them, packed, to emit(j0, u32x4).  Every kernel that quantises a vector
// (insert, query staging, lookahead check, calibration pairs) goes through
// row_norm and quantise8, so equal inputs quantise to identical bits wherever
// they are stored or compared.
// ---------------------------------------------------------------------------
__device__ inline double row_norm(const void* row, int dtype, int d, bool live, int lane) {
    double ss = 0.0;
    if (live) {
        for (int j0 = lane * 8; j0 < d; j0 += 512) {
            double v[8];
            load8(row, dtype, d, j0, v);
#pragma unroll
            for (int e = 0; e < 8; ++e)
                if (j0 + e < d) ss += v[e] * v[e];
        }
    }
    ss = wave_sum_f64(ss);
    return __builtin_sqrt(ss);
}

// Columns j0 .. j0+7 of the normalised row as packed bfloat16 (zeros beyond d, for a zero norm or dead rows).
__device__ inline u32x4 quantise8(const void* row, int dtype, int d, int j0, double n, bool live) {
    uint16_t h[8];
    float v[8];
    if (live && j0 < d && n != 0.0) load8f(row, dtype, d, j0, v);
    const float rnf = quotient_rcp_f32(n);
#pragma unroll
    for (int e = 0; e < 8; ++e) {
        const int j = j0 + e;
        h[e] = 0;
        if (live && j < d && n != 0.0) h[e] = bf16_rne_quotient(v[e], n, rnf);
    }
    u32x4 w;
    w.x = (uint32_t)h[0] | ((uint32_t)h[1] << 16);
    w.y = (uint32_t)h[2] | ((uint32_t)h[3] << 16);
    w.z = (uint32_t)h[4] | ((uint32_t)h[5] << 16);
    w.w = (uint32_t)h[6] | ((uint32_t)h[7] << 16);
    return w;
}

template <class Emit>
__device__ inline void normalise_row(const void* row, int dtype, int d, int d_pad, bool live, int lane, Emit emit) {
    const double n = row_norm(row, dtype, d, live, lane);
    for (int j0 = lane * 8; j0 < d_pad; j0 += 512) emit(j0, quantise8(row, dtype, d, j0, n, live));
}

// A row held in registers: lane l keeps columns l*8 + 512 c .. +7 for c < NC (zeros beyond d, and for rows that
// are not live), the columns row_norm and quantise8 give lane l.
template <int NC>
__device__ __forceinline__ void row_to_regs(const char* src, int dtype, int d, bool live, int lane, float (&x)[NC][8]) {
#pragma unroll
    for (int c = 0; c < NC; ++c) {
        if (live) {
            load8f(src, dtype, d, lane * 8 + 512 * c, x[c]);
        } else {
#pragma unroll
            for (int e = 0; e < 8; ++e) x[c][e] = 0.0f;
        }
    }
}

// Its norm, the squares summed in the order row_norm uses (the zeros it skips add nothing), so the two agree
// bit for bit.
template <int NC>
__device__ __forceinline__ double regs_norm(const float (&x)[NC][8]) {
    double ss = 0.0;
#pragma unroll
    for (int c = 0; c < NC; ++c)
#pragma unroll
        for (int e = 0; e < 8; ++e) ss += (double)x[c][e] * (double)x[c][e];
    return __builtin_sqrt(wave_sum_f64(ss));
}

// Columns j0 .. j0+7 of the row in registers (x = its c-th piece) rounded as quantise8 rounds them.
__device__ __forceinline__ u32x4 regs_quantise8(const float (&x)[8], int j0, int d, double n, float rnf, bool live) {
    uint32_t h[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) h[e] = (live && j0 + e < d && n != 0.0) ? bf16_rne_quotient(x[e], n, rnf) : 0u;
    u32x4 w;
    w.x = h[0] | (h[1] << 16);
    w.y = h[2] | (h[3] << 16);
    w.z = h[4] | (h[5] << 16);
    w.w = h[6] | (h[7] << 16);
    return w;
}

// Dot product of two packed bfloat16 chunks, accumulated into acc in float32 in column order.  bf16 x bf16
// products are exact in float.
__device__ inline float dot8_bf16(u32x4 a, u32x4 b, float acc) {
    const uint32_t av[4] = {a.x, a.y, a.z, a.w}, bv[4] = {b.x, b.y, b.z, b.w};
#pragma unroll
    for (int t = 0; t < 4; ++t) {
        acc += __uint_as_float(av[t] << 16) * __uint_as_float(bv[t] << 16);
        acc += __uint_as_float(av[t] & 0xFFFF0000u) * __uint_as_float(bv[t] & 0xFFFF0000u);
    }
    return acc;
}

// ---------------------------------------------------------------------------
// Top-1 candidates as one 64-bit key: high word = the score's bits mapped so
// that unsigned order equals float order, low word = ~index.  The unsigned
// maximum is then "highest score, lowest index among equal scores": a total
// order, so any merge order gives the same winner.  -0 is folded onto +0
// first so that equal scores compare equal.
// ---------------------------------------------------------------------------
__device__ inline uint32_t order_f32(float f) {
    const uint32_t u = __float_as_uint(f + 0.0f);
    return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}
__device__ inline float unorder_f32(uint32_t o) {
    return __uint_as_float((o & 0x80000000u) ? (o & 0x7FFFFFFFu) : ~o);
}
__device__ inline uint64_t pack_top1(float s, int32_t idx) {
    return ((uint64_t)order_f32(s) << 32) | (uint64_t)(0xFFFFFFFFu - (uint32_t)idx);
}
__device__ inline int32_t unpack_idx(uint64_t p) { return (int32_t)(0xFFFFFFFFu - (uint32_t)(p & 0xFFFFFFFFu)); }
__device__ inline float unpack_score(uint64_t p) { return unorder_f32((uint32_t)(p >> 32)); }

__device__ inline f32x4 mfma16x16x32(u32x4 a, u32x4 b, f32x4 c) {
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, a), __builtin_bit_cast(bf16x8, b), c,
                                                   0, 0, 0);
}

}  // namespace lacache
