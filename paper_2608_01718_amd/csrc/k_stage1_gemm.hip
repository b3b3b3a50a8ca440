// k_stage1_gemm.hip -- stage 1 for large batches.
//
// Interim form: the batch is processed in slices of up to 64 queries by the
// streaming kernel (every slice re-reads the keys).
#include "common.hpp"
#include "launch.hpp"

namespace lacache {

int stream_max_qg(int d_pad);

hipError_t launch_stage1_gemm(const uint16_t* keys, const uint16_t* qt, int B, int n_rows, int d_pad, uint64_t* part,
                              int num_cu, int* P_out, hipStream_t s) {
    const int slice = 16 * stream_max_qg(d_pad);
    if (slice == 0) return hipErrorInvalidValue;
    int P = 0;
    for (int b0 = 0; b0 < B; b0 += slice) {
        const int nb = (B - b0) < slice ? (B - b0) : slice;
        // P depends only on n_rows, so slice 0 (written at part + 0) fixes the stride of the later ones
        const uint16_t* q = qt + (int64_t)(b0 / 16) * (d_pad / 32) * 512;
        hipError_t e = launch_stage1_stream(keys, q, nb, n_rows, d_pad, part + (int64_t)b0 * P, num_cu, &P, s);
        if (e != hipSuccess) return e;
    }
    *P_out = P;
    return hipSuccess;
}

}  // namespace lacache
