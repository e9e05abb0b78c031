// Output-stationary gather -> MFMA GEMM over flattened (offset, channel) chunks.
#pragma once

#include "common.hpp"

namespace ssconv {

// True when gather_mfma handles the shape (ca a multiple of 8, at most 128 offsets).
bool gather_mfma_supported(ssconv_dtype dt, int ca, int cb, int K);

// out[order ? order[p] : p][:] = sum_s Bt[s] (cb x ca) . src[nbr[s][p]] for p < n_pos.
// src [*, ca], Bt [K][cb][ca] and out [*, cb] in dt; nbr [K][n_pos] (-1 = absent).
int gather_mfma(const void* src, ssconv_dtype dt, int ca, const void* Bt, int cb, const int32_t* nbr,
                const int32_t* order, int64_t n_pos, int K, void* out, hipStream_t st);

}  // namespace ssconv
