// Output-stationary gather -> MFMA GEMM over flattened (offset, channel) chunks.
#pragma once

#include "common.hpp"

namespace ssconv {

struct NormSink;

// True when gather_mfma handles the shape (ca a multiple of 8, at most 128 offsets).
bool gather_mfma_supported(ssconv_dtype dt, int ca, int cb, int K);

// out[order ? order[p] : p][:] = sum_s Bt[s] (cb x ca) . src[nbr[s][p]] for p < n_pos.
// src [*, ca], Bt [K][cb][ca] and out [*, cb] in dt; nbr [K][n_pos] (-1 = absent).
// Offset splits (fp32 partials added in split order) take their partials from sc (nullptr: the
// device memory cache); with a fixed scratch region the split count is lowered until they fit.
// sink (optional): the kernel that writes out also leaves the Norm statistics of out there (norm.hpp).
int gather_mfma(const void* src, int64_t n_src, ssconv_dtype dt, int ca, const void* Bt, int cb, const int32_t* nbr,
                const int32_t* order, int64_t n_pos, int K, void* out, hipStream_t st, CallScratch* sc = nullptr,
                NormSink* sink = nullptr);

// bf16 kernel with 256-row tiles and packed kappa (gather_bf16.hip).
bool gather_bf16_supported(int64_t n_src, int ca, int cb, int K);

// Bp[s][k/8][n][k%8] (bf16) from Bt[s'][n][k] (transposed = false) or from W[s'][k][n]
// (transposed = true), s' = s, or K-1-s when mirrored; for k < ca, n < cb; ca a multiple of 8.
int pack_b_bf16(const void* W, int K, int ca, int cb, bool transposed, bool mirror, void* Bp, hipStream_t st);

// out[order ? order[p] : p][:] = sum_s Bt[s] (cb x ca) . src[nbr[s][p]] with Bt given packed as above;
// src holds n_src rows.  sink (optional): the tiles also leave the Norm statistics of out there.
int gather_bf16(const void* src, int64_t n_src, int ca, const void* Bp, int cb, const int32_t* nbr,
                const int32_t* order, int64_t n_pos, int K, void* out, hipStream_t st, NormSink* sink = nullptr);

}  // namespace ssconv
