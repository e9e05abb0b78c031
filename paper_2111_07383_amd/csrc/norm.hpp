// Steerable normalisation (Sec. 3.3, Eq. 11): the forward statistics, shared between the Norm
// kernels and the convolution kernels that accumulate them while they write the convolution's
// output (the fused Norm epilogue of ssconv_forward_norm).
//
// Statistics layout: per-channel fp64 sums of the stored output values over row blocks b,
// part[(c * nblk + b) * 2 + q], q = 0: sum of x, q = 1: sum of x^2.  A fixed reduction then adds
// the blocks of each channel (norm_forward_finish), so the result does not depend on scheduling.
#pragma once

#include "common.hpp"

namespace ssconv {

constexpr int kNormThreads = 256;
constexpr int kNormMaxChunks = 4;                       // channels per row <= 4 * 256
constexpr int kNormMaxChannels = kNormMaxChunks * kNormThreads;

// Row blocks of the separate statistics pass over y [n, C]: blocks of rpb rows.  vec: thread t
// holds the 16 bytes of channels (t % nv) * VEC .. of rows r0 + t / nv + k G (nv = C / VEC vectors
// per row, G = 256 / nv row groups); else, for C <= 256, G = 256 / C row groups of C threads
// (thread t: channel t % C, rows r0 + t / C + k G), for C > 256 one group, thread t holding
// channels t + 256 j.  Rows are added in row order, the G groups then in group order.
struct NormStatsPlan {
  int C, G, NC, nblk;
  int64_t rpb;
  bool vec;
};
NormStatsPlan norm_stats_plan(ssconv_dtype dt, const void* y, int64_t n, int C);

// Device bytes of the statistics workspace of C channels over nblk row blocks: the partial sums
// (at its start), the channel sums and the per-channel coefficients.
size_t norm_ws_bytes(int C, int64_t nblk);

// Where a producing kernel leaves the statistics: it takes ws (norm_ws_bytes(C, nblk) bytes, from
// sc, nullptr: the device memory cache) and sets nblk; nblk == 0 means no kernel did, and the
// caller runs the separate pass.  The caller gives ws back.
struct NormSink {
  int C = 0;
  CallScratch* sc = nullptr;
  int64_t nblk = 0;
  char* ws = nullptr;
};
int norm_sink_take(NormSink* s, int64_t nblk, hipStream_t st);

// The partial sums (at the start of ws, plan.nblk blocks) by a pass over y [n, C].
int norm_forward_sums(ssconv_dtype dt, const void* y, int64_t n, const NormStatsPlan& p, char* ws, hipStream_t st);
// From the partial sums of nblk row blocks in ws: channel sums, coefficients, and z = Norm(y)
// (z may alias y).
int norm_forward_finish(const FieldTab& f, ssconv_dtype dt, const void* y, int64_t n, double eps, int64_t nblk,
                        char* ws, void* z, hipStream_t st);
// Argument checks of the Norm entry points (field table of the channels, eps > 0, size limits).
int norm_check_fields(const ssconv_fields* fields, ssconv_dtype dt, int64_t n, double eps, FieldTab* f);

// ---------------------------------------------------------------------------------------------
// Row-block statistics for the kernels that produce an output row by row (the pair-list reduce,
// the offset-split reduce): a workgroup of kStatsThreads threads owns rows [b * rpb, (b+1) * rpb);
// thread t < G * nv (nv = C / VEC vectors of VEC columns, G = kStatsThreads / nv) owns vector
// t % nv of the rows r0 + t / nv + k G, so its column sums stay in registers; the G row groups are
// then added in group order.
// ---------------------------------------------------------------------------------------------
constexpr int kStatsThreads = 512;
constexpr int kStatsRowsPerThread = 2;  // rows per thread (measured: 1 row gave more partials and no gain)

struct StatsRows {
  int G;
  int64_t rpb, nblk;
};
// false when C / VEC exceeds the workgroup (then the statistics come from the separate pass).
inline bool stats_rows_plan(int64_t n, int C, int VEC, StatsRows* p) {
  const int nv = C / VEC;
  if (C % VEC != 0 || nv < 1 || nv > kStatsThreads || n <= 0) return false;
  p->G = kStatsThreads / nv;
  p->rpb = (int64_t)p->G * kStatsRowsPerThread;
  p->nblk = (n + p->rpb - 1) / p->rpb;
  return p->nblk < ((int64_t)1 << 31);
}

// row_fn(r, v, val) computes row r's VEC columns v * VEC .., stores them and returns the stored
// values in val (as float); the sums are taken of those values.
template <int VEC, typename RowFn>
__device__ __forceinline__ void stats_rows(int C, int64_t n, int G, int64_t rpb, RowFn&& row_fn,
                                           double* __restrict__ part) {
  __shared__ double red[2 * VEC][kStatsThreads];
  const int nv = C / VEC, t = threadIdx.x;
  const int64_t r0 = (int64_t)blockIdx.x * rpb;
  const int64_t r1 = r0 + rpb < n ? r0 + rpb : n;
  const int v = t % nv, grp = t / nv;
  double s[2 * VEC];
#pragma unroll
  for (int q = 0; q < 2 * VEC; ++q) s[q] = 0.0;
  if (grp < G) {
    for (int64_t r = r0 + grp; r < r1; r += G) {
      float val[VEC];
      row_fn(r, v, val);
#pragma unroll
      for (int k = 0; k < VEC; ++k) {
        const double d = val[k];
        s[2 * k] += d;
        s[2 * k + 1] = fma(d, d, s[2 * k + 1]);
      }
    }
  }
#pragma unroll
  for (int q = 0; q < 2 * VEC; ++q) red[q][t] = s[q];
  __syncthreads();
  for (int e = t; e < C; e += kStatsThreads) {
    const int vv = e / VEC, k = e % VEC;
    double a = 0.0, b = 0.0;
    for (int j = 0; j < G; ++j) {
      a += red[2 * k][j * nv + vv];
      b += red[2 * k + 1][j * nv + vv];
    }
    part[((int64_t)e * gridDim.x + blockIdx.x) * 2] = a;
    part[((int64_t)e * gridDim.x + blockIdx.x) * 2 + 1] = b;
  }
}

}  // namespace ssconv
