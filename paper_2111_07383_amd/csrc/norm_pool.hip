// Steerable normalisation (Sec. 3.3, Eq. 11) and sparse 2x2x2 average pooling (the footnote of
// Sec. 3.1: downsampling is a stride-1 convolution followed by average pooling).
//
// Norm: every irreducible field is normalised on its own with population statistics over all n
// rows (so that a field is only ever multiplied by a scalar, which keeps it equivariant):
//   l = 0:  y = (f - mean) / sqrt(var + eps)
//   l > 0:  y = f / sqrt(mean over rows of |f|^2 + eps)
// Four launches, all bandwidth-bound: per-block channel sums in fp64 over fixed row ranges,
// one workgroup per channel adding the block sums in a fixed tree order (deterministic, no
// atomics), one thread per field turning the sums into per-channel coefficients, and an
// elementwise pass.  The backward pass is the exact gradient (the statistics depend on x): the
// same launches with four sums per channel (x, x^2, g, g x), then dx = A g + B (x - M) + C.
//
// Pooling runs on a rule book built with ksize 2, stride 2 (offsets {-1, 0}^3 under 2x - y = s):
// nbr[s][x] holds the active sites of the window 2x + {0,1}^3.  Forward: one pass per output row,
// the members added in offset order, times 1/8 (the dense average over the zero-filled window).
// Backward: every input lies in exactly one window, so each input row is written once with its
// window's gradient / 8.
#include <algorithm>

#include "norm.hpp"

namespace ssconv {
namespace {

constexpr int kThreads = kNormThreads;
constexpr int kMaxBlocks = 512;   // two workgroups per compute unit for the sums
constexpr int kMaxChunks = kNormMaxChunks;
constexpr int kMaxChannels = kNormMaxChannels;

// Vector of VEC elements moved as one 16-byte access (VEC = 1: scalar).
template <typename T, int VEC>
struct Vec {
  T e[VEC];
};

template <typename T, int VEC>
__device__ __forceinline__ Vec<T, VEC> vload(const T* p) {
  Vec<T, VEC> v;
  if constexpr (VEC * sizeof(T) == 16) {
    *reinterpret_cast<uint4*>(v.e) = *reinterpret_cast<const uint4*>(p);
  } else {
#pragma unroll
    for (int k = 0; k < VEC; ++k) v.e[k] = p[k];
  }
  return v;
}

template <typename T, int VEC>
__device__ __forceinline__ void vstore(T* p, const Vec<T, VEC>& v) {
  if constexpr (VEC * sizeof(T) == 16) {
    *reinterpret_cast<uint4*>(p) = *reinterpret_cast<const uint4*>(v.e);
  } else {
#pragma unroll
    for (int k = 0; k < VEC; ++k) p[k] = v.e[k];
  }
}

// ---------------------------------------------------------------------------------------------
// Norm
// ---------------------------------------------------------------------------------------------

// Channel sums of rows [b*rpb, min(n, (b+1)*rpb)) for block b, in fp64:
//   q = 0: x, q = 1: x^2, and with NQ = 4 also q = 2: g, q = 3: g x.
// Threads: for C <= 256, G = 256/C row groups of C threads (thread t: channel t % C, rows
// r0 + t/C + k G); for C > 256, one group, thread t holds channels t + 256 j.  Consecutive
// threads read consecutive addresses.  Output part[(c * nblk + b) * NQ + q].
template <typename T, int NQ>
__global__ __launch_bounds__(kThreads) void norm_sums_kernel(const T* __restrict__ x, const T* __restrict__ g,
                                                             int64_t n, int C, int G, int NC, int64_t rpb,
                                                             double* __restrict__ part) {
  __shared__ double red[NQ][kThreads];
  const int t = threadIdx.x, nblk = gridDim.x;
  const int64_t r0 = (int64_t)blockIdx.x * rpb;
  const int64_t r1 = min(n, r0 + rpb);
  const int grp = NC == 1 ? t / C : 0;
  double acc[kMaxChunks][NQ];
#pragma unroll
  for (int j = 0; j < kMaxChunks; ++j)
#pragma unroll
    for (int q = 0; q < NQ; ++q) acc[j][q] = 0.0;
#pragma unroll
  for (int j = 0; j < kMaxChunks; ++j) {
    if (j >= NC) break;
    const int c = NC == 1 ? t % C : t + j * kThreads;
    if (grp >= G || c >= C) break;
    int64_t r = r0 + grp;
    // four rows' loads issued together, then added in row order
    for (; r + 3 * (int64_t)G < r1; r += 4 * (int64_t)G) {
      float v[4], w[4];
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        v[k] = DT<T>::to_f(x[(r + k * (int64_t)G) * C + c]);
        if (NQ == 4) w[k] = DT<T>::to_f(g[(r + k * (int64_t)G) * C + c]);
      }
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        const double dv = v[k];
        acc[j][0] += dv;
        acc[j][1] = fma(dv, dv, acc[j][1]);
        if (NQ == 4) {
          const double dw = w[k];
          acc[j][2] += dw;
          acc[j][3] = fma(dw, dv, acc[j][3]);
        }
      }
    }
    for (; r < r1; r += G) {
      const double dv = DT<T>::to_f(x[r * C + c]);
      acc[j][0] += dv;
      acc[j][1] = fma(dv, dv, acc[j][1]);
      if (NQ == 4) {
        const double dw = DT<T>::to_f(g[r * C + c]);
        acc[j][2] += dw;
        acc[j][3] = fma(dw, dv, acc[j][3]);
      }
    }
  }
  if (NC == 1 && G > 1) {
    // add the G row groups of each channel in group order
#pragma unroll
    for (int q = 0; q < NQ; ++q) red[q][t] = acc[0][q];
    __syncthreads();
    if (t < C) {
#pragma unroll
      for (int q = 0; q < NQ; ++q) {
        double s = 0.0;
        for (int k = 0; k < G; ++k) s += red[q][k * C + t];
        part[((int64_t)t * nblk + blockIdx.x) * NQ + q] = s;
      }
    }
    return;
  }
#pragma unroll
  for (int j = 0; j < kMaxChunks; ++j) {
    if (j >= NC) break;
    const int c = NC == 1 ? t : t + j * kThreads;
    if (c >= C) break;
#pragma unroll
    for (int q = 0; q < NQ; ++q) part[((int64_t)c * nblk + blockIdx.x) * NQ + q] = acc[j][q];
  }
}

// One workgroup per channel: sums[c][q] = sum over blocks of part, thread t taking blocks t, t+256
// and a fixed halving tree across threads.
template <int NQ>
__global__ __launch_bounds__(kThreads) void norm_reduce_kernel(const double* __restrict__ part, int nblk,
                                                               double* __restrict__ sums) {
  __shared__ double red[NQ][kThreads];
  const int c = blockIdx.x, t = threadIdx.x;
  double a[NQ];
#pragma unroll
  for (int q = 0; q < NQ; ++q) a[q] = 0.0;
  for (int b = t; b < nblk; b += kThreads)
#pragma unroll
    for (int q = 0; q < NQ; ++q) a[q] += part[((int64_t)c * nblk + b) * NQ + q];
#pragma unroll
  for (int q = 0; q < NQ; ++q) red[q][t] = a[q];
  __syncthreads();
  for (int w = kThreads / 2; w >= 1; w >>= 1) {
    if (t < w)
#pragma unroll
      for (int q = 0; q < NQ; ++q) red[q][t] += red[q][t + w];
    __syncthreads();
  }
  if (t < NQ) sums[(int64_t)c * NQ + t] = red[t][0];
}

__device__ __forceinline__ int entry_of(const FieldTab& f, int field) {
  int e = 0;
  while (e + 1 < f.n && field >= f.f0[e + 1]) ++e;
  return e;
}

// Per-channel coefficients (A, B, M, C) from the sums of each field:
//   forward  y  = A (x - M)
//   backward dx = A g + B (x - M) + C
// l = 0: M = mean, A = r = 1/sqrt(var + eps); backward B = -r^2 mean(g xh), C = -r mean(g) with
//        xh = (x - M) r  (the gradient of Eq. 11 through mean and variance);
// l > 0: M = 0, A = r = 1/sqrt(nu + eps), nu = mean |f|^2; backward B = -(r^3 / n) sum(g . f), C = 0.
template <int NQ>
__global__ void norm_coef_kernel(FieldTab f, const double* __restrict__ sums, int64_t n, double eps,
                                 float4* __restrict__ coef) {
  const int n_fields = f.f0[f.n];
  const double inv_n = 1.0 / (double)n;
  for (int field = blockIdx.x * blockDim.x + threadIdx.x; field < n_fields; field += gridDim.x * blockDim.x) {
    const int e = entry_of(f, field), l = f.l[e], d = 2 * l + 1;
    const int c0 = f.ch0[e] + (field - f.f0[e]) * d;
    if (l == 0) {
      const double* S = sums + (int64_t)c0 * NQ;
      const double mean = S[0] * inv_n;
      const double var = fmax(S[1] * inv_n - mean * mean, 0.0);
      const double r = 1.0 / sqrt(var + eps);
      float4 k = make_float4((float)r, 0.f, (float)mean, 0.f);
      if (NQ == 4) {
        const double mg = S[2] * inv_n;
        const double mgxh = r * (S[3] * inv_n - mean * mg);
        k.y = (float)(-r * r * mgxh);
        k.w = (float)(-r * mg);
      }
      coef[c0] = k;
    } else {
      double nu = 0.0, sgf = 0.0;
      for (int c = 0; c < d; ++c) {
        nu += sums[(int64_t)(c0 + c) * NQ + 1];
        if (NQ == 4) sgf += sums[(int64_t)(c0 + c) * NQ + 3];
      }
      const double r = 1.0 / sqrt(nu * inv_n + eps);
      const float B = NQ == 4 ? (float)(-(r * r * r * inv_n) * sgf) : 0.f;
      for (int c = 0; c < d; ++c) coef[c0 + c] = make_float4((float)r, B, 0.f, 0.f);
    }
  }
}

// Elementwise pass over rows [b*rpb, ...): VEC consecutive channels of one row per access
// (C % VEC == 0).  kBwd: dx = A g + B (x - M) + C; else y = A (x - M).  The output may alias x
// (and g) element for element.
template <typename T, int VEC, bool kBwd>
__global__ __launch_bounds__(kThreads) void norm_apply_kernel(const T* x, const T* g, int64_t n, int C, int64_t rpb,
                                                              const float4* __restrict__ coef, T* y) {
  const int64_t r0 = (int64_t)blockIdx.x * rpb;
  const int64_t r1 = min(n, r0 + rpb);
  if (r0 >= r1) return;
  const int64_t base = r0 * C;
  const int nv = (int)((r1 - r0) * C / VEC);
  for (int v = threadIdx.x; v < nv; v += kThreads) {
    const int e = v * VEC;
    const int c = e % C;
    const Vec<T, VEC> xv = vload<T, VEC>(x + base + e);
    Vec<T, VEC> gv;
    if (kBwd) gv = vload<T, VEC>(g + base + e);
    Vec<T, VEC> out;
#pragma unroll
    for (int k = 0; k < VEC; ++k) {
      const float4 q = coef[c + k];
      const float xm = DT<T>::to_f(xv.e[k]) - q.z;
      const float r = kBwd ? fmaf(q.x, DT<T>::to_f(gv.e[k]), fmaf(q.y, xm, q.w)) : q.x * xm;
      out.e[k] = DT<T>::from_f(r);
    }
    vstore<T, VEC>(y + base + e, out);
  }
}

// Channel-stationary vector layout (C % VEC == 0, nv = C / VEC <= 256): thread t < G * nv
// (G = 256 / nv row groups) owns the VEC channels v * VEC .. of vector v = t % nv in rows
// r0 + t / nv + k G, so its coefficients and sums stay in registers and every access is 16 bytes.
template <typename T, int VEC>
struct VecIO {
  static __device__ __forceinline__ void load(const T* p, float* f) {
    const Vec<T, VEC> a = vload<T, VEC>(p);
#pragma unroll
    for (int k = 0; k < VEC; ++k) f[k] = DT<T>::to_f(a.e[k]);
  }
  static __device__ __forceinline__ void store(T* p, const float* f) {
    Vec<T, VEC> a;
#pragma unroll
    for (int k = 0; k < VEC; ++k) a.e[k] = DT<T>::from_f(f[k]);
    vstore<T, VEC>(p, a);
  }
};

// Channel sums as norm_sums_kernel, in the vector layout: rows added in row order per thread,
// four rows' loads issued together; the G groups then added in group order.
template <typename T, int VEC, int NQ>
__global__ __launch_bounds__(kThreads) void norm_sums_vec_kernel(const T* __restrict__ x, const T* __restrict__ g,
                                                                 int64_t n, int C, int G, int64_t rpb,
                                                                 double* __restrict__ part) {
  __shared__ double red[VEC][kThreads];
  const int nv = C / VEC, t = threadIdx.x, v = t % nv, grp = t / nv, nblk = gridDim.x;
  const int64_t r0 = (int64_t)blockIdx.x * rpb;
  const int64_t r1 = min(n, r0 + rpb);
  double acc[NQ][VEC];
#pragma unroll
  for (int q = 0; q < NQ; ++q)
#pragma unroll
    for (int k = 0; k < VEC; ++k) acc[q][k] = 0.0;
  if (grp < G) {
    const int64_t c0 = (int64_t)v * VEC;
    int64_t r = r0 + grp;
    for (; r + 3 * (int64_t)G < r1; r += 4 * (int64_t)G) {
      float xv[4][VEC], gv[4][VEC];
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        VecIO<T, VEC>::load(x + (r + i * (int64_t)G) * C + c0, xv[i]);
        if (NQ == 4) VecIO<T, VEC>::load(g + (r + i * (int64_t)G) * C + c0, gv[i]);
      }
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int k = 0; k < VEC; ++k) {
          const double dv = xv[i][k];
          acc[0][k] += dv;
          acc[1][k] = fma(dv, dv, acc[1][k]);
          if (NQ == 4) {
            const double dw = gv[i][k];
            acc[2][k] += dw;
            acc[3][k] = fma(dw, dv, acc[3][k]);
          }
        }
    }
    for (; r < r1; r += G) {
      float xv[VEC], gv[VEC];
      VecIO<T, VEC>::load(x + r * C + c0, xv);
      if (NQ == 4) VecIO<T, VEC>::load(g + r * C + c0, gv);
#pragma unroll
      for (int k = 0; k < VEC; ++k) {
        const double dv = xv[k];
        acc[0][k] += dv;
        acc[1][k] = fma(dv, dv, acc[1][k]);
        if (NQ == 4) {
          const double dw = gv[k];
          acc[2][k] += dw;
          acc[3][k] = fma(dw, dv, acc[3][k]);
        }
      }
    }
  }
#pragma unroll
  for (int q = 0; q < NQ; ++q) {
#pragma unroll
    for (int k = 0; k < VEC; ++k) red[k][t] = acc[q][k];
    __syncthreads();
    for (int e = t; e < C; e += kThreads) {
      const int vv = e / VEC, k = e % VEC;
      double sum = 0.0;
      for (int j = 0; j < G; ++j) sum += red[k][j * nv + vv];
      part[((int64_t)e * nblk + blockIdx.x) * NQ + q] = sum;
    }
    __syncthreads();
  }
}

// The elementwise pass in the vector layout, each thread's coefficients loaded once.  The output
// may alias x (and g) element for element.
template <typename T, int VEC, bool kBwd>
__global__ __launch_bounds__(kThreads) void norm_apply_vec_kernel(const T* x, const T* g, int64_t n, int C, int G,
                                                                  int64_t rpb, const float4* __restrict__ coef,
                                                                  T* y) {
  const int nv = C / VEC, t = threadIdx.x, v = t % nv, grp = t / nv;
  if (grp >= G) return;
  const int64_t c0 = (int64_t)v * VEC;
  float4 q[VEC];
#pragma unroll
  for (int k = 0; k < VEC; ++k) q[k] = coef[c0 + k];
  const int64_t r0 = (int64_t)blockIdx.x * rpb;
  const int64_t r1 = min(n, r0 + rpb);
  int64_t r = r0 + grp;
  for (; r + 3 * (int64_t)G < r1; r += 4 * (int64_t)G) {
    float xv[4][VEC], gv[4][VEC];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      VecIO<T, VEC>::load(x + (r + i * (int64_t)G) * C + c0, xv[i]);
      if (kBwd) VecIO<T, VEC>::load(g + (r + i * (int64_t)G) * C + c0, gv[i]);
    }
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      float o[VEC];
#pragma unroll
      for (int k = 0; k < VEC; ++k) {
        const float xm = xv[i][k] - q[k].z;
        o[k] = kBwd ? fmaf(q[k].x, gv[i][k], fmaf(q[k].y, xm, q[k].w)) : q[k].x * xm;
      }
      VecIO<T, VEC>::store(y + (r + i * (int64_t)G) * C + c0, o);
    }
  }
  for (; r < r1; r += G) {
    float xv[VEC], gv[VEC], o[VEC];
    VecIO<T, VEC>::load(x + r * C + c0, xv);
    if (kBwd) VecIO<T, VEC>::load(g + r * C + c0, gv);
#pragma unroll
    for (int k = 0; k < VEC; ++k) {
      const float xm = xv[k] - q[k].z;
      o[k] = kBwd ? fmaf(q[k].x, gv[k], fmaf(q[k].y, xm, q[k].w)) : q[k].x * xm;
    }
    VecIO<T, VEC>::store(y + r * C + c0, o);
  }
}

struct NormPlan {
  int C, G, NC, nblk;
  int64_t rpb;
};

// The vector layout where it applies: VEC elements of 16 bytes, nv = C / VEC <= 256 (else the
// scalar layout of norm_sums_kernel / norm_apply_kernel).
template <typename T>
bool vec_layout(int C, const void* a, const void* b, const void* c) {
  constexpr int V = 16 / sizeof(T);
  return C % V == 0 && C / V <= kThreads && aligned16(a) && (!b || aligned16(b)) && (!c || aligned16(c));
}

// Row blocks of the vector-layout sums: at least four row steps of each thread, at most
// kMaxVecBlocks blocks.
constexpr int kMaxVecBlocks = 1024;
template <typename T>
NormPlan norm_vec_plan(int64_t n, int C) {
  constexpr int V = 16 / sizeof(T);
  NormPlan p;
  p.C = C;
  p.NC = 1;
  p.G = kThreads / (C / V);
  const int64_t want = (n + 4 * (int64_t)p.G - 1) / (4 * (int64_t)p.G);
  p.nblk = (int)std::max<int64_t>(1, std::min<int64_t>(kMaxVecBlocks, want));
  p.rpb = (n + p.nblk - 1) / p.nblk;
  p.nblk = (int)((n + p.rpb - 1) / p.rpb);
  return p;
}

NormPlan norm_plan(int64_t n, int C) {
  NormPlan p;
  p.C = C;
  p.NC = (C + kThreads - 1) / kThreads;
  p.G = p.NC == 1 ? kThreads / C : 1;
  // at least 16 row steps of each thread per block, at most kMaxBlocks blocks
  const int64_t want = (n + 16 * (int64_t)p.G - 1) / (16 * (int64_t)p.G);
  p.nblk = (int)std::max<int64_t>(1, std::min<int64_t>(kMaxBlocks, want));
  p.rpb = (n + p.nblk - 1) / p.nblk;
  p.nblk = (int)((n + p.rpb - 1) / p.rpb);
  return p;
}

template <typename T, bool kBwd>
int launch_apply(const void* x, const void* g, int64_t n, int C, const float4* coef, void* y, hipStream_t st) {
  constexpr int V = 16 / sizeof(T);
  if (vec_layout<T>(C, x, kBwd ? g : nullptr, y)) {
    // four row steps of each thread per block
    const int G = kThreads / (C / V);
    const int64_t rpb = 4 * (int64_t)G;
    norm_apply_vec_kernel<T, V, kBwd><<<cdiv(n, rpb), kThreads, 0, st>>>((const T*)x, (const T*)g, n, C, G, rpb, coef,
                                                                          (T*)y);
    SSC_HIP(hipGetLastError());
    return SSCONV_OK;
  }
  // rows per block: about 4096 elements per workgroup
  const int64_t rpb = std::max<int64_t>(1, 4096 / C);
  const unsigned nb = cdiv(n, rpb);
  const bool vec = C % V == 0 && aligned16(x) && aligned16(y) && (!kBwd || aligned16(g));
  if (vec)
    norm_apply_kernel<T, V, kBwd><<<nb, kThreads, 0, st>>>((const T*)x, (const T*)g, n, C, rpb, coef, (T*)y);
  else
    norm_apply_kernel<T, 1, kBwd><<<nb, kThreads, 0, st>>>((const T*)x, (const T*)g, n, C, rpb, coef, (T*)y);
  SSC_HIP(hipGetLastError());
  return SSCONV_OK;
}

template <typename T, int NQ>
int norm_run(const FieldTab& f, const void* x, const void* g, int64_t n, double eps, void* y, hipStream_t st) {
  const int C = f.ch0[f.n];
  const bool vec = vec_layout<T>(C, x, NQ == 4 ? g : nullptr, nullptr);
  const NormPlan p = vec ? norm_vec_plan<T>(n, C) : norm_plan(n, C);
  const size_t part_b = ((size_t)C * p.nblk * NQ * 8 + 255) & ~(size_t)255;
  const size_t sums_b = ((size_t)C * NQ * 8 + 255) & ~(size_t)255;
  char* ws = nullptr;
  SSC_TRY(dev_alloc((void**)&ws, part_b + sums_b + (size_t)C * 16, st));
  double* part = (double*)ws;
  double* sums = (double*)(ws + part_b);
  float4* coef = (float4*)(ws + part_b + sums_b);
  if (vec)
    norm_sums_vec_kernel<T, 16 / sizeof(T), NQ><<<p.nblk, kThreads, 0, st>>>((const T*)x, (const T*)g, n, C, p.G,
                                                                             p.rpb, part);
  else
    norm_sums_kernel<T, NQ><<<p.nblk, kThreads, 0, st>>>((const T*)x, (const T*)g, n, C, p.G, p.NC, p.rpb, part);
  norm_reduce_kernel<NQ><<<C, kThreads, 0, st>>>(part, p.nblk, sums);
  const int n_fields = f.f0[f.n];
  norm_coef_kernel<NQ><<<cdiv(n_fields, 64), 64, 0, st>>>(f, sums, n, eps, coef);
  int rc = SSCONV_OK;
  if (hipGetLastError() != hipSuccess) rc = fail(SSCONV_E_HIP, "norm statistics launch failed");
  if (rc == SSCONV_OK) rc = launch_apply<T, NQ == 4>(x, g, n, C, coef, y, st);
  dev_free(ws, st);
  return rc;
}

}  // namespace

NormStatsPlan norm_stats_plan(ssconv_dtype dt, const void* y, int64_t n, int C) {
  const bool vec = dt == SSCONV_F32 ? vec_layout<float>(C, y, nullptr, nullptr)
                                    : vec_layout<uint16_t>(C, y, nullptr, nullptr);
  const NormPlan q = !vec ? norm_plan(n, C) : dt == SSCONV_F32 ? norm_vec_plan<float>(n, C)
                                                               : norm_vec_plan<uint16_t>(n, C);
  NormStatsPlan p;
  p.C = q.C, p.G = q.G, p.NC = q.NC, p.nblk = q.nblk, p.rpb = q.rpb, p.vec = vec;
  return p;
}

static size_t up256(size_t b) { return (b + 255) & ~(size_t)255; }

size_t norm_ws_bytes(int C, int64_t nblk) {
  return up256((size_t)C * nblk * 2 * 8) + up256((size_t)C * 2 * 8) + (size_t)C * 16;
}

int norm_sink_take(NormSink* s, int64_t nblk, hipStream_t st) {
  void* p = nullptr;
  SSC_TRY(scratch_take(s->sc, &p, norm_ws_bytes(s->C, nblk), st));
  s->ws = (char*)p;
  s->nblk = nblk;
  return SSCONV_OK;
}

int norm_forward_sums(ssconv_dtype dt, const void* y, int64_t n, const NormStatsPlan& p, char* ws, hipStream_t st) {
  double* part = (double*)ws;
  if (p.vec && dt == SSCONV_F32)
    norm_sums_vec_kernel<float, 4, 2><<<p.nblk, kThreads, 0, st>>>((const float*)y, nullptr, n, p.C, p.G, p.rpb, part);
  else if (p.vec)
    norm_sums_vec_kernel<uint16_t, 8, 2><<<p.nblk, kThreads, 0, st>>>((const uint16_t*)y, nullptr, n, p.C, p.G, p.rpb,
                                                                     part);
  else if (dt == SSCONV_F32)
    norm_sums_kernel<float, 2><<<p.nblk, kThreads, 0, st>>>((const float*)y, nullptr, n, p.C, p.G, p.NC, p.rpb, part);
  else
    norm_sums_kernel<uint16_t, 2><<<p.nblk, kThreads, 0, st>>>((const uint16_t*)y, nullptr, n, p.C, p.G, p.NC, p.rpb,
                                                               part);
  SSC_HIP(hipGetLastError());
  return SSCONV_OK;
}

int norm_forward_finish(const FieldTab& f, ssconv_dtype dt, const void* y, int64_t n, double eps, int64_t nblk,
                        char* ws, void* z, hipStream_t st) {
  const int C = f.ch0[f.n];
  const size_t part_b = up256((size_t)C * nblk * 2 * 8), sums_b = up256((size_t)C * 2 * 8);
  double* part = (double*)ws;
  double* sums = (double*)(ws + part_b);
  float4* coef = (float4*)(ws + part_b + sums_b);
  norm_reduce_kernel<2><<<C, kThreads, 0, st>>>(part, (int)nblk, sums);
  norm_coef_kernel<2><<<cdiv(f.f0[f.n], 64), 64, 0, st>>>(f, sums, n, eps, coef);
  SSC_HIP(hipGetLastError());
  return dt == SSCONV_F32 ? launch_apply<float, false>(y, nullptr, n, C, coef, z, st)
                          : launch_apply<uint16_t, false>(y, nullptr, n, C, coef, z, st);
}

namespace {

// ---------------------------------------------------------------------------------------------
// Pooling
// ---------------------------------------------------------------------------------------------

// Thread per (output row, VEC channels): out = (sum of the window's members in offset order) / 8.
template <typename T, int VEC>
__global__ __launch_bounds__(kThreads) void pool_fwd_kernel(const T* __restrict__ x, int C,
                                                            const int32_t* __restrict__ nbr, int64_t n_out,
                                                            T* __restrict__ y) {
  const int nv = C / VEC;
  const int64_t i = (int64_t)blockIdx.x * kThreads + threadIdx.x;
  if (i >= n_out * nv) return;
  const int64_t o = i / nv;
  const int v = (int)(i - o * nv);
  int32_t m[8];
#pragma unroll
  for (int s = 0; s < 8; ++s) m[s] = nbr[(int64_t)s * n_out + o];
  float acc[VEC];
#pragma unroll
  for (int k = 0; k < VEC; ++k) acc[k] = 0.f;
#pragma unroll
  for (int s = 0; s < 8; ++s) {
    if (m[s] < 0) continue;
    const Vec<T, VEC> a = vload<T, VEC>(x + (int64_t)m[s] * C + v * VEC);
#pragma unroll
    for (int k = 0; k < VEC; ++k) acc[k] += DT<T>::to_f(a.e[k]);
  }
  Vec<T, VEC> out;
#pragma unroll
  for (int k = 0; k < VEC; ++k) out.e[k] = DT<T>::from_f(acc[k] * 0.125f);
  vstore<T, VEC>(y + o * C + v * VEC, out);
}

// Thread per (output row, VEC channels): every member of the window receives grad_out / 8.
template <typename T, int VEC>
__global__ __launch_bounds__(kThreads) void pool_bwd_kernel(const T* __restrict__ dy, int C,
                                                            const int32_t* __restrict__ nbr, int64_t n_out,
                                                            T* __restrict__ dx) {
  const int nv = C / VEC;
  const int64_t i = (int64_t)blockIdx.x * kThreads + threadIdx.x;
  if (i >= n_out * nv) return;
  const int64_t o = i / nv;
  const int v = (int)(i - o * nv);
  const Vec<T, VEC> a = vload<T, VEC>(dy + o * C + v * VEC);
  Vec<T, VEC> out;
#pragma unroll
  for (int k = 0; k < VEC; ++k) out.e[k] = DT<T>::from_f(DT<T>::to_f(a.e[k]) * 0.125f);
#pragma unroll
  for (int s = 0; s < 8; ++s) {
    const int32_t m = nbr[(int64_t)s * n_out + o];
    if (m >= 0) vstore<T, VEC>(dx + (int64_t)m * C + v * VEC, out);
  }
}

template <typename T, bool kBwd>
int pool_run(const void* src, int C, const ssconv_rulebook* rb, void* dst, hipStream_t st) {
  constexpr int V = 16 / sizeof(T);
  const bool vec = C % V == 0 && aligned16(src) && aligned16(dst);
  const int vw = vec ? V : 1;
  const int64_t items = rb->n_out * (int64_t)(C / vw);
  const unsigned nb = cdiv(items, kThreads);
  if (kBwd) {
    if (vec)
      pool_bwd_kernel<T, V><<<nb, kThreads, 0, st>>>((const T*)src, C, rb->nbr, rb->n_out, (T*)dst);
    else
      pool_bwd_kernel<T, 1><<<nb, kThreads, 0, st>>>((const T*)src, C, rb->nbr, rb->n_out, (T*)dst);
  } else {
    if (vec)
      pool_fwd_kernel<T, V><<<nb, kThreads, 0, st>>>((const T*)src, C, rb->nbr, rb->n_out, (T*)dst);
    else
      pool_fwd_kernel<T, 1><<<nb, kThreads, 0, st>>>((const T*)src, C, rb->nbr, rb->n_out, (T*)dst);
  }
  SSC_HIP(hipGetLastError());
  return SSCONV_OK;
}

int check_pool(ssconv_dtype dt, int C, ssconv_rulebook_t rb, const void* a, const void* b) {
  if (dt != SSCONV_F32 && dt != SSCONV_BF16) return fail(SSCONV_E_DTYPE, "unsupported dtype %d", (int)dt);
  if (!rb) return fail(SSCONV_E_INVALID, "NULL rule book");
  SSC_TRY(rulebook_settle(rb));
  if (rb->ksize != 2 || rb->stride != 2)
    return fail(SSCONV_E_INVALID, "pooling needs a rule book built with ksize 2, stride 2");
  if (C < 1) return fail(SSCONV_E_INVALID, "channels must be positive");
  if ((rb->n_in > 0 && !a) || (rb->n_out > 0 && !b)) return fail(SSCONV_E_INVALID, "NULL feature buffer");
  if ((int64_t)C * std::max(rb->n_in, rb->n_out) >= ((int64_t)1 << 40))
    return fail(SSCONV_E_INVALID, "feature matrix too large");
  return SSCONV_OK;
}

int check_norm(const ssconv_fields* fields, ssconv_dtype dt, int64_t n, double eps, FieldTab* f) {
  if (dt != SSCONV_F32 && dt != SSCONV_BF16) return fail(SSCONV_E_DTYPE, "unsupported dtype %d", (int)dt);
  if (n < 0) return fail(SSCONV_E_INVALID, "n must be >= 0");
  if (!(eps > 0.0)) return fail(SSCONV_E_INVALID, "eps must be positive");
  SSC_TRY(make_fieldtab(fields, f));
  const int C = f->ch0[f->n];
  if (C < 1 || C > kMaxChannels) return fail(SSCONV_E_INVALID, "norm supports 1..%d channels (got %d)", kMaxChannels, C);
  if (n * (int64_t)C >= ((int64_t)1 << 40)) return fail(SSCONV_E_INVALID, "feature matrix too large");
  return SSCONV_OK;
}

}  // namespace

int norm_check_fields(const ssconv_fields* fields, ssconv_dtype dt, int64_t n, double eps, FieldTab* f) {
  return check_norm(fields, dt, n, eps, f);
}

}  // namespace ssconv

using namespace ssconv;

extern "C" int ssconv_norm_forward(const ssconv_fields* fields, const void* x, ssconv_dtype dtype, int64_t n,
                                   double eps, void* y, hipStream_t stream) {
  FieldTab f;
  SSC_TRY(check_norm(fields, dtype, n, eps, &f));
  if (n == 0) return SSCONV_OK;
  if (!x || !y) return fail(SSCONV_E_INVALID, "NULL feature buffer");
  if (dtype == SSCONV_F32) return norm_run<float, 2>(f, x, nullptr, n, eps, y, stream);
  return norm_run<uint16_t, 2>(f, x, nullptr, n, eps, y, stream);
}

extern "C" int ssconv_norm_backward(const ssconv_fields* fields, const void* x, const void* dy, ssconv_dtype dtype,
                                    int64_t n, double eps, void* dx, hipStream_t stream) {
  FieldTab f;
  SSC_TRY(check_norm(fields, dtype, n, eps, &f));
  if (n == 0) return SSCONV_OK;
  if (!x || !dy || !dx) return fail(SSCONV_E_INVALID, "NULL feature buffer");
  if (dtype == SSCONV_F32) return norm_run<float, 4>(f, x, dy, n, eps, dx, stream);
  return norm_run<uint16_t, 4>(f, x, dy, n, eps, dx, stream);
}

extern "C" int ssconv_pool_forward(const void* feats, ssconv_dtype dtype, int channels, ssconv_rulebook_t rb,
                                   void* out, hipStream_t stream) {
  SSC_TRY(check_pool(dtype, channels, rb, feats, out));
  if (rb->n_out == 0) return SSCONV_OK;
  if (dtype == SSCONV_F32) return pool_run<float, false>(feats, channels, rb, out, stream);
  return pool_run<uint16_t, false>(feats, channels, rb, out, stream);
}

extern "C" int ssconv_pool_backward(const void* grad_out, ssconv_dtype dtype, int channels, ssconv_rulebook_t rb,
                                    void* grad_feats, hipStream_t stream) {
  SSC_TRY(check_pool(dtype, channels, rb, grad_feats, grad_out));
  if (rb->n_out == 0) return SSCONV_OK;
  if (dtype == SSCONV_F32) return pool_run<float, true>(grad_out, channels, rb, grad_feats, stream);
  return pool_run<uint16_t, true>(grad_out, channels, rb, grad_feats, stream);
}
