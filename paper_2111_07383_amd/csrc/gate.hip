// Gated nonlinearity (Sec. 3.3, Eq. 12): ReLU on scalar fields, Sigmoid(gate) * f on
// fields of order l > 0, the gate being an extra scalar channel of the producing
// convolution (one per l > 0 field, appended after the fields in field order).
// One thread per (site, field); elementwise and bandwidth-bound.
#include "common.hpp"

namespace ssconv {
namespace {

struct GateTab {
  FieldTab f;
  int gate0[SSCONV_MAX_ENTRIES];  // gate index of the first field of each entry (l > 0 entries)
  int C, G, n_fields;
};

__device__ __forceinline__ int find_entry(const FieldTab& t, int field) {
  int e = 0;
  while (e + 1 < t.n && field >= t.f0[e + 1]) ++e;
  return e;
}

__device__ __forceinline__ float sigmoidf(float x) { return 1.f / (1.f + __expf(-x)); }

template <typename T>
__global__ void gate_fwd_kernel(GateTab t, const T* __restrict__ x, int64_t n, T* __restrict__ y) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= n * t.n_fields) return;
  const int64_t row = i / t.n_fields;
  const int field = (int)(i % t.n_fields);
  const int e = find_entry(t.f, field), l = t.f.l[e], d = 2 * l + 1;
  const int c0 = t.f.ch0[e] + (field - t.f.f0[e]) * d;
  const T* xr = x + row * (t.C + t.G);
  T* yr = y + row * t.C;
  if (l == 0) {
    const float v = DT<T>::to_f(xr[c0]);
    yr[c0] = DT<T>::from_f(v > 0.f ? v : 0.f);
  } else {
    const float sg = sigmoidf(DT<T>::to_f(xr[t.C + t.gate0[e] + field - t.f.f0[e]]));
    for (int c = 0; c < d; ++c) yr[c0 + c] = DT<T>::from_f(sg * DT<T>::to_f(xr[c0 + c]));
  }
}

template <typename T>
__global__ void gate_bwd_kernel(GateTab t, const T* __restrict__ x, const T* __restrict__ dy, int64_t n,
                                T* __restrict__ dx) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= n * t.n_fields) return;
  const int64_t row = i / t.n_fields;
  const int field = (int)(i % t.n_fields);
  const int e = find_entry(t.f, field), l = t.f.l[e], d = 2 * l + 1;
  const int c0 = t.f.ch0[e] + (field - t.f.f0[e]) * d;
  const T* xr = x + row * (t.C + t.G);
  const T* dyr = dy + row * t.C;
  T* dxr = dx + row * (t.C + t.G);
  if (l == 0) {
    const float v = DT<T>::to_f(xr[c0]);
    dxr[c0] = DT<T>::from_f(v > 0.f ? DT<T>::to_f(dyr[c0]) : 0.f);
  } else {
    const int gc = t.C + t.gate0[e] + field - t.f.f0[e];
    const float sg = sigmoidf(DT<T>::to_f(xr[gc]));
    float dot = 0.f;
    for (int c = 0; c < d; ++c) {
      const float g = DT<T>::to_f(dyr[c0 + c]);
      dot = fmaf(g, DT<T>::to_f(xr[c0 + c]), dot);
      dxr[c0 + c] = DT<T>::from_f(g * sg);
    }
    dxr[gc] = DT<T>::from_f(dot * sg * (1.f - sg));
  }
}

int make_gatetab(const ssconv_fields* f, GateTab* t) {
  SSC_TRY(make_fieldtab(f, &t->f));
  t->C = t->f.ch0[t->f.n];
  t->n_fields = t->f.f0[t->f.n];
  int g = 0;
  for (int e = 0; e < t->f.n; ++e) {
    t->gate0[e] = g;
    if (t->f.l[e] > 0) g += t->f.mult[e];
  }
  t->G = g;
  return SSCONV_OK;
}

}  // namespace
}  // namespace ssconv

using namespace ssconv;

extern "C" int ssconv_gate_forward(const ssconv_fields* fields, const void* x, ssconv_dtype dtype, int64_t n, void* y,
                                   hipStream_t stream) {
  if (dtype != SSCONV_F32 && dtype != SSCONV_BF16) return fail(SSCONV_E_DTYPE, "unsupported dtype");
  if (n < 0 || (n > 0 && (!x || !y))) return fail(SSCONV_E_INVALID, "bad arguments");
  GateTab t;
  SSC_TRY(make_gatetab(fields, &t));
  const int64_t work = n * t.n_fields;
  if (work == 0) return SSCONV_OK;
  if (dtype == SSCONV_F32)
    gate_fwd_kernel<float><<<cdiv(work, 256), 256, 0, stream>>>(t, (const float*)x, n, (float*)y);
  else
    gate_fwd_kernel<uint16_t><<<cdiv(work, 256), 256, 0, stream>>>(t, (const uint16_t*)x, n, (uint16_t*)y);
  SSC_HIP(hipGetLastError());
  return SSCONV_OK;
}

extern "C" int ssconv_gate_backward(const ssconv_fields* fields, const void* x, const void* dy, ssconv_dtype dtype,
                                    int64_t n, void* dx, hipStream_t stream) {
  if (dtype != SSCONV_F32 && dtype != SSCONV_BF16) return fail(SSCONV_E_DTYPE, "unsupported dtype");
  if (n < 0 || (n > 0 && (!x || !dy || !dx))) return fail(SSCONV_E_INVALID, "bad arguments");
  GateTab t;
  SSC_TRY(make_gatetab(fields, &t));
  const int64_t work = n * t.n_fields;
  if (work == 0) return SSCONV_OK;
  if (dtype == SSCONV_F32)
    gate_bwd_kernel<float><<<cdiv(work, 256), 256, 0, stream>>>(t, (const float*)x, (const float*)dy, n, (float*)dx);
  else
    gate_bwd_kernel<uint16_t><<<cdiv(work, 256), 256, 0, stream>>>(t, (const uint16_t*)x, (const uint16_t*)dy, n,
                                                                  (uint16_t*)dx);
  SSC_HIP(hipGetLastError());
  return SSCONV_OK;
}
