// Kernel synthesis (Sec. 3.2.1, Eq. 7 with the block matrix of Eq. 9) and its adjoint.
//
// W[s][o][i] = sum_q w[off(field(o), field(i)) + q] * B^{k l}_q[s][a][b], one thread per
// element of W so the dominant cost -- writing W -- is a coalesced stream.
// The adjoint dw[off + q] = sum_{s,a,b} dW[s][o][i] B_q[s][a][b] uses one
// workgroup per (out field, in field) pair with a fixed reduction order; dW comes
// field-pair-blocked (dw_block_pos), so a pair's values are one contiguous run.
#include "synth.hpp"

namespace ssconv {

int make_synth_args(const ssconv_basis_desc* d, SynthArgs* a) {
  int nq[SSCONV_MAX_L + 1][SSCONV_MAX_L + 1];
  int64_t base[SSCONV_MAX_L + 1][SSCONV_MAX_L + 1];
  int64_t floats = 0;
  SSC_TRY(basis_nq_table(d, nq, base, &floats));
  SSC_TRY(make_fieldtab(&d->in, &a->in));
  SSC_TRY(make_fieldtab(&d->out, &a->out));
  a->K = d->ksize * d->ksize * d->ksize;
  a->cin = a->in.ch0[a->in.n];
  a->cout = a->out.ch0[a->out.n];
  for (int k = 0; k <= SSCONV_MAX_L; ++k) {
    int64_t r = 0;
    for (int e = 0; e < a->in.n; ++e) r += (int64_t)a->in.mult[e] * nq[k][a->in.l[e]];
    a->rowsz[k] = r;
    for (int l = 0; l <= SSCONV_MAX_L; ++l) {
      a->nq[k][l] = nq[k][l];
      a->base[k][l] = base[k][l];
    }
  }
  // coefficient offset of the first field of every out entry
  int64_t off = 0;
  for (int e = 0; e < a->out.n; ++e) {
    a->row0[e] = off;
    off += (int64_t)a->out.mult[e] * a->rowsz[a->out.l[e]];
  }
  a->n_coeff = off;
  a->n_out_fields = a->out.f0[a->out.n];
  a->n_in_fields = a->in.f0[a->in.n];
  return SSCONV_OK;
}

namespace {

struct ChanInfo {
  int entry, field, comp, l;
};

__device__ __forceinline__ ChanInfo chan_info(const FieldTab& t, int c) {
  int e = 0;
  while (e + 1 < t.n && c >= t.ch0[e + 1]) ++e;
  const int d = 2 * t.l[e] + 1, r = c - t.ch0[e];
  return ChanInfo{e, r / d, r % d, t.l[e]};
}

// Offset of the first coefficient of the (out field (eo, fo), in field (ei, fi)) block.
__device__ __forceinline__ int64_t coeff_off(const SynthArgs& a, int eo, int fo, int k, int ei, int fi) {
  int64_t off = a.row0[eo] + (int64_t)fo * a.rowsz[k];
  for (int e = 0; e < ei; ++e) off += (int64_t)a.in.mult[e] * a.nq[k][a.in.l[e]];
  return off + (int64_t)fi * a.nq[k][a.in.l[ei]];
}

// Loads of the coefficients and basis values of one element are issued kQL at a time with no
// dependence between them, so an element costs one memory round trip per kQL basis functions.
constexpr int kQL = 8;

// grid (ceil(cout * cin / 256), K): the workgroup row is one offset s, so the element index fits
// in 32 bits and the (out, in) channel split is one 32-bit division.
template <typename T>
__global__ __launch_bounds__(256) void synth_kernel(SynthArgs a, const float* __restrict__ basis,
                                                    const float* __restrict__ coeffs, T* __restrict__ W) {
  const int plane = a.cout * a.cin;
  const int idx = blockIdx.x * 256 + threadIdx.x;
  if (idx >= plane) return;
  const int s = blockIdx.y;
  const int co = idx / a.cin, ci = idx - co * a.cin;
  const ChanInfo o = chan_info(a.out, co), i = chan_info(a.in, ci);
  const int k = o.l, l = i.l, dk = 2 * k + 1, dl = 2 * l + 1;
  const int nq = a.nq[k][l];
  const float* cp = coeffs + coeff_off(a, o.entry, o.field, k, i.entry, i.field);
  const float* bp = basis + a.base[k][l] + ((int64_t)s * dk + o.comp) * dl + i.comp;
  const int64_t qstride = (int64_t)a.K * dk * dl;
  float acc = 0.f;
  for (int q0 = 0; q0 < nq; q0 += kQL) {
    float cv[kQL], bv[kQL];
#pragma unroll
    for (int j = 0; j < kQL; ++j) {
      const bool ok = q0 + j < nq;
      cv[j] = ok ? cp[q0 + j] : 0.f;
      bv[j] = ok ? bp[(q0 + j) * qstride] : 0.f;
    }
#pragma unroll
    for (int j = 0; j < kQL; ++j)
      if (q0 + j < nq) acc = fmaf(cv[j], bv[j], acc);
  }
  W[(int64_t)s * plane + idx] = DT<T>::from_f(acc);
}

// One workgroup per (in field, out field) pair; its coefficients are done 16 at a time in
// registers: thread partial sums over the block's elements in a fixed order, a fixed butterfly
// within each wavefront, then the four wavefront sums added in order (independent of scheduling).
constexpr int kQB = 16;  // coefficients per pass (every (k, l) block of the workloads fits one pass)
constexpr int kEU = 4;   // elements per thread per step, their loads issued together

__global__ __launch_bounds__(256) void synth_adjoint_kernel(SynthArgs a, const float* __restrict__ basis,
                                                            const float* __restrict__ dW, float* __restrict__ dcoef) {
  __shared__ float red[4][kQB];
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int fi_all = blockIdx.x, fo_all = blockIdx.y;
  int eo = 0, ei = 0;
  while (eo + 1 < a.out.n && fo_all >= a.out.f0[eo + 1]) ++eo;
  while (ei + 1 < a.in.n && fi_all >= a.in.f0[ei + 1]) ++ei;
  const int fo = fo_all - a.out.f0[eo], fi = fi_all - a.in.f0[ei];
  const int k = a.out.l[eo], l = a.in.l[ei], dk = 2 * k + 1, dl = 2 * l + 1;
  const int nq = a.nq[k][l];
  if (nq == 0) return;  // uniform per workgroup
  const int ro = a.out.ch0[eo] + fo * dk, cc = a.in.ch0[ei] + fi * dl;
  const int64_t off = coeff_off(a, eo, fo, k, ei, fi);
  const int n = a.K * dk * dl;
  const int64_t qstride = (int64_t)a.K * dk * dl;
  const float* bp = basis + a.base[k][l];
  const int64_t blk = (int64_t)a.K * ((int64_t)ro * a.cin + (int64_t)dk * cc);  // dW is field-pair-blocked
  for (int q0 = 0; q0 < nq; q0 += kQB) {
    float acc[kQB];
#pragma unroll
    for (int j = 0; j < kQB; ++j) acc[j] = 0.f;
    for (int e0 = threadIdx.x; e0 < n; e0 += 256 * kEU) {
      float g[kEU], bv[kEU][kQB];
#pragma unroll
      for (int u = 0; u < kEU; ++u) {
        const int e = e0 + u * 256;
        const bool ok = e < n;
        g[u] = ok ? dW[blk + e] : 0.f;
#pragma unroll
        for (int j = 0; j < kQB; ++j) bv[u][j] = (ok && q0 + j < nq) ? bp[(q0 + j) * qstride + e] : 0.f;
      }
#pragma unroll
      for (int u = 0; u < kEU; ++u)
#pragma unroll
        for (int j = 0; j < kQB; ++j) acc[j] = fmaf(g[u], bv[u][j], acc[j]);
    }
#pragma unroll
    for (int j = 0; j < kQB; ++j) {
      if (q0 + j >= nq) break;  // uniform per workgroup: no butterflies for absent coefficients
      float v = acc[j];
#pragma unroll
      for (int m = 32; m >= 1; m >>= 1) v += __shfl_xor(v, m);
      if (lane == 0) red[w][j] = v;
    }
    __syncthreads();
    if (threadIdx.x < kQB && q0 + (int)threadIdx.x < nq) {
      const int j = threadIdx.x;
      dcoef[off + q0 + j] = ((red[0][j] + red[1][j]) + red[2][j]) + red[3][j];
    }
    __syncthreads();
  }
}

// The same sums with one wavefront per (out field, in field) pair, four pairs per workgroup, for
// small offset counts (a pair's K*(2k+1)*(2l+1) values are then at most a few hundred): four times
// as many pairs in flight per compute unit and no workgroup barrier.  Lane partial sums in element
// order, then the fixed butterfly.
__global__ __launch_bounds__(256) void synth_adjoint_wave_kernel(SynthArgs a, const float* __restrict__ basis,
                                                                 const float* __restrict__ dW,
                                                                 float* __restrict__ dcoef) {
  const int lane = threadIdx.x & 63;
  const int pair = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (pair >= a.n_in_fields * a.n_out_fields) return;  // uniform per wavefront
  const int fi_all = pair % a.n_in_fields, fo_all = pair / a.n_in_fields;
  int eo = 0, ei = 0;
  while (eo + 1 < a.out.n && fo_all >= a.out.f0[eo + 1]) ++eo;
  while (ei + 1 < a.in.n && fi_all >= a.in.f0[ei + 1]) ++ei;
  const int fo = fo_all - a.out.f0[eo], fi = fi_all - a.in.f0[ei];
  const int k = a.out.l[eo], l = a.in.l[ei], dk = 2 * k + 1, dl = 2 * l + 1;
  const int nq = a.nq[k][l];
  if (nq == 0) return;
  const int ro = a.out.ch0[eo] + fo * dk, cc = a.in.ch0[ei] + fi * dl;
  const int64_t off = coeff_off(a, eo, fo, k, ei, fi);
  const int n = a.K * dk * dl;
  const int64_t qstride = (int64_t)a.K * dk * dl;
  const float* bp = basis + a.base[k][l];
  const int64_t blk = (int64_t)a.K * ((int64_t)ro * a.cin + (int64_t)dk * cc);
  for (int q0 = 0; q0 < nq; q0 += kQB) {
    float acc[kQB];
#pragma unroll
    for (int j = 0; j < kQB; ++j) acc[j] = 0.f;
    for (int e0 = lane; e0 < n; e0 += 64 * kEU) {
      float g[kEU], bv[kEU][kQB];
#pragma unroll
      for (int u = 0; u < kEU; ++u) {
        const int e = e0 + u * 64;
        const bool ok = e < n;
        g[u] = ok ? dW[blk + e] : 0.f;
#pragma unroll
        for (int j = 0; j < kQB; ++j) bv[u][j] = (ok && q0 + j < nq) ? bp[(q0 + j) * qstride + e] : 0.f;
      }
#pragma unroll
      for (int u = 0; u < kEU; ++u)
#pragma unroll
        for (int j = 0; j < kQB; ++j) acc[j] = fmaf(g[u], bv[u][j], acc[j]);
    }
    float mine = 0.f;  // lane j keeps coefficient j's sum
#pragma unroll
    for (int j = 0; j < kQB; ++j) {
      if (q0 + j >= nq) break;  // uniform per wavefront: no butterflies for absent coefficients
      float v = acc[j];
#pragma unroll
      for (int m = 32; m >= 1; m >>= 1) v += __shfl_xor(v, m);
      if (lane == j) mine = v;
    }
    if (lane < kQB && q0 + lane < nq) dcoef[off + q0 + lane] = mine;
  }
}

}  // namespace

int launch_synth(const SynthArgs& a, const float* basis, const float* coeffs, ssconv_dtype dt, void* W,
                 hipStream_t st) {
  const int64_t plane = (int64_t)a.cout * a.cin;
  if (plane == 0 || a.K == 0) return SSCONV_OK;
  if (plane > 0x7fffffffll) return fail(SSCONV_E_INVALID, "Cout * Cin must be below 2^31");
  const dim3 g((unsigned)cdiv(plane, 256), (unsigned)a.K);
  if (dt == SSCONV_F32)
    synth_kernel<float><<<g, 256, 0, st>>>(a, basis, coeffs, (float*)W);
  else
    synth_kernel<uint16_t><<<g, 256, 0, st>>>(a, basis, coeffs, (uint16_t*)W);
  SSC_HIP(hipGetLastError());
  return SSCONV_OK;
}

int launch_synth_adjoint(const SynthArgs& a, const float* basis, const float* dW, float* dcoef, hipStream_t st) {
  if (a.n_coeff == 0) return SSCONV_OK;
  if (a.K <= 27) {
    const int64_t pairs = (int64_t)a.n_in_fields * a.n_out_fields;
    synth_adjoint_wave_kernel<<<(unsigned)cdiv(pairs, 4), 256, 0, st>>>(a, basis, dW, dcoef);
  } else {
    dim3 g(a.n_in_fields, a.n_out_fields);
    synth_adjoint_kernel<<<g, 256, 0, st>>>(a, basis, dW, dcoef);
  }
  SSC_HIP(hipGetLastError());
  return SSCONV_OK;
}

}  // namespace ssconv

using namespace ssconv;

extern "C" int ssconv_synth_kernel(const ssconv_basis_desc* desc, const float* basis, const float* coeffs,
                                   ssconv_dtype w_dtype, void* W, hipStream_t stream) {
  if (w_dtype != SSCONV_F32 && w_dtype != SSCONV_BF16) return fail(SSCONV_E_DTYPE, "unsupported W dtype");
  if (!basis || !coeffs || !W) return fail(SSCONV_E_INVALID, "NULL device pointer");
  SynthArgs a;
  SSC_TRY(make_synth_args(desc, &a));
  return launch_synth(a, basis, coeffs, w_dtype, W, stream);
}
