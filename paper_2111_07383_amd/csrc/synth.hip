// Kernel synthesis (Sec. 3.2.1, Eq. 7 with the block matrix of Eq. 9) and its adjoint.
//
// W[s][o][i] = sum_q w[off(field(o), field(i)) + q] * B^{k l}_q[s][a][b], one wavefront per
// (out field, in field) block of W: the block's coefficients and table entries are the same for
// every lane (scalar loads), its K(2k+1)(2l+1) elements spread over the lanes.
// The adjoint dw[off + q] = sum_{s,a,b} dW[s][o][i] B_q[s][a][b] uses one wavefront (or one
// workgroup) per (out field, in field) pair with a fixed reduction order; dW comes
// field-pair-blocked (dw_block_pos), so a pair's values are one contiguous run.
#include <algorithm>

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
  for (int eo = 0; eo < a->out.n; ++eo) {
    const int k = a->out.l[eo];
    int64_t c0 = a->row0[eo];
    for (int ei = 0; ei < a->in.n; ++ei) {
      const int l = a->in.l[ei];
      if (a->rowsz[k] > 0x7fffffffll) return fail(SSCONV_E_INVALID, "coefficient row too long");
      a->ep[eo][ei] = EntryPair{c0, a->base[k][l], (int)a->rowsz[k], a->nq[k][l], k, l};
      c0 += (int64_t)a->in.mult[ei] * a->nq[k][l];
    }
  }
  a->n_out_fields = a->out.f0[a->out.n];
  a->n_in_fields = a->in.f0[a->in.n];
  return SSCONV_OK;
}

namespace {

// Entry holding field f (f0 ascends, entries past n hold the field count): counted over every
// table slot, so with f uniform across the wavefront the table is read by scalar loads.
__device__ __forceinline__ int field_entry(const FieldTab& t, int f) {
  int e = 0;
#pragma unroll
  for (int j = 1; j < SSCONV_MAX_ENTRIES; ++j) e += f >= t.f0[j];
  return e;
}

// Basis values of kSU elements are loaded kQL functions at a time with no dependence between
// them, so a lane's elements cost one memory round trip per kQL basis functions.
constexpr int kQL = 8;
constexpr int kSU = 4;

// nch wavefronts per (out field, in field) pair, four per workgroup: wavefront c of a pair takes
// the block's elements [c span, (c + 1) span) in (s, a, b) order (e = (s (2k+1) + a)(2l+1) + b,
// the basis layout; span a multiple of 64 kSU, nch span covering the layer's largest block), lane
// t the elements t, t + 64, ... of that chunk, kSU per pass, and writes W[s][ro + a][cc + b]; the
// sum over q runs in q order for every element.
template <typename T>
__global__ __launch_bounds__(256) void synth_kernel(SynthArgs a, const float* __restrict__ basis,
                                                    const float* __restrict__ coeffs, T* __restrict__ W, int nch,
                                                    int span) {
  const int lane = threadIdx.x & 63;
  const int wid = __builtin_amdgcn_readfirstlane(blockIdx.x * 4 + (threadIdx.x >> 6));
  const int pair = wid / nch, chunk = wid - pair * nch;
  if (pair >= a.n_in_fields * a.n_out_fields) return;  // uniform per wavefront
  const int fi_all = pair % a.n_in_fields, fo_all = pair / a.n_in_fields;
  const int eo = field_entry(a.out, fo_all), ei = field_entry(a.in, fi_all);
  const EntryPair& ep = a.ep[eo][ei];
  const int fo = fo_all - a.out.f0[eo], fi = fi_all - a.in.f0[ei];
  const int k = ep.k, l = ep.l, dk = 2 * k + 1, dl = 2 * l + 1, dkl = dk * dl;
  const int nq = ep.nq;
  const int ro = a.out.ch0[eo] + fo * dk, cc = a.in.ch0[ei] + fi * dl;
  const float* cp = coeffs + ep.coff0 + (int64_t)fo * ep.rowsz + (int64_t)fi * nq;
  const float* bp = basis + ep.base;
  const int n = a.K * dkl;
  const int64_t qstride = n;
  const int64_t plane = (int64_t)a.cout * a.cin;
  const int e_end = min(n, (chunk + 1) * span);
  for (int e0 = chunk * span + lane; e0 < e_end; e0 += 64 * kSU) {
    float acc[kSU];
#pragma unroll
    for (int u = 0; u < kSU; ++u) acc[u] = 0.f;
    for (int q0 = 0; q0 < nq; q0 += kQL) {
      float cv[kQL], bv[kSU][kQL];
#pragma unroll
      for (int j = 0; j < kQL; ++j) cv[j] = q0 + j < nq ? cp[q0 + j] : 0.f;
#pragma unroll
      for (int u = 0; u < kSU; ++u) {
        const int e = e0 + u * 64;
#pragma unroll
        for (int j = 0; j < kQL; ++j) bv[u][j] = (e < n && q0 + j < nq) ? bp[(q0 + j) * qstride + e] : 0.f;
      }
#pragma unroll
      for (int u = 0; u < kSU; ++u)
#pragma unroll
        for (int j = 0; j < kQL; ++j)
          if (q0 + j < nq) acc[u] = fmaf(cv[j], bv[u][j], acc[u]);
    }
#pragma unroll
    for (int u = 0; u < kSU; ++u) {
      const int e = e0 + u * 64;
      if (e >= n) break;
      const int s = e / dkl, r = e - s * dkl, ca = r / dl, cb = r - ca * dl;
      W[(int64_t)s * plane + (int64_t)(ro + ca) * a.cin + cc + cb] = DT<T>::from_f(acc[u]);
    }
  }
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
  const int eo = field_entry(a.out, fo_all), ei = field_entry(a.in, fi_all);
  const EntryPair& ep = a.ep[eo][ei];
  const int fo = fo_all - a.out.f0[eo], fi = fi_all - a.in.f0[ei];
  const int k = ep.k, l = ep.l, dk = 2 * k + 1, dl = 2 * l + 1;
  const int nq = ep.nq;
  if (nq == 0) return;  // uniform per workgroup
  const int ro = a.out.ch0[eo] + fo * dk, cc = a.in.ch0[ei] + fi * dl;
  const int64_t off = ep.coff0 + (int64_t)fo * ep.rowsz + (int64_t)fi * nq;
  const int n = a.K * dk * dl;
  const int64_t qstride = (int64_t)a.K * dk * dl;
  const float* bp = basis + ep.base;
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
      if (q0 + j < nq) {  // uniform per workgroup: no butterflies for absent coefficients
        float v = acc[j];
#pragma unroll
        for (int m = 32; m >= 1; m >>= 1) v += __shfl_xor(v, m);
        if (lane == 0) red[w][j] = v;
      }
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
// order, then the fixed butterfly.  Eight coefficients per pass (the 3^3 layers' blocks hold at most
// a few): 68 registers instead of 118 let seven wavefronts share a SIMD, so the 6400 pairs of a
// 208-channel layer fit one round of wavefront slots instead of two (15 us against 18).
constexpr int kQW = 8;
__global__ __launch_bounds__(256) void synth_adjoint_wave_kernel(SynthArgs a, const float* __restrict__ basis,
                                                                 const float* __restrict__ dW,
                                                                 float* __restrict__ dcoef) {
  const int lane = threadIdx.x & 63;
  const int pair = __builtin_amdgcn_readfirstlane(blockIdx.x * 4 + (threadIdx.x >> 6));
  if (pair >= a.n_in_fields * a.n_out_fields) return;  // uniform per wavefront
  const int fi_all = pair % a.n_in_fields, fo_all = pair / a.n_in_fields;
  const int eo = field_entry(a.out, fo_all), ei = field_entry(a.in, fi_all);
  const EntryPair& ep = a.ep[eo][ei];
  const int fo = fo_all - a.out.f0[eo], fi = fi_all - a.in.f0[ei];
  const int k = ep.k, l = ep.l, dk = 2 * k + 1, dl = 2 * l + 1;
  const int nq = ep.nq;
  if (nq == 0) return;
  const int ro = a.out.ch0[eo] + fo * dk, cc = a.in.ch0[ei] + fi * dl;
  const int64_t off = ep.coff0 + (int64_t)fo * ep.rowsz + (int64_t)fi * nq;
  const int n = a.K * dk * dl;
  const int64_t qstride = (int64_t)a.K * dk * dl;
  const float* bp = basis + ep.base;
  const int64_t blk = (int64_t)a.K * ((int64_t)ro * a.cin + (int64_t)dk * cc);
  for (int q0 = 0; q0 < nq; q0 += kQW) {
    float acc[kQW];
#pragma unroll
    for (int j = 0; j < kQW; ++j) acc[j] = 0.f;
    for (int e0 = lane; e0 < n; e0 += 64 * kEU) {
      float g[kEU], bv[kEU][kQW];
#pragma unroll
      for (int u = 0; u < kEU; ++u) {
        const int e = e0 + u * 64;
        const bool ok = e < n;
        g[u] = ok ? dW[blk + e] : 0.f;
#pragma unroll
        for (int j = 0; j < kQW; ++j) bv[u][j] = (ok && q0 + j < nq) ? bp[(q0 + j) * qstride + e] : 0.f;
      }
#pragma unroll
      for (int u = 0; u < kEU; ++u)
#pragma unroll
        for (int j = 0; j < kQW; ++j) acc[j] = fmaf(g[u], bv[u][j], acc[j]);
    }
    float mine = 0.f;  // lane j keeps coefficient j's sum
#pragma unroll
    for (int j = 0; j < kQW; ++j) {
      if (q0 + j < nq) {  // uniform per wavefront: no butterflies for absent coefficients
        float v = acc[j];
#pragma unroll
        for (int m = 32; m >= 1; m >>= 1) v += __shfl_xor(v, m);
        if (lane == j) mine = v;
      }
    }
    if (lane < kQW && q0 + lane < nq) dcoef[off + q0 + lane] = mine;
  }
}

}  // namespace

int launch_synth(const SynthArgs& a, const float* basis, const float* coeffs, ssconv_dtype dt, void* W,
                 hipStream_t st) {
  const int64_t plane = (int64_t)a.cout * a.cin;
  if (plane == 0 || a.K == 0) return SSCONV_OK;
  if (plane > 0x7fffffffll) return fail(SSCONV_E_INVALID, "Cout * Cin must be below 2^31");
  const int64_t pairs = (int64_t)a.n_in_fields * a.n_out_fields;
  int kmax = 0, lmax = 0;
  for (int e = 0; e < a.out.n; ++e) kmax = std::max(kmax, a.out.l[e]);
  for (int e = 0; e < a.in.n; ++e) lmax = std::max(lmax, a.in.l[e]);
  // chunks per pair: enough for one pass per wavefront over the largest block, but no more than
  // one round of the chip's wavefront slots holds (256 CUs x 4 SIMDs x 8): past that, extra
  // wavefronts only repeat the per-pair setup (6400 pairs of up to 675 elements: one chunk,
  // 16 us against 17.5 with three; 1600 pairs of up to 3125 elements: five chunks of three
  // passes, 16-18 us, against 36 us for one chunk of thirteen)
  const int64_t one_pass = cdiv((int64_t)a.K * (2 * kmax + 1) * (2 * lmax + 1), 64 * kSU);
  const int nch = (int)std::max<int64_t>(1, std::min<int64_t>(one_pass, 8192 / std::max<int64_t>(pairs, 1)));
  const int span = (int)(cdiv(one_pass, nch) * 64 * kSU);  // elements per chunk, whole passes
  if (pairs * nch > 0x7fffffffll) return fail(SSCONV_E_INVALID, "too many field pairs for the synthesis launch");
  const unsigned g = (unsigned)cdiv(pairs * nch, 4);
  if (dt == SSCONV_F32)
    synth_kernel<float><<<g, 256, 0, st>>>(a, basis, coeffs, (float*)W, nch, span);
  else
    synth_kernel<uint16_t><<<g, 256, 0, st>>>(a, basis, coeffs, (uint16_t*)W, nch, span);
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
