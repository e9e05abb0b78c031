// Sparse steerable convolution on matrix cores (Sec. 3.2.3, the feature update of Alg. 1) and its adjoint.
//
// gather_gemm: output-stationary implicit GEMM.  A workgroup owns BM = 64 output
// rows x BN = 16*WNB output channels and accumulates, in MFMA accumulators,
//     out[x] = sum_s sum_{y = nbr[s][x]} kappa(s) feats[y]
// over the offsets present in its rows (an offset with no neighbour in the
// tile is skipped entirely; missing rows of a present offset are zero-filled).
// Feature rows are gathered with 16-byte loads into LDS tiles of 32 channels;
// kappa(s) is staged transposed so both MFMA operands are read as contiguous
// 8-element runs.  Each output element is written exactly once: no atomics.
// The feature gradient is the same kernel on (grad_out, kappa^T, transposed
// neighbour map).
//
// dw_gemm: dkappa(s) = sum_{(x,y) in R_s} grad_out[x] feats[y]^T, a gather-gather
// GEMM over the compact pair list of each offset, split along the pairs into
// fixed chunks whose partial sums are reduced in a fixed order (deterministic).
//
// MFMA: fp32 uses v_mfma_f32_16x16x4f32 (eight K-steps per 32-channel chunk,
// lane group g = lane/16 taking channels 8g..8g+7), bf16 uses the gfx950
// v_mfma_f32_16x16x32_bf16 (one step per chunk).  Any assignment of channels
// to K-steps is valid as long as both operands use the same one.
#include <algorithm>

#include "conv.hpp"
#include "norm.hpp"
#include "gather_mfma.hpp"
#include "kgrad_mfma.hpp"

namespace ssconv {

namespace {

typedef float f4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));

constexpr int kNT = 256;
constexpr int BM = 64;
constexpr int BK = 32;

template <typename T>
struct Cfg {
  static constexpr int VE = 16 / (int)sizeof(T);     // elements per 16-byte vector
  static constexpr int VPR = BK / VE;                // vectors per 32-element row chunk
  static constexpr int ROW = BK + VE;                // padded LDS row (elements): +16 bytes
};

template <typename T>
__device__ __forceinline__ uint4 load_vec(const T* __restrict__ p, int avail, bool vec_ok) {
  if (vec_ok && avail >= Cfg<T>::VE) return *reinterpret_cast<const uint4*>(p);
  T tmp[Cfg<T>::VE];
#pragma unroll
  for (int e = 0; e < Cfg<T>::VE; ++e) tmp[e] = e < avail ? p[e] : T(0);
  uint4 r;
  __builtin_memcpy(&r, tmp, 16);
  return r;
}

// One 32-element K chunk: acc += A_frag x B_frag for a 16x16 block.
__device__ __forceinline__ void mma_chunk(f4& acc, const float* a, const float* b) {
  const uint4 a0 = *reinterpret_cast<const uint4*>(a), a1 = *reinterpret_cast<const uint4*>(a + 4);
  const uint4 b0 = *reinterpret_cast<const uint4*>(b), b1 = *reinterpret_cast<const uint4*>(b + 4);
  const float av[8] = {__uint_as_float(a0.x), __uint_as_float(a0.y), __uint_as_float(a0.z), __uint_as_float(a0.w),
                       __uint_as_float(a1.x), __uint_as_float(a1.y), __uint_as_float(a1.z), __uint_as_float(a1.w)};
  const float bv[8] = {__uint_as_float(b0.x), __uint_as_float(b0.y), __uint_as_float(b0.z), __uint_as_float(b0.w),
                       __uint_as_float(b1.x), __uint_as_float(b1.y), __uint_as_float(b1.z), __uint_as_float(b1.w)};
#pragma unroll
  for (int t = 0; t < 8; ++t) acc = __builtin_amdgcn_mfma_f32_16x16x4f32(av[t], bv[t], acc, 0, 0, 0);
}

__device__ __forceinline__ void mma_chunk(f4& acc, const uint16_t* a, const uint16_t* b) {
  const uint4 ar = *reinterpret_cast<const uint4*>(a), br = *reinterpret_cast<const uint4*>(b);
  bf16x8 av, bv;
  __builtin_memcpy(&av, &ar, 16);
  __builtin_memcpy(&bv, &br, 16);
  acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(av, bv, acc, 0, 0, 0);
}

// ---------------------------------------------------------------------------
// output-stationary gather GEMM (forward and feature gradient)
// ---------------------------------------------------------------------------
template <typename T, int WNB>
__global__ __launch_bounds__(kNT) void gather_gemm(const T* __restrict__ src, int ca, const T* __restrict__ Bt,
                                                   int cb, const int32_t* __restrict__ nbr, int64_t n_rows, int K,
                                                   T* __restrict__ out) {
  using C = Cfg<T>;
  constexpr int BN = 16 * WNB;
  constexpr int AV = BM * C::VPR / kNT;                 // A vectors per thread (2 f32 / 1 bf16)
  constexpr int BV = (BN * C::VPR + kNT - 1) / kNT;     // B vectors per thread (upper bound)
  __shared__ __attribute__((aligned(16))) T As[BM * C::ROW];
  __shared__ __attribute__((aligned(16))) T Bs[BN * C::ROW];
  __shared__ uint32_t smask[4];

  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6, g = lane >> 4, r16 = lane & 15;
  const int64_t p0 = (int64_t)blockIdx.x * BM;
  const int n0 = blockIdx.y * BN;
  const bool vec_ok = (ca % C::VE) == 0;

  if (tid < 4) smask[tid] = 0;
  __syncthreads();
  for (int s = w; s < K; s += 4) {
    const int64_t p = p0 + lane;
    const int idx = p < n_rows ? nbr[(int64_t)s * n_rows + p] : -1;
    const uint64_t any = __ballot(idx >= 0);
    if (lane == 0 && any) atomicOr(&smask[s >> 5], 1u << (s & 31));
  }
  __syncthreads();
  const uint32_t mk[4] = {smask[0], smask[1], smask[2], smask[3]};

  f4 acc[WNB];
#pragma unroll
  for (int nb = 0; nb < WNB; ++nb) acc[nb] = f4{0.f, 0.f, 0.f, 0.f};

  for (int s = 0; s < K; ++s) {
    if (!((mk[s >> 5] >> (s & 31)) & 1u)) continue;
    int aidx[AV];
#pragma unroll
    for (int j = 0; j < AV; ++j) {
      const int r = (tid + kNT * j) / C::VPR;
      const int64_t p = p0 + r;
      aidx[j] = p < n_rows ? nbr[(int64_t)s * n_rows + p] : -1;
    }
    const T* Bs_s = Bt + (int64_t)s * cb * ca;
    for (int k0 = 0; k0 < ca; k0 += BK) {
      uint4 av[AV], bv[BV];
#pragma unroll
      for (int j = 0; j < AV; ++j) {
        const int v = tid + kNT * j, cv = v % C::VPR, col = k0 + cv * C::VE;
        av[j] = (aidx[j] >= 0 && col < ca) ? load_vec(src + (int64_t)aidx[j] * ca + col, ca - col, vec_ok)
                                          : make_uint4(0, 0, 0, 0);
      }
#pragma unroll
      for (int j = 0; j < BV; ++j) {
        const int v = tid + kNT * j, n = v / C::VPR, cv = v % C::VPR, col = k0 + cv * C::VE;
        bv[j] = (v < BN * C::VPR && n0 + n < cb && col < ca)
                    ? load_vec(Bs_s + (int64_t)(n0 + n) * ca + col, ca - col, vec_ok)
                    : make_uint4(0, 0, 0, 0);
      }
      __syncthreads();
#pragma unroll
      for (int j = 0; j < AV; ++j) {
        const int v = tid + kNT * j, r = v / C::VPR, cv = v % C::VPR;
        *reinterpret_cast<uint4*>(&As[r * C::ROW + cv * C::VE]) = av[j];
      }
#pragma unroll
      for (int j = 0; j < BV; ++j) {
        const int v = tid + kNT * j, n = v / C::VPR, cv = v % C::VPR;
        if (v < BN * C::VPR) *reinterpret_cast<uint4*>(&Bs[n * C::ROW + cv * C::VE]) = bv[j];
      }
      __syncthreads();
      const T* a = &As[(16 * w + r16) * C::ROW + 8 * g];
#pragma unroll
      for (int nb = 0; nb < WNB; ++nb) mma_chunk(acc[nb], a, &Bs[(16 * nb + r16) * C::ROW + 8 * g]);
    }
  }

#pragma unroll
  for (int nb = 0; nb < WNB; ++nb) {
    const int col = n0 + 16 * nb + r16;
    if (col >= cb) continue;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int64_t row = p0 + 16 * w + 4 * g + i;
      if (row < n_rows) out[row * cb + col] = DT<T>::from_f(acc[nb][i]);
    }
  }
}

// ---------------------------------------------------------------------------
// dkappa partials: gather-gather GEMM over the pair list of one offset
// ---------------------------------------------------------------------------
template <typename T, int WNB>
__global__ __launch_bounds__(kNT) void dw_gemm(const T* __restrict__ G, int cout, const T* __restrict__ F, int cin,
                                               const int32_t* __restrict__ pairs,
                                               const int64_t* __restrict__ pair_off, int K, int ntn, int nsplit,
                                               float* __restrict__ part) {
  using C = Cfg<T>;
  constexpr int BN = 16 * WNB;
  constexpr int VA = BM / C::VE;   // vectors per gathered grad row segment (64 channels)
  constexpr int VB = BN / C::VE;   // vectors per gathered feature row segment
  __shared__ __attribute__((aligned(16))) T At[BM * C::ROW];   // [m = out channel][k = pair]
  __shared__ __attribute__((aligned(16))) T Bs[BN * C::ROW];   // [n = in channel][k = pair]
  __shared__ int2 sp[BK];

  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6, g = lane >> 4, r16 = lane & 15;
  const int mt = blockIdx.x / ntn, nt = blockIdx.x % ntn;
  const int split = blockIdx.y, s = blockIdx.z;
  const int m0 = mt * BM, n0 = nt * BN;
  const int64_t off = pair_off[s], cnt = pair_off[s + 1] - off;
  const int64_t beg = off + cnt * split / nsplit, end = off + cnt * (split + 1) / nsplit;
  const bool vec_a = (cout % C::VE) == 0, vec_b = (cin % C::VE) == 0;

  f4 acc[WNB];
#pragma unroll
  for (int nb = 0; nb < WNB; ++nb) acc[nb] = f4{0.f, 0.f, 0.f, 0.f};

  for (int64_t kb = beg; kb < end; kb += BK) {
    __syncthreads();
    if (tid < BK) sp[tid] = (kb + tid < end) ? reinterpret_cast<const int2*>(pairs)[kb + tid] : make_int2(-1, -1);
    __syncthreads();
    // A: BK pairs x 64 out channels, stored transposed
    for (int v = tid; v < BK * VA; v += kNT) {
      const int k = v / VA, cv = v % VA, col = m0 + cv * C::VE;
      const int o = sp[k].x;
      uint4 x = (o >= 0 && col < cout) ? load_vec(G + (int64_t)o * cout + col, cout - col, vec_a) : make_uint4(0, 0, 0, 0);
      T e[C::VE];
      __builtin_memcpy(e, &x, 16);
#pragma unroll
      for (int q = 0; q < C::VE; ++q) At[(cv * C::VE + q) * C::ROW + k] = e[q];
    }
    for (int v = tid; v < BK * VB; v += kNT) {
      const int k = v / VB, cv = v % VB, col = n0 + cv * C::VE;
      const int i = sp[k].y;
      uint4 x = (i >= 0 && col < cin) ? load_vec(F + (int64_t)i * cin + col, cin - col, vec_b) : make_uint4(0, 0, 0, 0);
      T e[C::VE];
      __builtin_memcpy(e, &x, 16);
#pragma unroll
      for (int q = 0; q < C::VE; ++q) Bs[(cv * C::VE + q) * C::ROW + k] = e[q];
    }
    __syncthreads();
    const T* a = &At[(16 * w + r16) * C::ROW + 8 * g];
#pragma unroll
    for (int nb = 0; nb < WNB; ++nb) mma_chunk(acc[nb], a, &Bs[(16 * nb + r16) * C::ROW + 8 * g]);
  }

  float* dst = part + ((int64_t)split * K + s) * cout * cin;
#pragma unroll
  for (int nb = 0; nb < WNB; ++nb) {
    const int col = n0 + 16 * nb + r16;
    if (col >= cin) continue;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int row = m0 + 16 * w + 4 * g + i;
      if (row < cout) dst[(int64_t)row * cin + col] = acc[nb][i];
    }
  }
}

// dW (field-pair-blocked, dw_block_pos) = sum of the splits' [K][cout][cin] partials, in split order.
__global__ void reduce_splits(const float* __restrict__ part, int nsplit, int64_t n, FieldTab fout, FieldTab fin,
                              int K, int cin, int cout, float* __restrict__ dst) {
  const int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (e >= n) return;
  float acc = 0.f;
  for (int j = 0; j < nsplit; ++j) acc += part[(int64_t)j * n + e];
  const int64_t plane = (int64_t)cin * cout;
  const int s = (int)(e / plane), r = (int)(e - s * plane), o = r / cin, i = r - o * cin;
  dst[dw_block_pos(fout, fin, K, cin, s, o, i)] = acc;
}

template <typename T>
__global__ void transpose_kernel(const T* __restrict__ W, int K, int rows, int cols, int mirror, T* __restrict__ Wt) {
  // W [K][rows][cols] -> Wt [K][cols][rows], offsets reversed (Wt[s] = W[K-1-s]^T) when mirror
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int64_t per = (int64_t)rows * cols;
  if (i >= per * K) return;
  const int64_t s = i / per, r = i % per;
  const int c = (int)(r / rows), rr = (int)(r % rows);
  Wt[i] = W[(mirror ? K - 1 - s : s) * per + (int64_t)rr * cols + c];
}

__global__ void fill_i32(int32_t* __restrict__ p, int64_t n, int32_t v) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) p[i] = v;
}

__global__ void invert_nbr(const int32_t* __restrict__ nbr, int64_t n_out, int K, int64_t n_in,
                           int32_t* __restrict__ nbrT) {
  const int64_t p = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int s = blockIdx.y;
  if (p >= n_out) return;
  const int i = nbr[(int64_t)s * n_out + p];
  if (i >= 0) nbrT[(int64_t)s * n_in + i] = (int32_t)p;
}

template <typename T, int WNB>
void launch_gg(const void* src, int ca, const void* Bt, int cb, const int32_t* nbr, int64_t n_rows, int K, void* out,
               hipStream_t st) {
  dim3 grid(cdiv(n_rows, BM), cdiv(cb, 16 * WNB));
  gather_gemm<T, WNB><<<grid, kNT, 0, st>>>((const T*)src, ca, (const T*)Bt, cb, nbr, n_rows, K, (T*)out);
}

// Picks the N-tile width (in 16-column blocks) for cb output channels.
int pick_wnb(int cb) {
  const int blocks = (cb + 15) / 16;
  if (blocks <= 8) return blocks;
  // split wide outputs into near-equal tiles of at most 8 blocks
  const int tiles = (blocks + 7) / 8;
  return (blocks + tiles - 1) / tiles;
}

template <typename T>
int dispatch_gg(const void* src, int64_t n_src, int ca, const void* Bt, int cb, const int32_t* nbr, int64_t n_rows, int K,
                void* out, hipStream_t st, CallScratch* sc = nullptr, NormSink* sink = nullptr) {
  const ssconv_dtype dt = sizeof(T) == 4 ? SSCONV_F32 : SSCONV_BF16;
  if (gather_mfma_supported(dt, ca, cb, K))
    return gather_mfma(src, n_src, dt, ca, Bt, cb, nbr, nullptr, n_rows, K, out, st, sc, sink);
  switch (pick_wnb(cb)) {
    case 1: launch_gg<T, 1>(src, ca, Bt, cb, nbr, n_rows, K, out, st); break;
    case 2: launch_gg<T, 2>(src, ca, Bt, cb, nbr, n_rows, K, out, st); break;
    case 3: launch_gg<T, 3>(src, ca, Bt, cb, nbr, n_rows, K, out, st); break;
    case 4: launch_gg<T, 4>(src, ca, Bt, cb, nbr, n_rows, K, out, st); break;
    case 5: launch_gg<T, 5>(src, ca, Bt, cb, nbr, n_rows, K, out, st); break;
    case 6: launch_gg<T, 6>(src, ca, Bt, cb, nbr, n_rows, K, out, st); break;
    case 7: launch_gg<T, 7>(src, ca, Bt, cb, nbr, n_rows, K, out, st); break;
    default: launch_gg<T, 8>(src, ca, Bt, cb, nbr, n_rows, K, out, st); break;
  }
  SSC_HIP(hipGetLastError());
  return SSCONV_OK;
}

template <typename T, int WNB>
void launch_dw(const void* G, int cout, const void* F, int cin, const int32_t* pairs, const int64_t* pair_off, int K,
               int nsplit, float* part, hipStream_t st) {
  const int ntm = (int)cdiv(cout, BM), ntn = (int)cdiv(cin, 16 * WNB);
  dim3 grid(ntm * ntn, nsplit, K);
  dw_gemm<T, WNB><<<grid, kNT, 0, st>>>((const T*)G, cout, (const T*)F, cin, pairs, pair_off, K, ntn, nsplit, part);
}

template <typename T>
int dispatch_dw(const void* G, int cout, const void* F, int cin, const int32_t* pairs, const int64_t* pair_off, int K,
                int nsplit, float* part, hipStream_t st) {
  switch (pick_wnb(cin)) {
    case 1: launch_dw<T, 1>(G, cout, F, cin, pairs, pair_off, K, nsplit, part, st); break;
    case 2: launch_dw<T, 2>(G, cout, F, cin, pairs, pair_off, K, nsplit, part, st); break;
    case 3: launch_dw<T, 3>(G, cout, F, cin, pairs, pair_off, K, nsplit, part, st); break;
    case 4: launch_dw<T, 4>(G, cout, F, cin, pairs, pair_off, K, nsplit, part, st); break;
    case 5: launch_dw<T, 5>(G, cout, F, cin, pairs, pair_off, K, nsplit, part, st); break;
    case 6: launch_dw<T, 6>(G, cout, F, cin, pairs, pair_off, K, nsplit, part, st); break;
    case 7: launch_dw<T, 7>(G, cout, F, cin, pairs, pair_off, K, nsplit, part, st); break;
    default: launch_dw<T, 8>(G, cout, F, cin, pairs, pair_off, K, nsplit, part, st); break;
  }
  SSC_HIP(hipGetLastError());
  return SSCONV_OK;
}

}  // namespace

static bool use_bf16_kernel(ssconv_dtype dt, int64_t n_src, int ca, int cb, int K) {
  return dt == SSCONV_BF16 && debug_gather_variant() != 5 && gather_bf16_supported(n_src, ca, cb, K);
}

// Records the timing-hook events (ssconv_debug_set option 4) around one kernel launch.
struct KernelTimer {
  hipEvent_t start = nullptr, stop = nullptr;
  hipStream_t st;
  bool on;
  explicit KernelTimer(hipStream_t s) : st(s), on(debug_timing_events(&start, &stop)) {
    if (on) (void)hipEventRecord(start, st);
  }
  ~KernelTimer() {
    if (on) (void)hipEventRecord(stop, st);
  }
};

int conv_forward(const void* feats, ssconv_dtype dt, int cin, const ssconv_rulebook* rb, const void* W, int cout,
                 void* out, hipStream_t st, CallScratch* sc, NormSink* sink) {
  if (rb->n_out == 0) return SSCONV_OK;
  // the pair-list path needs its Y buffer; with a fixed scratch region too small for it the
  // output-stationary kernel runs instead (same sums, another order of the fp32 additions)
  const bool pair_fits = !(sc && sc->fixed()) || pair_path_bytes(rb, cin, cout, rb->n_out) <= sc->left();
  if (dt == SSCONV_F32 && pair_fits && pair_path_wins(rb, dt, cin, cout, rb->n_out)) {
    void* ws = nullptr;
    SSC_TRY(scratch_take(sc, &ws, pair_path_bytes(rb, cin, cout, rb->n_out), st));
    int rc;
    {
      KernelTimer timer(st);
      rc = pair_gemm(feats, cin, W, cout, rb, 1, out, rb->n_out, ws, st, sink);
    }
    scratch_give(sc, ws, st);
    return rc;
  }
  if (dt == SSCONV_F32) {
    KernelTimer timer(st);
    return dispatch_gg<float>(feats, rb->n_in, cin, W, cout, rb->nbr, rb->n_out, rb->K, out, st, sc, sink);
  }
  if (use_bf16_kernel(dt, rb->n_in, cin, cout, rb->K)) {
    // kappa packed for the bf16 kernel in a stream-ordered scratch buffer
    void* Bp = nullptr;
    SSC_TRY(scratch_take(sc, &Bp, (size_t)rb->K * cin * cout * 2, st));
    int rc = pack_b_bf16(W, rb->K, cin, cout, false, false, Bp, st);
    if (rc == SSCONV_OK) {
      KernelTimer timer(st);
      rc = gather_bf16(feats, rb->n_in, cin, Bp, cout, rb->nbr, nullptr, rb->n_out, rb->K, out, st, sink);
    }
    scratch_give(sc, Bp, st);
    return rc;
  }
  KernelTimer timer(st);
  return dispatch_gg<uint16_t>(feats, rb->n_in, cin, W, cout, rb->nbr, rb->n_out, rb->K, out, st, sc, sink);
}

// The convolution with the Norm of its output (Sec. 3.3, Eq. 11).  The kernel that writes y also
// leaves its per-channel sums (the output-stationary kernels per row tile, the pair-list and
// offset-split reduces per row block), so the Norm needs no pass of its own over y before the
// elementwise one; the other paths (the generic fallback kernel, an input set without rows) leave
// none and the separate statistics pass runs instead.
int conv_forward_norm(const void* feats, ssconv_dtype dt, int cin, const ssconv_rulebook* rb, const void* W, int cout,
                      const FieldTab& f, double eps, void* y, void* z, hipStream_t st) {
  const int64_t n = rb->n_out;
  if (n == 0) return SSCONV_OK;
  NormSink sink;
  sink.C = cout;
  int rc;
  if (rb->n_in == 0) {
    rc = hipMemsetAsync(y, 0, (size_t)n * cout * dtype_bytes(dt), st) == hipSuccess
             ? SSCONV_OK
             : fail(SSCONV_E_HIP, "clearing the output failed");
  } else {
    rc = conv_forward(feats, dt, cin, rb, W, cout, y, st, nullptr, &sink);
  }
  if (rc == SSCONV_OK && sink.nblk == 0) {
    const NormStatsPlan p = norm_stats_plan(dt, y, n, cout);
    rc = norm_sink_take(&sink, p.nblk, st);
    if (rc == SSCONV_OK) rc = norm_forward_sums(dt, y, n, p, sink.ws, st);
  }
  if (rc == SSCONV_OK) rc = norm_forward_finish(f, dt, y, n, eps, sink.nblk, sink.ws, z, st);
  if (sink.ws) dev_free(sink.ws, st);
  return rc;
}

int dw_nsplit(const ssconv_rulebook* rb) {
  int64_t mx = 0;
  for (int s = 0; s < rb->K; ++s) mx = std::max(mx, rb->pair_off[s + 1] - rb->pair_off[s]);
  int64_t ns = mx / 2048;
  if (ns < 1) ns = 1;
  if (ns > 16) ns = 16;
  return (int)ns;
}

static size_t align256(size_t b) { return (b + 255) & ~(size_t)255; }

// The bf16 kernel gradient cuts the pair lists into work units, one per compute unit (measured on
// the 128^3 208-channel layer: 512 units ran the gradient no faster and doubled the partials to add).
constexpr int kKgradUnits = 256;

static bool use_kgrad_units(const ssconv_rulebook* rb, ssconv_dtype dt, int cin, int cout) {
  if (dt == SSCONV_F32) return kgrad_f32_units_ok(rb, cin, cout);
  return debug_gather_variant() != 6 && kgrad_supported(dt, cin, cout) && rb->K <= kKgradMaxK &&
         (int64_t)rb->n_in * cin * 2 < ((int64_t)1 << 31) && (int64_t)rb->n_out * cout * 2 < ((int64_t)1 << 31);
}

// Work units of the kernel gradient: bf16 ~256 (one workgroup each, launched in row order), fp32
// enough wavefront tasks for one round of the wavefront slots.
static KgradUnits plan_units(const ssconv_rulebook* rb, ssconv_dtype dt, int cin, int cout) {
  if (dt == SSCONV_F32) return kgrad_units(rb, kgrad_f32_units_want(rb, cin, cout), false);
  return kgrad_units(rb, kKgradUnits, true);
}

BwdLayout bwd_layout(const ssconv_rulebook* rb, ssconv_dtype dt, int cin, int cout) {
  BwdLayout L;
  const size_t K = rb->K, sz = dtype_bytes(dt);
  size_t nparts;  // fp32 partial tiles of cout x cin
  if (use_kgrad_units(rb, dt, cin, cout)) {
    nparts = (size_t)plan_units(rb, dt, cin, cout).nunits;
  } else {
    L.nsplit = kgrad_supported(dt, cin, cout) ? kgrad_plan(rb, dt, cin, cout).nsplit : dw_nsplit(rb);
    nparts = (size_t)L.nsplit * K;
  }
  size_t o = 0;
  L.pair_feats = dt == SSCONV_F32 && rb->n_in > 0 && pair_path_wins(rb, dt, cout, cin, rb->n_in);
  L.nbrT = o;  // inverse neighbour map: only generated output sets on the gather kernels need one
  if (!rb->submanifold && !L.pair_feats) o += align256(K * (size_t)rb->n_in * 4);
  L.pair = o;
  if (L.pair_feats) o += align256(pair_path_bytes(rb, cout, cin, rb->n_in));
  L.Wt = o;
  o += align256(K * (size_t)cin * cout * sz);
  L.part = o;
  o += align256(nparts * cin * cout * 4);
  L.dW = o;
  o += align256(K * (size_t)cin * cout * 4);
  L.total = o;
  return L;
}

// The feature gradient is the gather GEMM over the transposed neighbour map with kappa^T.  For a
// submanifold layer the transposed map is the map itself with the offsets reversed (y = x - d(s)
// holds exactly when x = y - d(K-1-s), d(K-1-s) = -d(s), on the same site set), so it runs on the
// forward map with kappa^T stored in reversed offset order and no inverse map is built.
int conv_backward_feats(const void* grad_out, ssconv_dtype dt, int cin, int cout, const ssconv_rulebook* rb,
                        const void* W, void* grad_feats, char* ws, const BwdLayout& L, hipStream_t st) {
  if (rb->n_in == 0) return SSCONV_OK;
  if (L.pair_feats) {
    // kappa^T in the same offset order: the pairs of R_s are walked with their roles swapped
    const int64_t nw = (int64_t)rb->K * cin * cout;
    transpose_kernel<float><<<cdiv(nw, 256), 256, 0, st>>>((const float*)W, rb->K, cout, cin, false,
                                                            (float*)(ws + L.Wt));
    SSC_HIP(hipGetLastError());
    KernelTimer timer(st);
    return pair_gemm(grad_out, cout, ws + L.Wt, cin, rb, 0, grad_feats, rb->n_in, ws + L.pair, st);
  }
  const bool mirror = rb->submanifold != 0;
  const int32_t* nbrT = rb->nbr;
  void* Wt = ws + L.Wt;
  const int K = rb->K;
  if (!mirror) {
    int32_t* inv = (int32_t*)(ws + L.nbrT);
    const int64_t nT = (int64_t)K * rb->n_in;
    fill_i32<<<cdiv(nT, 256), 256, 0, st>>>(inv, nT, -1);
    if (rb->n_out > 0) {
      dim3 gi(cdiv(rb->n_out, 256), K);
      invert_nbr<<<gi, 256, 0, st>>>(rb->nbr, rb->n_out, K, rb->n_in, inv);
    }
    nbrT = inv;
  }
  const int64_t nw = (int64_t)K * cin * cout;
  if (dt == SSCONV_F32) {
    transpose_kernel<float><<<cdiv(nw, 256), 256, 0, st>>>((const float*)W, K, cout, cin, mirror, (float*)Wt);
    SSC_HIP(hipGetLastError());
    KernelTimer timer(st);
    return dispatch_gg<float>(grad_out, rb->n_out, cout, Wt, cin, nbrT, rb->n_in, K, grad_feats, st);
  }
  if (use_bf16_kernel(dt, rb->n_out, cout, cin, K)) {
    // kappa^T packed for the bf16 kernel: Bp[s][o/8][i][o%8] = W[s'][o][i], s' = s or K-1-s
    SSC_TRY(pack_b_bf16(W, K, cout, cin, true, mirror, Wt, st));
    KernelTimer timer(st);
    return gather_bf16(grad_out, rb->n_out, cout, Wt, cin, nbrT, nullptr, rb->n_in, K, grad_feats, st);
  }
  transpose_kernel<uint16_t><<<cdiv(nw, 256), 256, 0, st>>>((const uint16_t*)W, K, cout, cin, mirror, (uint16_t*)Wt);
  SSC_HIP(hipGetLastError());
  KernelTimer timer(st);
  return dispatch_gg<uint16_t>(grad_out, rb->n_out, cout, Wt, cin, nbrT, rb->n_in, K, grad_feats, st);
}

int conv_backward_dw(const void* feats, const void* grad_out, ssconv_dtype dt, int cin, int cout,
                     const ssconv_rulebook* rb, const FieldTab& fout, const FieldTab& fin, char* ws,
                     const BwdLayout& L, float** dW_out, hipStream_t st, hipStream_t* tail) {
  float* part = (float*)(ws + L.part);
  float* dW = (float*)(ws + L.dW);
  *dW_out = dW;
  if (tail) *tail = st;
  const int K = rb->K;
  const int64_t n = (int64_t)K * cin * cout;
  if (use_kgrad_units(rb, dt, cin, cout)) {
    const KgradUnits units = plan_units(rb, dt, cin, cout);
    if (dt == SSCONV_F32)
      SSC_TRY(kgrad_f32(grad_out, feats, cin, cout, rb, units, part, st));
    else
      SSC_TRY(kgrad_bf16(grad_out, rb->n_out, feats, rb->n_in, cin, cout, rb, units, part, st));
    hipStream_t rst = st;
    if (tail) {
      SSC_TRY(aux_fork(st, &rst));
      *tail = rst;
    }
    return reduce_units(part, units, cin, cout, fout, fin, dW, rst);
  }
  if (kgrad_supported(dt, cin, cout))
    SSC_TRY(kgrad_partials(grad_out, feats, dt, cin, cout, rb, kgrad_plan(rb, dt, cin, cout), part, st));
  else if (dt == SSCONV_F32)
    SSC_TRY(dispatch_dw<float>(grad_out, cout, feats, cin, rb->pairs, rb->pair_off_dev, K, L.nsplit, part, st));
  else
    SSC_TRY(dispatch_dw<uint16_t>(grad_out, cout, feats, cin, rb->pairs, rb->pair_off_dev, K, L.nsplit, part, st));
  reduce_splits<<<cdiv(n, 256), 256, 0, st>>>(part, L.nsplit, n, fout, fin, K, cin, cout, dW);
  SSC_HIP(hipGetLastError());
  return SSCONV_OK;
}

}  // namespace ssconv
