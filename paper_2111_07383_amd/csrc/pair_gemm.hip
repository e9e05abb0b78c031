// Pair-list GEMM for sparse fp32 layers (Sec. 3.2.3, the feature update of Alg. 1 taken offset by
// offset over the rule book R_s, as the paper states it).
//
// When the sites have few active neighbours (a stride-2 layer over sparse points, a 3x3x3 layer on
// isolated voxels, a 5x5x5 layer on a thin surface), the output-stationary kernel spends most of
// its matrix-core time on the zero rows of absent neighbours.  This path does only the useful
// products, in two deterministic passes:
//   pass 1  Y[p] = src[row(p)] B[s]^T for every pair p of every R_s: one wavefront task = 32 pairs
//           of one offset x up to 128 columns, v_mfma_f32_16x16x4f32, operands straight from
//           global memory (a lane fetches 16 bytes of its pair's row per 16-channel step; B, one
//           offset's kernel, stays in L1/L2 for all tasks of that offset);
//   pass 2  dst[r] = sum over s, in offset order, of Y[map[s][r]] (map: the pair of R_s whose
//           destination row is r, or -1), so every destination row is written once, no atomics.
// Forward: row(p) = input row, dst = output rows, B = kappa.  Feature gradient: row(p) = output
// row, dst = input rows, B = kappa^T.  The price is the Y traffic (pairs x columns x 4 bytes, written
// and read once), so the path is taken only when the cost model below says it wins.
#include <algorithm>

#include "conv.hpp"
#include "norm.hpp"

namespace ssconv {
namespace {

typedef float f4 __attribute__((ext_vector_type(4)));

constexpr int kThreads = 256;
constexpr int kTaskPairs = 32;                 // pairs per wavefront task (two 16-row MFMA blocks)
constexpr int kMaxOffsets = 125;

struct TaskTab {
  int64_t off[kMaxOffsets + 1];  // wavefront tasks of offset s: [off[s], off[s+1])
};

// Quads (4 channels) per offset in the packed B: ca / 4 rounded up to whole 16-channel steps.
__host__ __device__ __forceinline__ int packed_quads(int ca) { return (ca + 15) / 16 * 4; }

// B packed channel-quad-major, Bp[s][c/4][n][4] = B[s][n][c], zero past ca, so that the 16 lanes
// of a lane group fetch one contiguous 256-byte run per fragment instead of 16 scattered lines.
__global__ void pair_pack_b(const float* __restrict__ Bt, int K, int cb, int ca, float* __restrict__ Bp) {
  const int c4n = packed_quads(ca);
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int64_t total = (int64_t)K * c4n * cb;
  if (i >= total) return;
  const int n = (int)(i % cb);
  const int64_t sc = i / cb;
  const int c4 = (int)(sc % c4n), s = (int)(sc / c4n);
  const float* b = Bt + ((int64_t)s * cb + n) * ca + 4 * c4;
  float4 v;
  v.x = 4 * c4 + 0 < ca ? b[0] : 0.f;
  v.y = 4 * c4 + 1 < ca ? b[1] : 0.f;
  v.z = 4 * c4 + 2 < ca ? b[2] : 0.f;
  v.w = 4 * c4 + 3 < ca ? b[3] : 0.f;
  reinterpret_cast<float4*>(Bp)[i] = v;
}

template <int NB>
__global__ __launch_bounds__(kThreads) void pair_gemm_kernel(const float* __restrict__ src, int ca,
                                                             const float* __restrict__ Bp, int cb,
                                                             const int2* __restrict__ pairs,
                                                             const int64_t* __restrict__ pair_off, int K, TaskTab tt,
                                                             int sel_in, float* __restrict__ Y) {
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6, g = lane >> 4, m = lane & 15;
  const int64_t task = (int64_t)blockIdx.x * 4 + w;
  if (task >= tt.off[K]) return;  // no barrier below
  // the offset whose task range holds this task (empty ranges cannot hold it)
  int lo = 0, hi = K;
  while (hi - lo > 1) {
    const int mid = (lo + hi) >> 1;
    if (tt.off[mid] <= task) lo = mid;
    else hi = mid;
  }
  const int s = lo;
  const int64_t beg = pair_off[s], cnt = pair_off[s + 1] - beg;
  const int64_t q0 = (task - tt.off[s]) * kTaskPairs;  // first pair of the task within R_s
  const bool v0 = q0 + m < cnt, v1 = q0 + 16 + m < cnt;
  int r0 = 0, r1 = 0;
  if (v0) {
    const int2 pr = pairs[beg + q0 + m];
    r0 = sel_in ? pr.y : pr.x;
  }
  if (v1) {
    const int2 pr = pairs[beg + q0 + 16 + m];
    r1 = sel_in ? pr.y : pr.x;
  }
  const float4* A0 = reinterpret_cast<const float4*>(src + (int64_t)r0 * ca);
  const float4* A1 = reinterpret_cast<const float4*>(src + (int64_t)r1 * ca);
  const int nq = ca / 4, c4n = packed_quads(ca);
  const int n0 = blockIdx.y * 16 * NB;
  // this lane's B quads: Bp[s][q][min(n0 + 16 nb + m, cb - 1)] for quad q = c0/4 + g
  const float4* B4 = reinterpret_cast<const float4*>(Bp) + (int64_t)s * c4n * cb;
  int col[NB];
#pragma unroll
  for (int nb = 0; nb < NB; ++nb) col[nb] = min(n0 + 16 * nb + m, cb - 1);

  f4 acc0[NB], acc1[NB];
#pragma unroll
  for (int nb = 0; nb < NB; ++nb) acc0[nb] = acc1[nb] = f4{0.f, 0.f, 0.f, 0.f};

  // 16 channels per step: lane group g holds channels c0+4g..c0+4g+3 of its row, MFMA step t takes
  // channel c0+4g+t from both operands (any channel-to-step assignment is valid if A and B agree).
  // Both operands of the next step are fetched while this step's MFMAs run.  No load is masked:
  // a pair past the end of R_s reads row 0 and a column past cb reads column cb - 1 (neither
  // result is stored), and channels past ca meet the zero padding of the packed B (the A quad
  // read there is quad 0 of the same row).
  float4 a0 = A0[g < nq ? g : 0], a1 = A1[g < nq ? g : 0];
  float4 b[NB];
#pragma unroll
  for (int nb = 0; nb < NB; ++nb) b[nb] = B4[(int64_t)g * cb + col[nb]];
  for (int q0c = 0; q0c < c4n; q0c += 4) {  // q0c = c0 / 4
    const int qn = q0c + 4 + g;             // this lane's quad of the next step
    const int qa = qn < nq ? qn : 0, qb = qn < c4n ? qn : 0;
    const float4 a0n = A0[qa], a1n = A1[qa];
    float4 bn[NB];
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) bn[nb] = B4[(int64_t)qb * cb + col[nb]];
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) {
      acc0[nb] = __builtin_amdgcn_mfma_f32_16x16x4f32(a0.x, b[nb].x, acc0[nb], 0, 0, 0);
      acc1[nb] = __builtin_amdgcn_mfma_f32_16x16x4f32(a1.x, b[nb].x, acc1[nb], 0, 0, 0);
      acc0[nb] = __builtin_amdgcn_mfma_f32_16x16x4f32(a0.y, b[nb].y, acc0[nb], 0, 0, 0);
      acc1[nb] = __builtin_amdgcn_mfma_f32_16x16x4f32(a1.y, b[nb].y, acc1[nb], 0, 0, 0);
      acc0[nb] = __builtin_amdgcn_mfma_f32_16x16x4f32(a0.z, b[nb].z, acc0[nb], 0, 0, 0);
      acc1[nb] = __builtin_amdgcn_mfma_f32_16x16x4f32(a1.z, b[nb].z, acc1[nb], 0, 0, 0);
      acc0[nb] = __builtin_amdgcn_mfma_f32_16x16x4f32(a0.w, b[nb].w, acc0[nb], 0, 0, 0);
      acc1[nb] = __builtin_amdgcn_mfma_f32_16x16x4f32(a1.w, b[nb].w, acc1[nb], 0, 0, 0);
    }
    a0 = a0n;
    a1 = a1n;
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) b[nb] = bn[nb];
  }
  // accumulator lane layout: rows 4g..4g+3 of the 16-row block, column m
#pragma unroll
  for (int nb = 0; nb < NB; ++nb) {
    const int col = n0 + 16 * nb + m;
    if (col >= cb) continue;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int64_t qa = q0 + 4 * g + i, qb = qa + 16;
      if (qa < cnt) Y[(beg + qa) * cb + col] = acc0[nb][i];
      if (qb < cnt) Y[(beg + qb) * cb + col] = acc1[nb][i];
    }
  }
}

__global__ void pair_map_fill(int32_t* __restrict__ map, int64_t n) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) map[i] = -1;
}

// map[s][row] = p for every pair p of R_s, row = its destination row (the output row when the
// source rows are input rows, sel_in = 1, else the input row); a destination row takes at most
// one pair per offset, so every entry is written at most once.
__global__ void pair_map_scatter(const int2* __restrict__ pairs, const int64_t* __restrict__ pair_off, int sel_in,
                                 int64_t n_dst, int32_t* __restrict__ map) {
  const int s = blockIdx.y;
  const int64_t beg = pair_off[s], end = pair_off[s + 1];
  for (int64_t p = beg + (int64_t)blockIdx.x * blockDim.x + threadIdx.x; p < end; p += (int64_t)gridDim.x * blockDim.x) {
    const int2 pr = pairs[p];
    map[(int64_t)s * n_dst + (sel_in ? pr.x : pr.y)] = (int32_t)p;
  }
}

// acc = sum over s of Y[map[s][r]][VEC columns from v * VEC]; eight offsets' map entries and rows
// are fetched together, then added in offset order (absent pairs add 0).
template <int VEC>
__device__ __forceinline__ void pair_row(const float* __restrict__ Y, int cb, const int32_t* __restrict__ map, int K,
                                         int64_t n_dst, int64_t r, int v, float* acc) {
#pragma unroll
  for (int k = 0; k < VEC; ++k) acc[k] = 0.f;
  for (int s0 = 0; s0 < K; s0 += 8) {
    int p[8];
#pragma unroll
    for (int j = 0; j < 8; ++j) p[j] = s0 + j < K ? map[(int64_t)(s0 + j) * n_dst + r] : -1;
    float y[8][VEC];
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      if (p[j] >= 0) {
        if constexpr (VEC == 4) {
          const float4 t = *reinterpret_cast<const float4*>(Y + (int64_t)p[j] * cb + v * 4);
          y[j][0] = t.x, y[j][1] = t.y, y[j][2] = t.z, y[j][3] = t.w;
        } else {
#pragma unroll
          for (int k = 0; k < VEC; ++k) y[j][k] = Y[(int64_t)p[j] * cb + v * VEC + k];
        }
      } else {
#pragma unroll
        for (int k = 0; k < VEC; ++k) y[j][k] = 0.f;
      }
    }
#pragma unroll
    for (int j = 0; j < 8; ++j)
#pragma unroll
      for (int k = 0; k < VEC; ++k) acc[k] += y[j][k];
  }
}

template <int VEC>
__device__ __forceinline__ void store_row(float* __restrict__ dst, int cb, int64_t r, int v, const float* acc) {
  if constexpr (VEC == 4) {
    *reinterpret_cast<float4*>(dst + r * cb + v * 4) = make_float4(acc[0], acc[1], acc[2], acc[3]);
  } else {
#pragma unroll
    for (int k = 0; k < VEC; ++k) dst[r * cb + v * VEC + k] = acc[k];
  }
}

// dst[r][VEC columns] = pair_row, one thread per (row, vector).
template <int VEC>
__global__ __launch_bounds__(kThreads) void pair_reduce_kernel(const float* __restrict__ Y, int cb,
                                                               const int32_t* __restrict__ map, int K, int64_t n_dst,
                                                               float* __restrict__ dst) {
  const int nv = cb / VEC;
  const int64_t i = (int64_t)blockIdx.x * kThreads + threadIdx.x;
  if (i >= n_dst * nv) return;
  const int64_t r = i / nv;
  const int v = (int)(i - r * nv);
  float acc[VEC];
  pair_row<VEC>(Y, cb, map, K, n_dst, r, v, acc);
  store_row<VEC>(dst, cb, r, v, acc);
}

// The same rows (same values, same order of addition) in row blocks, with the Norm statistics of
// what it writes (part, in the row-block layout of stats_rows).
template <int VEC>
__global__ __launch_bounds__(kStatsThreads) void pair_reduce_stats_kernel(const float* __restrict__ Y, int cb,
                                                                          const int32_t* __restrict__ map, int K,
                                                                          int64_t n_dst, int G, int64_t rpb,
                                                                          float* __restrict__ dst,
                                                                          double* __restrict__ part) {
  stats_rows<VEC>(
      cb, n_dst, G, rpb,
      [&](int64_t r, int v, float* acc) {
        pair_row<VEC>(Y, cb, map, K, n_dst, r, v, acc);
        store_row<VEC>(dst, cb, r, v, acc);
      },
      part);
}

template <int NB>
void launch_pair_gemm(dim3 grid, const float* src, int ca, const float* Bt, int cb, const ssconv_rulebook* rb,
                      const TaskTab& tt, int sel_in, float* Y, hipStream_t st) {
  pair_gemm_kernel<NB><<<grid, kThreads, 0, st>>>(src, ca, Bt, cb, reinterpret_cast<const int2*>(rb->pairs),
                                                  rb->pair_off_dev, rb->K, tt, sel_in, Y);
}

}  // namespace

bool pair_path_supported(const ssconv_rulebook* rb, ssconv_dtype dt, int ca, int cb) {
  return dt == SSCONV_F32 && ca % 4 == 0 && rb->K <= kMaxOffsets && rb->n_pairs > 0 &&
         rb->n_pairs < ((int64_t)1 << 31) && (int64_t)rb->n_pairs * cb < ((int64_t)1 << 40);
}

// Cost model (measured rates on MI355X): the output-stationary kernels execute about
// pairs / density rows of MFMA work at ~100 TFLOP/s, density = pairs / (destination rows x
// offsets) (a tile of 128 rows holds nearly every offset, so its zero rows follow the density);
// this path does the useful products at ~80 TFLOP/s and moves Y (written, read) plus the gathered
// rows at ~4 TB/s, plus ~8 us of launches.  Kernel-selection override 9 forces it, 10 forbids it.
bool pair_path_wins(const ssconv_rulebook* rb, ssconv_dtype dt, int ca, int cb, int64_t n_dst) {
  if (!pair_path_supported(rb, dt, ca, cb) || n_dst <= 0) return false;
  const int64_t v = debug_gather_variant();
  if (v == 9) return true;
  if (v != 0 && v != 11 && v != 12) return false;  // 10 and the others forbid it (11, 12 concern other kernels)
  const double P = (double)rb->n_pairs;
  const double density = std::min(1.0, P / ((double)n_dst * rb->K));
  const double flops = 2.0 * P * ca * cb;
  const double t_os = flops / density / 100e12;
  const double t_pair = flops / 80e12 + P * (8.0 * cb + 4.0 * ca) / 4e12 + 8e-6;
  return t_pair < 0.85 * t_os;
}

static size_t y_bytes(const ssconv_rulebook* rb, int cb) { return ((size_t)rb->n_pairs * cb * 4 + 255) & ~(size_t)255; }
static size_t bp_bytes(const ssconv_rulebook* rb, int ca, int cb) {
  return ((size_t)rb->K * packed_quads(ca) * cb * 16 + 255) & ~(size_t)255;
}

size_t pair_path_bytes(const ssconv_rulebook* rb, int ca, int cb, int64_t n_dst) {
  return y_bytes(rb, cb) + bp_bytes(rb, ca, cb) + (size_t)rb->K * n_dst * 4;
}

// dst [n_dst, cb] fp32 from src [n_src, ca] fp32 over the rule book's pair lists; Bt [K][cb][ca].
// sel_in = 1: rows of src are the pairs' input rows (forward); 0: their output rows (gradient).
// ws: pair_path_bytes(rb, ca, cb, n_dst) bytes, 256-byte aligned.
int pair_gemm(const void* src, int ca, const void* Bt, int cb, const ssconv_rulebook* rb, int sel_in, void* dst,
              int64_t n_dst, void* ws, hipStream_t st, NormSink* sink) {
  const int K = rb->K;
  float* Y = (float*)ws;
  float* Bp = (float*)((char*)ws + y_bytes(rb, cb));
  int32_t* map = (int32_t*)((char*)ws + y_bytes(rb, cb) + bp_bytes(rb, ca, cb));
  TaskTab tt;
  tt.off[0] = 0;
  int64_t maxcnt = 0;
  for (int s = 0; s < K; ++s) {
    const int64_t cnt = rb->pair_off[s + 1] - rb->pair_off[s];
    tt.off[s + 1] = tt.off[s] + (cnt + kTaskPairs - 1) / kTaskPairs;
    maxcnt = std::max(maxcnt, cnt);
  }
  for (int s = K + 1; s <= kMaxOffsets; ++s) tt.off[s] = tt.off[K];
  const int64_t nmap = (int64_t)K * n_dst;
  pair_map_fill<<<cdiv(nmap, 256), 256, 0, st>>>(map, nmap);
  dim3 gs(std::min<unsigned>(cdiv(maxcnt, 256), 1024u), K);
  pair_map_scatter<<<gs, 256, 0, st>>>(reinterpret_cast<const int2*>(rb->pairs), rb->pair_off_dev, sel_in, n_dst, map);
  const int64_t nbp = (int64_t)K * packed_quads(ca) * cb;
  pair_pack_b<<<cdiv(nbp, 256), 256, 0, st>>>((const float*)Bt, K, cb, ca, Bp);
  // column blocks of 16: at most 8 per task (accumulators and two steps of B fragments then leave
  // room for three wavefronts per SIMD), the rest in further grid columns; small launches (few
  // pairs) split the columns further so that about 8192 wavefronts are in flight
  const int nblk16 = (cb + 15) / 16;
  const int64_t tasks = tt.off[K];
  int ngrp = (nblk16 + 7) / 8;
  while (ngrp < nblk16 && tasks * ngrp < 8192) ++ngrp;
  const int NB = (nblk16 + ngrp - 1) / ngrp;
  ngrp = (nblk16 + NB - 1) / NB;
  dim3 grid(cdiv(tasks, 4), ngrp);
  const float* S = (const float*)src;
  const float* B = Bp;
  switch (NB) {
    case 1: launch_pair_gemm<1>(grid, S, ca, B, cb, rb, tt, sel_in, Y, st); break;
    case 2: launch_pair_gemm<2>(grid, S, ca, B, cb, rb, tt, sel_in, Y, st); break;
    case 3: launch_pair_gemm<3>(grid, S, ca, B, cb, rb, tt, sel_in, Y, st); break;
    case 4: launch_pair_gemm<4>(grid, S, ca, B, cb, rb, tt, sel_in, Y, st); break;
    case 5: launch_pair_gemm<5>(grid, S, ca, B, cb, rb, tt, sel_in, Y, st); break;
    case 6: launch_pair_gemm<6>(grid, S, ca, B, cb, rb, tt, sel_in, Y, st); break;
    case 7: launch_pair_gemm<7>(grid, S, ca, B, cb, rb, tt, sel_in, Y, st); break;
    default: launch_pair_gemm<8>(grid, S, ca, B, cb, rb, tt, sel_in, Y, st); break;
  }
  const bool vec = cb % 4 == 0 && aligned16(dst);
  StatsRows sr;
  if (sink && stats_rows_plan(n_dst, cb, vec ? 4 : 1, &sr)) {
    SSC_TRY(norm_sink_take(sink, sr.nblk, st));
    double* part = (double*)sink->ws;
    if (vec)
      pair_reduce_stats_kernel<4><<<sr.nblk, kStatsThreads, 0, st>>>(Y, cb, map, K, n_dst, sr.G, sr.rpb, (float*)dst,
                                                                      part);
    else
      pair_reduce_stats_kernel<1><<<sr.nblk, kStatsThreads, 0, st>>>(Y, cb, map, K, n_dst, sr.G, sr.rpb, (float*)dst,
                                                                      part);
    SSC_HIP(hipGetLastError());
    return SSCONV_OK;
  }
  const int64_t items = n_dst * (vec ? cb / 4 : cb);
  if (vec)
    pair_reduce_kernel<4><<<cdiv(items, kThreads), kThreads, 0, st>>>(Y, cb, map, K, n_dst, (float*)dst);
  else
    pair_reduce_kernel<1><<<cdiv(items, kThreads), kThreads, 0, st>>>(Y, cb, map, K, n_dst, (float*)dst);
  SSC_HIP(hipGetLastError());
  return SSCONV_OK;
}

}  // namespace ssconv
