// Output-stationary gather -> MFMA GEMM with the reduction dimension flattened over
// the tile's active kernel offsets (Sec. 3.2.3, Alg. 1 feature update).
//
//   out[x] = sum_s kappa(s) in[nbr[s][x]]   for the output rows x of a tile
//
// A workgroup of NW wavefronts (8 for fp32, 4 for bf16) owns BM = NW*WMB*16 output
// rows and BN = WNB*16 output channels.  Its reduction dimension is the concatenation, over the
// offsets present in its rows, of the Cin input channels of each offset, cut
// into 32-wide chunks; a chunk may straddle two offsets, so no channel padding
// is paid per offset.
//
// Data movement (gfx950):
//   * the tile's neighbour indices for every offset are staged in LDS once;
//   * each chunk of gathered feature rows and of kappa(s) is fetched with
//     16-byte global->LDS DMA loads (global_load_lds_dwordx4) straight into
//     MFMA fragment order: lane l of a load lands at byte 16*l of a 1 KB
//     block, which is exactly the 16 bytes that lane l later feeds the MFMA;
//   * three stages: iteration c waits for the wavefront's own DMAs of chunk
//     c+1 (every wavefront issues the same number per stage: absent rows read
//     a zero line, surplus kappa slots load into a junk block), publishes them
//     with one barrier, and runs the MFMAs of chunk c from registers with the
//     fragment reads of chunk c+1 and the DMAs of chunk c+2 spread between the
//     column blocks;
//   * rows without a neighbour at an offset contribute zeros (measured on the
//     benchmark surfaces, skipping at 16-row granularity would save ~1% of the
//     MFMA work but costs branches around every MFMA).
// Every output element is written once (fp32, or rounded to bf16).
// fp32 uses v_mfma_f32_16x16x4f32 (8 steps per chunk; lane group g = lane/16
// takes channels 8g..8g+7, one per step), bf16 v_mfma_f32_16x16x32_bf16 (one
// step; lane group g supplies channels 8g..8g+7).
#include "gather_mfma.hpp"
#include "norm.hpp"
#include "lds_dma.hpp"

namespace ssconv {
namespace {

typedef float f4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));

constexpr int kBK = 32;
constexpr int kMaxK = 128;
constexpr int kLdsLimit = 160 * 1024;

__device__ __attribute__((aligned(64))) const uint4 g_zero_line[4] = {};


// acc += A x B for one 32-wide chunk; a and b are this lane's fragment vectors.
__device__ __forceinline__ void mma_frag(f4& acc, const uint4 (&a)[2], const uint4 (&b)[2]) {
  acc = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a[0].x), __uint_as_float(b[0].x), acc, 0, 0, 0);
  acc = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a[0].y), __uint_as_float(b[0].y), acc, 0, 0, 0);
  acc = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a[0].z), __uint_as_float(b[0].z), acc, 0, 0, 0);
  acc = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a[0].w), __uint_as_float(b[0].w), acc, 0, 0, 0);
  acc = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a[1].x), __uint_as_float(b[1].x), acc, 0, 0, 0);
  acc = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a[1].y), __uint_as_float(b[1].y), acc, 0, 0, 0);
  acc = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a[1].z), __uint_as_float(b[1].z), acc, 0, 0, 0);
  acc = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a[1].w), __uint_as_float(b[1].w), acc, 0, 0, 0);
}
__device__ __forceinline__ void mma_frag(f4& acc, const uint4 (&a)[1], const uint4 (&b)[1]) {
  bf16x8 av, bv;
  __builtin_memcpy(&av, &a[0], 16);
  __builtin_memcpy(&bv, &b[0], 16);
  acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(av, bv, acc, 0, 0, 0);
}

template <typename T, int WMB, int WNB, int S, int NW>
struct Shape {
  static constexpr int NT = 64 * NW;                     // NW wavefronts
  static constexpr int BM = NW * WMB * 16;
  static constexpr int BN = WNB * 16;
  static constexpr int VE = 16 / (int)sizeof(T);         // elements per 16-byte vector
  static constexpr int RV = 8 / VE;                      // 16-byte vectors per lane per chunk
  static constexpr int BJ = (WNB + NW - 1) / NW;         // kappa blocks loaded per wavefront per chunk
  static constexpr int ABYTES = NW * WMB * RV * 1024;    // gathered rows of one stage
  static constexpr int BBYTES = WNB * RV * 1024;         // kappa chunk of one stage
  static constexpr int STAGE = ABYTES + BBYTES;
  static constexpr int L = (WMB + BJ) * RV;              // DMA loads per wavefront per stage
};

// Neighbour-index table entries: 32-bit, or 16-bit (0xFFFF = none) when the source has fewer than
// 65535 rows, which halves the table for large offset counts.
template <typename IX>
__device__ __forceinline__ int ix_get(IX v) {
  if constexpr (sizeof(IX) == 2) return v == (IX)0xFFFF ? -1 : (int)v;
  return (int)v;
}

template <typename T, int WMB, int WNB, int S, int NW, typename IX, bool kStats>
__global__ __launch_bounds__(64 * NW) void gather_mfma_kernel(const T* __restrict__ src, int ca,
                                                          const T* __restrict__ Bt, int cb,
                                                          const int32_t* __restrict__ nbr,
                                                          const int32_t* __restrict__ order, int64_t n_pos, int K,
                                                          T* __restrict__ out, float* __restrict__ part,
                                                          double* __restrict__ stats) {
  using SH = Shape<T, WMB, WNB, S, NW>;
  constexpr int BM = SH::BM, RV = SH::RV, VE = SH::VE, BJ = SH::BJ, L = SH::L;
  // dynamic LDS only (base at LDS address 0): stages | junk | bmask | act | count | index table
  extern __shared__ __attribute__((aligned(16))) char smem[];
  char* stages = smem;                                                         // S * STAGE bytes
  char* junk = smem + S * SH::STAGE;                                           // 1 KB sink
  uint32_t* bmask = reinterpret_cast<uint32_t*>(junk + 1024);                  // [kMaxK]
  uint8_t* act = reinterpret_cast<uint8_t*>(bmask + kMaxK);                    // [kMaxK]
  int* n_act_p = reinterpret_cast<int*>(act + kMaxK);                          // [4]
  IX* idx_tab = reinterpret_cast<IX*>(n_act_p + 4);                            // [K][BM]

  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6, g = lane >> 4, r16 = lane & 15;
  const int64_t p0 = (int64_t)blockIdx.x * BM;
  const int n0 = blockIdx.y * SH::BN;

  // 1. neighbour indices of the tile (all offsets) and the 16-row blocks each offset touches
  for (int s = w; s < K; s += NW) {
    uint32_t m = 0;
#pragma unroll
    for (int j = 0; j < BM / 64; ++j) {
      const int64_t p = p0 + 64 * j + lane;
      const int idx = p < n_pos ? nbr[(int64_t)s * n_pos + p] : -1;
      idx_tab[s * BM + 64 * j + lane] = (IX)idx;
      const uint64_t b = __ballot(idx >= 0);
#pragma unroll
      for (int q = 0; q < 4; ++q)
        if ((b >> (16 * q)) & 0xffffull) m |= 1u << (4 * j + q);
    }
    if (lane == 0) bmask[s] = m;
  }
  __syncthreads();
  // 2. ordered list of the offsets present in the tile
  if (w == 0) {
    int base = 0;
    for (int s0 = 0; s0 < K; s0 += 64) {
      const int s = s0 + lane;
      const bool a = s < K && bmask[s] != 0;
      const uint64_t b = __ballot(a);
      if (a) act[base + __popcll(b & ((1ull << lane) - 1ull))] = (uint8_t)s;
      base += __popcll(b);
    }
    if (lane == 0) n_act_p[0] = base;
  }
  __syncthreads();
  // split z of gridDim.z takes its share of the present offsets, in order, and writes an fp32
  // partial (part != nullptr); the splits are added in order by split_reduce_kernel
  const int nsplit = gridDim.z, z = blockIdx.z;  // at most 8 splits of at most 128 offsets
  const int a0 = n_act_p[0] * z / nsplit;
  const int n_act = n_act_p[0] * (z + 1) / nsplit - a0;
  const int total = n_act * ca;
  const int nchunk = (total + kBK - 1) / kBK;

  // Gather state of this lane group's 8-channel run (flat position c*32 + 8g -> slot, channel):
  // per 16-row block a source pointer, per kappa slot a source pointer.  They advance by one
  // chunk per issue and are recomputed only when the run crosses into the next offset.
  int r_slot = 0, r_ch = 8 * g;
  while (r_ch >= ca && r_slot < n_act) r_ch -= ca, ++r_slot;
  const uint32_t stage0 = lds_addr(stages), junk_a = lds_addr(junk);
  const T* const zero = reinterpret_cast<const T*>(g_zero_line);
  const T* ap[WMB];
  const T* bp[BJ];
  bool alive[WMB], bok[BJ];

#define SSC_REFRESH()                                                                               \
  do {                                                                                              \
    const bool live_ = r_slot < n_act;                                                              \
    const int s_ = live_ ? act[a0 + r_slot] : 0;                                                    \
    _Pragma("unroll") for (int mb = 0; mb < WMB; ++mb) {                                            \
      const int idx_ = live_ ? ix_get(idx_tab[s_ * BM + 16 * (w * WMB + mb) + r16]) : -1;           \
      alive[mb] = idx_ >= 0;                                                                        \
      ap[mb] = alive[mb] ? src + (int64_t)idx_ * ca + r_ch : zero;                                  \
    }                                                                                               \
    _Pragma("unroll") for (int j = 0; j < BJ; ++j) {                                                \
      const int nb_ = w + NW * j;                                                                   \
      const int n_ = n0 + 16 * nb_ + r16;                                                           \
      bok[j] = nb_ < WNB && live_ && n_ < cb;                                                       \
      bp[j] = bok[j] ? Bt + ((int64_t)s_ * cb + n_) * ca + r_ch : zero;                             \
    }                                                                                               \
  } while (0)

  // DMA q of this wavefront for the chunk going into stage st_: q < WMB*RV -> row block q / RV,
  // vector q % RV; else kappa slot (q - WMB*RV) / RV (a slot past WNB loads into the junk block)
#define SSC_DMA(q_, st_)                                                                            \
  do {                                                                                              \
    const uint32_t abase_ = stage0 + (st_) * SH::STAGE;                                             \
    if ((q_) < WMB * RV) {                                                                          \
      const int mb_ = (q_) / RV, v_ = (q_) % RV;                                                    \
      dma16(ap[mb_] + (alive[mb_] ? v_ * VE : 0), abase_ + ((w * WMB + mb_) * RV + v_) * 1024);     \
    } else {                                                                                        \
      const int j_ = ((q_) - WMB * RV) / RV, v_ = ((q_) - WMB * RV) % RV;                           \
      const int nb_ = w + NW * j_;                                                                  \
      dma16(bp[j_] + (bok[j_] ? v_ * VE : 0),                                                       \
            nb_ < WNB ? abase_ + SH::ABYTES + (nb_ * RV + v_) * 1024 : junk_a);                     \
    }                                                                                               \
  } while (0)

#define SSC_ADVANCE()                                                                               \
  do {                                                                                              \
    r_ch += kBK;                                                                                    \
    if (r_ch >= ca) {                                                                               \
      while (r_ch >= ca) r_ch -= ca, ++r_slot;                                                      \
      SSC_REFRESH();                                                                                \
    } else {                                                                                        \
      _Pragma("unroll") for (int mb = 0; mb < WMB; ++mb) ap[mb] += alive[mb] ? kBK : 0;             \
      _Pragma("unroll") for (int j = 0; j < BJ; ++j) bp[j] += bok[j] ? kBK : 0;                     \
    }                                                                                               \
  } while (0)

#define SSC_ISSUE(c_)                                                                               \
  do {                                                                                              \
    _Pragma("unroll") for (int q = 0; q < L; ++q) SSC_DMA(q, (c_) % S);                             \
    SSC_ADVANCE();                                                                                  \
  } while (0)

  // fragment u of the chunk in stage base sb_: u < WMB*RV -> row block u / RV, vector u % RV;
  // else kappa block (u - WMB*RV) / RV
  constexpr int NR = (WMB + WNB) * RV;
#define SSC_FRAG(AF, BF, u_, sb_)                                                                   \
  do {                                                                                              \
    if ((u_) < WMB * RV)                                                                            \
      AF[(u_) / RV][(u_) % RV] =                                                                    \
          *reinterpret_cast<const uint4*>((sb_) + ((w * WMB + (u_) / RV) * RV + (u_) % RV) * 1024 + 16 * lane); \
    else                                                                                            \
      BF[((u_) - WMB * RV) / RV][((u_) - WMB * RV) % RV] =                                          \
          *reinterpret_cast<const uint4*>((sb_) + SH::ABYTES + ((u_) - WMB * RV) * 1024 + 16 * lane); \
  } while (0)

  SSC_REFRESH();

  f4 acc[WMB][WNB];
#pragma unroll
  for (int mb = 0; mb < WMB; ++mb)
#pragma unroll
    for (int nb = 0; nb < WNB; ++nb) acc[mb][nb] = f4{0.f, 0.f, 0.f, 0.f};

  // Software pipeline over the chunks (S = 3 or 4 stages): iteration c waits for this wavefront's
  // DMAs of chunk c+1 (chunk c+2's may stay in flight with four stages), publishes them with one
  // barrier, then runs the MFMAs of chunk c (fragments already
  // in registers) one column block at a time, with the fragment reads of chunk c+1 and the DMAs
  // of chunk c+S-1 spread between the blocks.  The stage refilled in iteration c held chunk c-1,
  // whose fragments were consumed by the MFMAs of iteration c-1, before this barrier.
  static_assert(S == 3 || S == 4, "the pipelined chunk loop is written for three or four stages");
  for (int c = 0; c < S - 1 && c < nchunk; ++c) SSC_ISSUE(c);
  uint4 fa0[WMB][RV], fb0[WNB][RV], fa1[WMB][RV], fb1[WNB][RV];
  if (nchunk > 0) {
    if (nchunk >= S - 1) wait_vm<L * (S - 2)>(); else wait_vm<0>();
    __syncthreads();
#pragma unroll
    for (int u = 0; u < NR; ++u) SSC_FRAG(fa0, fb0, u, stages);
  }
#define SSC_BODY(k_, AC, BC, AN, BN)                                                                \
  {                                                                                                 \
    const int cc_ = c + (k_);                                                                       \
    if (cc_ >= nchunk) break;                                                                       \
    if (cc_ + S - 2 < nchunk)                                                                       \
      wait_vm<L * (S - 3)>();                                                                       \
    else                                                                                            \
      wait_vm<0>();                                                                                 \
    __syncthreads();                                                                                \
    const bool rd_ = cc_ + 1 < nchunk;                                                              \
    const bool iss_ = cc_ + S - 1 < nchunk;                                                         \
    const int ks_ = (cc_ + S - 1) % S;                                                              \
    const char* sbr_ = stages + ((cc_ + 1) % S) * SH::STAGE;                                        \
    __builtin_amdgcn_sched_barrier(0);                                                              \
    _Pragma("unroll") for (int nb = 0; nb < WNB; ++nb) {                                            \
      _Pragma("unroll") for (int mb = 0; mb < WMB; ++mb) mma_frag(acc[mb][nb], AC[mb], BC[nb]);     \
      __builtin_amdgcn_sched_barrier(0);                                                            \
      if (rd_) {                                                                                    \
        _Pragma("unroll") for (int u = (nb * NR + WNB - 1) / WNB; u < ((nb + 1) * NR + WNB - 1) / WNB; ++u) \
          SSC_FRAG(AN, BN, u, sbr_);                                                                \
      }                                                                                             \
      if (iss_) {                                                                                   \
        _Pragma("unroll") for (int q = (nb * L + WNB - 1) / WNB; q < ((nb + 1) * L + WNB - 1) / WNB; ++q) \
          SSC_DMA(q, ks_);                                                                          \
      }                                                                                             \
      __builtin_amdgcn_sched_barrier(0);                                                            \
    }                                                                                               \
    if (iss_) SSC_ADVANCE();                                                                        \
  }
  for (int c = 0;; c += 2) {
    SSC_BODY(0, fa0, fb0, fa1, fb1)
    SSC_BODY(1, fa1, fb1, fa0, fb0)
  }
#undef SSC_BODY
#undef SSC_FRAG
#undef SSC_ADVANCE
#undef SSC_DMA
#undef SSC_ISSUE
#undef SSC_REFRESH

  if (part) {
#pragma unroll
    for (int mb = 0; mb < WMB; ++mb) {
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int64_t p = p0 + 16 * (w * WMB + mb) + 4 * g + i;
        if (p >= n_pos) continue;
        float* prow = part + ((int64_t)z * n_pos + p) * cb;
#pragma unroll
        for (int nb = 0; nb < WNB; ++nb) {
          const int col = n0 + 16 * nb + r16;
          if (col < cb) prow[col] = acc[mb][nb][i];
        }
      }
    }
    return;
  }
#pragma unroll
  for (int mb = 0; mb < WMB; ++mb) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int64_t p = p0 + 16 * (w * WMB + mb) + 4 * g + i;
      if (p >= n_pos) continue;
      const int64_t row = order ? order[p] : p;
      T* orow = out + row * cb;
#pragma unroll
      for (int nb = 0; nb < WNB; ++nb) {
        const int col = n0 + 16 * nb + r16;
        if (col < cb) orow[col] = DT<T>::from_f(acc[mb][nb][i]);
      }
    }
  }
  if constexpr (kStats) {
    // Norm statistics of the stored values, per column of the tile: each lane adds its rows in
    // row order, the four lane groups are added pairwise (the same sum in every lane), then the
    // wavefronts in wavefront order; stats[(col * row tiles + row tile) * 2 + q] in fp64
    static_assert(NW * SH::BN * 16 <= S * SH::STAGE, "the statistics exchange must fit the stage area");
    __syncthreads();  // every wavefront is past its last read of the stage area
    double* red = reinterpret_cast<double*>(stages);  // [NW][BN][2]
#pragma unroll
    for (int nb = 0; nb < WNB; ++nb) {
      double s1 = 0.0, s2 = 0.0;
#pragma unroll
      for (int mb = 0; mb < WMB; ++mb)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int64_t p = p0 + 16 * (w * WMB + mb) + 4 * g + i;
          if (p < n_pos) {
            const double v = DT<T>::to_f(DT<T>::from_f(acc[mb][nb][i]));
            s1 += v;
            s2 = fma(v, v, s2);
          }
        }
      s1 += __shfl_xor(s1, 16, 64);
      s2 += __shfl_xor(s2, 16, 64);
      s1 += __shfl_xor(s1, 32, 64);
      s2 += __shfl_xor(s2, 32, 64);
      if (g == 0) {
        red[(w * SH::BN + 16 * nb + r16) * 2] = s1;
        red[(w * SH::BN + 16 * nb + r16) * 2 + 1] = s2;
      }
    }
    __syncthreads();
    for (int c = tid; c < SH::BN; c += SH::NT) {
      const int col = n0 + c;
      if (col >= cb) continue;
      double a = 0.0, b = 0.0;
      for (int j = 0; j < NW; ++j) {
        a += red[(j * SH::BN + c) * 2];
        b += red[(j * SH::BN + c) * 2 + 1];
      }
      stats[((int64_t)col * gridDim.x + blockIdx.x) * 2] = a;
      stats[((int64_t)col * gridDim.x + blockIdx.x) * 2 + 1] = b;
    }
  }
}

// out[order ? order[p] : p][col] = sum over the splits, in split order, of part[z][p][col].
template <typename T>
__global__ __launch_bounds__(256) void split_reduce_kernel(const float* __restrict__ part, int nsplit, int64_t n_pos,
                                                           int cb, const int32_t* __restrict__ order,
                                                           T* __restrict__ out) {
  const int64_t e = (int64_t)blockIdx.x * 256 + threadIdx.x;
  const int64_t n = n_pos * cb;
  if (e >= n) return;
  float acc = part[e];
  for (int z = 1; z < nsplit; ++z) acc += part[(int64_t)z * n + e];
  const int64_t p = e / cb, col = e - p * cb;
  out[(order ? order[p] : p) * cb + col] = DT<T>::from_f(acc);
}

// The same sums in row blocks (the layout of stats_rows), with the Norm statistics of what it writes.
template <typename T, int VEC>
__global__ __launch_bounds__(kStatsThreads) void split_reduce_stats_kernel(const float* __restrict__ part, int nsplit,
                                                                           int64_t n_pos, int cb,
                                                                           const int32_t* __restrict__ order, int G,
                                                                           int64_t rpb, T* __restrict__ out,
                                                                           double* __restrict__ stats) {
  const int64_t n = n_pos * cb;
  stats_rows<VEC>(
      cb, n_pos, G, rpb,
      [&](int64_t p, int v, float* val) {
        const int64_t e = p * cb + v * VEC;
        T* o = out + (order ? order[p] : p) * cb + v * VEC;
#pragma unroll
        for (int k = 0; k < VEC; ++k) {
          float acc = part[e + k];
          for (int z = 1; z < nsplit; ++z) acc += part[(int64_t)z * n + e + k];
          const T q = DT<T>::from_f(acc);
          o[k] = q;
          val[k] = DT<T>::to_f(q);
        }
      },
      stats);
}

template <typename T, int WMB, int WNB, int S, int NW, typename IX>
size_t smem_bytes(int K) {
  using SH = Shape<T, WMB, WNB, S, NW>;
  return (size_t)S * SH::STAGE + 1024 + kMaxK * 5 + 16 + (size_t)K * SH::BM * sizeof(IX);
}

// Offset splits for a launch of `tiles` workgroups (one per compute unit at a time): the count in
// 1..8 (at most K) with the fewest rounds of the 256 compute units per unit of work, each split
// charged 3% for its own index loading and partial traffic; 1 when the tiles fill the chip.
int pick_nsplit(int64_t tiles, int K) {
  constexpr int64_t kCUs = 256;
  int best = 1;
  double best_cost = 1e30;
  for (int ns = 1; ns <= 8 && ns <= K; ++ns) {
    const double rounds = (double)((tiles * ns + kCUs - 1) / kCUs);
    const double cost = rounds / ns + 0.03 * (ns - 1);
    if (cost < best_cost - 1e-9) best_cost = cost, best = ns;
  }
  return best;
}

template <typename T, int WMB, int WNB, int S, int NW, typename IX>
int launch(const void* src, int ca, const void* Bt, int cb, const int32_t* nbr, const int32_t* order, int64_t n_pos,
           int K, void* out, hipStream_t st, CallScratch* sc, NormSink* sink) {
  using SH = Shape<T, WMB, WNB, S, NW>;
  const size_t smem = smem_bytes<T, WMB, WNB, S, NW, IX>(K);
  const int64_t mt = cdiv(n_pos, SH::BM), nt = cdiv(cb, SH::BN);
  int nsplit = debug_gather_variant() == 8 ? std::min(K, 3) : pick_nsplit(mt * nt, K);
  if (sc && sc->fixed())
    while (nsplit > 1 && (size_t)nsplit * n_pos * cb * 4 > sc->left()) --nsplit;
  if (nsplit == 1 && sink) {  // the tiles also sum the Norm statistics of what they write
    auto kern = gather_mfma_kernel<T, WMB, WNB, S, NW, IX, true>;
    SSC_HIP(hipFuncSetAttribute((const void*)kern, hipFuncAttributeMaxDynamicSharedMemorySize, (int)smem));
    SSC_TRY(norm_sink_take(sink, mt, st));
    kern<<<dim3(mt, nt, 1), SH::NT, smem, st>>>((const T*)src, ca, (const T*)Bt, cb, nbr, order, n_pos, K, (T*)out,
                                                 nullptr, (double*)sink->ws);
    SSC_HIP(hipGetLastError());
    return SSCONV_OK;
  }
  auto kern = gather_mfma_kernel<T, WMB, WNB, S, NW, IX, false>;
  SSC_HIP(hipFuncSetAttribute((const void*)kern, hipFuncAttributeMaxDynamicSharedMemorySize, (int)smem));
  if (nsplit == 1) {
    kern<<<dim3(mt, nt, 1), SH::NT, smem, st>>>((const T*)src, ca, (const T*)Bt, cb, nbr, order, n_pos, K, (T*)out,
                                                 nullptr, nullptr);
    SSC_HIP(hipGetLastError());
    return SSCONV_OK;
  }
  float* part = nullptr;
  SSC_TRY(scratch_take(sc, (void**)&part, (size_t)nsplit * n_pos * cb * 4, st));
  kern<<<dim3(mt, nt, nsplit), SH::NT, smem, st>>>((const T*)src, ca, (const T*)Bt, cb, nbr, order, n_pos, K,
                                                    (T*)out, part, nullptr);
  hipError_t e = hipGetLastError();
  int rc = SSCONV_OK;
  StatsRows sr;
  const int vec = cb % 4 == 0 ? 4 : 1;
  if (e == hipSuccess && sink && stats_rows_plan(n_pos, cb, vec, &sr)) {
    rc = norm_sink_take(sink, sr.nblk, st);
    if (rc == SSCONV_OK) {
      double* stats = (double*)sink->ws;
      if (vec == 4)
        split_reduce_stats_kernel<T, 4><<<sr.nblk, kStatsThreads, 0, st>>>(part, nsplit, n_pos, cb, order, sr.G,
                                                                            sr.rpb, (T*)out, stats);
      else
        split_reduce_stats_kernel<T, 1><<<sr.nblk, kStatsThreads, 0, st>>>(part, nsplit, n_pos, cb, order, sr.G,
                                                                            sr.rpb, (T*)out, stats);
      e = hipGetLastError();
    }
  } else if (e == hipSuccess) {
    split_reduce_kernel<T><<<cdiv(n_pos * cb, 256), 256, 0, st>>>(part, nsplit, n_pos, cb, order, (T*)out);
    e = hipGetLastError();
  }
  scratch_give(sc, part, st);
  if (rc != SSCONV_OK) return rc;
  if (e != hipSuccess) return fail(SSCONV_E_HIP, "gather launch: %s", hipGetErrorString(e));
  return SSCONV_OK;
}


// Tile configurations, best first; the first whose LDS footprint fits is used.
struct Cfg {
  int wmb, wnb, stages, nw;  // row blocks per wavefront, column blocks, LDS stages, wavefronts
  bool idx16;                // 16-bit neighbour-index table
};

template <typename T>
size_t cfg_smem(const Cfg& c, int K) {
  const int VE = 16 / (int)sizeof(T), RV = 8 / VE;
  return (size_t)c.stages * (c.nw * c.wmb + c.wnb) * RV * 1024 + 1024 + kMaxK * 5 + 16 +
         (size_t)K * c.nw * c.wmb * 16 * (c.idx16 ? 2 : 4);
}

int column_blocks(ssconv_dtype dt, int cb) {
  const int blocks = (cb + 15) / 16;
  if (dt == SSCONV_BF16) return blocks <= 4 ? 4 : blocks <= 8 ? 8 : blocks <= 13 ? 13 : 8;
  const int tiles = (blocks + 7) / 8;
  return (blocks + tiles - 1) / tiles;  // fp32: at most 8 column blocks per tile
}

bool pick_cfg(ssconv_dtype dt, int cb, int K, int64_t n_src, Cfg* out) {
  const int wnb = column_blocks(dt, cb);
  // fp32: eight wavefronts of 16 rows (two per SIMD, so one issues MFMAs while the other waits on
  // its DMAs, LDS reads or the barrier), four stages where the LDS allows, else four wavefronts
  // of 32 or 16 rows; a 16-bit index table when the source has fewer than 65535 rows
  const Cfg f32[] = {{1, wnb, 4, 8, true}, {1, wnb, 3, 8, true}, {1, wnb, 3, 8, false},
                     {2, wnb, 3, 4, false}, {1, wnb, 3, 4, false}};
  const Cfg b16[] = {{2, wnb, 3, 4, false}, {1, wnb, 3, 4, false}};
  const Cfg* list = dt == SSCONV_F32 ? f32 : b16;
  const int n = dt == SSCONV_F32 ? 5 : 2;
  for (int i = 0; i < n; ++i) {
    if (list[i].idx16 && n_src >= 0xFFFF) continue;
    const size_t need = dt == SSCONV_F32 ? cfg_smem<float>(list[i], K) : cfg_smem<uint16_t>(list[i], K);
    if (need <= (size_t)kLdsLimit) {
      *out = list[i];
      return true;
    }
  }
  return false;
}

template <typename T, int WMB, int S, int NW, typename IX>
int launch_wnb(int wnb, const void* src, int ca, const void* Bt, int cb, const int32_t* nbr, const int32_t* order,
               int64_t n_pos, int K, void* out, hipStream_t st, CallScratch* sc, NormSink* sink) {
  switch (wnb) {
    case 1: return launch<T, WMB, 1, S, NW, IX>(src, ca, Bt, cb, nbr, order, n_pos, K, out, st, sc, sink);
    case 2: return launch<T, WMB, 2, S, NW, IX>(src, ca, Bt, cb, nbr, order, n_pos, K, out, st, sc, sink);
    case 3: return launch<T, WMB, 3, S, NW, IX>(src, ca, Bt, cb, nbr, order, n_pos, K, out, st, sc, sink);
    case 4: return launch<T, WMB, 4, S, NW, IX>(src, ca, Bt, cb, nbr, order, n_pos, K, out, st, sc, sink);
    case 5: return launch<T, WMB, 5, S, NW, IX>(src, ca, Bt, cb, nbr, order, n_pos, K, out, st, sc, sink);
    case 6: return launch<T, WMB, 6, S, NW, IX>(src, ca, Bt, cb, nbr, order, n_pos, K, out, st, sc, sink);
    case 7: return launch<T, WMB, 7, S, NW, IX>(src, ca, Bt, cb, nbr, order, n_pos, K, out, st, sc, sink);
    case 8: return launch<T, WMB, 8, S, NW, IX>(src, ca, Bt, cb, nbr, order, n_pos, K, out, st, sc, sink);
    default: return launch<T, WMB, 13, S, NW, IX>(src, ca, Bt, cb, nbr, order, n_pos, K, out, st, sc, sink);
  }
}

}  // namespace

bool gather_mfma_supported(ssconv_dtype dt, int ca, int cb, int K) {
  Cfg c;  // the 32-bit index table fits whenever any configuration does
  return ca % 8 == 0 && ca >= 8 && K <= kMaxK && pick_cfg(dt, cb, K, INT64_MAX, &c);
}

int gather_mfma(const void* src, int64_t n_src, ssconv_dtype dt, int ca, const void* Bt, int cb, const int32_t* nbr,
                const int32_t* order, int64_t n_pos, int K, void* out, hipStream_t st, CallScratch* sc,
                NormSink* sink) {
  if (n_pos == 0) return SSCONV_OK;
  // tuning overrides (same results): 1 = four wavefronts of 32 rows, 2 = four of 16 rows,
  // 3 = no 16-bit index table, 8 = three offset splits (in launch)
  const int64_t variant = debug_gather_variant();
  Cfg c;
  if (!pick_cfg(dt, cb, K, variant == 3 ? INT64_MAX : n_src, &c))
    return fail(SSCONV_E_INVALID, "no gather tile fits the LDS for K=%d", K);
  if (variant == 1 && cfg_smem<float>({2, c.wnb, 3, 4, false}, K) <= (size_t)kLdsLimit) c = {2, c.wnb, 3, 4, false};
  if (variant == 2) c = {1, c.wnb, 3, 4, false};
#define SSC_GO(T, WMB, S, NW, IX) \
  return launch_wnb<T, WMB, S, NW, IX>(c.wnb, src, ca, Bt, cb, nbr, order, n_pos, K, out, st, sc, sink)
  if (dt == SSCONV_F32) {
    if (c.nw == 8 && c.idx16 && c.stages == 4) SSC_GO(float, 1, 4, 8, uint16_t);
    if (c.nw == 8 && c.idx16) SSC_GO(float, 1, 3, 8, uint16_t);
    if (c.nw == 8) SSC_GO(float, 1, 3, 8, int32_t);
    if (c.wmb == 2) SSC_GO(float, 2, 3, 4, int32_t);
    SSC_GO(float, 1, 3, 4, int32_t);
  }
  if (c.wmb == 2) SSC_GO(uint16_t, 2, 3, 4, int32_t);
  SSC_GO(uint16_t, 1, 3, 4, int32_t);
#undef SSC_GO
}

}  // namespace ssconv
