// bf16 output-stationary gather -> MFMA GEMM (Sec. 3.2.3, Alg. 1 feature update):
//
//   out[x] = sum_s kappa(s) in[nbr[s][x]]   for the 256 output rows x of a tile
//
// The reduction dimension is the concatenation, over the offsets present in the tile, of each
// offset's input channels, cut into 32-wide chunks (one v_mfma_f32_16x16x32_bf16 step each);
// a chunk may straddle two offsets, so no channel padding is paid per offset.
//
// Layout and data movement (gfx950), chosen from measurement:
//   * eight wavefronts, two per SIMD: row group wm = w % 4 (64 rows) x column group wn = w / 4
//     (ceil(NB/2) or floor(NB/2) 16-column blocks); the two wavefronts of a SIMD cover
//     complementary column groups, so with an odd block count the SIMD still does exactly the
//     tile's MFMA work, and one wavefront issues MFMAs while the other is stalled on issue;
//   * both operands reach LDS by DMA (16 bytes per lane, written at M0 + 16 * lane): gathered
//     rows with buffer DMA on 32-bit row offsets (an absent neighbour gets an offset past the
//     end of the buffer, which the hardware fills with zeros), kappa from a packed copy
//     Bp[K][ca/8][cb][8] so that a 16-column block of one chunk is four contiguous 256-byte
//     runs; no operand is loaded into registers asynchronously;
//   * four LDS stages: iteration c waits for its own DMAs of chunk c+1, publishes them with one
//     barrier, then runs the MFMAs of chunk c with the LDS fragment reads of chunk c+1 and the
//     four DMAs of chunk c+3 spread between the column blocks (issuing them in a burst stalls
//     the wavefront for the texture path's whole backlog);
//   * the row offsets of the tile are compacted per active offset once, and each lane reads the
//     next offset's rows ahead, so crossing into the next offset costs no LDS round trip;
//   * tiles are mapped XCD-contiguously (workgroups are dispatched round-robin over the 8 XCDs;
//     workgroup i runs tile (i % 8) * ceil(T / 8) + i / 8), so each XCD's L2 sees neighbouring
//     tiles, which share gathered rows;
//   * the epilogue stages each wavefront's rows in LDS and writes 16-byte pieces of rows.
#include "gather_mfma.hpp"
#include "lds_dma.hpp"
#include "norm.hpp"

namespace ssconv {
namespace {

typedef float f4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));

constexpr int kNT = 512;        // 8 wavefronts, two per SIMD
constexpr int kBM = 256;        // output rows per tile
constexpr int kBK = 32;         // reduction channels per chunk
constexpr int kD = 4;           // pipeline depth: LDS stages (gathered rows + kappa of one chunk)
constexpr int kMaxK = 128;
constexpr int kLdsLimit = 160 * 1024;

constexpr uint32_t kAbsent = 0x80000000u;         // row offset past any src: the DMA writes zeros
constexpr int kBufferWord3 = 0x00020000;          // buffer descriptor word 3 for gfx9-family raw loads

template <int NB>
struct GB {
  static constexpr int WN0 = (NB + 1) / 2;          // column blocks of column group 0
  static constexpr int WN1 = NB - WN0;              // ... and of column group 1
  static constexpr int ABYTES = (kBM / 16) * 1024;  // gathered rows of one chunk (16-row blocks)
  static constexpr int STAGE = ABYTES + NB * 1024;  // + kappa blocks
  static constexpr int L = 4;                       // DMAs per wavefront per chunk: 2 row blocks, 2 kappa slots
  static constexpr int PITCH = WN0 * 32 + 16;       // bytes per staged output row in the epilogue
};

template <int NB>
size_t bf16_smem(int K) {
  return (size_t)kD * GB<NB>::STAGE + 1024 + kMaxK * 5 + 16 + (size_t)K * kBM * 4;
}

// Workgroup i -> tile index such that each XCD (i % 8) runs a contiguous range of tiles.
__device__ __forceinline__ int64_t xcd_tile(int64_t i, int64_t total) {
  const int64_t x = i & 7, j = i >> 3, q = total >> 3, r = total & 7;
  return (x < r ? x * (q + 1) : r * (q + 1) + (x - r) * q) + j;
}

#pragma clang diagnostic push
#pragma clang diagnostic ignored "-Winline-asm"
// 16 bytes per lane at byte offset off of the buffer described by rsrc into LDS at byte
// lds + 16 * lane (buffer_load_dwordx4 with the LDS bit; an offset past the end of the buffer
// writes zeros).  One wait state separates the M0 write from the DMA.
__device__ __forceinline__ void dma16_buf(__amdgpu_buffer_rsrc_t rsrc, uint32_t off, uint32_t lds) {
  const uint32_t l = __builtin_amdgcn_readfirstlane(lds);
  asm volatile("s_mov_b32 m0, %0\n\ts_nop 0\n\tbuffer_load_dwordx4 %1, %2, 0 offen lds" ::"s"(l), "v"(off), "s"(rsrc)
               : "memory", "m0");
}
#pragma clang diagnostic pop

template <int NB, bool kStats>
__global__ __launch_bounds__(kNT) void gather_bf16_kernel(const uint16_t* __restrict__ src, int64_t src_bytes, int ca,
                                                          const uint16_t* __restrict__ Bp, int cb,
                                                          const int32_t* __restrict__ nbr,
                                                          const int32_t* __restrict__ order, int64_t n_pos, int K,
                                                          uint16_t* __restrict__ out, double* __restrict__ stats) {
  using G = GB<NB>;
  constexpr int WN0 = G::WN0, WN1 = G::WN1, L = G::L;
  extern __shared__ __attribute__((aligned(16))) char smem[];
  char* stages = smem;                                         // kD * STAGE bytes
  char* junk = smem + kD * G::STAGE;                           // 1 KB sink
  uint32_t* bmask = reinterpret_cast<uint32_t*>(junk + 1024);  // [kMaxK]
  uint8_t* act = reinterpret_cast<uint8_t*>(bmask + kMaxK);    // [kMaxK]
  int* n_act_p = reinterpret_cast<int*>(act + kMaxK);          // [4]
  uint32_t* rows = reinterpret_cast<uint32_t*>(n_act_p + 4);   // [K][kBM] byte offsets of gathered rows

  const int tid = threadIdx.x, lane = tid & 63, g = lane >> 4, r16 = lane & 15;
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6);  // wavefront index, scalar
  const int wm = w & 3, wn = w >> 2;  // row group and column group; SIMD w % 4 hosts (wm, 0), (wm, 1)
  const int64_t lin = (int64_t)blockIdx.y * gridDim.x + blockIdx.x;
  const int64_t t = xcd_tile(lin, (int64_t)gridDim.x * gridDim.y);
  const int64_t p0 = (t / gridDim.y) * kBM;
  const int n0 = (int)(t % gridDim.y) * NB * 16;
  const uint32_t row_bytes = (uint32_t)ca * 2u;

  // 1. neighbour rows of the tile (all offsets) as byte offsets into src (kAbsent: no neighbour)
  //    and whether each offset occurs in the tile; thread tid owns tile row tid % 256 for the
  //    offsets of parity tid / 256, and issues its loads in batches of 8 independent requests
  for (int s = tid; s < K; s += kNT) bmask[s] = 0u;
  __syncthreads();
  {
    const int r = tid & (kBM - 1), par = tid >> 8;
    const int64_t p = p0 + r;
    const bool in = p < n_pos;
    for (int s0 = par; s0 < K; s0 += 16) {
      int v[8];
#pragma unroll
      for (int j = 0; j < 8; ++j) v[j] = (in && s0 + 2 * j < K) ? nbr[(int64_t)(s0 + 2 * j) * n_pos + p] : -1;
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        if (s0 + 2 * j < K) {
          rows[(s0 + 2 * j) * kBM + r] = v[j] >= 0 ? (uint32_t)v[j] * row_bytes : kAbsent;
          if (v[j] >= 0) bmask[s0 + 2 * j] = 1u;
        }
      }
    }
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
  const int n_act = n_act_p[0];
  // 3. compact the row table to the active offsets (slot j <- offset act[j] >= j; each thread
  //    moves its own column in increasing j, so no entry is overwritten before it is read)
  if (tid < kBM)
    for (int j = 0; j < n_act; ++j) rows[j * kBM + tid] = rows[act[j] * kBM + tid];
  __syncthreads();
  const int nchunk = (n_act * ca + kBK - 1) / kBK;
  const int cg8 = ca / 8;

  // Gathered rows are fetched with buffer DMA (32-bit offsets; an offset past the end of src
  // writes zeros, which covers absent neighbours and the padding of the last chunk).
  const __amdgpu_buffer_rsrc_t src_rsrc =
      __builtin_amdgcn_make_buffer_rsrc(const_cast<uint16_t*>(src), (short)0, (int)src_bytes, kBufferWord3);

  // DMA duty of this wavefront per chunk: row blocks w and w + 8, kappa blocks w and w + 8.
  // This lane group's 8-channel run sits at flat position c*32 + 8g -> (slot, channel).  Per
  // row block the byte offset of this lane's row for the current slot, and the next slot's,
  // read ahead so that crossing into it needs no LDS round trip; per kappa block a byte offset
  // into Bp.  Offsets advance by one chunk per issue and are recomputed only when the run
  // crosses into the next offset.
  int r_slot = 0, r_ch = 8 * g;
  while (r_ch >= ca && r_slot < n_act) r_ch -= ca, ++r_slot;
  const uint32_t stage0 = lds_addr(stages), junk_a = lds_addr(junk);
  uint32_t arow[2], nrow[2], boff[2];
  bool bok[2];
  int s_cur = 0, s_nxt = 0, pslot = -1;
  const uint32_t bstep = 64u * (uint32_t)cb;  // packed kappa: +4 channel groups per chunk

#define SSB_PREFETCH()                                                                              \
  do {                                                                                              \
    pslot = r_slot + 1;                                                                             \
    const bool pl_ = pslot < n_act;                                                                 \
    s_nxt = pl_ ? act[pslot] : 0;                                                                   \
    _Pragma("unroll") for (int j = 0; j < 2; ++j)                                                   \
      nrow[j] = pl_ ? rows[pslot * kBM + 16 * (w + 8 * j) + r16] : kAbsent;                         \
  } while (0)

#define SSB_REFRESH()                                                                               \
  do {                                                                                              \
    const bool live_ = r_slot < n_act;                                                              \
    if (r_slot == pslot) {                                                                          \
      s_cur = s_nxt;                                                                                \
      _Pragma("unroll") for (int j = 0; j < 2; ++j) arow[j] = nrow[j];                              \
    } else {                                                                                        \
      s_cur = live_ ? act[r_slot] : 0;                                                              \
      _Pragma("unroll") for (int j = 0; j < 2; ++j)                                                 \
        arow[j] = live_ ? rows[r_slot * kBM + 16 * (w + 8 * j) + r16] : kAbsent;                    \
    }                                                                                               \
    _Pragma("unroll") for (int j = 0; j < 2; ++j) {                                                 \
      const int nb_ = w + 8 * j;                                                                    \
      const int n_ = n0 + 16 * nb_ + r16;                                                           \
      bok[j] = nb_ < NB && live_ && n_ < cb;                                                        \
      boff[j] = bok[j] ? (((uint32_t)s_cur * cg8 + (uint32_t)(r_ch >> 3)) * (uint32_t)cb + n_) * 16u : 0u; \
    }                                                                                               \
    SSB_PREFETCH();                                                                                 \
  } while (0)

  // DMA q (0, 1: row blocks; 2, 3: kappa slots) of the chunk going into LDS stage k_
#define SSB_DMA(q_, k_)                                                                             \
  do {                                                                                              \
    const int q__ = (q_);                                                                           \
    const uint32_t sbase_ = stage0 + (k_) * G::STAGE;                                               \
    if (q__ < 2) {                                                                                  \
      dma16_buf(src_rsrc, arow[q__ & 1] + 2u * r_ch, sbase_ + (w + 8 * (q__ & 1)) * 1024);          \
    } else {                                                                                        \
      const int nb_ = w + 8 * (q__ & 1);                                                            \
      dma16_off(Bp, boff[q__ & 1], nb_ < NB ? sbase_ + G::ABYTES + nb_ * 1024 : junk_a);            \
    }                                                                                               \
  } while (0)

#define SSB_ADVANCE()                                                                               \
  do {                                                                                              \
    r_ch += kBK;                                                                                    \
    if (r_ch >= ca) {                                                                               \
      while (r_ch >= ca) r_ch -= ca, ++r_slot;                                                      \
      SSB_REFRESH();                                                                                \
    } else {                                                                                        \
      _Pragma("unroll") for (int j = 0; j < 2; ++j) boff[j] += bok[j] ? bstep : 0u;                 \
    }                                                                                               \
  } while (0)

#define SSB_ISSUE(k_)                                                                               \
  do {                                                                                              \
    _Pragma("unroll") for (int q = 0; q < L; ++q) SSB_DMA(q, k_);                                   \
    SSB_ADVANCE();                                                                                  \
  } while (0)

  // fragments of the chunk in stage k_: this wavefront's four row blocks and its column blocks
#define SSB_READ(da_, db_, WNX, NOFF, k_)                                                           \
  do {                                                                                              \
    const char* sb_ = stages + (k_) * G::STAGE;                                                     \
    _Pragma("unroll") for (int mb = 0; mb < 4; ++mb)                                                \
      da_[mb] = *reinterpret_cast<const uint4*>(sb_ + (4 * wm + mb) * 1024 + 16 * lane);            \
    _Pragma("unroll") for (int nb = 0; nb < WNX; ++nb)                                              \
      db_[nb] = *reinterpret_cast<const uint4*>(sb_ + G::ABYTES + ((NOFF) + nb) * 1024 + 16 * lane); \
  } while (0)

  SSB_REFRESH();

  f4 acc[4][WN0];
#pragma unroll
  for (int mb = 0; mb < 4; ++mb)
#pragma unroll
    for (int nb = 0; nb < WN0; ++nb) acc[mb][nb] = f4{0.f, 0.f, 0.f, 0.f};

  if (nchunk > 0) SSB_ISSUE(0);
  if (nchunk > 1) SSB_ISSUE(1);
  if (nchunk > 2) SSB_ISSUE(2);

#define SSB_MMA(nb_, AC, BC)                                                                        \
  do {                                                                                              \
    bf16x8 bv_;                                                                                     \
    __builtin_memcpy(&bv_, &BC[nb_], 16);                                                           \
    _Pragma("unroll") for (int mb = 0; mb < 4; ++mb) {                                              \
      bf16x8 av_;                                                                                   \
      __builtin_memcpy(&av_, &AC[mb], 16);                                                          \
      acc[mb][nb_] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(av_, bv_, acc[mb][nb_], 0, 0, 0);      \
    }                                                                                               \
  } while (0)

  // Iteration c (stage k = c % kD): wait for this wavefront's DMA of chunk c+1, publish it with a
  // barrier (which also retires every LDS read of the stage refilled next: it was read two
  // chunks ago), read the fragments of chunk c+1, then the MFMAs of chunk c with the DMAs of
  // chunk c+kD-1 spread between the column blocks (DMA q after column block q), so that the
  // texture path drains while the matrix cores run.
#define SSB_BODY(k_, AC, BC, AN, BN, WNX, NOFF)                                                     \
  {                                                                                                 \
    const int cc_ = c + (k_);                                                                       \
    if (cc_ >= nchunk) break;                                                                       \
    if (cc_ + kD - 2 < nchunk)                                                                      \
      wait_vm<(kD - 3) * L>();                                                                      \
    else                                                                                            \
      wait_vm<0>();                                                                                 \
    __syncthreads();                                                                                \
    const bool rd_ = cc_ + 1 < nchunk;                                                              \
    const bool iss_ = cc_ + kD - 1 < nchunk;                                                        \
    constexpr int ks_ = ((k_) + kD - 1) % kD;                                                       \
    const char* sbr_ = stages + (((k_) + 1) % kD) * G::STAGE;                                       \
    __builtin_amdgcn_sched_barrier(0);                                                              \
    _Pragma("unroll") for (int nb = 0; nb < WNX; ++nb) {                                            \
      SSB_MMA(nb, AC, BC);                                                                          \
      __builtin_amdgcn_sched_barrier(0);                                                            \
      if (rd_) {                                                                                    \
        /* two fragment reads of chunk c+1 per column block: row blocks first, then kappa */        \
        _Pragma("unroll") for (int u = 2 * nb; u < 2 * nb + 2; ++u) {                               \
          if (u < 4)                                                                                \
            AN[u & 3] = *reinterpret_cast<const uint4*>(sbr_ + (4 * wm + (u & 3)) * 1024 + 16 * lane); \
          else if (u - 4 < WNX)                                                                     \
            BN[(u - 4) % WNX] = *reinterpret_cast<const uint4*>(sbr_ + G::ABYTES + ((NOFF) + (u - 4) % WNX) * 1024 + 16 * lane); \
        }                                                                                           \
      }                                                                                             \
      if (nb < L && iss_) SSB_DMA(nb, ks_);                                                         \
      __builtin_amdgcn_sched_barrier(0);                                                            \
    }                                                                                               \
    if (rd_) {                                                                                      \
      _Pragma("unroll") for (int u = 2 * WNX; u < 4 + WNX; ++u)                                     \
        BN[(u - 4) % WNX] = *reinterpret_cast<const uint4*>(sbr_ + G::ABYTES + ((NOFF) + (u - 4) % WNX) * 1024 + 16 * lane); \
    }                                                                                               \
    _Pragma("unroll") for (int q = WNX; q < L; ++q)                                                 \
      if (iss_) SSB_DMA(q, ks_);                                                                    \
    if (iss_) SSB_ADVANCE();                                                                        \
  }

  // Four chunks per trip; the first body past the last chunk leaves the loop.
#define SSB_LOOP(WNX, NOFF)                                                                         \
  {                                                                                                 \
    uint4 fa0[4], fb0[WNX], fa1[4], fb1[WNX];                                                       \
    if (nchunk > 0) {                                                                               \
      if (nchunk > 2) wait_vm<2 * L>(); else wait_vm<0>();                                          \
      __syncthreads();                                                                              \
      SSB_READ(fa0, fb0, WNX, NOFF, 0);                                                             \
    }                                                                                               \
    for (int c = 0;; c += kD) {                                                                     \
      SSB_BODY(0, fa0, fb0, fa1, fb1, WNX, NOFF)                                                    \
      SSB_BODY(1, fa1, fb1, fa0, fb0, WNX, NOFF)                                                    \
      SSB_BODY(2, fa0, fb0, fa1, fb1, WNX, NOFF)                                                    \
      SSB_BODY(3, fa1, fb1, fa0, fb0, WNX, NOFF)                                                    \
    }                                                                                               \
  }

  static_assert(kD == 4, "the unrolled chunk loop is written for four stages");
  if constexpr (WN0 == WN1) {
    SSB_LOOP(WN0, wn * WN0)
  } else {
    if (wn == 0) {
      SSB_LOOP(WN0, 0)
    } else {
      SSB_LOOP(WN1, WN0)
    }
  }
#undef SSB_LOOP
#undef SSB_BODY
#undef SSB_MMA
#undef SSB_READ
#undef SSB_ISSUE
#undef SSB_ADVANCE
#undef SSB_DMA
#undef SSB_REFRESH
#undef SSB_PREFETCH

  // Epilogue: each wavefront stages its rows, 32 at a time, as bf16 in LDS (row pitch padded so
  // the 2-byte writes of the four row groups fall in distinct banks) and writes them back as
  // 16-byte pieces of its column range of the output rows.
  static_assert(kNT / 64 * 32 * G::PITCH <= kD * G::STAGE, "epilogue staging must fit the stage area");
  __syncthreads();  // every wavefront is done with the stage area
  char* const ep = stages + w * 32 * G::PITCH;
  const int nbc = wn == 0 ? WN0 : WN1;
  const int col0 = n0 + 16 * WN0 * wn;
  const bool vec = (cb & 7) == 0;
#pragma unroll
  for (int half = 0; half < 2; ++half) {
#pragma unroll
    for (int m2 = 0; m2 < 2; ++m2) {
      const int mb = 2 * half + m2;
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int nb = 0; nb < WN0; ++nb)
          if (nb < nbc)
            *reinterpret_cast<uint16_t*>(ep + (16 * m2 + 4 * g + i) * G::PITCH + (16 * nb + r16) * 2) =
                f32_to_bf16_rne(acc[mb][nb][i]);
    }
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
    const int pieces = 2 * nbc;  // 16-byte pieces per staged row
    for (int e = lane; e < 32 * pieces; e += 64) {
      const int r = e / pieces, q = e - r * pieces;
      const int64_t p = p0 + 64 * wm + 32 * half + r;
      const int col = col0 + 8 * q;
      if (p >= n_pos || col >= cb) continue;
      const int64_t row = order ? order[p] : p;
      uint16_t* dst = out + row * cb + col;
      const char* srcp = ep + r * G::PITCH + q * 16;
      if (vec) {
        *reinterpret_cast<uint4*>(dst) = *reinterpret_cast<const uint4*>(srcp);
      } else {
        const int n = cb - col < 8 ? cb - col : 8;
        for (int j = 0; j < n; ++j) dst[j] = reinterpret_cast<const uint16_t*>(srcp)[j];
      }
    }
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
  }
  if constexpr (kStats) {
    // Norm statistics of the stored (bf16) values, per column of the tile: each lane adds its 16
    // rows in row order, the four lane groups are added pairwise (the same sum in every lane),
    // then the four row groups in order; stats[(col * row tiles + row tile) * 2 + q] in fp64
    static_assert(4 * NB * 16 * 16 <= kD * G::STAGE, "the statistics exchange must fit the stage area");
    __syncthreads();  // every wavefront is done with its staged rows
    double* red = reinterpret_cast<double*>(stages);  // [4 row groups][NB * 16 columns][2]
#pragma unroll
    for (int nb = 0; nb < WN0; ++nb) {
      if (nb >= nbc) break;
      double s1 = 0.0, s2 = 0.0;
#pragma unroll
      for (int mb = 0; mb < 4; ++mb)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int64_t p = p0 + 64 * wm + 16 * mb + 4 * g + i;
          if (p < n_pos) {
            const double v = bf16_to_f32(f32_to_bf16_rne(acc[mb][nb][i]));
            s1 += v;
            s2 = fma(v, v, s2);
          }
        }
      s1 += __shfl_xor(s1, 16, 64);
      s2 += __shfl_xor(s2, 16, 64);
      s1 += __shfl_xor(s1, 32, 64);
      s2 += __shfl_xor(s2, 32, 64);
      if (g == 0) {
        const int c = 16 * WN0 * wn + 16 * nb + r16;
        red[(wm * NB * 16 + c) * 2] = s1;
        red[(wm * NB * 16 + c) * 2 + 1] = s2;
      }
    }
    __syncthreads();
    const int64_t mt = t / gridDim.y;
    for (int c = tid; c < NB * 16; c += kNT) {
      const int col = n0 + c;
      if (col >= cb) continue;
      double a = 0.0, b = 0.0;
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        a += red[(j * NB * 16 + c) * 2];
        b += red[(j * NB * 16 + c) * 2 + 1];
      }
      stats[((int64_t)col * gridDim.x + mt) * 2] = a;
      stats[((int64_t)col * gridDim.x + mt) * 2 + 1] = b;
    }
  }
}

// Bp[s][k/8][n][k%8] from kappa given as Bt[s'][n][k] (transposed = 0) or as W[s'][k][n]
// (transposed = 1), s' = s or K-1-s (mirror); one thread per 16-byte output vector.
__global__ void pack_b_kernel(const uint16_t* __restrict__ W, int K, int ca, int cb, int transposed, int mirror,
                              uint16_t* __restrict__ Bp) {
  const int64_t v = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int cg8 = ca / 8;
  const int64_t total = (int64_t)K * cg8 * cb;
  if (v >= total) return;
  const int n = (int)(v % cb);
  const int kg = (int)((v / cb) % cg8);
  const int64_t s = mirror ? K - 1 - v / ((int64_t)cb * cg8) : v / ((int64_t)cb * cg8);
  uint4 o;
  if (!transposed) {
    o = *reinterpret_cast<const uint4*>(W + (s * cb + n) * ca + 8 * kg);
  } else {
    uint16_t e[8];
#pragma unroll
    for (int j = 0; j < 8; ++j) e[j] = W[(s * ca + 8 * kg + j) * cb + n];
    __builtin_memcpy(&o, e, 16);
  }
  *reinterpret_cast<uint4*>(Bp + v * 8) = o;
}

template <int NB>
int launch_bf16(const void* src, int64_t src_bytes, int ca, const void* Bp, int cb, const int32_t* nbr, const int32_t* order,
                int64_t n_pos, int K, void* out, hipStream_t st, NormSink* sink) {
  const size_t smem = bf16_smem<NB>(K);
  auto kern = sink ? gather_bf16_kernel<NB, true> : gather_bf16_kernel<NB, false>;
  SSC_HIP(hipFuncSetAttribute((const void*)kern, hipFuncAttributeMaxDynamicSharedMemorySize, (int)smem));
  dim3 grid(cdiv(n_pos, kBM), cdiv(cb, NB * 16));
  double* stats = nullptr;
  if (sink) {
    SSC_TRY(norm_sink_take(sink, grid.x, st));
    stats = (double*)sink->ws;
  }
  kern<<<grid, kNT, smem, st>>>((const uint16_t*)src, src_bytes, ca, (const uint16_t*)Bp, cb, nbr, order, n_pos, K,
                                (uint16_t*)out, stats);
  SSC_HIP(hipGetLastError());
  return SSCONV_OK;
}

// Column blocks per tile: the instantiated width that covers cb in the fewest, most even tiles.
int bf16_nb(int cb) {
  const int blocks = (cb + 15) / 16;
  const int tiles = (blocks + 13) / 14;
  const int per = (blocks + tiles - 1) / tiles;
  return per <= 4 ? 4 : per <= 8 ? 8 : per <= 13 ? 13 : 14;
}

size_t bf16_smem_for(int nb, int K) {
  switch (nb) {
    case 4: return bf16_smem<4>(K);
    case 8: return bf16_smem<8>(K);
    case 13: return bf16_smem<13>(K);
    default: return bf16_smem<14>(K);
  }
}

}  // namespace

bool gather_bf16_supported(int64_t n_src, int ca, int cb, int K) {
  // 32-bit byte offsets: every gathered row and every packed kappa entry below 2^31
  return ca % 8 == 0 && ca >= 8 && cb >= 1 && K >= 1 && K <= kMaxK && n_src >= 0 &&
         n_src * ca * 2 < ((int64_t)1 << 31) && (int64_t)K * ca * cb * 2 < ((int64_t)1 << 31) &&
         bf16_smem_for(bf16_nb(cb), K) <= (size_t)kLdsLimit;
}

int pack_b_bf16(const void* W, int K, int ca, int cb, bool transposed, bool mirror, void* Bp, hipStream_t st) {
  const int64_t total = (int64_t)K * (ca / 8) * cb;
  if (total == 0) return SSCONV_OK;
  pack_b_kernel<<<cdiv(total, 256), 256, 0, st>>>((const uint16_t*)W, K, ca, cb, transposed ? 1 : 0, mirror ? 1 : 0,
                                                   (uint16_t*)Bp);
  SSC_HIP(hipGetLastError());
  return SSCONV_OK;
}

int gather_bf16(const void* src, int64_t n_src, int ca, const void* Bp, int cb, const int32_t* nbr,
                const int32_t* order, int64_t n_pos, int K, void* out, hipStream_t st, NormSink* sink) {
  if (n_pos == 0) return SSCONV_OK;
  if (!gather_bf16_supported(n_src, ca, cb, K))
    return fail(SSCONV_E_INVALID, "bf16 gather kernel does not support this shape (K=%d)", K);
  const int64_t sb = n_src * ca * 2;
  switch (bf16_nb(cb)) {
    case 4: return launch_bf16<4>(src, sb, ca, Bp, cb, nbr, order, n_pos, K, out, st, sink);
    case 8: return launch_bf16<8>(src, sb, ca, Bp, cb, nbr, order, n_pos, K, out, st, sink);
    case 13: return launch_bf16<13>(src, sb, ca, Bp, cb, nbr, order, n_pos, K, out, st, sink);
    default: return launch_bf16<14>(src, sb, ca, Bp, cb, nbr, order, n_pos, K, out, st, sink);
  }
}

}  // namespace ssconv
