// Gradient of the kernel tensor (the adjoint of Alg. 1's feature update):
//
//   dkappa(s)[o][i] = sum_{(x, y) in R_s} grad_out[x][o] * feats[y][i]
//
// a GEMM per offset whose reduction runs over the compact pair list R_s.
//
// fp32 (v_mfma_f32_16x16x4f32): the A operand of lane l is A[m = l%16][k = l/16]
// and the B operand B[k = l/16][n = l%16], so a step of the reduction takes 4 pairs
// and each lane group reads 16 consecutive channels of ONE gathered row.  Each
// wavefront owns a (16*WMB out channels) x (16*WNB in channels) tile of one offset
// and a contiguous slice of its pairs, and stages the rows of its steps in a
// private LDS ring (four steps deep, no barriers): one 1 KB DMA (buffer_load ...
// lds) fetches 16 granules of 4 channels of all 4 pairs of a step, pair-minor, so a
// lane fetches the same pair row in every DMA of a step and reads its operands
// without bank conflicts; the slice's pair indices are staged 128 at a time.
// Every slice writes its own partial tile; the partials are summed in a fixed order
// afterwards (deterministic, no atomics).  Sources of 2 GB or more use a variant
// that loads the rows straight into registers one step ahead.
//
// bf16 (v_mfma_f32_16x16x32_bf16): each lane's operand holds 8 consecutive PAIRS of
// one channel, i.e. the transpose of the row layout.  Gathered rows are DMA'd
// (global_load_lds_dwordx4) into LDS row-major, 32 pairs per stage, and the operands
// are read with ds_read_b64_tr_b16: within a 16-lane group, output lane i / slot j
// receives element i%4 of the 8 bytes addressed by source lane 4j + i/4, so source
// lane L pointing at row (base + L/4), channel (c0 + 4*(L%4)) delivers pairs
// base..base+3 of channel c0 + i.  Two such reads form one MFMA operand.  The
// pair indices of a slice are staged in LDS 1024 at a time.
#include <algorithm>

#include "kgrad_mfma.hpp"
#include "lds_dma.hpp"

namespace ssconv {
namespace {

typedef float f4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef short s4 __attribute__((ext_vector_type(4)));

__device__ __attribute__((aligned(64))) const uint4 g_zero16[4] = {};


__device__ __forceinline__ s4 tr_read(uint32_t lds_byte) {
  return __builtin_amdgcn_ds_read_tr16_b64_v4i16((__attribute__((address_space(3))) s4*)(uintptr_t)lds_byte);
}

// bf16 tile: 2 x 2 wavefronts, each W x W blocks of 16 x 16 -> a (32W) x (32W) tile of dkappa(s).
template <int W, int S>
struct KgB {
  static constexpr int TW = 32 * W;            // tile width in channels (each side)
  static constexpr int GR = TW / 8;            // 16-byte granules of one row segment
  static constexpr int RS = GR + 1;            // granules per LDS row (one pad granule)
  static constexpr int NDMA = (32 * RS + 63) / 64;   // DMA instructions per operand per stage
  static constexpr int OPB = NDMA * 1024;      // bytes per operand per stage
  static constexpr int STAGE = 2 * OPB;
  static constexpr int PW = (2 * NDMA + 3) / 4;      // DMA instructions per wavefront per stage
  static constexpr int PBLK = 1024;            // pair indices staged per block
  static constexpr int SMEM = S * STAGE + 1024 + PBLK * 8;
};

template <int W, int S>
__global__ __launch_bounds__(256) void kgrad_bf16_kernel(const uint16_t* __restrict__ G, int cout,
                                                         const uint16_t* __restrict__ F, int cin,
                                                         const int2* __restrict__ pairs,
                                                         const int64_t* __restrict__ pair_off, int K, int mtiles,
                                                         int ntiles, int nsplit, float* __restrict__ part) {
  using C = KgB<W, S>;
  extern __shared__ __attribute__((aligned(16))) char smem[];
  char* stages = smem;
  char* junk = smem + S * C::STAGE;
  int2* pblk = reinterpret_cast<int2*>(junk + 1024);
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6, g = lane >> 4, r16 = lane & 15;
  const int wm = w >> 1, wn = w & 1;

  const int nt = blockIdx.x % ntiles;
  const int mt = (blockIdx.x / ntiles) % mtiles;
  const int split = (blockIdx.x / (ntiles * mtiles)) % nsplit;
  const int s = blockIdx.x / (ntiles * mtiles * nsplit);
  const int m0 = mt * C::TW, n0 = nt * C::TW;
  const int64_t off = pair_off[s], cnt = pair_off[s + 1] - off;
  const int64_t beg = off + cnt * split / nsplit, end = off + cnt * (split + 1) / nsplit;
  const int64_t npairs = end - beg;
  const int nchunk = (int)((npairs + 31) / 32);
  const uint32_t stage0 = (uint32_t)(uintptr_t)stages, junk_a = (uint32_t)(uintptr_t)junk;

  // pair indices: block b covers slice pairs [b*PBLK, (b+1)*PBLK); registers hold the next block
  constexpr int PPT = C::PBLK / 256;
  int2 preg[PPT];
#define SSC_LOAD_PAIRS(b_)                                                                 \
  _Pragma("unroll") for (int q = 0; q < PPT; ++q) {                                        \
    const int64_t k_ = (int64_t)(b_) * C::PBLK + q * 256 + tid;                            \
    preg[q] = k_ < npairs ? pairs[beg + k_] : make_int2(-1, -1);                           \
  }
#define SSC_STORE_PAIRS()                                                                  \
  _Pragma("unroll") for (int q = 0; q < PPT; ++q) pblk[q * 256 + tid] = preg[q];

  SSC_LOAD_PAIRS(0);
  SSC_STORE_PAIRS();
  SSC_LOAD_PAIRS(1);
  __syncthreads();

  // one stage: rows of 32 pairs for both operands, DMA'd row-major with RS granules per row
#define SSC_ISSUE(c_)                                                                      \
  do {                                                                                     \
    const uint32_t base_ = stage0 + ((c_) % S) * C::STAGE;                                 \
    _Pragma("unroll") for (int j = 0; j < C::PW; ++j) {                                    \
      const int d_ = w + 4 * j;                                                            \
      const bool isF_ = d_ >= C::NDMA;                                                     \
      const int dd_ = isF_ ? d_ - C::NDMA : d_;                                            \
      const int pos_ = dd_ * 64 + lane;                                                    \
      const int row_ = pos_ / C::RS, gcv_ = pos_ % C::RS;                                  \
      const int64_t kk_ = (int64_t)(c_) * 32 + row_;                                       \
      const void* src_ = g_zero16;                                                         \
      if (d_ < 2 * C::NDMA && row_ < 32 && gcv_ < C::GR && kk_ < npairs) {                 \
        const int2 pr_ = pblk[kk_ % C::PBLK];                                              \
        const int ch_ = (isF_ ? n0 : m0) + 8 * gcv_;                                       \
        if (!isF_ && ch_ < cout) src_ = G + (int64_t)pr_.x * cout + ch_;                   \
        if (isF_ && ch_ < cin) src_ = F + (int64_t)pr_.y * cin + ch_;                      \
      }                                                                                    \
      dma16(src_, d_ < 2 * C::NDMA ? base_ + (isF_ ? C::OPB : 0) + dd_ * 1024 : junk_a);   \
    }                                                                                      \
  } while (0)

  f4 acc[W][W];
#pragma unroll
  for (int i = 0; i < W; ++i)
#pragma unroll
    for (int j = 0; j < W; ++j) acc[i][j] = f4{0.f, 0.f, 0.f, 0.f};

  for (int c = 0; c < S - 1 && c < nchunk; ++c) SSC_ISSUE(c);
  for (int c = 0; c < nchunk; ++c) {
    if (c + S - 2 < nchunk) wait_vm<C::PW * (S - 2)>(); else wait_vm<0>();
    __syncthreads();
    const int cn = c + S - 1;                       // chunk to issue now
    if (cn < nchunk) {
      if (cn % (C::PBLK / 32) == 0 && cn > 0) {     // first chunk of a new pair block
        __syncthreads();                            // every lane has issued from the old block
        SSC_STORE_PAIRS();
        SSC_LOAD_PAIRS(cn / (C::PBLK / 32) + 1);
        __syncthreads();
      }
      SSC_ISSUE(cn);
    }
    // operands of stage c via transpose reads: row base = 8g + 4h + L/4, column 4*(L%4)
    const uint32_t sb = stage0 + (c % S) * C::STAGE;
    const int rsel = 8 * g + (r16 >> 2);
    const int csel = 4 * (r16 & 3);
    bf16x8 a[W], b[W];
#pragma unroll
    for (int i = 0; i < W; ++i) {
      const int ca = (wm * W + i) * 16 + csel, cbn = (wn * W + i) * 16 + csel;
      s4 a0 = tr_read(sb + (rsel * C::RS) * 16 + ca * 2);
      s4 a1 = tr_read(sb + ((rsel + 4) * C::RS) * 16 + ca * 2);
      s4 b0 = tr_read(sb + C::OPB + (rsel * C::RS) * 16 + cbn * 2);
      s4 b1 = tr_read(sb + C::OPB + ((rsel + 4) * C::RS) * 16 + cbn * 2);
      short t[8] = {a0[0], a0[1], a0[2], a0[3], a1[0], a1[1], a1[2], a1[3]};
      short u[8] = {b0[0], b0[1], b0[2], b0[3], b1[0], b1[1], b1[2], b1[3]};
      __builtin_memcpy(&a[i], t, 16);
      __builtin_memcpy(&b[i], u, 16);
    }
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int i = 0; i < W; ++i)
#pragma unroll
      for (int j = 0; j < W; ++j) acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a[i], b[j], acc[i][j], 0, 0, 0);
  }
#undef SSC_ISSUE
#undef SSC_LOAD_PAIRS
#undef SSC_STORE_PAIRS

  float* dst = part + ((int64_t)split * K + s) * cout * cin;
#pragma unroll
  for (int i = 0; i < W; ++i)
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const int m = m0 + (wm * W + i) * 16 + 4 * g + e;
      if (m >= cout) continue;
#pragma unroll
      for (int j = 0; j < W; ++j) {
        const int n = n0 + (wn * W + j) * 16 + r16;
        if (n < cin) dst[(int64_t)m * cin + n] = acc[i][j][e];
      }
    }
}

template <int WMB, int WNB>
__global__ __launch_bounds__(256) void kgrad_f32_kernel(const float* __restrict__ G, int cout,
                                                        const float* __restrict__ F, int cin,
                                                        const int2* __restrict__ pairs,
                                                        const int64_t* __restrict__ pair_off, int K, int mtiles,
                                                        int ntiles, int nsplit, float* __restrict__ part) {
  const int lane = threadIdx.x & 63, g = lane >> 4, r16 = lane & 15;
  const int64_t task = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  const int64_t ntask = (int64_t)K * nsplit * mtiles * ntiles;
  if (task >= ntask) return;  // uniform per wavefront
  const int nt = (int)(task % ntiles);
  const int mt = (int)((task / ntiles) % mtiles);
  const int split = (int)((task / ((int64_t)ntiles * mtiles)) % nsplit);
  const int s = (int)(task / ((int64_t)ntiles * mtiles * nsplit));
  const int m0 = mt * 16 * WMB, n0 = nt * 16 * WNB;
  const int64_t off = pair_off[s], cnt = pair_off[s + 1] - off;
  const int64_t beg = off + cnt * split / nsplit, end = off + cnt * (split + 1) / nsplit;

  bool mok[WMB], nok[WNB];
#pragma unroll
  for (int mb = 0; mb < WMB; ++mb) mok[mb] = m0 + 16 * mb + r16 < cout;
#pragma unroll
  for (int nb = 0; nb < WNB; ++nb) nok[nb] = n0 + 16 * nb + r16 < cin;
  const float* Gc = G + m0 + r16;  // this lane's out-channel column
  const float* Fc = F + n0 + r16;  // this lane's in-channel column

  f4 acc[WMB][WNB];
#pragma unroll
  for (int mb = 0; mb < WMB; ++mb)
#pragma unroll
    for (int nb = 0; nb < WNB; ++nb) acc[mb][nb] = f4{0.f, 0.f, 0.f, 0.f};

  auto pair_at = [&](int64_t k) -> int2 { return k < end ? pairs[k] : make_int2(-1, -1); };
  float a0[WMB], b0[WNB], a1[WMB], b1[WNB];
#define SSC_ROWS(a_, b_, p_)                                                              \
  do {                                                                                    \
    _Pragma("unroll") for (int mb = 0; mb < WMB; ++mb)                                    \
      a_[mb] = (p_.x >= 0 && mok[mb]) ? Gc[(int64_t)p_.x * cout + 16 * mb] : 0.f;         \
    _Pragma("unroll") for (int nb = 0; nb < WNB; ++nb)                                    \
      b_[nb] = (p_.y >= 0 && nok[nb]) ? Fc[(int64_t)p_.y * cin + 16 * nb] : 0.f;          \
  } while (0)
#define SSC_MMA(a_, b_)                                                                   \
  do {                                                                                    \
    _Pragma("unroll") for (int mb = 0; mb < WMB; ++mb)                                    \
      _Pragma("unroll") for (int nb = 0; nb < WNB; ++nb)                                  \
        acc[mb][nb] = __builtin_amdgcn_mfma_f32_16x16x4f32(a_[mb], b_[nb], acc[mb][nb], 0, 0, 0); \
  } while (0)

  // steps of 4 pairs; lane group g takes pair k0 + g.  Rows of step t+1 and the pair
  // indices of step t+2 are in flight while step t runs on the matrix cores.
  int2 pn = pair_at(beg + 4 + g);
  {
    const int2 p0 = pair_at(beg + g);
    SSC_ROWS(a0, b0, p0);
  }
  for (int64_t k0 = beg; k0 < end; k0 += 4) {
    SSC_ROWS(a1, b1, pn);
    pn = pair_at(k0 + 8 + g);
    SSC_MMA(a0, b0);
#pragma unroll
    for (int mb = 0; mb < WMB; ++mb) a0[mb] = a1[mb];
#pragma unroll
    for (int nb = 0; nb < WNB; ++nb) b0[nb] = b1[nb];
  }
#undef SSC_ROWS
#undef SSC_MMA

  float* dst = part + ((int64_t)split * K + s) * cout * cin;
#pragma unroll
  for (int mb = 0; mb < WMB; ++mb)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int m = m0 + 16 * mb + 4 * g + i;
      if (m >= cout) continue;
#pragma unroll
      for (int nb = 0; nb < WNB; ++nb)
        if (nok[nb]) dst[(int64_t)m * cin + n0 + 16 * nb + r16] = acc[mb][nb][i];
    }
}

// Column blocks (16 channels) per tile: up to 8, near-equal tiles.
int tile_blocks(int c) {
  const int blocks = (c + 15) / 16;
  const int tiles = (blocks + 7) / 8;
  return (blocks + tiles - 1) / tiles;
}

int round_wb(int b) { return b <= 1 ? 1 : b <= 2 ? 2 : b <= 4 ? 4 : b <= 7 ? 7 : 8; }

// ---------------------------------------------------------------------------
// fp32 with a per-wavefront LDS ring
// ---------------------------------------------------------------------------
constexpr uint32_t kAbsentRow = 0x80000000u;  // byte offset past any buffer: the DMA writes zeros
constexpr int kBufWord3 = 0x00020000;         // buffer descriptor word 3 for gfx9-family raw loads
constexpr int kFD = 4;                        // LDS stages (steps of 4 pairs) per wavefront

template <int WMB, int WNB>
struct KF {
  static constexpr int LG = (WMB + 3) / 4;        // grad_out DMAs per step (16 granules each)
  static constexpr int LF = (WNB + 3) / 4;        // feats DMAs per step
  static constexpr int L = LG + LF;
  static constexpr int STEP = L * 1024;           // LDS bytes per step
  static constexpr int WAVE = 2 * 1024 + kFD * STEP;  // pair ring (2 x 128 pairs) + stages
  static constexpr int SMEM = 4 * WAVE;
};

#pragma clang diagnostic push
#pragma clang diagnostic ignored "-Winline-asm"
// 16 bytes per lane from byte offset off + IMM of the buffer rsrc into LDS at lds + 16 * lane.  The
// MUBUF immediate offset is added to the LDS address as well, so M0 is set IMM bytes lower.
template <int IMM>
__device__ __forceinline__ void dma_buf_imm(__amdgpu_buffer_rsrc_t rsrc, uint32_t off, uint32_t lds) {
  static_assert(IMM >= 0 && IMM < 4096, "MUBUF immediate offset");
  const uint32_t l = __builtin_amdgcn_readfirstlane(lds - IMM);
  asm volatile("s_mov_b32 m0, %0\n\ts_nop 0\n\tbuffer_load_dwordx4 %1, %2, 0 offen offset:%3 lds" ::"s"(l), "v"(off),
               "s"(rsrc), "n"(IMM)
               : "memory", "m0");
}
#pragma clang diagnostic pop

// DMA block j (0 or 1) of a step: channels 64 j .. 64 j + 63 of the tile
__device__ __forceinline__ void dma_blk(int j, __amdgpu_buffer_rsrc_t rsrc, uint32_t off, uint32_t lds) {
  if (j == 0)
    dma_buf_imm<0>(rsrc, off, lds);
  else
    dma_buf_imm<256>(rsrc, off, lds);
}

template <int WMB, int WNB>
__global__ __launch_bounds__(256) void kgrad_f32_lds_kernel(const float* __restrict__ G, int64_t g_rows, int cout,
                                                            const float* __restrict__ F, int64_t f_rows, int cin,
                                                            const int2* __restrict__ pairs,
                                                            const int64_t* __restrict__ pair_off, KgradUnits units,
                                                            int mtiles, int ntiles, float* __restrict__ part) {
  using C = KF<WMB, WNB>;
  static_assert(C::LG <= 2 && C::LF <= 2, "at most two DMA blocks per operand");
  extern __shared__ __attribute__((aligned(16))) char smem[];
  const int lane = threadIdx.x & 63, g = lane >> 4, r16 = lane & 15;
  const int w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  // task = (work unit u: a slice of one offset's pairs, output tile)
  const int task = blockIdx.x * 4 + w;
  if (task >= units.nunits * mtiles * ntiles) return;  // whole wavefront; the kernel has no barriers
  const int nt = task % ntiles;
  const int mt = (task / ntiles) % mtiles;
  const int u = task / (ntiles * mtiles);
  int s = 0;
  while (s + 1 < units.K && units.uoff[s + 1] <= u) ++s;
  const int j = u - units.uoff[s], ns = units.uoff[s + 1] - units.uoff[s];
  const int m0 = mt * 16 * WMB, n0 = nt * 16 * WNB;
  const int64_t off = pair_off[s], cnt = pair_off[s + 1] - off;
  const int64_t beg = off + cnt * j / ns, end = off + cnt * (j + 1) / ns;
  const int npairs = (int)(end - beg);
  const int nstep = (npairs + 3) / 4;

  char* const wl = smem + w * C::WAVE;  // [2][128] int2 pair ring, then kFD stages
  const uint32_t pr_a = lds_addr(wl), st_a = pr_a + 2048;
  const __amdgpu_buffer_rsrc_t g_rsrc =
      __builtin_amdgcn_make_buffer_rsrc(const_cast<float*>(G), (short)0, (int)(g_rows * cout * 4), kBufWord3);
  const __amdgpu_buffer_rsrc_t f_rsrc =
      __builtin_amdgcn_make_buffer_rsrc(const_cast<float*>(F), (short)0, (int)(f_rows * cin * 4), kBufWord3);
  const __amdgpu_buffer_rsrc_t p_rsrc = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<int2*>(pairs + beg), (short)0, npairs * 8, kBufWord3);

  // DMA lane l: pair l % 4 of the step, granule (4 channels) l / 4 of the DMA block
  const int pl = lane & 3, gl = lane >> 2;
  const uint32_t g_stat = (uint32_t)(m0 + 4 * gl) * 4u, f_stat = (uint32_t)(n0 + 4 * gl) * 4u;
  const uint32_t g_rowb = (uint32_t)cout * 4u, f_rowb = (uint32_t)cin * 4u;
  // operand reads: lane (r16, g) takes channel 16 mb + r16 of pair g -> granule 4 mb + r16 / 4
  const uint32_t rd_lane = (uint32_t)((r16 >> 2) * 64 + g * 16 + (r16 & 3) * 4);
  const int nblk = (npairs + 127) / 128;

#define KF_PAIRS(b_) dma_buf_imm<0>(p_rsrc, (uint32_t)(b_) * 1024u + 16u * lane, pr_a + ((b_) & 1) * 1024)

  // step t_: refill the pair ring when entering a new block of 32 steps, look up this lane's pair,
  // then the step's DMAs into stage t_ % kFD
#define KF_ISSUE(t_)                                                                                \
  do {                                                                                              \
    if (((t_) & 31) == 0 && (t_) > 0 && ((t_) >> 5) + 1 < nblk) KF_PAIRS(((t_) >> 5) + 1);          \
    const int pi_ = 4 * (t_) + pl;                                                                  \
    const int2 pv_ = *reinterpret_cast<const int2*>(wl + ((pi_ >> 7) & 1) * 1024 + (pi_ & 127) * 8);\
    const bool ok_ = pi_ < npairs;                                                                  \
    const uint32_t gb_ = ok_ ? (uint32_t)pv_.x * g_rowb + g_stat : kAbsentRow;                      \
    const uint32_t fb_ = ok_ ? (uint32_t)pv_.y * f_rowb + f_stat : kAbsentRow;                      \
    const uint32_t sb_ = st_a + ((t_) % kFD) * C::STEP;                                             \
    _Pragma("unroll") for (int j = 0; j < C::LG; ++j) dma_blk(j, g_rsrc, gb_, sb_ + j * 1024);      \
    _Pragma("unroll") for (int j = 0; j < C::LF; ++j) dma_blk(j, f_rsrc, fb_, sb_ + (C::LG + j) * 1024); \
  } while (0)

  bool mok[WMB], nok[WNB];
#pragma unroll
  for (int mb = 0; mb < WMB; ++mb) mok[mb] = m0 + 16 * mb + r16 < cout;
#pragma unroll
  for (int nb = 0; nb < WNB; ++nb) nok[nb] = n0 + 16 * nb + r16 < cin;

  f4 acc[WMB][WNB];
#pragma unroll
  for (int mb = 0; mb < WMB; ++mb)
#pragma unroll
    for (int nb = 0; nb < WNB; ++nb) acc[mb][nb] = f4{0.f, 0.f, 0.f, 0.f};

  if (nblk > 0) KF_PAIRS(0);
  if (nblk > 1) KF_PAIRS(1);
  wait_vm<0>();
  for (int t = 0; t < kFD - 1 && t < nstep; ++t) KF_ISSUE(t);
  for (int t = 0; t < nstep; ++t) {
    // this wavefront's DMAs of step t have landed (later steps may stay in flight)
    if (t + kFD - 2 < nstep)
      wait_vm<C::L * (kFD - 2)>();
    else
      wait_vm<0>();
    const char* sb = wl + 2048 + (t % kFD) * C::STEP;
    float a[WMB], b[WNB];
#pragma unroll
    for (int mb = 0; mb < WMB; ++mb) {
      const float v = *reinterpret_cast<const float*>(sb + (mb >> 2) * 1024 + (mb & 3) * 256 + rd_lane);
      a[mb] = mok[mb] ? v : 0.f;
    }
#pragma unroll
    for (int nb = 0; nb < WNB; ++nb) {
      const float v = *reinterpret_cast<const float*>(sb + (C::LG + (nb >> 2)) * 1024 + (nb & 3) * 256 + rd_lane);
      b[nb] = nok[nb] ? v : 0.f;
    }
    // the stage refilled now held step t-1, whose operands were consumed by its MFMAs
    if (t + kFD - 1 < nstep) KF_ISSUE(t + kFD - 1);
#pragma unroll
    for (int mb = 0; mb < WMB; ++mb)
#pragma unroll
      for (int nb = 0; nb < WNB; ++nb)
        acc[mb][nb] = __builtin_amdgcn_mfma_f32_16x16x4f32(a[mb], b[nb], acc[mb][nb], 0, 0, 0);
  }
#undef KF_ISSUE
#undef KF_PAIRS

  float* dst = part + (int64_t)u * cout * cin;
#pragma unroll
  for (int mb = 0; mb < WMB; ++mb)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int m = m0 + 16 * mb + 4 * g + i;
      if (m >= cout) continue;
#pragma unroll
      for (int nb = 0; nb < WNB; ++nb)
        if (nok[nb]) dst[(int64_t)m * cin + n0 + 16 * nb + r16] = acc[mb][nb][i];
    }
}

template <int WMB, int WNB>
void launch_f32_lds(dim3 grid, const float* G, int64_t g_rows, int cout, const float* F, int64_t f_rows, int cin,
                    const int2* pairs, const int64_t* pair_off, const KgradUnits& units, int mt, int nt, float* part,
                    hipStream_t st) {
  auto kern = kgrad_f32_lds_kernel<WMB, WNB>;
  (void)hipFuncSetAttribute((const void*)kern, hipFuncAttributeMaxDynamicSharedMemorySize, KF<WMB, WNB>::SMEM);
  kern<<<grid, 256, KF<WMB, WNB>::SMEM, st>>>(G, g_rows, cout, F, f_rows, cin, pairs, pair_off, units, mt, nt, part);
}

template <int WMB>
void launch_f32_lds_n(int wnb, dim3 grid, const float* G, int64_t g_rows, int cout, const float* F, int64_t f_rows,
                      int cin, const int2* pairs, const int64_t* pair_off, const KgradUnits& units, int mt, int nt,
                      float* part, hipStream_t st) {
  switch (wnb) {
    case 1: launch_f32_lds<WMB, 1>(grid, G, g_rows, cout, F, f_rows, cin, pairs, pair_off, units, mt, nt, part, st); break;
    case 2: launch_f32_lds<WMB, 2>(grid, G, g_rows, cout, F, f_rows, cin, pairs, pair_off, units, mt, nt, part, st); break;
    case 4: launch_f32_lds<WMB, 4>(grid, G, g_rows, cout, F, f_rows, cin, pairs, pair_off, units, mt, nt, part, st); break;
    case 7: launch_f32_lds<WMB, 7>(grid, G, g_rows, cout, F, f_rows, cin, pairs, pair_off, units, mt, nt, part, st); break;
    default: launch_f32_lds<WMB, 8>(grid, G, g_rows, cout, F, f_rows, cin, pairs, pair_off, units, mt, nt, part, st); break;
  }
}

template <int WMB>
void launch_f32_n(int wnb, dim3 grid, const float* G, int cout, const float* F, int cin, const int2* pairs,
                  const int64_t* pair_off, int K, int mt, int nt, int nsplit, float* part, hipStream_t st) {
  switch (wnb) {
    case 1: kgrad_f32_kernel<WMB, 1><<<grid, 256, 0, st>>>(G, cout, F, cin, pairs, pair_off, K, mt, nt, nsplit, part); break;
    case 2: kgrad_f32_kernel<WMB, 2><<<grid, 256, 0, st>>>(G, cout, F, cin, pairs, pair_off, K, mt, nt, nsplit, part); break;
    case 4: kgrad_f32_kernel<WMB, 4><<<grid, 256, 0, st>>>(G, cout, F, cin, pairs, pair_off, K, mt, nt, nsplit, part); break;
    case 7: kgrad_f32_kernel<WMB, 7><<<grid, 256, 0, st>>>(G, cout, F, cin, pairs, pair_off, K, mt, nt, nsplit, part); break;
    default: kgrad_f32_kernel<WMB, 8><<<grid, 256, 0, st>>>(G, cout, F, cin, pairs, pair_off, K, mt, nt, nsplit, part); break;
  }
}

}  // namespace

KgradPlan kgrad_plan(const ssconv_rulebook* rb, ssconv_dtype dt, int cin, int cout) {
  KgradPlan p;
  if (dt == SSCONV_F32) {
    p.wmb = round_wb(tile_blocks(cout));
    p.wnb = round_wb(tile_blocks(cin));
    // few pairs (at least ~256 per work unit, so few units): when the (unit, tile) tasks number
    // under 1024, most SIMDs idle while each wavefront runs its tile's MFMAs serially, so the
    // output rows are cut into 4-block tiles (the gathered input rows are then read once per
    // tile, from L2)
    const int64_t units = std::max<int64_t>(rb->K, rb->n_pairs / 256);
    const int64_t tiles_now = (int64_t)((cout + 16 * p.wmb - 1) / (16 * p.wmb)) * ((cin + 16 * p.wnb - 1) / (16 * p.wnb));
    if (p.wmb >= 7 && units * tiles_now < 1024) p.wmb = 4;
    p.mtiles = (cout + 16 * p.wmb - 1) / (16 * p.wmb);
    p.ntiles = (cin + 16 * p.wnb - 1) / (16 * p.wnb);
  } else {
    // square 2x2-wavefront tiles of 32W channels, W in {2, 4, 7}
    const int need = (std::max(cout, cin) + 31) / 32;
    p.wmb = p.wnb = need <= 2 ? 2 : need <= 4 ? 4 : 7;
    p.mtiles = (cout + 32 * p.wmb - 1) / (32 * p.wmb);
    p.ntiles = (cin + 32 * p.wnb - 1) / (32 * p.wnb);
  }
  int64_t mx = 1;
  for (int s = 0; s < rb->K; ++s) mx = std::max(mx, rb->pair_off[s + 1] - rb->pair_off[s]);
  // fp32: at most 4096 wavefronts, i.e. two full rounds of the 2048 wavefront slots (256 CUs x
  // two four-wavefront workgroups): rounding up would start a third, nearly empty round.  bf16:
  // about 512 workgroups.  At least 256 pairs per slice, at most 64 slices.
  const int64_t tiles = (int64_t)rb->K * p.mtiles * p.ntiles;
  int64_t ns = dt == SSCONV_F32 ? 4096 / tiles : (512 + tiles - 1) / tiles;
  ns = std::min<int64_t>(ns, std::max<int64_t>(1, mx / 256));
  p.nsplit = (int)std::max<int64_t>(1, std::min<int64_t>(ns, 64));
  return p;
}

int kgrad_partials(const void* grad_out, const void* feats, ssconv_dtype dt, int cin, int cout,
                   const ssconv_rulebook* rb, const KgradPlan& p, float* part, hipStream_t st) {
  const int64_t ntask = (int64_t)rb->K * p.nsplit * p.mtiles * p.ntiles;
  if (ntask == 0) return SSCONV_OK;
  const int2* pairs = reinterpret_cast<const int2*>(rb->pairs);
  if (dt == SSCONV_BF16) {
    const uint16_t* G = (const uint16_t*)grad_out;
    const uint16_t* F = (const uint16_t*)feats;
    dim3 g1((unsigned)ntask);
#define SSC_KB(Wv)                                                                                    \
  do {                                                                                                \
    auto kern = kgrad_bf16_kernel<Wv, 3>;                                                             \
    SSC_HIP(hipFuncSetAttribute((const void*)kern, hipFuncAttributeMaxDynamicSharedMemorySize, KgB<Wv, 3>::SMEM)); \
    kern<<<g1, 256, KgB<Wv, 3>::SMEM, st>>>(G, cout, F, cin, pairs, rb->pair_off_dev, rb->K, p.mtiles, p.ntiles, \
                                            p.nsplit, part);                                          \
  } while (0)
    if (p.wmb == 2) SSC_KB(2);
    else if (p.wmb == 4) SSC_KB(4);
    else SSC_KB(7);
#undef SSC_KB
    SSC_HIP(hipGetLastError());
    return SSCONV_OK;
  }
  dim3 grid(cdiv(ntask, 4));
  const float* G = (const float*)grad_out;
  const float* F = (const float*)feats;
  switch (p.wmb) {
    case 1: launch_f32_n<1>(p.wnb, grid, G, cout, F, cin, pairs, rb->pair_off_dev, rb->K, p.mtiles, p.ntiles, p.nsplit, part, st); break;
    case 2: launch_f32_n<2>(p.wnb, grid, G, cout, F, cin, pairs, rb->pair_off_dev, rb->K, p.mtiles, p.ntiles, p.nsplit, part, st); break;
    case 4: launch_f32_n<4>(p.wnb, grid, G, cout, F, cin, pairs, rb->pair_off_dev, rb->K, p.mtiles, p.ntiles, p.nsplit, part, st); break;
    case 7: launch_f32_n<7>(p.wnb, grid, G, cout, F, cin, pairs, rb->pair_off_dev, rb->K, p.mtiles, p.ntiles, p.nsplit, part, st); break;
    default: launch_f32_n<8>(p.wnb, grid, G, cout, F, cin, pairs, rb->pair_off_dev, rb->K, p.mtiles, p.ntiles, p.nsplit, part, st); break;
  }
  SSC_HIP(hipGetLastError());
  return SSCONV_OK;
}

bool kgrad_f32_units_ok(const ssconv_rulebook* rb, int cin, int cout) {
  return rb->K <= kKgradMaxK && (int64_t)rb->n_out * cout * 4 < ((int64_t)1 << 31) &&
         (int64_t)rb->n_in * cin * 4 < ((int64_t)1 << 31) && debug_gather_variant() != 7;
}

int kgrad_f32_units_want(const ssconv_rulebook* rb, int cin, int cout) {
  const KgradPlan p = kgrad_plan(rb, SSCONV_F32, cin, cout);
  // one full round of the 2048 wavefront slots (256 CUs x two four-wavefront workgroups): measured
  // against 1024, 1536, 3072 and 4096 tasks, fewer partials to add up outweigh the balance of
  // two rounds (C2 step -12 us, C5 -215 us against 4096)
  const int64_t slots = std::max(1, 2048 / (p.mtiles * p.ntiles));
  // at least ~256 pairs per unit: below that the partial tiles (written once, added up again)
  // outweigh the gathered rows of the unit (C6: 1024 units of ~83 pairs made 35 MB of partials)
  const int64_t by_pairs = std::max<int64_t>(rb->K, rb->n_pairs / 256);
  return (int)std::max<int64_t>(1, std::min(slots, by_pairs));
}

int kgrad_f32(const void* grad_out, const void* feats, int cin, int cout, const ssconv_rulebook* rb,
              const KgradUnits& units, float* part, hipStream_t st) {
  if (units.nunits == 0) return SSCONV_OK;
  const KgradPlan p = kgrad_plan(rb, SSCONV_F32, cin, cout);
  const int64_t ntask = (int64_t)units.nunits * p.mtiles * p.ntiles;
  dim3 grid(cdiv(ntask, 4));
  const int2* pairs = reinterpret_cast<const int2*>(rb->pairs);
  const float* G = (const float*)grad_out;
  const float* F = (const float*)feats;
  const int64_t g_rows = rb->n_out, f_rows = rb->n_in;
  switch (p.wmb) {
    case 1: launch_f32_lds_n<1>(p.wnb, grid, G, g_rows, cout, F, f_rows, cin, pairs, rb->pair_off_dev, units, p.mtiles, p.ntiles, part, st); break;
    case 2: launch_f32_lds_n<2>(p.wnb, grid, G, g_rows, cout, F, f_rows, cin, pairs, rb->pair_off_dev, units, p.mtiles, p.ntiles, part, st); break;
    case 4: launch_f32_lds_n<4>(p.wnb, grid, G, g_rows, cout, F, f_rows, cin, pairs, rb->pair_off_dev, units, p.mtiles, p.ntiles, part, st); break;
    case 7: launch_f32_lds_n<7>(p.wnb, grid, G, g_rows, cout, F, f_rows, cin, pairs, rb->pair_off_dev, units, p.mtiles, p.ntiles, part, st); break;
    default: launch_f32_lds_n<8>(p.wnb, grid, G, g_rows, cout, F, f_rows, cin, pairs, rb->pair_off_dev, units, p.mtiles, p.ntiles, part, st); break;
  }
  SSC_HIP(hipGetLastError());
  return SSCONV_OK;
}

}  // namespace ssconv
