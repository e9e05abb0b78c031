// bf16 gradient of the kernel tensor (the adjoint of Alg. 1's feature update):
//
//   dkappa(s)[o][i] = sum_{(x, y) in R_s} grad_out[x][o] * feats[y][i]
//
// a GEMM per offset whose reduction runs over the compact pair list R_s.  The pair lists of
// all offsets are cut into work units of about equal length (several per offset, so that the
// units fill the chip evenly); each workgroup computes one (32W x 32W) tile of one offset over
// one unit and writes its own fp32 partial, and the partials of an offset are summed in a
// fixed order afterwards (deterministic, no atomics).
//
// v_mfma_f32_16x16x32_bf16 takes 8 consecutive PAIRS of one channel per lane, the transpose of
// the row layout.  A chunk of 32 pairs is staged in LDS per operand as 16-byte granule columns
// of 32 rows each; one 1 KB DMA (buffer_load ... lds on 32-bit row offsets: the tail of a unit
// reads past the end of the buffer, which writes zeros) fills granule column j with lanes 0-31
// and column j + H with lanes 32-63 (H = half the columns), so a lane fetches the same pair row
// in every DMA of a chunk: one pair-table read per chunk, and the DMAs of a chunk differ only in
// an immediate offset.  DMA blocks are padded to 1088 bytes so that the two columns read
// together (2i, 2i + 1) sit 16 banks apart.  The operands are read with ds_read_b64_tr_b16:
// within a 16-lane group, output lane i / slot j receives element i%4 of the 8 bytes addressed
// by source lane 4j + i/4, so source lane L pointing at row (base + L/4), channel
// (c0 + 4*(L%4)) delivers pairs base..base+3 of channel c0 + i; two such reads form one operand.
//
// Pipeline (four LDS stages): iteration c waits for its own DMAs of chunk c+1, publishes them
// with one barrier, then runs the MFMAs of chunk c with the transpose reads of chunk c+1 and the
// DMAs of chunk c+3 spread between them.  Wavefronts 0-1 fetch grad_out rows, 2-3 feats rows.
// The unit's pair indices are staged in LDS in blocks of 1024, double-buffered and DMA'd one
// block ahead.
#include <algorithm>
#include <utility>
#include <vector>

#include "kgrad_mfma.hpp"
#include "lds_dma.hpp"

namespace ssconv {
namespace {

typedef float f4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef short s4 __attribute__((ext_vector_type(4)));

constexpr uint32_t kAbsent = 0x80000000u;  // row offset past any buffer: the DMA writes zeros
constexpr int kBufferWord3 = 0x00020000;   // buffer descriptor word 3 for gfx9-family raw loads
constexpr int kS = 4;                      // LDS stages
constexpr int kPBLK = 1024;                // pair indices per staged block

// Operand staging in LDS.  Quad layout (kQuad, the default): granule quad j (channels 32j .. 32j
// + 31 of the tile) of the chunk's 32 rows is 2 KB, row r at 64 r, the granule of position p at
// 16 (p ^ 2 ((r / 8) % 2)) (the swizzle keeps the 32 lanes served together by a transpose read on
// distinct banks); one DMA fills a quad for 16 rows, so a lane fetches 16 bytes of a 64-byte piece
// of one row.  Column layout: granule column j (16 bytes of 32 rows, 512 B) in block j % H, half
// j / H, blocks padded to 1088 bytes; one DMA fills a block with two 16-byte pieces of 32 rows.
// Measured on gathered 416-byte rows (1 KB DMAs, 80 MB table): 64-byte pieces moved 24-27 B/ns
// per CU, 16-byte pieces 11-15.
template <int W, bool kQuad = true>
struct KB {
  static constexpr int TW = 32 * W;                 // tile width in channels (each side)
  static constexpr int H = 2 * W;                   // DMA blocks per operand (two granule columns each)
  static constexpr int BLK = 1024 + 64;             // bytes per DMA block (padded), column layout
  static constexpr int OPB = kQuad ? 2 * W * 1024 : H * BLK;  // bytes per operand per stage
  static constexpr int STAGE = 2 * OPB;
  static constexpr int PW = W;                      // DMAs per wavefront per chunk
  static_assert(W <= 7, "DMA immediate offsets are instantiated for up to 7 blocks per wavefront");
  static constexpr int SMEM = kS * STAGE + 2 * kPBLK * 8;
};

#pragma clang diagnostic push
#pragma clang diagnostic ignored "-Winline-asm"
// 16 bytes per lane at byte offset off + IMM of the buffer rsrc into LDS at lds + IMM + 16 * lane
// (the immediate offset applies to both addresses).
template <int IMM>
__device__ __forceinline__ void dma16_buf(__amdgpu_buffer_rsrc_t rsrc, uint32_t off, uint32_t lds) {
  static_assert(IMM >= 0 && IMM < 4096, "MUBUF immediate offset");
  const uint32_t l = __builtin_amdgcn_readfirstlane(lds);
  asm volatile("s_mov_b32 m0, %0\n\ts_nop 0\n\tbuffer_load_dwordx4 %1, %2, 0 offen offset:%3 lds" ::"s"(l), "v"(off),
               "s"(rsrc), "n"(IMM)
               : "memory", "m0");
}
#pragma clang diagnostic pop

// dma16_buf with immediate offset 64 q; q is a constant once the callers' loops are unrolled
__device__ __forceinline__ void dma16_buf_q64(int q, __amdgpu_buffer_rsrc_t rsrc, uint32_t off, uint32_t lds) {
  switch (q) {
    case 0: dma16_buf<0>(rsrc, off, lds); break;
    case 1: dma16_buf<64>(rsrc, off, lds); break;
    case 2: dma16_buf<128>(rsrc, off, lds); break;
    case 3: dma16_buf<192>(rsrc, off, lds); break;
    case 4: dma16_buf<256>(rsrc, off, lds); break;
    case 5: dma16_buf<320>(rsrc, off, lds); break;
    default: dma16_buf<384>(rsrc, off, lds); break;
  }
}

// dma16_buf with immediate offset 16 q; q is a constant once the callers' loops are unrolled
__device__ __forceinline__ void dma16_buf_q(int q, __amdgpu_buffer_rsrc_t rsrc, uint32_t off, uint32_t lds) {
  switch (q) {
    case 0: dma16_buf<0>(rsrc, off, lds); break;
    case 1: dma16_buf<16>(rsrc, off, lds); break;
    case 2: dma16_buf<32>(rsrc, off, lds); break;
    case 3: dma16_buf<48>(rsrc, off, lds); break;
    case 4: dma16_buf<64>(rsrc, off, lds); break;
    case 5: dma16_buf<80>(rsrc, off, lds); break;
    default: dma16_buf<96>(rsrc, off, lds); break;
  }
}

// Workgroups are dispatched round-robin over the 8 XCDs: launch index i runs on XCD i % 8, which
// takes slot positions (i % 8) * ceil(n / 8) + i / 8, a contiguous range per XCD.
__device__ __forceinline__ int xcd_slot(int i, int n) {
  const int x = i & 7, j = i >> 3, q = n >> 3, r = n & 7;
  return (x < r ? x * (q + 1) : r * (q + 1) + (x - r) * q) + j;
}

__device__ __forceinline__ s4 tr_read(uint32_t lds) {
  return __builtin_amdgcn_ds_read_tr16_b64_v4i16((__attribute__((address_space(3))) s4*)(uintptr_t)lds);
}

template <int W, bool kQuad>
__global__ __launch_bounds__(256) void kgrad_bf16_kernel(const uint16_t* __restrict__ G, int64_t g_rows, int cout,
                                                         const uint16_t* __restrict__ F, int64_t f_rows, int cin,
                                                         const int2* __restrict__ pairs,
                                                         const int64_t* __restrict__ pair_off, KgradUnits units,
                                                         int mtiles, int ntiles, float* __restrict__ part) {
  using C = KB<W, kQuad>;
  extern __shared__ __attribute__((aligned(16))) char smem[];
  char* stages = smem;
  char* pblk = smem + kS * C::STAGE;  // [2][kPBLK] int2
  const int tid = threadIdx.x, lane = tid & 63, g = lane >> 4, r16 = lane & 15;
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm = w >> 1, wn = w & 1;

  // launch slot -> work unit (XCD-contiguous over the row-sorted order) -> (offset s, slice of
  // R_s), tile (mt, nt)
  const int tile = blockIdx.x % (mtiles * ntiles);
  const int u = units.order[xcd_slot(blockIdx.x / (mtiles * ntiles), units.nunits)];
  int s = 0;
  while (s + 1 < units.K && units.uoff[s + 1] <= u) ++s;
  const int j = u - units.uoff[s], ns = units.uoff[s + 1] - units.uoff[s];
  const int nt = tile % ntiles, mt = tile / ntiles;
  const int m0 = mt * C::TW, n0 = nt * C::TW;
  const int64_t off = pair_off[s], cnt = pair_off[s + 1] - off;
  const int64_t beg = off + cnt * j / ns, end = off + cnt * (j + 1) / ns;
  const int npairs = (int)(end - beg);
  const int nchunk = (npairs + 31) / 32;

  const __amdgpu_buffer_rsrc_t g_rsrc =
      __builtin_amdgcn_make_buffer_rsrc(const_cast<uint16_t*>(G), (short)0, (int)(g_rows * cout * 2), kBufferWord3);
  const __amdgpu_buffer_rsrc_t f_rsrc =
      __builtin_amdgcn_make_buffer_rsrc(const_cast<uint16_t*>(F), (short)0, (int)(f_rows * cin * 2), kBufferWord3);
  // the unit's pair list as a byte buffer (past its end: zeros, i.e. row 0 -- masked below)
  const __amdgpu_buffer_rsrc_t p_rsrc = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<int2*>(pairs + beg), (short)0, npairs * 8, kBufferWord3);
  const uint32_t stage0 = lds_addr(stages), pblk_a = lds_addr(pblk);

  // DMA duty: wavefronts 0-1 fetch grad_out (operand 0), 2-3 feats (operand 1).  Quad layout:
  // wavefront w fills quads 0 .. W - 1 of rows 16 (w % 2) .. + 15, lane l: row 16 (w % 2) + l / 4,
  // granule gq = (l % 4) ^ swizzle of the quad.  Column layout: blocks jb .. jb + W - 1,
  // jb = W * (w % 2), lane l: row l % 32, granule column (block + H * (l / 32)).
  const bool isF = w >= 2;
  const int jb = W * (w & 1);
  const int prow = kQuad ? 16 * (w & 1) + (lane >> 2) : lane & 31;
  const int gq = (lane & 3) ^ (((prow >> 3) & 1) << 1);
  const __amdgpu_buffer_rsrc_t x_rsrc = isF ? f_rsrc : g_rsrc;
  const uint32_t x_rowb = (uint32_t)(isF ? cin : cout) * 2u;
  const uint32_t x_stat = (uint32_t)(isF ? n0 : m0) * 2u +
                          16u * (uint32_t)(kQuad ? gq : jb + C::H * (lane >> 5));
  // DMA q of this lane fetches channels (isF ? n0 : m0) + 8 (4q + gq) .. + 7 (column layout: + 8 (jb
  // + q + H (lane / 32))); a granule past the operand's channels (the tile is padded to 32 W) is
  // not fetched (offset past the end: zeros; the products it feeds are never stored)
  uint32_t gvalid = 0;
  {
    const int ch = isF ? cin : cout;
    const int c0 = (isF ? n0 : m0) + 8 * (kQuad ? gq : jb + C::H * (lane >> 5));
#pragma unroll
    for (int q = 0; q < C::PW; ++q) gvalid |= (c0 + 8 * (kQuad ? 4 * q : q) < ch ? 1u : 0u) << q;
  }
  // + stage * STAGE + q * (quad: 2048, column: BLK)
  const uint32_t m0_base = stage0 + (isF ? C::OPB : 0) + (kQuad ? (w & 1) * 1024 : jb * C::BLK);
  const uint32_t p_ent = (uint32_t)prow * 8u + (isF ? 4u : 0u);        // this lane's index in a chunk's pairs

  // pair block b (slice pairs [b*kPBLK, (b+1)*kPBLK)) into buffer b % 2: 8 KB per block, two
  // 1 KB DMAs per wavefront
#define SSK_PAIRS(b_)                                                                               \
  do {                                                                                              \
    _Pragma("unroll") for (int i_ = 0; i_ < 2; ++i_) {                                              \
      const int blk_ = w + 4 * i_;                                                                  \
      dma16_buf<0>(p_rsrc, (uint32_t)((b_) * kPBLK * 8 + blk_ * 1024 + 16 * lane),                  \
                   pblk_a + ((b_) & 1) * kPBLK * 8 + blk_ * 1024);                                  \
    }                                                                                               \
  } while (0)

  // byte offset of this lane's row in chunk c_ (kAbsent past the unit's end).  Pair k = c_*32 +
  // row of the slice sits in buffer (c_ / 32) % 2 at entry (c_ % 32)*32 + row (32 chunks per block).
#define SSK_ROW(dst_, c_)                                                                           \
  do {                                                                                              \
    const uint32_t pb_ = ((uint32_t)(c_) >> 5 & 1u) * (kPBLK * 8) + ((uint32_t)(c_) & 31u) * 256u;  \
    const int v_ = *reinterpret_cast<const int*>(pblk + pb_ + p_ent);                               \
    dst_ = (prow < npairs - (c_) * 32) ? (uint32_t)v_ * x_rowb + x_stat : kAbsent;                  \
  } while (0)

  // DMA q of this wavefront (quad q; column layout: block jb + q) into stage k_, from row offset
  // ro_.  The MUBUF immediate offset (64 q; column layout: 16 q) is added to the LDS address as
  // well, so M0 is set that much lower.
#define SSK_DMA(q_, ro_, k_)                                                                        \
  do {                                                                                              \
    const uint32_t src_ = ((gvalid >> (q_)) & 1u) ? (ro_) : kAbsent;                                \
    if constexpr (kQuad)                                                                            \
      dma16_buf_q64(q_, x_rsrc, src_, m0_base + (k_) * C::STAGE + (q_) * (2048 - 64));              \
    else                                                                                            \
      dma16_buf_q(q_, x_rsrc, src_, m0_base + (k_) * C::STAGE + (q_) * (C::BLK - 16));              \
  } while (0)

  // operands of the chunk in stage k_ via transpose reads: rows R = 8g + 4h + L/4, channel
  // 16 bi + 4 (L % 4) for MFMA block bi = wm * W + i (grad_out; feats: wn * W + i), i.e. granule
  // J = 2 bi + (L % 4) / 2, byte 8 ((L % 4) % 2).  Quad layout: quad bi / 2, row R, position
  // 2 ((bi % 2) ^ (g % 2)) + (L % 4) / 2 (R / 8 = g).  Column layout: block 2i + (L % 4) / 2, half
  // wm (wn), row R.
  const uint32_t rd_lane =
      kQuad ? (uint32_t)((8 * g + (r16 >> 2)) * 64 + ((r16 & 3) >> 1) * 16 + (r16 & 1) * 8)
            : (uint32_t)((((r16 & 3) >> 1) * C::BLK) + (8 * g + (r16 >> 2)) * 16 + ((r16 & 1) * 8));
  const uint32_t gx = (uint32_t)(g & 1) * 32u;  // quad layout: the swizzle bit of this lane's rows
  const uint32_t rd_a = stage0 + (kQuad ? 0u : wm * 512u) + rd_lane;
  const uint32_t rd_b = stage0 + C::OPB + (kQuad ? 0u : wn * 512u) + rd_lane;
  // byte offset of MFMA block bi_ (wave-uniform) in the quad layout; h = 1 adds 4 rows (256 B)
#define SSK_QOFF(bi_) ((uint32_t)((bi_) >> 1) * 2048u + ((((uint32_t)(bi_) & 1u) * 32u) ^ gx))
#define SSK_READ(da_, db_, i_, k_)                                                                  \
  do {                                                                                              \
    const uint32_t oa_ = (k_) * C::STAGE + (kQuad ? SSK_QOFF(wm * W + (i_)) : 2 * (i_) * C::BLK);   \
    const uint32_t ob_ = (k_) * C::STAGE + (kQuad ? SSK_QOFF(wn * W + (i_)) : 2 * (i_) * C::BLK);   \
    const uint32_t hs_ = kQuad ? 256u : 64u;                                                        \
    const s4 a0_ = tr_read(rd_a + oa_);                                                             \
    const s4 a1_ = tr_read(rd_a + oa_ + hs_);                                                       \
    const s4 b0_ = tr_read(rd_b + ob_);                                                             \
    const s4 b1_ = tr_read(rd_b + ob_ + hs_);                                                       \
    da_[i_] = __builtin_bit_cast(bf16x8, __builtin_shufflevector(a0_, a1_, 0, 1, 2, 3, 4, 5, 6, 7)); \
    db_[i_] = __builtin_bit_cast(bf16x8, __builtin_shufflevector(b0_, b1_, 0, 1, 2, 3, 4, 5, 6, 7)); \
  } while (0)

  // Accumulators start at zero through a value the compiler cannot fold (npairs >= 0), each from
  // its own expression: a single shared zero makes the register allocator merge the initial
  // accumulators and then copy them apart on every path into the chunk loop.
  f4 acc[W][W];
  {
    const float z = __uint_as_float((uint32_t)__builtin_amdgcn_readfirstlane(npairs < 0 ? 1 : 0));
#pragma unroll
    for (int i = 0; i < W; ++i)
#pragma unroll
      for (int jj = 0; jj < W; ++jj) {
        const float zi = z * (float)(i * W + jj + 1);
        acc[i][jj] = f4{zi, zi, zi, zi};
      }
  }

  constexpr int L = C::PW;  // row DMAs per wavefront per chunk (pair-block DMAs only add to waits)
  const int nblk = (npairs + kPBLK - 1) / kPBLK;
  // prologue: pair blocks 0 and 1, then the rows of chunks 0..2
  if (nblk > 0) SSK_PAIRS(0);
  if (nblk > 1) SSK_PAIRS(1);
  wait_vm<0>();
  __syncthreads();
#pragma unroll
  for (int c = 0; c < kS - 1; ++c)
    if (c < nchunk) {
      uint32_t ro;
      SSK_ROW(ro, c);
#pragma unroll
      for (int q = 0; q < L; ++q) SSK_DMA(q, ro, c);
    }

  // The barrier of iteration c needs no LDS fence: the transpose reads of a chunk are consumed
  // by its MFMAs before the next barrier, and its stage is refilled only two barriers later.
#define SSK_BODY(k_, AC, BC, AN, BN)                                                                \
  if (c + (k_) < nchunk) {                                                                          \
    const int cc_ = c + (k_);                                                                       \
    if (cc_ + kS - 2 < nchunk)                                                                      \
      wait_vm<(kS - 3) * L>();                                                                      \
    else                                                                                            \
      wait_vm<0>();                                                                                 \
    asm volatile("s_barrier" ::: "memory");                                                         \
    const bool rd_ = cc_ + 1 < nchunk;                                                              \
    const int ci_ = cc_ + kS - 1; /* chunk whose rows are issued now */                             \
    const bool iss_ = ci_ < nchunk;                                                                 \
    /* entering pair block b at the issue side: block b+1 goes into the other buffer, whose */      \
    /* entries (block b-1) were all read by issues before this iteration's barrier */               \
    if (iss_ && (ci_ % (kPBLK / 32)) == 0 && ci_ / (kPBLK / 32) + 1 < nblk)                         \
      SSK_PAIRS(ci_ / (kPBLK / 32) + 1);                                                            \
    constexpr int ks_ = ((k_) + kS - 1) % kS, kr_ = ((k_) + 1) % kS;                                \
    uint32_t ro_ = kAbsent;                                                                         \
    if (iss_) SSK_ROW(ro_, ci_);                                                                    \
    __builtin_amdgcn_sched_barrier(0);                                                              \
    _Pragma("unroll") for (int i = 0; i < W; ++i) {                                                 \
      _Pragma("unroll") for (int jj = 0; jj < W; ++jj)                                              \
        acc[i][jj] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(AC[i], BC[jj], acc[i][jj], 0, 0, 0);   \
      __builtin_amdgcn_sched_barrier(0);                                                            \
      if (rd_) SSK_READ(AN, BN, i, kr_);                                                            \
      if (iss_) SSK_DMA(i, ro_, ks_);                                                               \
      __builtin_amdgcn_sched_barrier(0);                                                            \
    }                                                                                               \
  }

  bf16x8 a0[W], b0[W], a1[W], b1[W];
  if (nchunk > 0) {
    if (nchunk > 2) wait_vm<2 * L>(); else wait_vm<0>();
    __syncthreads();
#pragma unroll
    for (int i = 0; i < W; ++i) SSK_READ(a0, b0, i, 0);
  }
  static_assert(kS == 4, "the unrolled chunk loop is written for four stages");
  static_assert(L == W, "one DMA per row block of the MFMA loop");
  for (int c = 0; c < nchunk; c += kS) {
    SSK_BODY(0, a0, b0, a1, b1)
    SSK_BODY(1, a1, b1, a0, b0)
    SSK_BODY(2, a0, b0, a1, b1)
    SSK_BODY(3, a1, b1, a0, b0)
  }
#undef SSK_BODY
#undef SSK_QOFF
#undef SSK_READ
#undef SSK_DMA
#undef SSK_ROW
#undef SSK_PAIRS

  float* dst = part + (int64_t)u * cout * cin;
#pragma unroll
  for (int i = 0; i < W; ++i)
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const int m = m0 + (wm * W + i) * 16 + 4 * g + e;
      if (m >= cout) continue;
#pragma unroll
      for (int jj = 0; jj < W; ++jj) {
        const int n = n0 + (wn * W + jj) * 16 + r16;
        if (n < cin) dst[(int64_t)m * cin + n] = acc[i][jj][e];
      }
    }
}

// dW[s] (field-pair-blocked, dw_block_pos) = sum of offset s's unit partials ([cout][cin]) in unit
// order.  A thread takes VEC consecutive elements of one row (cin % VEC == 0) and loads sixteen
// units' values before adding them in order, so the partials stream instead of one round trip
// per unit.
template <int VEC>
__global__ __launch_bounds__(256) void reduce_units_kernel(const float* __restrict__ part, KgradUnits units, int cin,
                                                           int cout, FieldTab fout, FieldTab fin,
                                                           float* __restrict__ dW) {
  const int e = (blockIdx.x * blockDim.x + threadIdx.x) * VEC;
  const int s = blockIdx.y;
  const int64_t n = (int64_t)cin * cout;
  if (e >= n) return;
  float acc[VEC];
#pragma unroll
  for (int k = 0; k < VEC; ++k) acc[k] = 0.f;
  // batches of 16 units: every load issued (a unit past the offset's last reads that last unit
  // again and contributes +0, which leaves the sum unchanged: it never holds -0), then the adds in
  // unit order
  const int u0 = units.uoff[s], u1 = units.uoff[s + 1];
  for (int u = u0; u < u1; u += 16) {
    float v[16][VEC];
#pragma unroll
    for (int j = 0; j < 16; ++j) {
      const float* p = part + (int64_t)min(u + j, u1 - 1) * n + e;
      if constexpr (VEC == 4) {
        const float4 t = *reinterpret_cast<const float4*>(p);
        v[j][0] = t.x, v[j][1] = t.y, v[j][2] = t.z, v[j][3] = t.w;
      } else {
        v[j][0] = *p;
      }
    }
#pragma unroll
    for (int j = 0; j < 16; ++j)
#pragma unroll
      for (int k = 0; k < VEC; ++k) acc[k] += u + j < u1 ? v[j][k] : 0.f;
  }
  const int o = e / cin;
#pragma unroll
  for (int k = 0; k < VEC; ++k) dW[dw_block_pos(fout, fin, units.K, cin, s, o, e + k - o * cin)] = acc[k];
}

}  // namespace

KgradUnits kgrad_units(const ssconv_rulebook* rb, int want, bool ordered) {
  KgradUnits u;
  u.K = rb->K;
  const int K = rb->K;
  const int cap = ordered ? kKgradMaxUnits : kKgradMaxUnitsF32;
  int64_t total = 0;
  for (int s = 0; s < K; ++s) total += rb->pair_off[s + 1] - rb->pair_off[s];
  want = std::min(std::max(want, K), cap);
  int n[kKgradMaxK];
  double rem[kKgradMaxK];
  int sum = 0;
  for (int s = 0; s < K; ++s) {
    const double quota = total > 0 ? (double)(rb->pair_off[s + 1] - rb->pair_off[s]) * want / (double)total : 0.0;
    n[s] = std::max(1, (int)quota);
    rem[s] = quota - n[s];
    sum += n[s];
  }
  // largest remainders first (the floors leave fewer than K units to hand out, one per offset at
  // most); ties by offset, so the split is deterministic
  int by_rem[kKgradMaxK];
  for (int s = 0; s < K; ++s) by_rem[s] = s;
  std::stable_sort(by_rem, by_rem + K, [&](int a, int b) { return rem[a] > rem[b]; });
  for (int i = 0; i < K && sum < want && rem[by_rem[i]] > 0.0; ++i) ++n[by_rem[i]], ++sum;
  while (sum > cap) {  // the one-unit minimum can overshoot: trim the largest offsets
    int big = 0;
    for (int s = 1; s < K; ++s)
      if (n[s] > n[big]) big = s;
    --n[big];
    --sum;
  }
  u.uoff[0] = 0;
  for (int s = 0; s < K; ++s) u.uoff[s + 1] = u.uoff[s] + n[s];
  u.nunits = u.uoff[K];
  if (!ordered) return u;
  // launch order: by the centre of each unit's slice along R_s (pairs are sorted by output row),
  // ties by offset -- a stable order, so the launch is deterministic
  std::vector<std::pair<double, int>> key(u.nunits);
  for (int s = 0; s < K; ++s)
    for (int j = 0; j < n[s]; ++j) key[u.uoff[s] + j] = {(j + 0.5) / n[s], u.uoff[s] + j};
  std::stable_sort(key.begin(), key.end(),
                   [](const std::pair<double, int>& a, const std::pair<double, int>& b) { return a.first < b.first; });
  for (int i = 0; i < u.nunits; ++i) u.order[i] = (uint16_t)key[i].second;
  return u;
}

int reduce_units(const float* part, const KgradUnits& units, int cin, int cout, const FieldTab& fout,
                 const FieldTab& fin, float* dW, hipStream_t st) {
  const int64_t n = (int64_t)cin * cout;
  if (n == 0 || units.K == 0) return SSCONV_OK;
  if (cin % 4 == 0)
    reduce_units_kernel<4><<<dim3(cdiv(n / 4, 256), units.K), 256, 0, st>>>(part, units, cin, cout, fout, fin, dW);
  else
    reduce_units_kernel<1><<<dim3(cdiv(n, 256), units.K), 256, 0, st>>>(part, units, cin, cout, fout, fin, dW);
  SSC_HIP(hipGetLastError());
  return SSCONV_OK;
}

int kgrad_bf16_tile(int cin, int cout) {
  const int need = (std::max(cout, cin) + 31) / 32;
  return need <= 2 ? 2 : need <= 4 ? 4 : 7;
}

int kgrad_bf16(const void* grad_out, int64_t n_out, const void* feats, int64_t n_in, int cin, int cout,
               const ssconv_rulebook* rb, const KgradUnits& units, float* part, hipStream_t st) {
  if (units.nunits == 0) return SSCONV_OK;
  const int W = kgrad_bf16_tile(cin, cout);
  const int mtiles = (cout + 32 * W - 1) / (32 * W), ntiles = (cin + 32 * W - 1) / (32 * W);
  dim3 grid((unsigned)(units.nunits * mtiles * ntiles));
  const int2* pairs = reinterpret_cast<const int2*>(rb->pairs);
  // override 12: the column layout (same operands in the MFMAs, same results bit for bit)
  const bool quad = debug_gather_variant() != 12;
#define SSK_LAUNCH(Wv)                                                                              \
  do {                                                                                              \
    auto kern = quad ? kgrad_bf16_kernel<Wv, true> : kgrad_bf16_kernel<Wv, false>;                  \
    const int smem = quad ? KB<Wv, true>::SMEM : KB<Wv, false>::SMEM;                               \
    SSC_HIP(hipFuncSetAttribute((const void*)kern, hipFuncAttributeMaxDynamicSharedMemorySize, smem)); \
    kern<<<grid, 256, smem, st>>>((const uint16_t*)grad_out, n_out, cout, (const uint16_t*)feats, n_in, cin, \
                                  pairs, rb->pair_off_dev, units, mtiles, ntiles, part);            \
  } while (0)
  if (W == 2) SSK_LAUNCH(2);
  else if (W == 4) SSK_LAUNCH(4);
  else SSK_LAUNCH(7);
#undef SSK_LAUNCH
  SSC_HIP(hipGetLastError());
  return SSCONV_OK;
}

}  // namespace ssconv
