// Kernel-tensor gradient: per-offset GEMM over the pair lists, split along the pairs.
#pragma once

#include "common.hpp"

namespace ssconv {

struct KgradPlan {
  int wmb = 1, wnb = 1;        // 16-channel blocks per wavefront tile (out, in)
  int mtiles = 1, ntiles = 1;  // tiles covering Cout and Cin
  int nsplit = 1;              // pair slices per offset (one partial each)
};

// fp32 handles any channel counts; bf16 needs multiples of 8 channels and at most 224 per side.
inline bool kgrad_supported(ssconv_dtype dt, int cin, int cout) {
  return dt == SSCONV_F32 || (cin % 8 == 0 && cout % 8 == 0 && cin <= 224 && cout <= 224);
}

KgradPlan kgrad_plan(const ssconv_rulebook* rb, ssconv_dtype dt, int cin, int cout);

// Work units of the bf16 kernel gradient: offset s owns units uoff[s] .. uoff[s+1]-1, which cut
// its pair list R_s into near-equal slices (passed to the kernels by value).
// Units are launched in `order`: sorted by the position of their slice along the output rows
// and handed out XCD-contiguously, so the units of all offsets over one stretch of rows run on
// one XCD together and share its L2 for the gathered rows.
constexpr int kKgradMaxK = 125;  // ksize <= 5
constexpr int kKgradMaxUnits = 512;      // bf16 (launch order recorded)
constexpr int kKgradMaxUnitsF32 = 4096;  // fp32 (one wavefront per unit and tile)
struct KgradUnits {
  int K = 0, nunits = 0;
  int uoff[kKgradMaxK + 1] = {};
  uint16_t order[kKgradMaxUnits] = {};
};

// Units for the rule book: about `want` in total (at least one per offset, at most
// kKgradMaxUnits when `ordered`, else kKgradMaxUnitsF32), distributed over the offsets in
// proportion to their pair counts (largest remainders); `ordered` also records the launch order.
KgradUnits kgrad_units(const ssconv_rulebook* rb, int want, bool ordered);

// fp32 kernel gradient over work units (per-wavefront LDS ring): usable when every row offset
// fits 31 bits; the unit count that fills one round of wavefront slots.
bool kgrad_f32_units_ok(const ssconv_rulebook* rb, int cin, int cout);
int kgrad_f32_units_want(const ssconv_rulebook* rb, int cin, int cout);
int kgrad_f32(const void* grad_out, const void* feats, int cin, int cout, const ssconv_rulebook* rb,
              const KgradUnits& units, float* part, hipStream_t st);

// bf16 tile width (in 32-channel steps of the 2x2 wavefront grid) for cin x cout.
int kgrad_bf16_tile(int cin, int cout);

// part[u][o][i] (fp32) = sum over unit u's slice of R_s of grad_out[x][o] feats[y][i]; grad_out
// holds n_out rows, feats n_in rows.
int kgrad_bf16(const void* grad_out, int64_t n_out, const void* feats, int64_t n_in, int cin, int cout,
               const ssconv_rulebook* rb, const KgradUnits& units, float* part, hipStream_t st);

// dW[s][:] = sum over the units of offset s of part[u][:] (n = cout * cin per unit), fixed order.
// dW (field-pair-blocked, dw_block_pos) from the unit partials, each offset's in unit order.
int reduce_units(const float* part, const KgradUnits& units, int cin, int cout, const FieldTab& fout,
                 const FieldTab& fin, float* dW, hipStream_t st);

// part[split][s][o][i] (fp32) = sum over the split's slice of R_s of grad_out[x][o] feats[y][i].
int kgrad_partials(const void* grad_out, const void* feats, ssconv_dtype dt, int cin, int cout,
                   const ssconv_rulebook* rb, const KgradPlan& p, float* part, hipStream_t st);

}  // namespace ssconv
