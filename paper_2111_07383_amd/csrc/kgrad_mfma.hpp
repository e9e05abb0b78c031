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

// part[split][s][o][i] (fp32) = sum over the split's slice of R_s of grad_out[x][o] feats[y][i].
int kgrad_partials(const void* grad_out, const void* feats, ssconv_dtype dt, int cin, int cout,
                   const ssconv_rulebook* rb, const KgradPlan& p, float* part, hipStream_t st);

}  // namespace ssconv
