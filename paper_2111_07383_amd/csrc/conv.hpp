// Internal interface of the gather-GEMM kernels.
#pragma once

#include "common.hpp"

namespace ssconv {

struct NormSink;

struct BwdLayout {
  size_t nbrT = 0, Wt = 0, part = 0, dW = 0, pair = 0, total = 0;  // byte offsets in the workspace
  int nsplit = 1;
  bool pair_feats = false;  // feature gradient on the pair-list path
};

// Pair-list GEMM for sparse fp32 layers (pair_gemm.hip).
bool pair_path_supported(const ssconv_rulebook* rb, ssconv_dtype dt, int ca, int cb);
bool pair_path_wins(const ssconv_rulebook* rb, ssconv_dtype dt, int ca, int cb, int64_t n_dst);
size_t pair_path_bytes(const ssconv_rulebook* rb, int ca, int cb, int64_t n_dst);
// sink (optional): the reduce pass also leaves the Norm statistics of dst there (norm.hpp).
int pair_gemm(const void* src, int ca, const void* Bt, int cb, const ssconv_rulebook* rb, int sel_in, void* dst,
              int64_t n_dst, void* ws, hipStream_t st, NormSink* sink = nullptr);

// sc: where the call's scratch comes from (nullptr: the device memory cache).  sink (optional):
// the kernel that writes out also leaves the Norm statistics of out there where it can.
int conv_forward(const void* feats, ssconv_dtype dt, int cin, const ssconv_rulebook* rb, const void* W, int cout,
                 void* out, hipStream_t st, CallScratch* sc = nullptr, NormSink* sink = nullptr);
// y = the convolution, z = Norm(y) over the fields f of the output channels (z may alias y).
int conv_forward_norm(const void* feats, ssconv_dtype dt, int cin, const ssconv_rulebook* rb, const void* W, int cout,
                      const FieldTab& f, double eps, void* y, void* z, hipStream_t st);
BwdLayout bwd_layout(const ssconv_rulebook* rb, ssconv_dtype dt, int cin, int cout);
int conv_backward_feats(const void* grad_out, ssconv_dtype dt, int cin, int cout, const ssconv_rulebook* rb,
                        const void* W, void* grad_feats, char* ws, const BwdLayout& L, hipStream_t st);
// Kernel gradient dW in the field-pair-blocked layout (dw_block_pos) of the fields fout, fin.
// With tail given, a balanced-unit kernel gradient forks its reduction onto the library's second
// stream (aux_fork after the partials are queued on st) and *tail receives the stream dW is
// complete on (st when nothing was forked); the caller joins it.
int conv_backward_dw(const void* feats, const void* grad_out, ssconv_dtype dt, int cin, int cout,
                     const ssconv_rulebook* rb, const FieldTab& fout, const FieldTab& fin, char* ws,
                     const BwdLayout& L, float** dW_out, hipStream_t st, hipStream_t* tail = nullptr);

}  // namespace ssconv
