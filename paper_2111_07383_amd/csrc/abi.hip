// C ABI entry points of the convolution: argument checks and launches.
#include <algorithm>
#include <mutex>

#include "conv.hpp"
#include "norm.hpp"
#include "synth.hpp"

using namespace ssconv;

namespace {

int check_conv_args(const void* a, const void* b, ssconv_dtype dt, int cin, int cout, ssconv_rulebook_t rb,
                    const void* W) {
  if (dt != SSCONV_F32 && dt != SSCONV_BF16) return fail(SSCONV_E_DTYPE, "unsupported dtype %d", (int)dt);
  if (!rb) return fail(SSCONV_E_INVALID, "NULL rule book");
  if ((rb->ksize & 1) == 0) return fail(SSCONV_E_INVALID, "a ksize-2 rule book holds pooling windows (ssconv_pool_*)");
  if (cin < 1 || cout < 1) return fail(SSCONV_E_INVALID, "channel counts must be positive");
  if (!W) return fail(SSCONV_E_INVALID, "NULL kernel tensor");
  if (!aligned16(W) || (a && !aligned16(a)) || (b && !aligned16(b)))
    return fail(SSCONV_E_INVALID, "device buffers must be 16-byte aligned");
  return SSCONV_OK;
}

}  // namespace

extern "C" int ssconv_forward(const void* feats, ssconv_dtype dtype, int cin, ssconv_rulebook_t rb, const void* W,
                              int cout, void* out, hipStream_t stream) {
  SSC_TRY(check_conv_args(feats, out, dtype, cin, cout, rb, W));
  // fp32 picks its kernel from the pair counts; bf16 needs only the neighbour map, so it may run
  // on an asynchronous build that has not been settled yet
  if (dtype != SSCONV_BF16) SSC_TRY(rulebook_settle(rb));
  if ((rb->n_in > 0 && !feats) || (rb->n_out > 0 && !out)) return fail(SSCONV_E_INVALID, "NULL feature buffer");
  if (rb->n_in == 0 && rb->n_out > 0) {
    SSC_HIP(hipMemsetAsync(out, 0, (size_t)rb->n_out * cout * dtype_bytes(dtype), stream));
    return SSCONV_OK;
  }
  return conv_forward(feats, dtype, cin, rb, W, cout, out, stream);
}

extern "C" int ssconv_forward_norm(const void* feats, ssconv_dtype dtype, int cin, ssconv_rulebook_t rb,
                                   const void* W, const ssconv_fields* fields_out, double eps, void* y, void* z,
                                   hipStream_t stream) {
  if (!fields_out) return fail(SSCONV_E_INVALID, "NULL field table");
  FieldTab f;
  SSC_TRY(norm_check_fields(fields_out, dtype, rb ? rb->n_out : 0, eps, &f));
  const int cout = f.ch0[f.n];
  SSC_TRY(check_conv_args(feats, y, dtype, cin, cout, rb, W));
  if (dtype != SSCONV_BF16) SSC_TRY(rulebook_settle(rb));
  if (z && !aligned16(z)) return fail(SSCONV_E_INVALID, "device buffers must be 16-byte aligned");
  if ((rb->n_in > 0 && !feats) || (rb->n_out > 0 && (!y || !z))) return fail(SSCONV_E_INVALID, "NULL feature buffer");
  return conv_forward_norm(feats, dtype, cin, rb, W, cout, f, eps, y, z, stream);
}

// ---------------------------------------------------------------------------
// allocation-free forward
// ---------------------------------------------------------------------------
// The scratch of ssconv_forward_noalloc: one fixed region per device, part of the library's code
// object (each device that loads the library holds its own copy until the process ends).  Host
// code never uses this name as a device address: it is a host-side stand-in; the device address
// comes from hipGetSymbolAddress, taken once per device with that device current.
static __device__ __align__(256) char scratch[SSCONV_NOALLOC_SCRATCH_BYTES];

namespace {

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
char* g_scratch_ptr[kMaxDevices] = {};

// Device address of this device's scratch region (looked up on the first call per device).
int scratch_region(char** out) {
  int dev = 0;
  SSC_HIP(hipGetDevice(&dev));
  if (dev < 0 || dev >= kMaxDevices) return fail(SSCONV_E_INVALID, "device %d is beyond the %d supported", dev, kMaxDevices);
  std::lock_guard<std::mutex> lk(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* p = nullptr;
    SSC_HIP(hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)));
    if (!p) return fail(SSCONV_E_HIP, "hipGetSymbolAddress returned no address for the scratch region");
    g_scratch_ptr[dev] = (char*)p;
  }
  *out = g_scratch_ptr[dev];
  return SSCONV_OK;
}

__global__ void zero_halves_kernel(uint16_t* __restrict__ p, int64_t n) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) p[i] = 0u;
}

}  // namespace

extern "C" int ssconv_forward_noalloc(const void* feats, ssconv_dtype dtype, int cin, ssconv_rulebook_t rb,
                                      const void* W, int cout, void* out, hipStream_t stream) {
  SSC_TRY(check_conv_args(feats, out, dtype, cin, cout, rb, W));
  if (dtype != SSCONV_BF16) SSC_TRY(rulebook_settle(rb));
  if ((rb->n_in > 0 && !feats) || (rb->n_out > 0 && !out)) return fail(SSCONV_E_INVALID, "NULL feature buffer");
  if (rb->n_out == 0) return SSCONV_OK;
  if (rb->n_in == 0) {  // no input rows: every output row is 0 (a fill kernel, no memset node)
    const int64_t halves = (int64_t)rb->n_out * cout * (int64_t)dtype_bytes(dtype) / 2;  // exactly the buffer
    zero_halves_kernel<<<cdiv(halves, 256), 256, 0, stream>>>((uint16_t*)out, halves);
    SSC_HIP(hipGetLastError());
    return SSCONV_OK;
  }
  CallScratch sc;
  SSC_TRY(scratch_region(&sc.base));
  sc.cap = SSCONV_NOALLOC_SCRATCH_BYTES;
  return conv_forward(feats, dtype, cin, rb, W, cout, out, stream, &sc);
}

extern "C" size_t ssconv_backward_workspace_size(ssconv_rulebook_t rb, ssconv_dtype dtype, int cin, int cout) {
  if (!rb || cin < 1 || cout < 1) return 0;
  if (rulebook_settle(rb) != SSCONV_OK) return 0;
  return bwd_layout(rb, dtype, cin, cout).total;
}

extern "C" int ssconv_backward(const void* feats, const void* grad_out, ssconv_dtype dtype, int cin, int cout,
                               ssconv_rulebook_t rb, const void* W, const ssconv_basis_desc* desc, const float* basis,
                               void* grad_feats, float* grad_coeffs, void* workspace, size_t ws_bytes,
                               hipStream_t stream) {
  SSC_TRY(check_conv_args(feats, grad_out, dtype, cin, cout, rb, W));
  SSC_TRY(rulebook_settle(rb));
  if (grad_feats && !aligned16(grad_feats)) return fail(SSCONV_E_INVALID, "grad_feats must be 16-byte aligned");
  const BwdLayout L = bwd_layout(rb, dtype, cin, cout);
  if (!workspace || ws_bytes < L.total || (reinterpret_cast<uintptr_t>(workspace) & 255))
    return fail(SSCONV_E_INVALID, "workspace must be 256-byte aligned and hold %zu bytes", L.total);
  if ((rb->n_out > 0 && !grad_out) || (rb->n_in > 0 && !feats)) return fail(SSCONV_E_INVALID, "NULL input buffer");
  SynthArgs sa;
  if (grad_coeffs) {
    if (!basis) return fail(SSCONV_E_INVALID, "basis is required for the coefficient gradient");
    SSC_TRY(make_synth_args(desc, &sa));
    if (sa.cin != cin || sa.cout != cout || sa.K != rb->K)
      return fail(SSCONV_E_INVALID, "basis descriptor does not match cin/cout/ksize");
  }
  char* ws = (char*)workspace;
  // The coefficient gradient (kernel gradient, its reduction, the synthesis adjoint) does not
  // depend on the feature gradient.  When the feature gradient takes the pair-list path (a chain
  // of small launches) the coefficient gradient runs on the library's second stream, forked from
  // and joined back to the caller's, so the two overlap (disjoint workspace regions).  Next to
  // the fp32 output-stationary gather kernel only its tail is forked: the kernel gradient runs on
  // the caller's stream, then its reduction and the synthesis adjoint (small, memory-bound) run
  // on the second stream next to the feature gradient (C2 backward 1.437 -> 1.424 ms).  Next to
  // the bf16 gather nothing is forked: the tail cost it 0.802 -> 0.809 ms (C4 backward), and the
  // whole coefficient gradient made the two slow each other down (C4 step 1.49 -> 1.56 ms).
  // Kernel-selection override 11 switches both forks off.
  hipStream_t dw_stream = stream;
  const bool both = grad_feats && grad_coeffs && rb->n_out > 0 && debug_gather_variant() != 11;
  const bool fork = both && L.pair_feats;
  const bool fork_tail = both && !L.pair_feats && rb->n_in > 0 && dtype == SSCONV_F32;
  bool need_join = fork;
  if (fork) SSC_TRY(aux_fork(stream, &dw_stream));
  int rc = SSCONV_OK;
  if (grad_coeffs) {
    float* dW = nullptr;
    hipStream_t tail = dw_stream;
    rc = conv_backward_dw(feats, grad_out, dtype, cin, cout, rb, sa.out, sa.in, ws, L, &dW, dw_stream,
                          fork_tail ? &tail : nullptr);
    if (fork_tail && tail != stream) {
      dw_stream = tail;
      need_join = true;
    }
    if (rc == SSCONV_OK) rc = launch_synth_adjoint(sa, basis, dW, grad_coeffs, dw_stream);
  }
  if (rc == SSCONV_OK && grad_feats) {
    if (rb->n_out == 0 && rb->n_in > 0) {
      if (hipMemsetAsync(grad_feats, 0, (size_t)rb->n_in * cin * dtype_bytes(dtype), stream) != hipSuccess)
        rc = fail(SSCONV_E_HIP, "hipMemsetAsync failed");
    } else {
      rc = conv_backward_feats(grad_out, dtype, cin, cout, rb, W, grad_feats, ws, L, stream);
    }
  }
  if (need_join) {
    const int jr = aux_join(stream, dw_stream);  // always joined, so nothing stays pending on the side stream
    if (rc == SSCONV_OK) rc = jr;
  }
  return rc;
}
