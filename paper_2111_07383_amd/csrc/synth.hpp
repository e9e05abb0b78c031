// Kernel synthesis arguments shared by the synthesis and backward entry points.
#pragma once

#include "common.hpp"

namespace ssconv {

// Basis layout tables computed on the host (basis_host.cpp).
int validate_desc(const ssconv_basis_desc* d);
int basis_nq_table(const ssconv_basis_desc* d, int nq[SSCONV_MAX_L + 1][SSCONV_MAX_L + 1],
                   int64_t base[SSCONV_MAX_L + 1][SSCONV_MAX_L + 1], int64_t* total_floats);

// Per (out entry, in entry) block: what a wavefront needs once it knows its two entries.
struct EntryPair {
  int64_t coff0;  // coefficient offset of the (first out field, first in field) block
  int64_t base;   // float offset of the (k, l) block in the basis buffer
  int rowsz;      // coefficients per out field of order k (step from one out field to the next)
  int nq;         // basis elements per (k, l), the step from one in field to the next
  int k, l;
};

struct SynthArgs {
  FieldTab in, out;
  EntryPair ep[SSCONV_MAX_ENTRIES][SSCONV_MAX_ENTRIES];
  int K, cin, cout;
  int n_out_fields, n_in_fields;
  int nq[SSCONV_MAX_L + 1][SSCONV_MAX_L + 1];       // basis elements per (k, l)
  int64_t base[SSCONV_MAX_L + 1][SSCONV_MAX_L + 1];  // float offset of the (k, l) block in the basis buffer
  int64_t rowsz[SSCONV_MAX_L + 1];                   // coefficients per out field of order k
  int64_t row0[SSCONV_MAX_ENTRIES];                  // coefficient offset of each out entry
  int64_t n_coeff;
};

int make_synth_args(const ssconv_basis_desc* d, SynthArgs* a);
int launch_synth(const SynthArgs& a, const float* basis, const float* coeffs, ssconv_dtype dt, void* W,
                 hipStream_t st);
// dW in the field-pair-blocked layout of dw_block_pos.
int launch_synth_adjoint(const SynthArgs& a, const float* basis, const float* dW, float* dcoef, hipStream_t st);

}  // namespace ssconv
