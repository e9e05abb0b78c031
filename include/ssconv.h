/*
 * ssconv.h -- C ABI of the MI355X (gfx950) Sparse Steerable Convolution library.
 *
 * Sparse Steerable Convolution (SS-Conv, Lin et al., NeurIPS 2021,
 * arXiv 2111.07383) convolves a sparse tensor (H_n, F_n) -- a hash table of
 * active voxel sites and a feature matrix whose rows follow it -- with a
 * rotation-steerable kernel kappa to give (H_{n+1}, F_{n+1}) (Sec. 3.2).
 * The library implements the three steps of Sec. 3.2:
 *   1. rule book construction (Sec. 3.2.2 site state, the rule-book part of
 *      Alg. 1 in Sec. 3.2.3) over a GPU coordinate hash table;
 *   2. kernel synthesis as a linear combination of steerable basis kernels
 *      (Sec. 3.2.1, Eq. 7-9);
 *   3. the feature update of Alg. 1 as an output-stationary
 *      gather -> matrix-core GEMM -> single write per output row;
 * plus the exact adjoint (feature and coefficient gradients) and the gated
 * nonlinearity of Sec. 3.3 (Eq. 12).
 *
 * Conventions shared by every call
 *  - Pointers are DEVICE pointers unless marked (host).  The caller owns every
 *    buffer it passes and every stream; the library owns only the internal
 *    buffers of a rule book handle.
 *  - Every call returns 0 (SSCONV_OK) or a negative SSCONV_E_* code and never
 *    throws; ssconv_last_error() gives a message (thread-local).  On error no
 *    handle is returned (the out-handle is set to NULL).
 *  - Work is enqueued on the given stream and is asynchronous, except
 *    ssconv_build_rulebook, which synchronises the stream to size its
 *    outputs and to report device-detected errors (ssconv_build_rulebook_async
 *    defers that for submanifold layers), and the calls that settle such a
 *    build.
 *  - Sites are int32 (b, x, y, z) with 0 <= x < grid[0], 0 <= y < grid[1],
 *    0 <= z < grid[2], b >= 0 and (max b + 1) * grid[0]*grid[1]*grid[2] < 2^32.
 *  - Kernel offsets s = (dx, dy, dz) in S = {-h..ksize-1-h}^3, h = ksize/2
 *    ({-h..h}^3 for the odd convolution kernels), are indexed
 *    s_idx = ((dx+h)*ksize + (dy+h))*ksize + (dz+h)   (Sec. 3.2, Eq. 6).
 *  - Channel layout (Sec. 3.1, Eq. 5): a feature row stacks irreducible fields
 *    in the order of an ssconv_fields list; the fields of one entry are
 *    consecutive and each field's 2l+1 components are contiguous, ordered
 *    m = -l..l in the real spherical-harmonic basis (no Condon-Shortley phase;
 *    Y_1 is proportional to (y, z, x)).
 *  - Feature matrices are row-major [rows, channels]; row r of F_n belongs to
 *    site r of H_n (Sec. 3.2).
 *  - The kernel tensor W is kappa(s) of Eq. 9 for every offset, stored
 *    row-major [ksize^3][Cout][Cin]: out_row(x) = sum_s kappa(s) in_row(y).
 */
#ifndef SSCONV_H
#define SSCONV_H

#include <stddef.h>
#include <stdint.h>

#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

/* ---- status codes ------------------------------------------------------- */
#define SSCONV_OK 0
#define SSCONV_E_INVALID (-1)   /* bad argument (null pointer, bad size/flag/alignment) */
#define SSCONV_E_BOUNDS (-2)    /* a site lies outside the grid or the 32-bit key space */
#define SSCONV_E_DUPLICATE (-3) /* the same site appears twice in the input */
#define SSCONV_E_HASH_FULL (-4) /* hash table capacity exhausted (only with a forced capacity) */
#define SSCONV_E_NOMEM (-5)     /* device allocation failed */
#define SSCONV_E_HIP (-6)       /* a HIP runtime call failed */
#define SSCONV_E_DTYPE (-7)     /* unsupported dtype */

typedef enum { SSCONV_F32 = 0, SSCONV_BF16 = 1 } ssconv_dtype;

#define SSCONV_MAX_ENTRIES 8
#define SSCONV_MAX_L 4
#define SSCONV_MAX_SHELLS 8

/* A feature type: entries (l[e], mult[e]) in channel order (Sec. 3.1, Eq. 5).
 * Channels = sum_e mult[e] * (2 l[e] + 1).  0 <= l[e] <= SSCONV_MAX_L. */
typedef struct {
  int n;
  int l[SSCONV_MAX_ENTRIES];
  int mult[SSCONV_MAX_ENTRIES];
} ssconv_fields;

/* Basis of one layer (Sec. 3.2.1, Eq. 8): for every out field (order k) and in
 * field (order l), elements kappa^{kl,Jm} for J = |k-l| .. min(k+l, jmax) and
 * every radial shell m, with phi^m(r) = exp(-(r - shells[m])^2 / (2 eps^2)).
 * jmax < 0 means no band limit.  Each element is normalised to unit Frobenius
 * norm over (offset, row, column) with its first entry of magnitude above
 * 1e-3 of its maximum made positive; elements that vanish on the grid
 * (J > 0 on a 1x1x1 kernel) are left out. */
typedef struct {
  ssconv_fields in, out;
  int ksize;
  int n_shells;
  double shells[SSCONV_MAX_SHELLS];
  double eps;
  int jmax;
} ssconv_basis_desc;

typedef struct ssconv_rulebook* ssconv_rulebook_t;

const char* ssconv_last_error(void);
const char* ssconv_version(void);

/* Device memory the library allocates (rule book buffers, the packed bf16 kernel
 * of ssconv_forward) comes from a per-process cache: a freed block is kept with
 * the stream that freed it and reused, on that stream at once (stream order),
 * on another stream after that stream waits for an event recorded at reuse on
 * the freeing stream; up to 8 GB of free blocks are kept, beyond that the
 * oldest are freed stream-ordered on their freeing stream.  A stream that
 * frees library memory (destroys a rule book, runs a call with temporaries)
 * must therefore stay valid while the cache holds the block: until
 * ssconv_empty_cache, or for the life of the process.  ssconv_empty_cache
 * synchronises each free block's stream and releases every free block (blocks
 * in use are untouched); ssconv_cached_bytes returns the bytes held in free
 * blocks.  Both are safe to call at any time. */
int ssconv_empty_cache(void);
int64_t ssconv_cached_bytes(void);

/* ---- steerable basis (host) ---------------------------------------------
 * Sec. 3.2.1, Eq. 7-8.  Computed on the host in fp64 from Clebsch-Gordan
 * coefficients (Racah's formula) carried to the real harmonic basis.
 *
 * ssconv_basis_info: number of floats of the basis buffer and number of
 * learned coefficients (sum over field pairs of the block's element count;
 * without vanishing elements M (2 min(k,l)+1) per block when J is uncapped).
 *
 * ssconv_basis_build: fills (host) basis[basis_floats] as fp32.  Layout: for
 * every distinct out order k (ascending) and distinct in order l (ascending):
 * [nq(k,l)][ksize^3][2k+1][2l+1], elements ordered (J ascending, shell).
 *
 * Coefficient layout (ssconv_synth_kernel / ssconv_backward): for every out
 * field i, every in field j (channel order), the nq(k_i, l_j) weights
 * w^{k l, J m} in element order. */
int ssconv_basis_info(const ssconv_basis_desc* desc /*host*/, int64_t* basis_floats /*host*/,
                      int64_t* n_coeff /*host*/);
int ssconv_basis_build(const ssconv_basis_desc* desc /*host*/, float* basis /*host*/);

/* ---- rule book (Sec. 3.2.2, Eq. 10; Sec. 3.2.3, rule book of Alg. 1) -----
 * coords: [n, 4] int32 (b, x, y, z), n >= 0, no duplicates.
 * grid (host): input grid extent per axis.  ksize: odd, 1..5, or 2 with
 * stride 2 (the 2x2x2 pooling windows of ssconv_pool_*, offsets {-1, 0}^3).
 * stride: 1 or 2.  submanifold = 1 keeps H_{n+1} = H_n (stride must be 1, rows
 * unchanged); otherwise H_{n+1} = { x : exists y in H_n, stride*x - y in S }
 * clipped to the output grid ceil(grid/stride), rows in lexicographic
 * (b, x, y, z) order.  Pairs satisfy stride*x - y = s and never cross b.
 * The call synchronises `stream` and returns a handle that owns all device
 * buffers (coordinate hash tables, neighbour map, per-offset pair lists);
 * they are freed by ssconv_rulebook_destroy, stream-ordered on `stream`,
 * which must still be valid then.  Errors: E_INVALID, E_BOUNDS,
 * E_DUPLICATE, E_HASH_FULL, E_NOMEM, E_HIP. */
int ssconv_build_rulebook(const int32_t* coords, int64_t n, const int32_t* grid /*host [3]*/,
                          int ksize, int stride, int submanifold, hipStream_t stream,
                          ssconv_rulebook_t* out /*host*/);
/* The same build without its final synchronisation, for submanifold layers
 * (generated output sets synchronise as ssconv_build_rulebook does, since the
 * output count sizes their buffers): the handle is returned as soon as the
 * build's kernels and the read-back of its pair counts are queued on `stream`.
 * The pair counts, and the errors the device detects (E_BOUNDS, E_DUPLICATE,
 * E_HASH_FULL), reach the host when the build is settled: by
 * ssconv_rulebook_wait, or by the first call that needs them (rulebook info,
 * pairs and hash, backward and its workspace size, fp32 forwards, pooling,
 * interpolation), which then returns that error.  The neighbour map is complete
 * on `stream`, so a bf16 forward and the map and site copies may be queued
 * before the build is settled; if the build then reports an error, their
 * results are undefined (never an access out of bounds: every map entry is a
 * row of the input or -1).  Argument errors and allocation failures are
 * returned at once, as by ssconv_build_rulebook. */
int ssconv_build_rulebook_async(const int32_t* coords, int64_t n, const int32_t* grid /*host [3]*/,
                                int ksize, int stride, int submanifold, hipStream_t stream,
                                ssconv_rulebook_t* out /*host*/);
/* Settles an asynchronous build (blocks the host until its read-back has
 * arrived) and returns the build's result; a synchronous build returns
 * SSCONV_OK.  Every later call returns the same result. */
int ssconv_rulebook_wait(ssconv_rulebook_t rb);

/* n_in, n_out (host) and, if non-NULL, pair_counts (host [ksize^3]) = |R_s|. */
int ssconv_rulebook_info(ssconv_rulebook_t rb, int64_t* n_in, int64_t* n_out,
                         int64_t* pair_counts);
/* Copies H_{n+1} as [n_out, 4] int32 into dst. */
int ssconv_rulebook_out_coords(ssconv_rulebook_t rb, int32_t* dst, hipStream_t stream);
/* Copies all R_s concatenated in s_idx order as [P, 2] int32 (out row, in row)
 * into dst, P = sum of pair_counts; within R_s pairs follow the output rows. */
int ssconv_rulebook_pairs(ssconv_rulebook_t rb, int32_t* dst, hipStream_t stream);
/* Copies the neighbour map nbr[s_idx][out row] (in row or -1) as [ksize^3, n_out] int32. */
int ssconv_rulebook_neighbours(ssconv_rulebook_t rb, int32_t* dst, hipStream_t stream);
/* Copies a coordinate hash table (which = 0: H_n, 1: H_{n+1}) as its raw uint64
 * slots (key << 32 | row, key = ((b*G0 + x)*G1 + y)*G2 + z, empty = ~0) into dst
 * [capacity]; *capacity (host) is set when dst is NULL.  The table of a generated
 * output set (which = 1, non-submanifold) is not needed to build the rule book; it
 * is filled on the first call that asks for it, on stream, and that call then
 * synchronises with the host (SSCONV_E_HASH_FULL if it overflows). */
int ssconv_rulebook_hash(ssconv_rulebook_t rb, int which, uint64_t* dst, int64_t* capacity /*host*/,
                         hipStream_t stream);
void ssconv_rulebook_destroy(ssconv_rulebook_t rb);

/* ---- kernel synthesis (Sec. 3.2.1, Eq. 7 and Eq. 9) -----------------------
 * W[s][o][i] = sum over the basis elements q of the block holding out channel
 * o and in channel i of coeffs[q] * basis_q[s][a][b].  basis and coeffs are
 * fp32 device buffers in the layouts of ssconv_basis_build; W is written in
 * w_dtype (fp32, or bf16 rounded to nearest even from the fp32 sum). */
int ssconv_synth_kernel(const ssconv_basis_desc* desc /*host*/, const float* basis,
                        const float* coeffs, ssconv_dtype w_dtype, void* W, hipStream_t stream);

/* ---- forward (Sec. 3.2.3, feature update of Alg. 1) -----------------------
 * out[x] = sum_s sum_{(x,y) in R_s} kappa(s) feats[y], every output row written
 * exactly once (rows with no pair become 0).  feats [n_in, cin], W
 * [ksize^3, cout, cin], out [n_out, cout], all in `dtype` (bf16 inputs are
 * multiplied exactly and accumulated in fp32).  Buffers must be 16-byte
 * aligned.  feats and out must not overlap.  rb must have an odd ksize. */
int ssconv_forward(const void* feats, ssconv_dtype dtype, int cin, ssconv_rulebook_t rb,
                   const void* W, int cout, void* out, hipStream_t stream);

/* ---- allocation-free forward ----------------------------------------------
 * For callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc): the same
 * operation, arguments and results as ssconv_forward, but the call allocates
 * nothing — no hipMalloc / hipFree / hipMallocAsync, no library cache block.
 * The scratch the kernels need (the packed bf16 kernel, fp32 offset-split
 * partials, the pair-list path's buffers) is carved from one fixed region of
 * SSCONV_NOALLOC_SCRATCH_BYTES per device, built into the library and held by
 * every device the library runs on until the process ends.  Scratch use per
 * call: bf16 2*ksize^3*cin*cout bytes; fp32 nothing on the output-stationary
 * kernel (offset splits are reduced until their partials fit) and the
 * pair-list buffers only where they fit (otherwise the output-stationary
 * kernel runs: same sums, another order of the fp32 additions).
 * Errors: as ssconv_forward, plus SSCONV_E_INVALID when the call would need
 * more scratch than the region holds (bf16 with 2*ksize^3*cin*cout above it).
 * Every call on one device uses that device's one region: calls that overlap
 * in time on one device (another stream, another thread) race and give
 * undefined results; the region keeps the last call's contents, and nothing in
 * it needs to start at zero.  The device address is looked up on the first
 * call on each device (with that device current). */
#define SSCONV_NOALLOC_SCRATCH_BYTES (64u << 20)
int ssconv_forward_noalloc(const void* feats, ssconv_dtype dtype, int cin, ssconv_rulebook_t rb,
                           const void* W, int cout, void* out, hipStream_t stream);

/* ---- backward (adjoint of the forward and of the synthesis) ---------------
 * For L = <out, grad_out>:
 *   grad_feats[y] = sum_s sum_{(x,y) in R_s} kappa(s)^T grad_out[x]       (dtype)
 *   dW[s]        = sum_{(x,y) in R_s} grad_out[x] feats[y]^T             (fp32, in workspace)
 *   grad_coeffs[q] = sum_s <dW[s] block, basis_q[s]>                     (fp32)
 * grad_feats or grad_coeffs may be NULL to skip them (desc and basis may then
 * be NULL as well when grad_coeffs is NULL).  workspace: device scratch of at
 * least ssconv_backward_workspace_size bytes, 256-byte aligned; the result
 * is deterministic (no atomics in the reductions). */
size_t ssconv_backward_workspace_size(ssconv_rulebook_t rb, ssconv_dtype dtype, int cin, int cout);
int ssconv_backward(const void* feats, const void* grad_out, ssconv_dtype dtype, int cin, int cout,
                    ssconv_rulebook_t rb, const void* W, const ssconv_basis_desc* desc /*host*/,
                    const float* basis, void* grad_feats, float* grad_coeffs, void* workspace,
                    size_t ws_bytes, hipStream_t stream);

/* ---- gated nonlinearity (Sec. 3.3, Eq. 12) ---------------------------------
 * x: [n, C + G] where C = channels of `fields` and G = number of l > 0 fields
 * (the gate channels, appended after the fields in field order).
 * y: [n, C]: ReLU on l = 0 fields, sigmoid(gate) * f on l > 0 fields.
 * Backward: dx [n, C + G] from x and dy [n, C] (ReLU'(0) = 0). */
int ssconv_gate_forward(const ssconv_fields* fields /*host*/, const void* x, ssconv_dtype dtype,
                        int64_t n, void* y, hipStream_t stream);
int ssconv_gate_backward(const ssconv_fields* fields /*host*/, const void* x, const void* dy,
                         ssconv_dtype dtype, int64_t n, void* dx, hipStream_t stream);

/* ---- steerable normalisation (Sec. 3.3, Eq. 11) ------------------------------
 * x, y: [n, C] in `dtype`, C = channels of `fields` (1..1024).  Every field is
 * normalised on its own with population statistics over all n rows:
 *   l = 0:  y = (f - mean) / sqrt(var + eps)            (var: biased)
 *   l > 0:  y = f / sqrt(mean over rows of |f|^2 + eps)
 * No affine parameters.  Statistics are accumulated in fp64 in a fixed order
 * (deterministic); the elementwise step runs in fp32.  Backward: dx [n, C] =
 * the exact gradient of <y, dy> with respect to x (through the statistics).
 * y may alias x, and dx may alias x or dy, element for element.  n = 0 is a
 * no-op.  Temporary sums come from the library's device memory cache.
 * Errors: E_DTYPE, E_INVALID (fields, eps <= 0, null buffers), E_NOMEM, E_HIP. */
int ssconv_norm_forward(const ssconv_fields* fields /*host*/, const void* x, ssconv_dtype dtype, int64_t n,
                        double eps, void* y, hipStream_t stream);
int ssconv_norm_backward(const ssconv_fields* fields /*host*/, const void* x, const void* dy, ssconv_dtype dtype,
                         int64_t n, double eps, void* dx, hipStream_t stream);

/* ---- convolution followed by the steerable normalisation (Sec. 3.2.3, Alg. 1
 * feature update, then Sec. 3.3, Eq. 11) ----------------------------------------
 * y = ssconv_forward(feats, W) and z = the Norm of y over fields_out, as
 * ssconv_forward followed by ssconv_norm_forward(fields_out, y, eps, z) compute
 * them: y is the same (bit for bit), z agrees up to the order of the fp64
 * statistics sums.  The Norm's per-channel sums come out of the kernel that
 * writes y (per row tile of the output-stationary kernels, per row block of the
 * pair-list and offset-split reduces), so y is not read back before the
 * elementwise Norm step; the generic fallback kernel leaves none, and a
 * separate statistics pass then runs.  cout = channels of fields_out (1..1024);
 * feats [n_in, cin], W [ksize^3, cout, cin], y and z [n_out, cout], all in
 * `dtype`, 16-byte aligned.  z may alias y (y is then overwritten by z); y
 * stays the input of ssconv_norm_backward.  n_out = 0 is a no-op.  Temporary
 * sums come from the library's device memory cache.
 * Errors: as ssconv_forward and ssconv_norm_forward. */
int ssconv_forward_norm(const void* feats, ssconv_dtype dtype, int cin, ssconv_rulebook_t rb, const void* W,
                        const ssconv_fields* fields_out /*host*/, double eps, void* y, void* z,
                        hipStream_t stream);

/* ---- sparse average pooling (Sec. 3.1, footnote: downsampling is a stride-1
 * convolution followed by average pooling) -----------------------------------
 * rb must be built with ksize = 2, stride = 2, submanifold = 0: its offsets
 * are {-1, 0}^3 under 2x - y = s, so output x is active when an input lies in
 * the window 2x + {0,1}^3 (outputs = the distinct floor(y/2), lexicographic),
 * and nbr[s][x] lists the window's members.
 * Forward: out[x] = (sum of the window's active rows of feats) / 8, the dense
 * 2x2x2 average of the zero-filled grid at active outputs.  feats [n_in, C],
 * out [n_out, C].  Backward: grad_feats[y] = grad_out[x(y)] / 8 (every input
 * lies in exactly one window).  Sums in fp32, one rounding to bf16.
 * Errors: E_DTYPE, E_INVALID (not a pooling rule book, C < 1, null buffers),
 * E_HIP. */
int ssconv_pool_forward(const void* feats, ssconv_dtype dtype, int channels, ssconv_rulebook_t rb, void* out,
                        hipStream_t stream);
int ssconv_pool_backward(const void* grad_out, ssconv_dtype dtype, int channels, ssconv_rulebook_t rb,
                         void* grad_feats, hipStream_t stream);

/* ---- voxelisation (Sec. 4.1) -------------------------------------------------
 * A site is active when its grid cell encloses an input point; its feature is
 * the average of the features of the points its cell encloses (the paper's
 * points carry (R, G, B, 1); Feature-Steering merges re-voxelised sites the
 * same way).  The cell of point p is floor((p - origin) / voxel) per axis, the
 * subtraction and division in fp32 with round-to-nearest; points whose cell is
 * outside [0, grid) or whose coordinates are not finite are dropped.
 * points [n, 3] fp32; batch [n] int32 in [0, nbatch) or NULL (all 0);
 * feats [n, channels] fp32 (channels >= 0; NULL when 0); origin [3] and grid
 * [3] on the host; nbatch * grid volume < 2^32.
 * Outputs (caller buffers sized for n sites, the upper bound): coords_out
 * [n, 4] int32 (b, x, y, z), 16-byte aligned; feats_out [n, channels] fp32;
 * point_row [n] int32 = the site row of each point or -1 (may be NULL);
 * *n_sites (host) = the number of sites, rows [0, n_sites) are written in
 * lexicographic (b, x, y, z) order.  Averages add each cell's points in point
 * order in fp32 (deterministic).  Synchronises the stream once; temporaries
 * come from the device memory cache.  Errors: E_INVALID, E_BOUNDS (a batch
 * index outside [0, nbatch), or the key space exceeded), E_NOMEM, E_HIP; on
 * error the outputs are unspecified and *n_sites is 0. */
int ssconv_voxelize(const float* points, const int32_t* batch, const float* feats, int64_t n, int channels,
                    const float* origin /*host [3]*/, float voxel, const int32_t* grid /*host [3]*/, int nbatch,
                    int32_t* coords_out, float* feats_out, int32_t* point_row, int64_t* n_sites /*host*/,
                    hipStream_t stream);

/* ---- Wigner-D matrices (host; Sec. 3.1, Eq. 4-5) ----------------------------
 * D (host [(2l+1)^2], row-major) = D^l(rot) of the real harmonic basis used
 * throughout (Y^l(rot u) = D^l(rot) Y^l(u)), 0 <= l <= SSCONV_MAX_L; rot is a
 * host [9] row-major rotation.  A field of order l of a feature transforms as
 * f -> D^l(rot) f.  Errors: E_INVALID. */
int ssconv_wigner_d(int l, const double* rot /*host [9]*/, double* D /*host*/);

/* ---- Feature-Steering (Sec. 4.1) -------------------------------------------
 * Moves a sparse tensor (coords [n, 4], feats [n, C] fp32, C = channels of
 * `fields`) by the rigid motion p -> rot p + trans (rot: host [9] row-major
 * rotation, trans: host [3], world units): every field of order l is rotated
 * by its Wigner-D matrix D^l(rot) of the real harmonic basis (the block-diagonal
 * rho(rot) of Eq. 5, computed on the host by an exact quadrature), every site
 * is taken to the centre of its cell origin + (x + 1/2) voxel, moved, and the
 * moved points are re-voxelised exactly as ssconv_voxelize does (grid, nbatch,
 * dropping, lexicographic sites, averages of merged sites in a fixed order).
 * The centre and the moved point are computed in fp32 with every product and
 * sum rounded to nearest in the order ((r0 p0 + r1 p1) + r2 p2) + t.
 * Outputs as ssconv_voxelize: coords_out [n, 4], feats_out [n, C],
 * site_row [n] (new row of each input site or -1; may be NULL), *n_sites.
 * Errors: E_INVALID (fields, rot not orthonormal with det +1, non-finite
 * trans, null buffers), E_BOUNDS, E_NOMEM, E_HIP. */
int ssconv_steer(const int32_t* coords, const float* feats, int64_t n, const ssconv_fields* fields /*host*/,
                 const double* rot /*host [9]*/, const double* trans /*host [3]*/, const float* origin /*host [3]*/,
                 float voxel, const int32_t* grid /*host [3]*/, int nbatch, int32_t* coords_out, float* feats_out,
                 int32_t* site_row, int64_t* n_sites /*host*/, hipStream_t stream);

/* ---- Tensor-to-Point interpolation (Sec. 4.1) --------------------------------
 * rb: any rule book built on the sites (its input hash table and grid are
 * used); feats [n_in, channels] fp32 in its input rows.  points [m, 3] fp32,
 * batch [m] int32 or NULL (all 0), origin host [3], voxel > 0.
 * The features live at the cell centres origin + (x + 1/2) voxel and are zero
 * off the active sites; out [m, channels] = the trilinear interpolant of that
 * zero-filled grid at each point: u = (p - origin)/voxel - 1/2 in fp32,
 * x0 = floor(u), corner x0 + c weighted prod_a (c_a ? w_a : 1 - w_a) with
 * w = u - x0, corners inactive or outside the grid (or of another batch
 * entry) contributing nothing, corners added in the order 4cx + 2cy + cz.
 * Backward: grad_feats [n_in, channels] = the exact adjoint (every point
 * scatters weight * grad to its corners), summed per site in (point, corner)
 * order (deterministic, every row written).  Temporaries come from the device
 * memory cache.  Errors: E_INVALID (m >= 2^28, bad origin / voxel, null
 * buffers), E_NOMEM, E_HIP. */
int ssconv_interpolate(ssconv_rulebook_t rb, const float* feats, int channels, const float* points,
                       const int32_t* batch, int64_t m, const float* origin /*host [3]*/, float voxel, float* out,
                       hipStream_t stream);
int ssconv_interpolate_backward(ssconv_rulebook_t rb, const float* grad, int channels, const float* points,
                                const int32_t* batch, int64_t m, const float* origin /*host [3]*/, float voxel,
                                float* grad_feats, hipStream_t stream);

/* ---- test hooks --------------------------------------------------------
 * Forces failure paths from the host so they can be tested without faulting
 * a device: option 1 = hash capacity (slots) used by the next rule book builds
 * (0 restores automatic sizing); option 2 = make the N-th following device
 * allocation fail (0 disables); option 3 = kernel-selection override for
 * tuning sweeps and cross-checks (0 = automatic choice; 1, 2 = tile variants
 * of the generic gather-GEMM kernel; 3 = the generic kernel keeps 32-bit
 * neighbour indices in LDS; 5 = bf16 convolutions use the generic
 * gather-GEMM kernel instead of the bf16 pipeline kernel; 6 = the bf16 kernel
 * gradient uses per-offset splits instead of balanced work units; 7 = the
 * fp32 kernel gradient loads rows into registers instead of an LDS ring; 8 = the
 * generic gather-GEMM kernel splits every tile's offsets three ways (fp32
 * partials added in split order), which it otherwise does only when its tiles
 * leave compute units idle; 9 = fp32 convolutions take the pair-list path
 * (one GEMM per offset over R_s, then a per-row sum in offset order) wherever
 * it applies; 10 = never take it, which a cost model otherwise decides;
 * 11 = run the coefficient gradient of ssconv_backward on the caller's
 * stream instead of forking it onto the library's second stream (all of it
 * next to a pair-list feature gradient, its reduction and synthesis adjoint
 * next to the fp32 gather kernel); 12 = the bf16 kernel gradient stages its
 * operands as 16-byte granule columns instead of 64-byte quads (the same
 * results, bit for bit); results
 * agree within the dtype's tolerance for every value); option 4 = kernel
 * timing: a nonzero value switches it on and clears this thread's log, 0
 * switches it off; while on, every gather-GEMM kernel launch (the one of
 * ssconv_forward and the input-feature gradient one of ssconv_backward) is
 * bracketed by a pair of HIP events on its stream, up to 4096 launches per
 * thread, and nothing else of the call is timed.  Returns E_INVALID for
 * unknown options. */
int ssconv_debug_set(int option, int64_t value);

/* Kernel timing read-out: *count (host) = gather-GEMM launches timed on this
 * thread since option 4 was last switched on, *total_ms (host) = the sum of
 * their durations in milliseconds.  Waits for the last timed kernel.
 * E_INVALID if nothing was timed, E_HIP if the events fail. */
int ssconv_debug_kernel_ms(int64_t* count, float* total_ms);

#ifdef __cplusplus
}
#endif

#endif /* SSCONV_H */
