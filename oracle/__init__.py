"""CPU oracle for Sparse Steerable Convolution (SS-Conv, arXiv 2111.07383).

TEST INFRASTRUCTURE ONLY.  This package is a plain, slow, fp64 numpy statement
of what the SS-Conv hot path computes.  Only the test suite, the smoke check
and the benchmark's CPU-baseline leg may import it; the GPU library never
calls it and shares no code with it.

Modules
    sh        real spherical harmonics, Wigner-D matrices, the cube rotation group
    basis     steerable basis kernels on the s^3 grid (Sec. 3.2.1, Eq. 7-9)
    rulebook  output site sets and rule books (Sec. 3.2.2, Eq. 10; Sec. 3.2.3, Alg. 1)
    conv      kernel synthesis, sparse convolution forward/backward, dense
              reference convolution, gated nonlinearity (Alg. 1; Sec. 3.3, Eq. 12)
    norm_pool steerable normalisation (Sec. 3.3, Eq. 11) and 2x2x2 / stride-2
              sparse average pooling (footnote of Sec. 3.1), forward and backward
    voxel     point-cloud voxelisation with per-cell feature averaging (Sec. 4.1)
    steer     Feature-Steering: Wigner-D rotation of the fields, rigid motion of the
              site centres, re-voxelisation with averaging of merged sites (Sec. 4.1)
    interp    Tensor-to-Point: trilinear interpolation of the zero-filled site grid at
              points, and its adjoint (Sec. 4.1)

Readings of the paper that it takes (all pinned by invariants in tests/):
    real SH without Condon-Shortley phase, components ordered m = -l..l;
    Wigner-D defined by Y(R u) = D(R) Y(u);
    basis elements normalised to unit Frobenius norm over (offset, row, col)
    with the first significant entry positive;
    stride-2 pairing 2x - y = s (a zero-padded strided convolution);
    generated output sets in lexicographic (b, x, y, z) order;
    gate = extra scalar output channel of the same convolution;
    Norm: eps = 1e-5, population statistics over every active site, no affine;
    pooling divides window sums by 8 (zero-filled dense semantics);
    voxel cells floor((p - origin) / voxel) taken in fp32, points outside the
    grid dropped, sites lexicographic.

Parity status: every function here is pinned by at least one invariant test
(brute force, dense convolution, exact equivariance, adjointness, closed
forms); the paper prints no worked numerical example.
"""
