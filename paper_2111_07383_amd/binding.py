"""Thin PyTorch binding of the C ABI: device memory and streams come from torch,
every step of the computation runs in the HIP library.

Names follow the C entry points (``ssconv_build_rulebook`` -> ``build_rulebook``
etc.).  Tensors must live on the current HIP device; bf16 tensors map to
SSCONV_BF16 and fp32 tensors to SSCONV_F32.
"""
import ctypes
from ctypes import byref, c_float, c_int, c_int64, c_void_p
from typing import Optional, Sequence, Tuple

import numpy as np
import torch

from ._abi import BF16, F32, BasisDesc, Fields, check, lib

FieldList = Sequence[Tuple[int, int]]


def _stream(stream=None) -> c_void_p:
    s = torch.cuda.current_stream() if stream is None else stream
    return c_void_p(s.cuda_stream)


def _ptr(t: Optional[torch.Tensor]) -> c_void_p:
    return c_void_p(0 if t is None else t.data_ptr())


def _dtype(t: torch.Tensor) -> int:
    if t.dtype == torch.float32:
        return F32
    if t.dtype == torch.bfloat16:
        return BF16
    raise TypeError(f"unsupported dtype {t.dtype}")


def _need(t: torch.Tensor, name: str, dtype=None, shape=None):
    if not t.is_cuda:
        raise ValueError(f"{name} must be a device tensor")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    if dtype is not None and t.dtype != dtype:
        raise TypeError(f"{name} must be {dtype}, got {t.dtype}")
    if shape is not None and tuple(t.shape) != tuple(shape):
        raise ValueError(f"{name} must have shape {tuple(shape)}, got {tuple(t.shape)}")


def make_fields(fields: FieldList) -> Fields:
    f = Fields()
    f.n = len(fields)
    for e, (l, m) in enumerate(fields):
        f.l[e] = int(l)
        f.mult[e] = int(m)
    return f


def n_channels(fields: FieldList) -> int:
    return sum(m * (2 * l + 1) for l, m in fields)


def basis_desc(fields_in: FieldList, fields_out: FieldList, ksize: int, shells: Sequence[float],
               eps: float = 0.6, jmax: Optional[int] = None) -> BasisDesc:
    d = BasisDesc()
    d.in_ = make_fields(fields_in)
    d.out = make_fields(fields_out)
    d.ksize = int(ksize)
    d.n_shells = len(shells)
    for i, m in enumerate(shells):
        d.shells[i] = float(m)
    d.eps = float(eps)
    d.jmax = -1 if jmax is None else int(jmax)
    return d


def layer_desc(layer) -> BasisDesc:
    """Descriptor of a layer spec with fields_in/out, ksize, shells, eps, jmax attributes."""
    return basis_desc(layer.fields_in, layer.fields_out, layer.ksize, layer.shells, layer.eps, layer.jmax)


def basis_info(desc: BasisDesc) -> Tuple[int, int]:
    floats, ncoef = c_int64(), c_int64()
    check(lib().ssconv_basis_info(byref(desc), byref(floats), byref(ncoef)), "ssconv_basis_info")
    return floats.value, ncoef.value


def basis_build(desc: BasisDesc) -> np.ndarray:
    """Host-built basis (fp32 numpy, layout of ssconv_basis_build)."""
    n, _ = basis_info(desc)
    out = np.zeros(max(n, 1), np.float32)
    check(lib().ssconv_basis_build(byref(desc), out.ctypes.data_as(c_void_p)), "ssconv_basis_build")
    return out[:n]


class Rulebook:
    """Owner of an ssconv_rulebook_t (hash tables, neighbour map, pair lists).

    ``asynchronous``: ssconv_build_rulebook_async -- a submanifold build returns before its pair
    counts reach the host; ``pair_counts`` / ``n_pairs`` (and ``wait()``) settle it, and so does
    every library call that needs them."""

    def __init__(self, coords: torch.Tensor, grid, ksize: int, stride: int = 1, submanifold: bool = True,
                 stream=None, asynchronous: bool = False):
        _need(coords, "coords", torch.int32)
        if coords.dim() != 2 or coords.shape[1] != 4:
            raise ValueError("coords must be [n, 4] (b, x, y, z)")
        g = (c_int * 3)(*([int(grid)] * 3 if np.isscalar(grid) else [int(v) for v in grid]))
        h = c_void_p()
        self._h = None
        self.device = coords.device
        build = lib().ssconv_build_rulebook_async if asynchronous else lib().ssconv_build_rulebook
        check(build(_ptr(coords), coords.shape[0], g, int(ksize), int(stride), int(bool(submanifold)),
                    _stream(stream), byref(h)), "ssconv_build_rulebook")
        self._h = h
        self.ksize, self.K, self.stride, self.submanifold = ksize, ksize ** 3, stride, bool(submanifold)
        self._counts = None
        self.n_in = int(coords.shape[0])
        if self.submanifold:
            self.n_out = self.n_in
        else:
            self._settle()
        if not asynchronous:
            self._settle()

    def _settle(self):
        if self._counts is None:
            n_in, n_out = c_int64(), c_int64()
            counts = (c_int64 * self.K)()
            check(lib().ssconv_rulebook_info(self.handle, byref(n_in), byref(n_out), counts), "ssconv_rulebook_info")
            self.n_in, self.n_out = n_in.value, n_out.value
            self._counts = np.array(counts[:], np.int64)
        return self._counts

    def wait(self):
        """Settles an asynchronous build (raises its error, if any)."""
        check(lib().ssconv_rulebook_wait(self.handle), "ssconv_rulebook_wait")

    @property
    def pair_counts(self) -> np.ndarray:
        return self._settle()

    @property
    def n_pairs(self) -> int:
        return int(self._settle().sum())

    @property
    def handle(self) -> c_void_p:
        if self._h is None:
            raise RuntimeError("rule book has been destroyed")
        return self._h

    def out_coords(self, stream=None) -> torch.Tensor:
        t = torch.empty((self.n_out, 4), dtype=torch.int32, device=self.device)
        check(lib().ssconv_rulebook_out_coords(self.handle, _ptr(t), _stream(stream)), "ssconv_rulebook_out_coords")
        return t

    def pairs(self, stream=None) -> torch.Tensor:
        t = torch.empty((self.n_pairs, 2), dtype=torch.int32, device=self.device)
        check(lib().ssconv_rulebook_pairs(self.handle, _ptr(t), _stream(stream)), "ssconv_rulebook_pairs")
        return t

    def neighbours(self, stream=None) -> torch.Tensor:
        t = torch.empty((self.K, self.n_out), dtype=torch.int32, device=self.device)
        check(lib().ssconv_rulebook_neighbours(self.handle, _ptr(t), _stream(stream)), "ssconv_rulebook_neighbours")
        return t

    def hash_slots(self, which: int = 0, stream=None) -> torch.Tensor:
        cap = c_int64()
        check(lib().ssconv_rulebook_hash(self.handle, which, None, byref(cap), _stream(stream)), "ssconv_rulebook_hash")
        t = torch.empty((cap.value,), dtype=torch.int64, device=self.device)
        check(lib().ssconv_rulebook_hash(self.handle, which, _ptr(t), byref(cap), _stream(stream)),
              "ssconv_rulebook_hash")
        return t

    def close(self):
        if self._h is not None:
            lib().ssconv_rulebook_destroy(self._h)
            self._h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


def build_rulebook(coords, grid, ksize, stride=1, submanifold=True, stream=None) -> Rulebook:
    return Rulebook(coords, grid, ksize, stride, submanifold, stream)


def synth_kernel(desc: BasisDesc, basis: torch.Tensor, coeffs: torch.Tensor, dtype=torch.float32,
                 out: Optional[torch.Tensor] = None, stream=None) -> torch.Tensor:
    _need(basis, "basis", torch.float32)
    _need(coeffs, "coeffs", torch.float32)
    n_floats, n_coeff = basis_info(desc)
    if basis.numel() < n_floats or coeffs.numel() != n_coeff:
        raise ValueError(f"basis needs {n_floats} floats and coeffs {n_coeff} values")
    K = desc.ksize ** 3
    cin = sum(desc.in_.mult[e] * (2 * desc.in_.l[e] + 1) for e in range(desc.in_.n))
    cout = sum(desc.out.mult[e] * (2 * desc.out.l[e] + 1) for e in range(desc.out.n))
    if out is None:
        out = torch.empty((K, cout, cin), dtype=dtype, device=basis.device)
    _need(out, "W", dtype, (K, cout, cin))
    check(lib().ssconv_synth_kernel(byref(desc), _ptr(basis), _ptr(coeffs), _dtype(out), _ptr(out), _stream(stream)),
          "ssconv_synth_kernel")
    return out


def forward(feats: torch.Tensor, rb: Rulebook, W: torch.Tensor, out: Optional[torch.Tensor] = None,
            stream=None) -> torch.Tensor:
    _need(feats, "feats")
    _need(W, "W", feats.dtype)
    K, cout, cin = W.shape
    if feats.shape != (rb.n_in, cin):
        raise ValueError(f"feats must be [{rb.n_in}, {cin}]")
    if out is None:
        out = torch.empty((rb.n_out, cout), dtype=feats.dtype, device=feats.device)
    _need(out, "out", feats.dtype, (rb.n_out, cout))
    check(lib().ssconv_forward(_ptr(feats), _dtype(feats), cin, rb.handle, _ptr(W), cout, _ptr(out), _stream(stream)),
          "ssconv_forward")
    return out


def forward_noalloc(feats: torch.Tensor, rb: Rulebook, W: torch.Tensor, out: torch.Tensor, stream=None) -> torch.Tensor:
    """ssconv_forward_noalloc: forward into a caller-given out with no device allocation (scratch
    from the library's fixed per-device region)."""
    _need(feats, "feats")
    _need(W, "W", feats.dtype)
    K, cout, cin = W.shape
    if feats.shape != (rb.n_in, cin):
        raise ValueError(f"feats must be [{rb.n_in}, {cin}]")
    _need(out, "out", feats.dtype, (rb.n_out, cout))
    check(lib().ssconv_forward_noalloc(_ptr(feats), _dtype(feats), cin, rb.handle, _ptr(W), cout, _ptr(out),
                                       _stream(stream)), "ssconv_forward_noalloc")
    return out


NOALLOC_SCRATCH_BYTES = 64 << 20


def backward_workspace_size(rb: Rulebook, dtype: torch.dtype, cin: int, cout: int) -> int:
    return lib().ssconv_backward_workspace_size(rb.handle, BF16 if dtype == torch.bfloat16 else F32, cin, cout)


def backward(feats: torch.Tensor, grad_out: torch.Tensor, rb: Rulebook, W: torch.Tensor,
             desc: Optional[BasisDesc] = None, basis: Optional[torch.Tensor] = None,
             need_feats: bool = True, need_coeffs: bool = True, n_coeff: Optional[int] = None,
             workspace: Optional[torch.Tensor] = None, stream=None):
    """(grad_feats or None, grad_coeffs or None) for L = <forward(feats), grad_out>."""
    _need(feats, "feats")
    _need(grad_out, "grad_out", feats.dtype)
    _need(W, "W", feats.dtype)
    K, cout, cin = W.shape
    gf = torch.empty_like(feats) if need_feats else None
    gc = None
    if need_coeffs:
        if desc is None or basis is None:
            raise ValueError("desc and basis are required for the coefficient gradient")
        if n_coeff is None:
            n_coeff = basis_info(desc)[1]
        gc = torch.empty((n_coeff,), dtype=torch.float32, device=feats.device)
    ws_bytes = backward_workspace_size(rb, feats.dtype, cin, cout)
    if workspace is None or workspace.numel() < ws_bytes:
        workspace = torch.empty((max(ws_bytes, 256),), dtype=torch.uint8, device=feats.device)
    check(lib().ssconv_backward(_ptr(feats), _ptr(grad_out), _dtype(feats), cin, cout, rb.handle, _ptr(W),
                                byref(desc) if desc is not None else None, _ptr(basis), _ptr(gf), _ptr(gc),
                                _ptr(workspace), workspace.numel(), _stream(stream)),
          "ssconv_backward")
    return gf, gc


def gate_forward(fields: FieldList, x: torch.Tensor, out: Optional[torch.Tensor] = None, stream=None) -> torch.Tensor:
    _need(x, "x")
    f = make_fields(fields)
    C = n_channels(fields)
    if out is None:
        out = torch.empty((x.shape[0], C), dtype=x.dtype, device=x.device)
    check(lib().ssconv_gate_forward(byref(f), _ptr(x), _dtype(x), x.shape[0], _ptr(out), _stream(stream)),
          "ssconv_gate_forward")
    return out


def gate_backward(fields: FieldList, x: torch.Tensor, dy: torch.Tensor, stream=None) -> torch.Tensor:
    _need(x, "x")
    _need(dy, "dy", x.dtype)
    f = make_fields(fields)
    dx = torch.empty_like(x)
    check(lib().ssconv_gate_backward(byref(f), _ptr(x), _ptr(dy), _dtype(x), x.shape[0], _ptr(dx), _stream(stream)),
          "ssconv_gate_backward")
    return dx


NORM_EPS = 1e-5


def norm_forward(fields: FieldList, x: torch.Tensor, eps: float = NORM_EPS, out: Optional[torch.Tensor] = None,
                 stream=None) -> torch.Tensor:
    """Steerable normalisation (Eq. 11) of x [n, C] with statistics over all rows."""
    _need(x, "x")
    f = make_fields(fields)
    if x.dim() != 2 or x.shape[1] != n_channels(fields):
        raise ValueError(f"x must be [n, {n_channels(fields)}]")
    if out is None:
        out = torch.empty_like(x)
    _need(out, "out", x.dtype, tuple(x.shape))
    check(lib().ssconv_norm_forward(byref(f), _ptr(x), _dtype(x), x.shape[0], float(eps), _ptr(out),
                                    _stream(stream)), "ssconv_norm_forward")
    return out


def forward_norm(feats: torch.Tensor, rb: Rulebook, W: torch.Tensor, fields_out: FieldList, eps: float = NORM_EPS,
                 y: Optional[torch.Tensor] = None, z: Optional[torch.Tensor] = None, stream=None):
    """ssconv_forward_norm: (y, z) = (forward(feats), norm_forward(fields_out, y)), the Norm's
    statistics taken by the kernel that writes y.  z may be y (then y is overwritten)."""
    _need(feats, "feats")
    _need(W, "W", feats.dtype)
    K, cout, cin = W.shape
    if feats.shape != (rb.n_in, cin):
        raise ValueError(f"feats must be [{rb.n_in}, {cin}]")
    if cout != n_channels(fields_out):
        raise ValueError(f"W has {cout} output channels; fields_out has {n_channels(fields_out)}")
    if y is None:
        y = torch.empty((rb.n_out, cout), dtype=feats.dtype, device=feats.device)
    if z is None:
        z = torch.empty_like(y)
    _need(y, "y", feats.dtype, (rb.n_out, cout))
    _need(z, "z", feats.dtype, (rb.n_out, cout))
    f = make_fields(fields_out)
    check(lib().ssconv_forward_norm(_ptr(feats), _dtype(feats), cin, rb.handle, _ptr(W), byref(f), float(eps), _ptr(y),
                                    _ptr(z), _stream(stream)), "ssconv_forward_norm")
    return y, z


def norm_backward(fields: FieldList, x: torch.Tensor, dy: torch.Tensor, eps: float = NORM_EPS,
                  stream=None) -> torch.Tensor:
    _need(x, "x")
    _need(dy, "dy", x.dtype, tuple(x.shape))
    if x.dim() != 2 or x.shape[1] != n_channels(fields):
        raise ValueError(f"x must be [n, {n_channels(fields)}]")
    f = make_fields(fields)
    dx = torch.empty_like(x)
    check(lib().ssconv_norm_backward(byref(f), _ptr(x), _ptr(dy), _dtype(x), x.shape[0], float(eps), _ptr(dx),
                                     _stream(stream)), "ssconv_norm_backward")
    return dx


def pool_forward(feats: torch.Tensor, rb: Rulebook, out: Optional[torch.Tensor] = None, stream=None) -> torch.Tensor:
    """2x2x2 average pooling over a rule book built with ksize 2, stride 2."""
    _need(feats, "feats")
    if feats.dim() != 2 or feats.shape[0] != rb.n_in:
        raise ValueError(f"feats must be [{rb.n_in}, C]")
    C = feats.shape[1]
    if out is None:
        out = torch.empty((rb.n_out, C), dtype=feats.dtype, device=feats.device)
    _need(out, "out", feats.dtype, (rb.n_out, C))
    check(lib().ssconv_pool_forward(_ptr(feats), _dtype(feats), C, rb.handle, _ptr(out), _stream(stream)),
          "ssconv_pool_forward")
    return out


def pool_backward(grad_out: torch.Tensor, rb: Rulebook, stream=None) -> torch.Tensor:
    _need(grad_out, "grad_out")
    if grad_out.dim() != 2 or grad_out.shape[0] != rb.n_out:
        raise ValueError(f"grad_out must be [{rb.n_out}, C]")
    C = grad_out.shape[1]
    gf = torch.empty((rb.n_in, C), dtype=grad_out.dtype, device=grad_out.device)
    check(lib().ssconv_pool_backward(_ptr(grad_out), _dtype(grad_out), C, rb.handle, _ptr(gf), _stream(stream)),
          "ssconv_pool_backward")
    return gf


def voxelize(points: torch.Tensor, feats: Optional[torch.Tensor] = None, batch: Optional[torch.Tensor] = None,
             nbatch: int = 1, origin=(0.0, 0.0, 0.0), voxel: float = 1.0, grid=64, stream=None):
    """Voxelisation with per-cell feature averaging (Sec. 4.1).  Returns (coords [m, 4] int32,
    averaged feats [m, C] fp32 or None, point_row [n] int32); with a batch tensor, nbatch
    must cover its indices."""
    _need(points, "points", torch.float32)
    if points.dim() != 2 or points.shape[1] != 3:
        raise ValueError("points must be [n, 3]")
    n = points.shape[0]
    C = 0
    if feats is not None:
        _need(feats, "feats", torch.float32)
        if feats.dim() != 2 or feats.shape[0] != n:
            raise ValueError(f"feats must be [{n}, C]")
        C = feats.shape[1]
    if batch is not None:
        _need(batch, "batch", torch.int32, (n,))
    g = (c_int * 3)(*([int(grid)] * 3 if np.isscalar(grid) else [int(v) for v in grid]))
    o = (c_float * 3)(*[float(v) for v in origin])
    coords = torch.empty((n, 4), dtype=torch.int32, device=points.device)
    fo = torch.empty((n, C), dtype=torch.float32, device=points.device) if C else None
    rows = torch.empty((n,), dtype=torch.int32, device=points.device)
    m = c_int64()
    check(lib().ssconv_voxelize(_ptr(points), _ptr(batch), _ptr(feats), n, C, o, float(voxel), g, int(nbatch),
                                _ptr(coords), _ptr(fo), _ptr(rows), byref(m), _stream(stream)), "ssconv_voxelize")
    k = m.value
    return coords[:k], (fo[:k] if fo is not None else None), rows


def wigner_d(l: int, rot) -> np.ndarray:
    """D^l(rot) of the real harmonic basis (host computation)."""
    d = 2 * int(l) + 1
    r = (ctypes.c_double * 9)(*[float(v) for v in np.asarray(rot, np.float64).reshape(9)])
    out = (ctypes.c_double * (d * d))()
    check(lib().ssconv_wigner_d(int(l), r, out), "ssconv_wigner_d")
    return np.array(out[:], np.float64).reshape(d, d)


def steer(coords: torch.Tensor, feats: torch.Tensor, fields: FieldList, rot, trans, nbatch: int = 1,
          origin=(0.0, 0.0, 0.0), voxel: float = 1.0, grid=64, stream=None):
    """Feature-Steering (Sec. 4.1) by p -> rot p + trans.  Returns (coords' [m, 4] int32,
    feats' [m, C] fp32, site_row [n] int32)."""
    _need(coords, "coords", torch.int32)
    _need(feats, "feats", torch.float32)
    n = coords.shape[0]
    C = n_channels(fields)
    if coords.dim() != 2 or coords.shape[1] != 4 or tuple(feats.shape) != (n, C):
        raise ValueError(f"coords must be [n, 4] and feats [n, {C}]")
    f = make_fields(fields)
    r = (ctypes.c_double * 9)(*[float(v) for v in np.asarray(rot, np.float64).reshape(9)])
    t = (ctypes.c_double * 3)(*[float(v) for v in np.asarray(trans, np.float64).reshape(3)])
    g = (c_int * 3)(*([int(grid)] * 3 if np.isscalar(grid) else [int(v) for v in grid]))
    o = (c_float * 3)(*[float(v) for v in origin])
    co = torch.empty((n, 4), dtype=torch.int32, device=coords.device)
    fo = torch.empty((n, C), dtype=torch.float32, device=coords.device)
    rows = torch.empty((n,), dtype=torch.int32, device=coords.device)
    m = c_int64()
    check(lib().ssconv_steer(_ptr(coords), _ptr(feats), n, byref(f), r, t, o, float(voxel), g, int(nbatch), _ptr(co),
                             _ptr(fo), _ptr(rows), byref(m), _stream(stream)), "ssconv_steer")
    k = m.value
    return co[:k], fo[:k], rows


def _interp_args(rb, points, batch, C):
    _need(points, "points", torch.float32)
    if points.dim() != 2 or points.shape[1] != 3:
        raise ValueError("points must be [m, 3]")
    if batch is not None:
        _need(batch, "batch", torch.int32, (points.shape[0],))
    if C < 1:
        raise ValueError("channels must be positive")


def interpolate(rb: Rulebook, feats: torch.Tensor, points: torch.Tensor, batch: Optional[torch.Tensor] = None,
                origin=(0.0, 0.0, 0.0), voxel: float = 1.0, stream=None) -> torch.Tensor:
    """Tensor-to-Point (Sec. 4.1): trilinear interpolation of the sites' features at points."""
    _need(feats, "feats", torch.float32)
    if feats.dim() != 2 or feats.shape[0] != rb.n_in:
        raise ValueError(f"feats must be [{rb.n_in}, C]")
    C = feats.shape[1]
    _interp_args(rb, points, batch, C)
    out = torch.empty((points.shape[0], C), dtype=torch.float32, device=points.device)
    o = (c_float * 3)(*[float(v) for v in origin])
    check(lib().ssconv_interpolate(rb.handle, _ptr(feats), C, _ptr(points), _ptr(batch), points.shape[0], o,
                                   float(voxel), _ptr(out), _stream(stream)), "ssconv_interpolate")
    return out


def interpolate_backward(rb: Rulebook, grad: torch.Tensor, points: torch.Tensor, batch: Optional[torch.Tensor] = None,
                         origin=(0.0, 0.0, 0.0), voxel: float = 1.0, stream=None) -> torch.Tensor:
    _need(grad, "grad", torch.float32)
    if grad.dim() != 2 or grad.shape[0] != points.shape[0]:
        raise ValueError("grad must be [m, C]")
    C = grad.shape[1]
    _interp_args(rb, points, batch, C)
    gf = torch.empty((rb.n_in, C), dtype=torch.float32, device=points.device)
    o = (c_float * 3)(*[float(v) for v in origin])
    check(lib().ssconv_interpolate_backward(rb.handle, _ptr(grad), C, _ptr(points), _ptr(batch), points.shape[0], o,
                                            float(voxel), _ptr(gf), _stream(stream)), "ssconv_interpolate_backward")
    return gf


def debug_set(option: int, value: int) -> None:
    check(lib().ssconv_debug_set(int(option), int(value)), "ssconv_debug_set")


def empty_cache() -> None:
    """Waits for and releases the library's cached free device blocks."""
    check(lib().ssconv_empty_cache(), "ssconv_empty_cache")


def cached_bytes() -> int:
    """Bytes held in the library's cached free device blocks."""
    return int(lib().ssconv_cached_bytes())


def debug_kernel_ms() -> Tuple[int, float]:
    """(launches, total ms) of the gather-GEMM kernels timed on this thread since
    debug_set(4, 1); waits for the last of them."""
    n, ms = c_int64(), c_float()
    check(lib().ssconv_debug_kernel_ms(byref(n), byref(ms)), "ssconv_debug_kernel_ms")
    return int(n.value), float(ms.value)
