"""A stack of SS-Conv layers with the gated nonlinearity between them (Sec. 3.2-3.3), and the
paper's downsampling block (stride-1 SS-Conv, Norm, gate, average pooling).

Every step calls the C ABI through ``binding``; this module only sequences the
calls and keeps what the backward pass needs.  A layer object provides
``fields_in``, ``fields_out`` (gate channels included when ``gated``),
``ksize``, ``stride``, ``submanifold``, ``shells``, ``eps``, ``jmax``, ``gated``.
"""
from dataclasses import dataclass, field
from typing import List, Optional

import torch

from . import binding as B


@dataclass
class LayerState:
    layer: object
    desc: object
    basis: torch.Tensor          # fp32 device basis of ssconv_basis_build
    coeffs: torch.Tensor         # fp32 device coefficients
    n_coeff: int
    grid: int                    # input grid extent
    rb: Optional[B.Rulebook] = None
    W: Optional[torch.Tensor] = None
    x: Optional[torch.Tensor] = None   # layer input features
    y: Optional[torch.Tensor] = None   # convolution output (before the gate)


def regular_fields(layer):
    """Output fields without the appended gate channels."""
    return tuple(layer.fields_out[:-1]) if layer.gated else tuple(layer.fields_out)


@dataclass
class Stack:
    layers: List[LayerState] = field(default_factory=list)
    dtype: torch.dtype = torch.float32

    @staticmethod
    def create(layer_specs, coeffs_list, grid: int, device, dtype=torch.float32) -> "Stack":
        st = Stack(dtype=dtype)
        g = grid
        for spec, w in zip(layer_specs, coeffs_list):
            desc = B.layer_desc(spec)
            basis = torch.from_numpy(B.basis_build(desc)).to(device)
            n_coeff = B.basis_info(desc)[1]
            c = torch.as_tensor(w, dtype=torch.float32).to(device)
            if c.numel() != n_coeff:
                raise ValueError(f"layer expects {n_coeff} coefficients, got {c.numel()}")
            st.layers.append(LayerState(spec, desc, basis, c, n_coeff, g))
            g = -(-g // spec.stride)
        return st

    def forward(self, coords: torch.Tensor, feats: torch.Tensor, overlap: bool = True):
        """Returns (output coords, output features); rule books are rebuilt every call.

        Rule books and kernels depend on coordinates and coefficients only (a generated output set
        comes from the rule book itself), so with ``overlap`` they are prepared on a side stream
        one layer ahead: the rule-book build of layer n+1, whose host synchronisation waits on
        the side stream only, is queued while layer n's convolution runs on the caller's stream
        (measured on the five-layer stack: 5.85 -> 5.76 ms per step; a host thread running the
        builds further ahead was slower, 6.3 ms)."""
        main = torch.cuda.current_stream()
        side = self._side() if overlap else main
        side.wait_stream(main)          # the caller's coordinates, and last call's uses of the rule books
        for L in self.layers:
            if L.rb is not None:
                L.rb.close()
                L.rb = None
        with torch.cuda.stream(side):
            self._prepare(0, coords)
        h, c = feats, coords
        for i, L in enumerate(self.layers):
            s = L.layer
            main.wait_stream(side)
            if side is not main:
                L.W.record_stream(main)
            L.x = h
            L.y = B.forward(h, L.rb, L.W)
            h = B.gate_forward(regular_fields(s), L.y) if s.gated else L.y
            if not s.submanifold:
                with torch.cuda.stream(side):
                    c = L.rb.out_coords()
                if side is not main:
                    c.record_stream(main)
            if i + 1 < len(self.layers):
                with torch.cuda.stream(side):
                    self._prepare(i + 1, c)
        return c, h

    def _side(self) -> torch.cuda.Stream:
        if getattr(self, "_side_stream", None) is None:
            self._side_stream = torch.cuda.Stream()   # default priority
        return self._side_stream

    def _prepare(self, i: int, coords: torch.Tensor):
        """Kernel and rule book of layer i on the current stream (a generated output set's build
        synchronises it; a submanifold build is settled by the first call that needs its counts)."""
        L = self.layers[i]
        s = L.layer
        L.W = B.synth_kernel(L.desc, L.basis, L.coeffs, self.dtype)
        L.rb = B.Rulebook(coords, L.grid, s.ksize, s.stride, s.submanifold, asynchronous=True)

    def backward(self, grad: torch.Tensor, need_input_grad: bool = True):
        """Returns (grad of the stack input or None, [grad_coeffs per layer])."""
        g = grad
        gcs = [None] * len(self.layers)
        for idx in range(len(self.layers) - 1, -1, -1):
            L = self.layers[idx]
            s = L.layer
            if s.gated:
                g = B.gate_backward(regular_fields(s), L.y, g)
            gf, gc = B.backward(L.x, g, L.rb, L.W, L.desc, L.basis, need_feats=(idx > 0 or need_input_grad),
                                need_coeffs=True, n_coeff=L.n_coeff)
            gcs[idx] = gc
            g = gf
        return g, gcs

    def close(self):
        if getattr(self, "_side_stream", None) is not None:
            self._side_stream.wait_stream(torch.cuda.current_stream())
        for L in self.layers:
            if L.rb is not None:
                L.rb.close()
                L.rb = None


@dataclass
class DownBlock:
    """The paper's downsampling block: a stride-1 submanifold SS-Conv, steerable Norm (Eq. 11)
    over every output field (gate channels included), the gated nonlinearity (Eq. 12), then
    2x2x2 average pooling (the footnote of Sec. 3.1).  The convolution and its Norm are one call
    (``forward_norm``: the kernel that writes the convolution output also sums its statistics).
    Rule books are rebuilt every call."""
    state: LayerState
    dtype: torch.dtype = torch.float32
    norm_eps: float = B.NORM_EPS
    pool_rb: Optional[B.Rulebook] = None
    z: Optional[torch.Tensor] = None     # normalised convolution output (input of the gate)

    @staticmethod
    def create(layer_spec, coeffs, grid: int, device, dtype=torch.float32) -> "DownBlock":
        if layer_spec.stride != 1 or not layer_spec.submanifold:
            raise ValueError("the block's convolution is a stride-1 submanifold SS-Conv")
        st = Stack.create([layer_spec], [coeffs], grid, device, dtype)
        return DownBlock(st.layers[0], dtype)

    def forward(self, coords: torch.Tensor, feats: torch.Tensor, overlap: bool = True):
        """Returns (pooled coords, pooled features).  The pooling rule book depends on the
        coordinates only: with ``overlap`` it is built on a side stream after the convolution,
        Norm and gate are queued, so its host synchronisations overlap them."""
        L, s = self.state, self.state.layer
        main = torch.cuda.current_stream()
        side = self._side() if overlap else main
        side.wait_stream(main)
        for rb in (L.rb, self.pool_rb):
            if rb is not None:
                rb.close()
        L.W = B.synth_kernel(L.desc, L.basis, L.coeffs, self.dtype)
        L.rb = B.Rulebook(coords, L.grid, s.ksize, 1, True, asynchronous=True)
        L.x = feats
        L.y, self.z = B.forward_norm(feats, L.rb, L.W, s.fields_out, self.norm_eps)
        h = B.gate_forward(regular_fields(s), self.z) if s.gated else self.z
        with torch.cuda.stream(side):
            self.pool_rb = B.Rulebook(coords, L.grid, 2, 2, False)
            pc = self.pool_rb.out_coords()
        main.wait_stream(side)
        if side is not main:
            pc.record_stream(main)
        return pc, B.pool_forward(h, self.pool_rb)

    def _side(self) -> torch.cuda.Stream:
        if getattr(self, "_side_stream", None) is None:
            self._side_stream = torch.cuda.Stream()   # default priority
        return self._side_stream

    def backward(self, grad: torch.Tensor, need_input_grad: bool = True):
        """Returns (grad of the block input or None, grad_coeffs)."""
        L, s = self.state, self.state.layer
        g = B.pool_backward(grad, self.pool_rb)
        if s.gated:
            g = B.gate_backward(regular_fields(s), self.z, g)
        g = B.norm_backward(s.fields_out, L.y, g, self.norm_eps)
        return B.backward(L.x, g, L.rb, L.W, L.desc, L.basis, need_feats=need_input_grad, need_coeffs=True,
                          n_coeff=L.n_coeff)

    def close(self):
        if getattr(self, "_side_stream", None) is not None:
            self._side_stream.wait_stream(torch.cuda.current_stream())
        for rb in (self.state.rb, self.pool_rb):
            if rb is not None:
                rb.close()
        self.state.rb = self.pool_rb = None
