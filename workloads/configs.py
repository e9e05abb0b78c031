"""The synthetic SS-Conv workloads (layer shapes, basis parameters, dtypes).

Field lists are ``((l, multiplicity), ...)`` in channel order: all fields of an
entry are consecutive and each field's ``2l+1`` components are contiguous.
Gated layers append one extra scalar (l = 0) output field per l > 0 field, after
the regular fields (the gate channels of the gated nonlinearity, Sec. 3.3,
Eq. 12).

Radial shells follow the paper's Plain12 setting ({m} = {0, 1}, epsilon = 0.6
for 3x3x3 kernels, Sec. 5.1) generalised to m in {0 .. (s-1)/2} for an s^3
kernel; the 16^3 workload uses shells at r in {0, 1, sqrt2, sqrt3}.
"""
from dataclasses import dataclass, field
from math import sqrt
from typing import Optional, Tuple

Fields = Tuple[Tuple[int, int], ...]


def n_channels(fields: Fields) -> int:
    return sum(m * (2 * l + 1) for l, m in fields)


def gate_fields(fields: Fields) -> Fields:
    """Regular fields plus one l = 0 gate channel per l > 0 field."""
    n_gates = sum(m for l, m in fields if l > 0)
    return tuple(fields) + (((0, n_gates),) if n_gates else ())


@dataclass(frozen=True)
class LayerSpec:
    ksize: int
    stride: int
    submanifold: bool
    fields_in: Fields
    fields_out: Fields          # as produced by the convolution (gates included)
    shells: Tuple[float, ...]
    eps: float = 0.6
    jmax: Optional[int] = None  # None: J runs over the full |k-l| .. k+l
    gated: bool = False         # gated nonlinearity applied to this layer's output

    @property
    def cin(self) -> int:
        return n_channels(self.fields_in)

    @property
    def cout(self) -> int:
        return n_channels(self.fields_out)

    @property
    def n_offsets(self) -> int:
        return self.ksize ** 3


@dataclass(frozen=True)
class WorkloadSpec:
    index: int
    name: str
    grid: int
    batch: int
    dtype: str                  # "f32" or "bf16"
    layers: Tuple[LayerSpec, ...]
    geometry: str
    params: dict = field(default_factory=dict, compare=False, hash=False)

    @property
    def seed(self) -> int:
        return 20211107 + self.index


L0 = lambda m: ((0, m),)  # noqa: E731
F_104 = ((0, 16), (1, 16), (2, 8))
F_208 = ((0, 32), (1, 32), (2, 16))

CONFIGS = {
    1: WorkloadSpec(
        1, "sphere16_k3_sub_4to8", 16, 1, "f32",
        (LayerSpec(3, 1, True, L0(4), ((0, 2), (1, 2)),
                   shells=(0.0, 1.0, sqrt(2.0), sqrt(3.0)), jmax=1),),
        geometry="sphere", params=dict(radius=6.0, tau=0.0)),
    2: WorkloadSpec(
        2, "ellipsoids64_k5_sub_104", 64, 1, "f32",
        (LayerSpec(5, 1, True, F_104, F_104, shells=(0.0, 1.0, 2.0), jmax=2),),
        geometry="ellipsoids", params=dict(n=4, axes=(8.0, 24.0), centre=(24.0, 40.0), tau=0.75)),
    3: WorkloadSpec(
        3, "objects64_b32_k3_s2_60to120", 64, 32, "f32",
        (LayerSpec(3, 2, False, ((0, 16), (1, 8), (2, 4)), ((0, 32), (1, 16), (2, 8)),
                   shells=(0.0, 1.0)),),
        geometry="objects_sparse", params=dict(extent=(8.0, 24.0), n_points=1024)),
    4: WorkloadSpec(
        4, "scene128_k3_sub_208_bf16", 128, 1, "bf16",
        (LayerSpec(3, 1, True, F_208, F_208, shells=(0.0, 1.0)),),
        geometry="scene", params=dict(n=16, axes=(8.0, 32.0), centre=(32.0, 96.0), tau=0.6)),
    5: WorkloadSpec(
        5, "stack5_objects64_b16", 64, 16, "f32",
        (LayerSpec(5, 1, True, L0(8), gate_fields(F_104), shells=(0.0, 1.0, 2.0), gated=True),
         LayerSpec(5, 1, True, F_104, gate_fields(F_208), shells=(0.0, 1.0, 2.0), gated=True),
         LayerSpec(3, 2, False, F_208, gate_fields(F_208), shells=(0.0, 1.0), gated=True),
         LayerSpec(3, 1, True, F_208, gate_fields(F_208), shells=(0.0, 1.0), gated=True),
         LayerSpec(3, 2, False, F_208, F_208, shells=(0.0, 1.0))),
        geometry="objects_dense", params=dict(extent=(8.0, 24.0), scale=0.555, margin=2)),
    # The paper's downsampling block on the objects of workload 3 (Sec. 3.1 footnote, Sec. 3.3):
    # stride-1 submanifold SS-Conv -> Norm (Eq. 11, over every output field, gates included)
    # -> gated nonlinearity (Eq. 12) -> 2x2x2 average pooling, 64^3 -> 32^3.
    6: WorkloadSpec(
        6, "objects64_b32_block_k3_sub_norm_gate_pool_60to120", 64, 32, "f32",
        (LayerSpec(3, 1, True, ((0, 16), (1, 8), (2, 4)), gate_fields(((0, 32), (1, 16), (2, 8))),
                   shells=(0.0, 1.0), gated=True),),
        geometry="objects_sparse", params=dict(extent=(8.0, 24.0), n_points=1024, norm=True, pool=True)),
    # Input voxelisation (Sec. 4.1): raw point clouds of 32 objects (the object recipe of
    # workload 3 with 16 384 area-uniform points each) carrying (R, G, B, 1), voxelised into a
    # 64^3 grid per object with per-cell feature averaging.  No convolution layer.
    7: WorkloadSpec(
        7, "points64_b32_voxelise_rgb1", 64, 32, "f32", (),
        geometry="points", params=dict(extent=(8.0, 24.0), n_points=16384)),
    # Feature-Steering (Sec. 4.1) of a backbone feature map: the ellipsoid scene recipe of
    # workload 2 (its own seed) with 104 channels of orders 0, 1, 2, moved by a seeded random
    # rotation about the grid centre and a translation of up to 2 voxels, then re-voxelised.
    8: WorkloadSpec(
        8, "steer_ellipsoids64_104", 64, 1, "f32",
        (LayerSpec(5, 1, True, F_104, F_104, shells=(0.0, 1.0, 2.0), jmax=2),),
        geometry="ellipsoids", params=dict(n=4, axes=(8.0, 24.0), centre=(24.0, 40.0), tau=0.75)),
    # Tensor-to-Point (Sec. 4.1): the feature map of workload 8's recipe (its own seed) read at 4
    # query points per site, each its cell centre plus U(-1, 1) voxels per axis.
    9: WorkloadSpec(
        9, "interp_ellipsoids64_104_4pps", 64, 1, "f32",
        (LayerSpec(5, 1, True, F_104, F_104, shells=(0.0, 1.0, 2.0), jmax=2),),
        geometry="ellipsoids", params=dict(n=4, axes=(8.0, 24.0), centre=(24.0, 40.0), tau=0.75, per_site=4)),
}


def get_config(i: int) -> WorkloadSpec:
    return CONFIGS[int(i)]
