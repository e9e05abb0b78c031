"""ctypes declarations of the C ABI in include/ssconv.h (argument marshalling only).

The shared library is built in-tree by ``paper_2111_07383_amd.build`` as
``libssconv.so`` next to this file.  There is no fallback: if the library is
missing, loading raises.
"""
import ctypes
import os
from ctypes import POINTER, c_char_p, c_double, c_float, c_int, c_int64, c_size_t, c_void_p

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libssconv.so")

OK = 0
E_INVALID, E_BOUNDS, E_DUPLICATE, E_HASH_FULL, E_NOMEM, E_HIP, E_DTYPE = -1, -2, -3, -4, -5, -6, -7
ERROR_NAMES = {E_INVALID: "E_INVALID", E_BOUNDS: "E_BOUNDS", E_DUPLICATE: "E_DUPLICATE",
               E_HASH_FULL: "E_HASH_FULL", E_NOMEM: "E_NOMEM", E_HIP: "E_HIP", E_DTYPE: "E_DTYPE"}
F32, BF16 = 0, 1
MAX_ENTRIES, MAX_L, MAX_SHELLS = 8, 4, 8


class Fields(ctypes.Structure):
    _fields_ = [("n", c_int), ("l", c_int * MAX_ENTRIES), ("mult", c_int * MAX_ENTRIES)]


class BasisDesc(ctypes.Structure):
    _fields_ = [("in_", Fields), ("out", Fields), ("ksize", c_int), ("n_shells", c_int),
                ("shells", c_double * MAX_SHELLS), ("eps", c_double), ("jmax", c_int)]


# name -> (restype, argtypes)
SIGNATURES = {
    "ssconv_last_error": (c_char_p, []),
    "ssconv_version": (c_char_p, []),
    "ssconv_empty_cache": (c_int, []),
    "ssconv_cached_bytes": (c_int64, []),
    "ssconv_basis_info": (c_int, [POINTER(BasisDesc), POINTER(c_int64), POINTER(c_int64)]),
    "ssconv_basis_build": (c_int, [POINTER(BasisDesc), c_void_p]),
    "ssconv_build_rulebook": (c_int, [c_void_p, c_int64, POINTER(c_int), c_int, c_int, c_int, c_void_p,
                                      POINTER(c_void_p)]),
    "ssconv_build_rulebook_async": (c_int, [c_void_p, c_int64, POINTER(c_int), c_int, c_int, c_int, c_void_p,
                                            POINTER(c_void_p)]),
    "ssconv_rulebook_wait": (c_int, [c_void_p]),
    "ssconv_rulebook_info": (c_int, [c_void_p, POINTER(c_int64), POINTER(c_int64), POINTER(c_int64)]),
    "ssconv_rulebook_out_coords": (c_int, [c_void_p, c_void_p, c_void_p]),
    "ssconv_rulebook_pairs": (c_int, [c_void_p, c_void_p, c_void_p]),
    "ssconv_rulebook_neighbours": (c_int, [c_void_p, c_void_p, c_void_p]),
    "ssconv_rulebook_hash": (c_int, [c_void_p, c_int, c_void_p, POINTER(c_int64), c_void_p]),
    "ssconv_rulebook_destroy": (None, [c_void_p]),
    "ssconv_synth_kernel": (c_int, [POINTER(BasisDesc), c_void_p, c_void_p, c_int, c_void_p, c_void_p]),
    "ssconv_forward": (c_int, [c_void_p, c_int, c_int, c_void_p, c_void_p, c_int, c_void_p, c_void_p]),
    "ssconv_forward_noalloc": (c_int, [c_void_p, c_int, c_int, c_void_p, c_void_p, c_int, c_void_p, c_void_p]),
    "ssconv_backward_workspace_size": (c_size_t, [c_void_p, c_int, c_int, c_int]),
    "ssconv_backward": (c_int, [c_void_p, c_void_p, c_int, c_int, c_int, c_void_p, c_void_p, POINTER(BasisDesc),
                                c_void_p, c_void_p, c_void_p, c_void_p, c_size_t, c_void_p]),
    "ssconv_gate_forward": (c_int, [POINTER(Fields), c_void_p, c_int, c_int64, c_void_p, c_void_p]),
    "ssconv_gate_backward": (c_int, [POINTER(Fields), c_void_p, c_void_p, c_int, c_int64, c_void_p, c_void_p]),
    "ssconv_norm_forward": (c_int, [POINTER(Fields), c_void_p, c_int, c_int64, c_double, c_void_p, c_void_p]),
    "ssconv_forward_norm": (c_int, [c_void_p, c_int, c_int, c_void_p, c_void_p, POINTER(Fields), c_double, c_void_p,
                                    c_void_p, c_void_p]),
    "ssconv_norm_backward": (c_int, [POINTER(Fields), c_void_p, c_void_p, c_int, c_int64, c_double, c_void_p,
                                     c_void_p]),
    "ssconv_pool_forward": (c_int, [c_void_p, c_int, c_int, c_void_p, c_void_p, c_void_p]),
    "ssconv_pool_backward": (c_int, [c_void_p, c_int, c_int, c_void_p, c_void_p, c_void_p]),
    "ssconv_voxelize": (c_int, [c_void_p, c_void_p, c_void_p, c_int64, c_int, POINTER(c_float), c_float,
                                POINTER(c_int), c_int, c_void_p, c_void_p, c_void_p, POINTER(c_int64), c_void_p]),
    "ssconv_wigner_d": (c_int, [c_int, POINTER(c_double), POINTER(c_double)]),
    "ssconv_steer": (c_int, [c_void_p, c_void_p, c_int64, POINTER(Fields), POINTER(c_double), POINTER(c_double),
                             POINTER(c_float), c_float, POINTER(c_int), c_int, c_void_p, c_void_p, c_void_p,
                             POINTER(c_int64), c_void_p]),
    "ssconv_interpolate": (c_int, [c_void_p, c_void_p, c_int, c_void_p, c_void_p, c_int64, POINTER(c_float), c_float,
                                   c_void_p, c_void_p]),
    "ssconv_interpolate_backward": (c_int, [c_void_p, c_void_p, c_int, c_void_p, c_void_p, c_int64, POINTER(c_float),
                                            c_float, c_void_p, c_void_p]),
    "ssconv_debug_set": (c_int, [c_int, c_int64]),
    "ssconv_debug_kernel_ms": (c_int, [POINTER(c_int64), POINTER(c_float)]),
}


class SSConvError(RuntimeError):
    def __init__(self, code: int, where: str, msg: str):
        super().__init__(f"{where}: {ERROR_NAMES.get(code, code)}: {msg}")
        self.code = code


_lib = None


def lib():
    """The loaded library (raises if it has not been built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing: build it with `python -m paper_2111_07383_amd.build`")
        L = ctypes.CDLL(LIB_PATH)
        for name, (res, args) in SIGNATURES.items():
            fn = getattr(L, name)
            fn.restype = res
            fn.argtypes = args
        _lib = L
    return _lib


def check(rc: int, where: str) -> None:
    if rc != OK:
        raise SSConvError(rc, where, lib().ssconv_last_error().decode())
