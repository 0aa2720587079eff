"""ctypes binding of libsobek_hip.so (argument marshalling only).

Every computation runs in the library's generated HIP kernels; there is no
Python or CPU fallback.  Loading fails loudly when the library is missing.
"""

from __future__ import annotations

import ctypes
import os
import re

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libsobek_hip.so")

LAYOUTS = {"ir_mul": 0, "mul_ir": 1}
NORMS = {"none": 0, "fan_in": 1}
MODES = {"uvw": 0, "uvu": 1}
DTYPES = {"f32": 0, "bf16_gemm": 1}
PASSES = {"fwd": 0, "bwd": 1, "dbwd": 2}
STATUS = {0: "OK", -1: "INVALID", -2: "UNSUPPORTED", -3: "SHAPE", -4: "ALIGN", -5: "WORKSPACE",
          -6: "HIP", -7: "INTERNAL", -8: "COMPILE"}


class SobekError(RuntimeError):
    def __init__(self, code, message):
        super().__init__(f"sobek error {code} ({STATUS.get(code, '?')}): {message}")
        self.code = code
        self.message = message

    def __reduce__(self):  # picklable across the build's worker processes
        return (SobekError, (self.code, self.message))


class Irrep(ctypes.Structure):
    _fields_ = [("mul", ctypes.c_int32), ("l", ctypes.c_int32), ("parity", ctypes.c_int32)]


_P = ctypes.c_void_p
_I64 = ctypes.c_int64
_SZ = ctypes.c_size_t
_INT = ctypes.c_int
_lib = None

_SIGNATURES = {
    "sobek_last_error": (ctypes.c_char_p, []),
    "sobek_version": (_INT, []),
    "sobek_plan_create": (_INT, [ctypes.POINTER(Irrep), _INT, _INT, ctypes.POINTER(Irrep), _INT, _INT, _INT, _INT,
                                 _INT, _INT, ctypes.POINTER(_P)]),
    "sobek_jit_compile": (_INT, [ctypes.POINTER(Irrep), _INT, _INT, ctypes.POINTER(Irrep), _INT, _INT, _INT, _INT,
                                 _INT, _INT]),
    "sobek_plan_source": (_INT, [ctypes.POINTER(Irrep), _INT, _INT, ctypes.POINTER(Irrep), _INT, _INT, _INT, _INT,
                                 _INT, _INT, ctypes.c_char_p, _SZ, ctypes.POINTER(_SZ)]),
    "sobek_plan_destroy": (_INT, [_P]),
    "sobek_plan_info": (_INT, [_P] + [ctypes.POINTER(_I64)] * 5),
    "sobek_plan_paths": (_INT, [_P, ctypes.POINTER(ctypes.c_int32), ctypes.POINTER(ctypes.c_int32),
                                ctypes.POINTER(ctypes.c_int32), ctypes.POINTER(_I64)]),
    "sobek_plan_cg": (_INT, [_P, _INT, ctypes.POINTER(ctypes.c_double)]),
    "sobek_cg_table": (_INT, [_INT, _INT, _INT, ctypes.POINTER(ctypes.c_double)]),
    "sobek_sh_table": (_INT, [_INT, _INT, ctypes.POINTER(ctypes.c_int32), ctypes.POINTER(ctypes.c_double),
                              ctypes.POINTER(ctypes.c_int32), _INT]),
    "sobek_graph_prepare_size": (_INT, [_I64, _I64, ctypes.POINTER(_SZ)]),
    "sobek_graph_prepare": (_INT, [_P, _P, _I64, _I64, _P, _SZ, ctypes.POINTER(_P), _P]),
    "sobek_graph_destroy": (_INT, [_P]),
    "sobek_graph_info": (_INT, [_P, ctypes.POINTER(_I64), ctypes.POINTER(_I64)]),
    "sobek_workspace_size": (_INT, [_P, _P, _INT, _SZ, ctypes.POINTER(_SZ)]),
    "sobek_conv_fwd": (_INT, [_P, _P, _P, _P, _P, _P, _P, _P, _SZ, _P]),
    "sobek_conv_bwd": (_INT, [_P, _P, _P, _P, _P, _P, _P, _P, _P, _P, _P, _P, _SZ, _P]),
    "sobek_conv_dbwd": (_INT, [_P, _P, _P, _P, _P, _P, _P, _P, _P, _P, _P, _P, _P, _P, _P, _P, _P, _SZ, _P]),
    "sobek_state_size": (_INT, [_P, _P, ctypes.POINTER(_SZ)]),
    "sobek_conv_fwd_save": (_INT, [_P, _P, _P, _P, _P, _P, _P, _P, _P, _SZ, _P]),
    "sobek_conv_bwd_saved": (_INT, [_P, _P, _P, _P, _P, _P, _P, _P, _P, _P, _P, _P, _P, _P, _SZ, _P]),
    "sobek_conv_dbwd_saved": (_INT, [_P, _P, _P, _P, _P, _P, _P, _P, _P, _P, _P, _P, _P, _P, _P, _P, _P, _P, _SZ,
                                     _P]),
    "sobek_plan_set_policy": (_INT, [_P, _INT]),
    "sobek_kept_size": (_INT, [_P, _P, ctypes.c_uint64, ctypes.POINTER(_SZ)]),
    "sobek_retention_select": (_INT, [_P, _P, _SZ, ctypes.POINTER(ctypes.c_uint64), ctypes.POINTER(_SZ)]),
    "sobek_conv_fwd_keep": (_INT, [_P, _P, _P, _P, _P, _P, _P, ctypes.c_uint64, _P, _P, _SZ, _P]),
    "sobek_conv_bwd_kept": (_INT, [_P, _P, _P, _P, _P, _P, _P, ctypes.c_uint64, _P, _P, _P, _P, _P, _P, _SZ, _P]),
    "sobek_materialized_workspace_size": (_INT, [_P, _P, _SZ, ctypes.POINTER(_SZ)]),
    "sobek_conv_fwd_materialized": (_INT, [_P, _P, _P, _P, _P, _P, _P, _P, _SZ, _P]),
    "sobek_profile_enable": (_INT, [_INT]),
    "sobek_profile_reset": (_INT, []),
    "sobek_profile_query": (_INT, [_INT, ctypes.c_char_p, _SZ, ctypes.POINTER(_I64), ctypes.POINTER(ctypes.c_double)]),
}

EXPORTED = tuple(_SIGNATURES)


def lib():
    """The loaded library (raises if it has not been built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing: build it with paper_2607_18074_amd/build.py "
                               "(there is no fallback implementation)")
        L = ctypes.CDLL(LIB_PATH)
        for name, (res, args) in _SIGNATURES.items():
            f = getattr(L, name)
            f.restype = res
            f.argtypes = args
        _lib = L
    return _lib


def check(rc):
    if rc != 0:
        msg = lib().sobek_last_error().decode(errors="replace")
        raise SobekError(rc, msg)


def parse_irreps(spec):
    """'8x0e+8x1o' or [(mul, l, parity)] -> list of (mul, l, parity)."""
    if not isinstance(spec, str):
        return [(int(m), int(l), int(p)) for (m, l, p) in spec]
    out = []
    for tok in spec.replace(" ", "").split("+"):
        if not tok:
            continue
        m = re.fullmatch(r"(?:(\d+)x)?(\d+)([eo])", tok)
        if m is None:
            raise ValueError(f"bad irrep token {tok!r}")
        out.append((int(m.group(1) or 1), int(m.group(2)), 1 if m.group(3) == "e" else -1))
    return out


def irrep_array(spec):
    v = parse_irreps(spec)
    arr = (Irrep * len(v))()
    for i, (m, l, p) in enumerate(v):
        arr[i] = Irrep(m, l, p)
    return arr, len(v)


def _sig_args(irreps_in, lmax, irreps_out, K, layout="ir_mul", normalization="none", mode="uvw", dtype="f32"):
    a, na = irrep_array(irreps_in)
    b, nb = irrep_array(irreps_out)
    return (a, na, int(lmax), b, nb, int(K), MODES[mode], LAYOUTS[layout], DTYPES[dtype], NORMS[normalization])


def jit_compile(irreps_in, lmax, irreps_out, K, layout="ir_mul", normalization="none", mode="uvw", dtype="f32"):
    """Generate and compile the kernels of a signature into the code-object cache (no GPU needed)."""
    check(lib().sobek_jit_compile(*_sig_args(irreps_in, lmax, irreps_out, K, layout, normalization, mode, dtype)))


def plan_source(irreps_in, lmax, irreps_out, K, layout="ir_mul", normalization="none", mode="uvw", dtype="f32"):
    """The full HIP source compiled for a signature."""
    args = _sig_args(irreps_in, lmax, irreps_out, K, layout, normalization, mode, dtype)
    need = _SZ(0)
    check(lib().sobek_plan_source(*args, None, 0, ctypes.byref(need)))
    buf = ctypes.create_string_buffer(need.value)
    check(lib().sobek_plan_source(*args, buf, need.value, ctypes.byref(need)))
    return buf.value.decode()


def cg_table(l1, l2, l3):
    import numpy as np
    n = (2 * l1 + 1) * (2 * l2 + 1) * (2 * l3 + 1)
    buf = (ctypes.c_double * n)()
    check(lib().sobek_cg_table(l1, l2, l3, buf))
    return np.array(buf).reshape(2 * l1 + 1, 2 * l2 + 1, 2 * l3 + 1)


def sh_table(l, m, max_terms=64):
    n = ctypes.c_int32(0)
    c = (ctypes.c_double * max_terms)()
    pw = (ctypes.c_int32 * (3 * max_terms))()
    check(lib().sobek_sh_table(l, m, ctypes.byref(n), c, pw, max_terms))
    return [(c[t], (pw[3 * t], pw[3 * t + 1], pw[3 * t + 2])) for t in range(n.value)]


def profile_enable(on=True):
    check(lib().sobek_profile_enable(1 if on else 0))


def profile_reset():
    check(lib().sobek_profile_reset())


def profile_read():
    """{kernel name: (launches, total ms)} of the launches recorded since the last reset."""
    out = {}
    idx = 0
    name = ctypes.create_string_buffer(256)
    n = _I64()
    ms = ctypes.c_double()
    while lib().sobek_profile_query(idx, name, 256, ctypes.byref(n), ctypes.byref(ms)) == 0:
        out[name.value.decode()] = (n.value, ms.value)
        idx += 1
    return out
