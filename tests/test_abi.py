"""CPU tests of the C ABI: exports, generator tables against the oracle, error paths.

No compute call is made here (there is no GPU); the kernels' code generation
and hipRTC compilation for gfx950 do run, since they need no device.
"""

import os
import re

import numpy as np
import pytest

from oracle import cg as ocg
from oracle import irreps as oir
from oracle import sh as osh
from paper_2607_18074_amd import _lib

HEADER = os.path.join(os.path.dirname(os.path.dirname(__file__)), "include", "sobek.h")


def header_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"^\s*(?:const\s+)?\w+\s*\*?\s*(sobek_\w+)\s*\(", text, flags=re.M)))


def test_library_exports_every_declared_function():
    L = _lib.lib()
    names = header_functions()
    assert len(names) >= 18
    for n in names:
        assert hasattr(L, n), n
    assert set(names) == set(_lib.EXPORTED)
    assert L.sobek_version() >= 1


def test_cg_tables_match_oracle():
    for l1 in range(4):
        for l2 in range(4):
            for l3 in range(abs(l1 - l2), min(l1 + l2, 3) + 1):
                np.testing.assert_allclose(_lib.cg_table(l1, l2, l3), ocg.real_cg(l1, l2, l3), atol=1e-14,
                                           err_msg=str((l1, l2, l3)))


def test_sh_tables_match_oracle():
    rng = np.random.default_rng(0)
    v = rng.normal(size=(30, 3))
    v /= np.linalg.norm(v, axis=1, keepdims=True)
    ref = osh.sh(3, v)
    k = 0
    for l in range(4):
        for m in range(-l, l + 1):
            val = np.zeros(len(v))
            for c, (a, b, d) in _lib.sh_table(l, m):
                assert a + b + d == l          # homogeneous of degree l
                val += c * v[:, 0] ** a * v[:, 1] ** b * v[:, 2] ** d
            np.testing.assert_allclose(val, ref[:, k], atol=1e-13, err_msg=f"l={l} m={m}")
            k += 1


def test_error_codes():
    with pytest.raises(_lib.SobekError) as e:
        _lib.plan_source("8x0e", 4, "8x0e", 8)            # lmax > 3
    assert e.value.code == -2
    with pytest.raises(_lib.SobekError) as e:
        _lib.plan_source("8x5e", 1, "8x0e", 8)            # l > 3
    assert e.value.code == -2
    with pytest.raises(_lib.SobekError) as e:
        _lib.plan_source("0x0e", 1, "8x0e", 8)            # multiplicity 0
    assert e.value.code == -1
    with pytest.raises(_lib.SobekError) as e:
        _lib.plan_source("8x0e", 1, "8x0o", 8)            # no path satisfies the selection rules
    assert e.value.code == -1
    with pytest.raises(_lib.SobekError) as e:
        _lib.plan_source("8x0e", 1, "8x1o", 0)            # K = 0
    assert e.value.code == -1
    with pytest.raises(_lib.SobekError) as e:
        _lib.plan_source("8x0e+4x1o", 1, "8x0e+4x1o", 4, mode="uvu")   # uvu path 0e x 1o -> 1o joins 8 and 4
    assert e.value.code == -1
    with pytest.raises(_lib.SobekError) as e:
        _lib.cg_table(1, 1, 3)                            # triangle rule
    assert e.value.code == -1
    import ctypes
    nb = ctypes.c_size_t()
    assert _lib.lib().sobek_graph_prepare_size(-1, 0, ctypes.byref(nb)) == -1
    assert _lib.lib().sobek_graph_prepare_size(10, 20, ctypes.byref(nb)) == 0 and nb.value >= 44 + 80


def test_generated_source_reflects_paths():
    src = _lib.plan_source("32x0e+32x1o+32x2e", 2, "32x0e+32x1o+32x2e", 8)
    prob_paths = oir.enumerate_paths(oir.parse_irreps("32x0e+32x1o+32x2e"), oir.sh_irreps(2),
                                     oir.parse_irreps("32x0e+32x1o+32x2e"))
    for t, p in enumerate(prob_paths):
        assert f"// path {t}: l_in={p['l_in']} l_sh={p['l_sh']} l_out={p['l_out']}" in src
    for kname in ("sobek_fwd_S", "sobek_fwd_dS", "sobek_bwd_E", "sobek_dbwd_E", "SB_GEMM_ENTRY(32)",
                  "sobek_gemm_sa_##BN", "sobek_ga_reduce", "sobek_sender_reduce"):
        assert kname in src
    # packed-FP32 instructions are never written by hand
    assert "v_pk_" not in src


def test_uvu_source_carries_channelwise_normalisation():
    # fan_in counts paths for uvu (3 paths reach 0e here) and C_in for uvw (3 * 8)
    su = _lib.plan_source("8x0e+8x1o+8x2e", 2, "8x0e+8x1o+8x2e", 4, "ir_mul", "fan_in", "uvu")
    sw = _lib.plan_source("8x0e+8x1o+8x2e", 2, "8x0e+8x1o+8x2e", 4, "ir_mul", "fan_in", "uvw")
    assert "alpha=%g" % (1 / np.sqrt(3)) in su and "alpha=%g" % (1 / np.sqrt(24)) in sw
    for kname in ("sobek_uvu_mix", "sobek_uvu_sbar", "sobek_uvu_ga"):
        assert kname in su


def test_jit_compiles_for_gfx950():
    _lib.jit_compile("8x0e+8x1o", 1, "8x0e+8x1o", 8)
    _lib.jit_compile("8x0e+8x1o", 1, "8x0e+8x1o", 8, "ir_mul", "fan_in", "uvu")
    _lib.jit_compile("3x0e+5x1o+2x2e+1x0o", 1, "4x0e+3x1o+2x2e+1x3e", 4, "mul_ir", "fan_in")


def test_bf16_gemm_option():
    sig = ("32x0e+32x1o+32x2e", 2, "32x0e+32x1o+32x2e", 8)
    s32 = _lib.plan_source(*sig)
    sbf = _lib.plan_source(*sig, "ir_mul", "none", "uvw", "bf16_gemm")
    # the bf16 GEMM text is added to bf16 plans only, and their state kernels store S in bf16:
    # removing the one and restoring the fp32 state type gives the fp32 source exactly
    here = os.path.dirname(os.path.abspath(__file__))
    with open(os.path.join(here, "..", "paper_2607_18074_amd", "csrc", "device", "gemm_bf16.hip")) as f:
        block = "\n" + f.read() + "\n"
    assert "__builtin_amdgcn_mfma_f32_16x16x32_bf16" in sbf and "SB_GEMM_VB_ENTRY(64)" in sbf
    assert "bf16" not in s32
    assert sbf.count(block) == 1
    rest = sbf.replace(block, "")
    # with it, one bf16 adjoint-state GEMM entry per output multiplicity that is a multiple of 32
    entries = re.findall(r'extern "C" __global__ __launch_bounds__\(256\) void sobek_gemm_sbar_cb(\d+)\(.*?\n}\n',
                         rest, re.S)
    assert entries == ["32"]
    rest = re.sub(r'extern "C" __global__ __launch_bounds__\(256\) void sobek_gemm_sbar_cb\d+\(.*?\n}\n', "", rest,
                  flags=re.S)
    assert rest.count("__bf16* __restrict__ S,") >= 4 and rest.count("__bf16* Sg = S") >= 1   # 3 kernels + the units
    assert rest.replace("__bf16* __restrict__ S,", "float* __restrict__ S,").replace("__bf16* Sg = S", "float* Sg = S") == s32
    # reduced precision is implemented for uvw plans whose multiplicities are multiples of 4
    for args in (("8x0e+8x1o", 1, "8x0e+8x1o", 4, "ir_mul", "none", "uvu", "bf16_gemm"),
                 ("6x0e+4x1o", 1, "6x0e+4x1o", 4, "ir_mul", "none", "uvw", "bf16_gemm")):
        with pytest.raises(_lib.SobekError) as e:
            _lib.plan_source(*args)
        assert e.value.code == -2
    with pytest.raises(KeyError):
        _lib.plan_source(*sig, "ir_mul", "none", "uvw", "f16")


def test_channelwise_state_free_source_is_separate():
    # a channelwise plan with the state-free kernels compiles them at creation and the
    # receiver-route kernels on first use; building only the first needs no GPU either
    os.environ["SOBEK_JIT_STATE_FREE_ONLY"] = "1"
    try:
        _lib.jit_compile("8x0e+8x1o", 1, "8x0e+8x1o", 4, "ir_mul", "none", "uvu")
    finally:
        del os.environ["SOBEK_JIT_STATE_FREE_ONLY"]
    src = _lib.plan_source("8x0e+8x1o", 1, "8x0e+8x1o", 4, "ir_mul", "none", "uvu")
    for kname in ("sobek_uvu_fwd", "sobek_uvu_wgrad", "sobek_fwd_S", "sobek_dbwd_E_r"):
        assert kname in src
