"""pytest plugin: run GPU test files on the CPU emulation build instead of the GPU.

    python -m pytest -p tests.emu.pytest_plugin tests/test_gpu_parity.py -k "not autograd"

The package's api module is replaced by tests.emu.harness (the same calls on guarded host
buffers), the binding's library handle by the emulation library, the test modules' _t/_n helpers by their harness equivalents, and the few torch calls the
tests make on device tensors (torch.empty/zeros/full with device="cuda", torch.cuda.synchronize,
torch.isfinite) by stand-ins.  Tests that go through torch autograd are not supported.
"""

import sys

import numpy as np

from tests.emu import harness as H
import paper_2607_18074_amd  # noqa: E402
from paper_2607_18074_amd import _lib  # noqa: E402

sys.modules["paper_2607_18074_amd.api"] = H
paper_2607_18074_amd.api = H
_lib.lib = H.lib   # the binding's helpers (launch profile, errors) call the emulation library

import torch  # noqa: E402

torch.cuda.is_available = lambda: True
torch.cuda.synchronize = lambda *a, **k: None


class _Stream:
    cuda_stream = 0


torch.cuda.current_stream = lambda *a, **k: _Stream()
_NP = {torch.float32: np.float32, torch.int32: np.int32, torch.uint8: np.uint8, None: np.float32}
_isfinite, _empty, _zeros, _full = torch.isfinite, torch.empty, torch.zeros, torch.full


def _on_device(device):
    return device is not None and "cuda" in str(device)


def _empty_f(*shape, dtype=None, device=None, **kw):
    if not _on_device(device):
        return _empty(*shape, dtype=dtype, device=device, **kw)
    shape = tuple(shape[0]) if len(shape) == 1 and isinstance(shape[0], (tuple, list)) else shape
    return H.Dev(shape, _NP[dtype], "torch.empty")


def _zeros_f(*shape, dtype=None, device=None, **kw):
    if not _on_device(device):
        return _zeros(*shape, dtype=dtype, device=device, **kw)
    return _empty_f(*shape, dtype=dtype, device=device).fill_(0)


def _full_f(size, value, dtype=None, device=None, **kw):
    if not _on_device(device):
        return _full(size, value, dtype=dtype, device=device, **kw)
    return H.Dev(tuple(size), _NP[dtype], "torch.full", value)


torch.empty, torch.zeros, torch.full = _empty_f, _zeros_f, _full_f
torch.isfinite = lambda t: _isfinite(torch.from_numpy(t.np())) if isinstance(t, H.Dev) else _isfinite(t)


def _t(a, dev=None):
    return None if a is None else H.dev(np.ascontiguousarray(a), "test input")


def _n(t):
    return None if t is None else t.np()


def pytest_collection_modifyitems(session, config, items):
    for it in items:
        mod = it.module
        if hasattr(mod, "_t"):
            mod._t = _t
        if hasattr(mod, "_n"):
            mod._n = _n
