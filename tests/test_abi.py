"""The C-ABI library loads and exports every symbol include/dmoe.h declares;
host-side validation works without a GPU (no compute calls here)."""
import ctypes
import os
import re

import pytest

from conftest import ROOT

HEADER = os.path.join(ROOT, "include", "dmoe.h")


def _declared():
    txt = open(HEADER).read()
    txt = re.sub(r"/\*.*?\*/", "", txt, flags=re.S)
    return sorted(set(re.findall(r"\b(dmoe_[a-z_]+)\s*\(", txt)))


@pytest.fixture(scope="module")
def lib():
    from paper_2002_04013_amd import abi
    if not os.path.exists(abi.LIB_PATH):
        pytest.fail("libdmoe.so not built: run `python -m paper_2002_04013_amd.build`")
    return abi


def test_header_lists_the_boundary():
    names = _declared()
    for n in ("dmoe_gate_topk", "dmoe_dispatch", "dmoe_expert_ffn_fwd", "dmoe_expert_ffn_bwd",
              "dmoe_combine", "dmoe_combine_bwd", "dmoe_gate_topk_bwd", "dmoe_dispatch_bwd",
              "dmoe_workspace_bytes", "dmoe_strerror"):
        assert n in names


def test_library_exports_every_declared_symbol(lib):
    raw = ctypes.CDLL(lib.LIB_PATH)
    for name in _declared():
        assert hasattr(raw, name), name
    assert sorted(lib.EXPORTS) == _declared()


def test_workspace_and_validation(lib):
    ok = lib.make_dims(4096, 1024, 4096, 2, 32, 4, "bf16", "gelu")
    assert lib.workspace_bytes(ok) > 0
    bad = [
        lib.make_dims(64, 64, 256, 0, 4, 2),        # d < 1
        lib.make_dims(64, 64, 256, 5, 2, 2),        # d > 4
        lib.make_dims(64, 64, 256, 2, 4, 17),       # k > N
        lib.make_dims(64, 64, 256, 2, 4, 9, "f32"), # k > 8 (unsupported)
        lib.make_dims(64, 60, 256, 2, 4, 2),        # D % 64
        lib.make_dims(64, 64, 250, 2, 4, 2),        # H % 64
        lib.make_dims(-1, 64, 256, 2, 4, 2),        # T < 0
        lib.make_dims(64, 64, 256, 2, 200, 2),      # d*M > 128
    ]
    for dims in bad:
        assert lib.workspace_bytes(dims) == 0
    # empty batch is valid
    assert lib.workspace_bytes(lib.make_dims(0, 64, 256, 2, 4, 2, "f32", "relu")) > 0


def test_null_arguments_rejected_on_host(lib):
    raw = lib.load()
    dims = lib.make_dims(64, 64, 256, 2, 4, 2, "f32", "relu")
    rc = raw.dmoe_gate_topk(ctypes.byref(dims), *([None] * 10))
    assert rc == -1
    rc = raw.dmoe_gate_topk(None, *([None] * 10))
    assert rc == -1
    assert lib.strerror(-1).startswith("invalid")
    assert lib.strerror(-2).startswith("unsupported")


def test_no_cpu_fallback_without_device(lib):
    import torch
    dims = lib.make_dims(8, 64, 64, 1, 4, 2, "f32", "relu")
    x = torch.zeros(8, 64)
    with pytest.raises(lib.DmoeError):
        lib.dmoe_combine(dims, x, torch.zeros(8, 2, dtype=torch.int32), torch.zeros(8, 2), x)
