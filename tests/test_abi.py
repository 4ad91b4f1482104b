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


def _fake(addr=1 << 20):
    """A 16-byte aligned non-null address; the calls below return before any device work."""
    return ctypes.c_void_p(addr)


def test_new_entry_points_validate_on_host(lib):
    raw = lib.load()
    F = lambda: ctypes.c_void_p(1 << 20)
    dims = lib.make_dims(64, 64, 256, 2, 4, 2, "bf16", "relu")
    # null parameter / activation structs
    rc = raw.dmoe_expert_ffblock_fwd(ctypes.byref(dims), F(), F(), None, None, F(), F(), None)
    assert rc == -1
    prm = lib.FFBlockParams(*[F() for _ in lib.FFBLOCK_PARAMS])
    acts = lib.FFBlockActs(*[F() for _ in lib.FFBLOCK_ACTS])
    # a missing gradient pointer in the struct is rejected
    grads = lib.FFBlockParams(*[F() for _ in lib.FFBLOCK_PARAMS])
    grads.W2 = None
    rc = raw.dmoe_expert_ffblock_bwd(ctypes.byref(dims), F(), F(), ctypes.byref(prm), ctypes.byref(acts), F(),
                                     F(), F(), F(), ctypes.byref(grads), F(), None)
    assert rc == -1
    # LayerNorm rows wider than the register-held row (bf16: 4096 values) are unsupported
    wide = lib.make_dims(64, 64, 8192, 2, 4, 2, "bf16", "relu")
    rc = raw.dmoe_expert_ffblock_fwd(ctypes.byref(wide), F(), F(), ctypes.byref(prm), ctypes.byref(acts), F(),
                                     F(), None)
    assert rc == -2
    rc = raw.dmoe_ln_act_fwd(ctypes.byref(wide), F(), F(), F(), F(), F(), F(), None)
    assert rc == -2
    # misaligned pointer
    rc = raw.dmoe_ln_act_fwd(ctypes.byref(dims), F(), ctypes.c_void_p((1 << 20) + 2), F(), F(), F(), F(), None)
    assert rc == -2
    # NaN step size for the fused SGD backward
    rc = raw.dmoe_expert_ffn_bwd_sgd(ctypes.byref(dims), *[F() for _ in range(10)], ctypes.c_float(float("nan")),
                                     F(), F(), F(), None)
    assert rc == -1
    # widths past the 32-bit tile addressing limit
    assert lib.workspace_bytes(lib.make_dims(64, 1 << 23, 256, 2, 4, 2)) == 0
    assert lib.workspace_bytes(lib.make_dims(64, 64, 1 << 23, 2, 4, 2)) == 0
    # token counts whose pair indices do not fit 32 bits (no overflow in the check itself)
    assert lib.workspace_bytes(lib.make_dims(1 << 28, 64, 256, 2, 4, 4)) == 0
    assert lib.workspace_bytes(lib.make_dims(1 << 62, 64, 256, 2, 4, 4)) == 0
    assert lib.workspace_bytes(lib.make_dims((1 << 28) - 1, 64, 256, 2, 4, 4)) > 0
    # unknown flag bits
    assert lib.workspace_bytes(lib.make_dims(64, 64, 256, 2, 4, 2, flags=4)) == 0


def test_gate_workspace_required_on_host(lib):
    """The gate's queue of tokens to recompute lives in the workspace: the MFMA path
    (bf16, d*M <= 96) and the alive-first TopK (either dtype) reject ws = NULL before
    any device work."""
    raw = lib.load()
    F = lambda: ctypes.c_void_p(1 << 20)
    for dt, flags in (("bf16", 0), ("bf16", lib.DMOE_FLAG_ALIVE_TOPK), ("f32", lib.DMOE_FLAG_ALIVE_TOPK)):
        dims = lib.make_dims(64, 64, 256, 2, 4, 2, dt, "relu", flags)
        rc = raw.dmoe_gate_topk(ctypes.byref(dims), F(), F(), None, None, F(), F(), None, None, None, None)
        assert rc == -1, (dt, flags)


@pytest.mark.parametrize("case,kw,rc", [
    ("T < 0", dict(T=-1), -1),
    ("D = 0", dict(D=0), -1),
    ("H = 0", dict(H=0), -1),
    ("d = 0", dict(d=0), -1),
    ("M = 0", dict(M=0), -1),
    ("k = 0", dict(k=0), -1),
    ("k > N", dict(d=1, M=2, k=3), -1),
    ("unknown dtype", dict(dtype=7), -1),
    ("unknown activation", dict(act=9), -1),
    ("unknown flag bit", dict(flags=0x80), -1),
    ("d > 4", dict(d=5, M=2), -2),
    ("N > 16384", dict(d=2, M=129), -2),
    ("k > 8", dict(d=2, M=4, k=9), -2),
    ("d M > 128", dict(d=2, M=65), -2),
    ("D not a multiple of 64", dict(D=96), -2),
    ("H not a multiple of 64", dict(H=200), -2),
    ("D above 2^22", dict(D=(1 << 22) + 64), -2),
    ("T k at 2^30", dict(T=1 << 28, k=4), -2),
])
def test_dims_rules_on_host(lib, case, kw, rc):
    """The supported-set rules of the header: each invalid dims is refused by the entry
    point before any device work (the pointers below are never dereferenced), and the
    workspace query answers 0 for it."""
    raw = lib.load()
    base = dict(T=64, D=64, H=256, d=2, M=4, k=2, dtype=lib.DMOE_BF16, act=lib.DMOE_RELU, flags=0)
    base.update(kw)
    dims = lib.Dims(*(int(base[f]) for f in ("T", "D", "H", "d", "M", "k", "dtype", "act", "flags")))
    got = raw.dmoe_gate_topk(ctypes.byref(dims), *[_fake() for _ in range(9)], None)
    assert got == rc, f"{case}: dmoe_gate_topk returned {got}, expected {rc}"
    assert lib.workspace_bytes(dims) == 0, case
    ok = lib.make_dims(64, 64, 256, 2, 4, 2, "bf16", "relu")
    assert lib.workspace_bytes(ok) > 0
