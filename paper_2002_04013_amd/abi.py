"""ctypes binding of libdmoe.so: the C ABI of include/dmoe.h, same names.

Argument marshalling only: torch tensors (device memory) are passed as raw
pointers together with the current HIP stream; every step runs in the HIP
kernels of the library.  There is no fallback: without the built library or a
GPU every call raises.
"""
import ctypes
import os

import torch

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG, "libdmoe.so")

DMOE_F32, DMOE_BF16 = 0, 1
DMOE_RELU, DMOE_GELU = 0, 1
DMOE_FLAG_GATE_EXACT = 1
DMOE_FLAG_ALIVE_TOPK = 2

# every extern "C" symbol the header declares
EXPORTS = (
    "dmoe_workspace_bytes", "dmoe_strerror", "dmoe_gate_topk", "dmoe_dispatch",
    "dmoe_expert_ffn_fwd", "dmoe_combine", "dmoe_combine_bwd", "dmoe_gate_topk_bwd",
    "dmoe_expert_ffn_bwd", "dmoe_dispatch_bwd", "dmoe_expert_ffn_bwd_recompute", "dmoe_expert_ffn_bwd_sgd",
    "dmoe_expert_ffblock_fwd", "dmoe_expert_ffblock_bwd", "dmoe_ln_act_fwd", "dmoe_ln_act_bwd",
    "dmoe_trace_begin", "dmoe_trace_end", "dmoe_expert_ffn_fwd_noalloc",
)

# parameters of the feed-forward block expert, in dmoe_ffblock_params order
FFBLOCK_PARAMS = ("W1", "b1", "g1", "be1", "W2", "b2", "g2", "be2", "W3", "b3")
FFBLOCK_ACTS = ("h1", "a1", "st1", "h2", "a2", "st2")


class DmoeError(RuntimeError):
    pass


class Dims(ctypes.Structure):
    _fields_ = [("T", ctypes.c_int64), ("D", ctypes.c_int64), ("H", ctypes.c_int64),
                ("d", ctypes.c_int32), ("M", ctypes.c_int32), ("k", ctypes.c_int32),
                ("dtype", ctypes.c_int32), ("act", ctypes.c_int32), ("flags", ctypes.c_int32)]


class FFBlockParams(ctypes.Structure):
    _fields_ = [(n, ctypes.c_void_p) for n in FFBLOCK_PARAMS]


class FFBlockActs(ctypes.Structure):
    _fields_ = [(n, ctypes.c_void_p) for n in FFBLOCK_ACTS]


def make_dims(T, D, H, d, M, k, dtype="bf16", act="gelu", flags=0):
    return Dims(int(T), int(D), int(H), int(d), int(M), int(k),
                DMOE_BF16 if dtype == "bf16" else DMOE_F32,
                DMOE_GELU if act == "gelu" else DMOE_RELU, int(flags))


_lib = None
_P = ctypes.c_void_p


def load(path=LIB_PATH):
    """Load libdmoe.so (once).  Raises if it has not been built."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise DmoeError(f"{path} is missing: build it with `python -m paper_2002_04013_amd.build`")
    lib = ctypes.CDLL(path)
    pd = ctypes.POINTER(Dims)
    sig = {
        "dmoe_workspace_bytes": (ctypes.c_size_t, [pd]),
        "dmoe_strerror": (ctypes.c_char_p, [ctypes.c_int]),
        "dmoe_gate_topk": (ctypes.c_int, [pd] + [_P] * 10),
        "dmoe_dispatch": (ctypes.c_int, [pd] + [_P] * 10),
        "dmoe_expert_ffn_fwd": (ctypes.c_int, [pd] + [_P] * 11),
        "dmoe_combine": (ctypes.c_int, [pd] + [_P] * 5),
        "dmoe_combine_bwd": (ctypes.c_int, [pd] + [_P] * 7),
        "dmoe_gate_topk_bwd": (ctypes.c_int, [pd] + [_P] * 10),
        "dmoe_expert_ffn_bwd": (ctypes.c_int, [pd] + [_P] * 16),
        "dmoe_dispatch_bwd": (ctypes.c_int, [pd] + [_P] * 7),
        "dmoe_expert_ffn_bwd_recompute": (ctypes.c_int, [pd] + [_P] * 16),
        "dmoe_expert_ffn_bwd_sgd": (ctypes.c_int, [pd] + [_P] * 10 + [ctypes.c_float] + [_P] * 4),
        "dmoe_expert_ffblock_fwd": (ctypes.c_int, [pd, _P, _P, ctypes.POINTER(FFBlockParams),
                                                   ctypes.POINTER(FFBlockActs), _P, _P, _P]),
        "dmoe_expert_ffblock_bwd": (ctypes.c_int, [pd, _P, _P, ctypes.POINTER(FFBlockParams),
                                                   ctypes.POINTER(FFBlockActs), _P, _P, _P, _P,
                                                   ctypes.POINTER(FFBlockParams), _P, _P]),
        "dmoe_ln_act_fwd": (ctypes.c_int, [pd] + [_P] * 7),
        "dmoe_ln_act_bwd": (ctypes.c_int, [pd] + [_P] * 10),
        "dmoe_trace_begin": (ctypes.c_int, [ctypes.POINTER(ctypes.c_void_p), ctypes.POINTER(ctypes.c_char_p),
                                            ctypes.c_int]),
        "dmoe_trace_end": (ctypes.c_int, []),
        "dmoe_expert_ffn_fwd_noalloc": (ctypes.c_int, [pd] + [_P] * 10),
    }
    for name, (res, args) in sig.items():
        fn = getattr(lib, name)
        fn.restype = res
        fn.argtypes = args
    _lib = lib
    return lib


def _ptr(t):
    if t is None:
        return None
    if not isinstance(t, torch.Tensor):
        raise TypeError("expected a torch.Tensor or None")
    if not t.is_cuda:
        raise DmoeError("libdmoe takes device tensors only")
    if not t.is_contiguous():
        raise DmoeError("libdmoe takes contiguous tensors only")
    return ctypes.c_void_p(t.data_ptr())


def _stream(stream=None):
    s = torch.cuda.current_stream() if stream is None else stream
    return ctypes.c_void_p(s.cuda_stream)


def _check(rc, name):
    if rc != 0:
        msg = load().dmoe_strerror(rc).decode()
        raise DmoeError(f"{name} failed: {msg} ({rc})")


def workspace_bytes(dims):
    return int(load().dmoe_workspace_bytes(ctypes.byref(dims)))


def strerror(code):
    return load().dmoe_strerror(int(code)).decode()


def dmoe_gate_topk(dims, x, Wg, bg, alive, idx, w, g=None, scores=None, ws=None, stream=None):
    _check(load().dmoe_gate_topk(ctypes.byref(dims), _ptr(x), _ptr(Wg), _ptr(bg), _ptr(alive),
                                 _ptr(idx), _ptr(w), _ptr(g), _ptr(scores), _ptr(ws),
                                 _stream(stream)), "dmoe_gate_topk")


def dmoe_dispatch(dims, x, idx, alive, counts, offsets, row_token, pos, x_perm, ws, stream=None):
    _check(load().dmoe_dispatch(ctypes.byref(dims), _ptr(x), _ptr(idx), _ptr(alive), _ptr(counts),
                                _ptr(offsets), _ptr(row_token), _ptr(pos), _ptr(x_perm), _ptr(ws),
                                _stream(stream)), "dmoe_dispatch")


def dmoe_expert_ffn_fwd(dims, offsets, x_perm, W1, b1, W2, b2, h, a, y_perm, ws, stream=None):
    _check(load().dmoe_expert_ffn_fwd(ctypes.byref(dims), _ptr(offsets), _ptr(x_perm), _ptr(W1),
                                      _ptr(b1), _ptr(W2), _ptr(b2), _ptr(h), _ptr(a), _ptr(y_perm),
                                      _ptr(ws), _stream(stream)), "dmoe_expert_ffn_fwd")


def dmoe_expert_ffn_fwd_noalloc(dims, offsets, x_perm, W1, b1, W2, b2, h, a, y_perm, stream=None):
    _check(load().dmoe_expert_ffn_fwd_noalloc(ctypes.byref(dims), _ptr(offsets), _ptr(x_perm), _ptr(W1),
                                              _ptr(b1), _ptr(W2), _ptr(b2), _ptr(h), _ptr(a), _ptr(y_perm),
                                              _stream(stream)), "dmoe_expert_ffn_fwd_noalloc")


def dmoe_combine(dims, y_perm, pos, w, y, stream=None):
    _check(load().dmoe_combine(ctypes.byref(dims), _ptr(y_perm), _ptr(pos), _ptr(w), _ptr(y),
                               _stream(stream)), "dmoe_combine")


def dmoe_combine_bwd(dims, dy, y_perm, pos, w, dy_perm, dw, stream=None):
    _check(load().dmoe_combine_bwd(ctypes.byref(dims), _ptr(dy), _ptr(y_perm), _ptr(pos), _ptr(w),
                                   _ptr(dy_perm), _ptr(dw), _stream(stream)), "dmoe_combine_bwd")


def dmoe_gate_topk_bwd(dims, x, idx, w, dw, alive, dg, dWg, dbg, ws, stream=None):
    _check(load().dmoe_gate_topk_bwd(ctypes.byref(dims), _ptr(x), _ptr(idx), _ptr(w), _ptr(dw),
                                     _ptr(alive), _ptr(dg), _ptr(dWg), _ptr(dbg), _ptr(ws),
                                     _stream(stream)), "dmoe_gate_topk_bwd")


def dmoe_expert_ffn_bwd(dims, offsets, counts, x_perm, h, a, dy_perm, W1, W2, dh, dx_perm, dW1, db1,
                        dW2, db2, ws, stream=None):
    _check(load().dmoe_expert_ffn_bwd(ctypes.byref(dims), _ptr(offsets), _ptr(counts), _ptr(x_perm),
                                      _ptr(h), _ptr(a), _ptr(dy_perm), _ptr(W1), _ptr(W2), _ptr(dh),
                                      _ptr(dx_perm), _ptr(dW1), _ptr(db1), _ptr(dW2), _ptr(db2),
                                      _ptr(ws), _stream(stream)), "dmoe_expert_ffn_bwd")


def dmoe_dispatch_bwd(dims, dx_perm, pos, idx, dg, Wg, dx, stream=None):
    _check(load().dmoe_dispatch_bwd(ctypes.byref(dims), _ptr(dx_perm), _ptr(pos), _ptr(idx), _ptr(dg),
                                    _ptr(Wg), _ptr(dx), _stream(stream)), "dmoe_dispatch_bwd")


def dmoe_expert_ffn_bwd_recompute(dims, offsets, counts, x_perm, W1, b1, W2, dy_perm, h, a, dx_perm, dW1, db1,
                                  dW2, db2, ws, stream=None):
    _check(load().dmoe_expert_ffn_bwd_recompute(ctypes.byref(dims), _ptr(offsets), _ptr(counts), _ptr(x_perm),
                                                _ptr(W1), _ptr(b1), _ptr(W2), _ptr(dy_perm), _ptr(h), _ptr(a),
                                                _ptr(dx_perm), _ptr(dW1), _ptr(db1), _ptr(dW2), _ptr(db2),
                                                _ptr(ws), _stream(stream)), "dmoe_expert_ffn_bwd_recompute")


def dmoe_expert_ffn_bwd_sgd(dims, offsets, counts, x_perm, h, a, dy_perm, W1, b1, W2, b2, lr, dh, dx_perm, ws,
                            stream=None):
    _check(load().dmoe_expert_ffn_bwd_sgd(ctypes.byref(dims), _ptr(offsets), _ptr(counts), _ptr(x_perm), _ptr(h),
                                          _ptr(a), _ptr(dy_perm), _ptr(W1), _ptr(b1), _ptr(W2), _ptr(b2),
                                          ctypes.c_float(lr), _ptr(dh), _ptr(dx_perm), _ptr(ws), _stream(stream)),
           "dmoe_expert_ffn_bwd_sgd")


def _block_params(t):
    """dict name -> device tensor (FFBLOCK_PARAMS) as a dmoe_ffblock_params struct."""
    return FFBlockParams(*[_ptr(t[n]) for n in FFBLOCK_PARAMS])


def _block_acts(t):
    return FFBlockActs(*[_ptr(t[n]) for n in FFBLOCK_ACTS])


def dmoe_expert_ffblock_fwd(dims, offsets, x_perm, params, acts, y_perm, ws, stream=None):
    """params: dict of the block parameters (FFBLOCK_PARAMS); acts: dict of the kept
    per-row tensors (FFBLOCK_ACTS)."""
    p, a = _block_params(params), _block_acts(acts)
    _check(load().dmoe_expert_ffblock_fwd(ctypes.byref(dims), _ptr(offsets), _ptr(x_perm), ctypes.byref(p),
                                          ctypes.byref(a), _ptr(y_perm), _ptr(ws), _stream(stream)),
           "dmoe_expert_ffblock_fwd")


def dmoe_expert_ffblock_bwd(dims, offsets, x_perm, params, acts, dy_perm, g1, g2, dx_perm, grads, ws, stream=None):
    """grads: dict of gradient tensors with the parameters' names and shapes."""
    p, a, g = _block_params(params), _block_acts(acts), _block_params(grads)
    _check(load().dmoe_expert_ffblock_bwd(ctypes.byref(dims), _ptr(offsets), _ptr(x_perm), ctypes.byref(p),
                                          ctypes.byref(a), _ptr(dy_perm), _ptr(g1), _ptr(g2), _ptr(dx_perm),
                                          ctypes.byref(g), _ptr(ws), _stream(stream)), "dmoe_expert_ffblock_bwd")


def dmoe_ln_act_fwd(dims, offsets, h, gamma, beta, a, stats, stream=None):
    _check(load().dmoe_ln_act_fwd(ctypes.byref(dims), _ptr(offsets), _ptr(h), _ptr(gamma), _ptr(beta), _ptr(a),
                                  _ptr(stats), _stream(stream)), "dmoe_ln_act_fwd")


def dmoe_ln_act_bwd(dims, offsets, h, stats, gamma, beta, da, dh, dgamma, dbeta, stream=None):
    _check(load().dmoe_ln_act_bwd(ctypes.byref(dims), _ptr(offsets), _ptr(h), _ptr(stats), _ptr(gamma),
                                  _ptr(beta), _ptr(da), _ptr(dh), _ptr(dgamma), _ptr(dbeta), _stream(stream)),
           "dmoe_ln_act_bwd")


class Trace:
    """Launch trace of the library (dmoe_trace_begin / dmoe_trace_end): every kernel the
    calls made inside the `with` block enqueue is followed by a record of the next of
    `capacity` timing events on its stream.  After the block, `kernels()` gives
    (name, milliseconds) per traced kernel once the stream has reached them."""

    def __init__(self, capacity=256, stream=None):
        self.stream = torch.cuda.current_stream() if stream is None else stream
        self.events = [torch.cuda.Event(enable_timing=True) for _ in range(capacity + 1)]
        for e in self.events:          # torch creates the HIP event on its first record
            e.record(self.stream)
        self._handles = (ctypes.c_void_p * capacity)(*[e.cuda_event for e in self.events[1:]])
        self._names = (ctypes.c_char_p * capacity)()
        self.capacity = capacity
        self.count = 0

    def __enter__(self):
        self.events[0].record(self.stream)
        _check(load().dmoe_trace_begin(self._handles, self._names, self.capacity), "dmoe_trace_begin")
        return self

    def __exit__(self, *exc):
        self.count = int(load().dmoe_trace_end())
        return False

    def kernels(self):
        self.events[-1].synchronize()
        n = min(self.count, self.capacity)
        return [(self._names[i].decode(), self.events[i].elapsed_time(self.events[i + 1])) for i in range(n)]
