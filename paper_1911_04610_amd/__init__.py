"""Python binding of libxpipe: XPipe's one-stage training step on MI355X.

The binding only marshals arguments to the C ABI declared in include/xpipe.h;
every step of the path runs in the library's HIP kernels.  PyTorch is used to
allocate device memory and to supply the HIP stream.  If the built library is
missing the import of any entry point raises: there is no CPU fallback.

Entry points (same names as the C ABI):
  xpipe_version_difference, xpipe_stage_query, Stage (xpipe_stage_create /
  _param_layout / _output_shape / xpipe_predict_weights / xpipe_stage_fwd /
  xpipe_stage_bwd / xpipe_adam_step / xpipe_rule_step / xpipe_stage_destroy /
  timing / recorded passes / xpipe_stage_run), xpipe_schedule, xpipe_predict_flat,
  xpipe_adam_flat, xpipe_rule_flat.
"""
from __future__ import annotations

import ctypes
import dataclasses
import os
from typing import List, Optional, Sequence

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libxpipe.so")

OK, EINVAL, ESTATE, EHIP, EUNSUPPORTED = 0, 1, 2, 3, 4
F32, BF16 = 0, 1
FWD, BWD = 0, 1
KEEP_PRED = 2
PRED_EQ3, PRED_ADAMDIR, PRED_LITERAL, PRED_SMOOTHED = 0, 1, 2, 3
RULE_MOMENTUM_SGD, RULE_RMSPROP = 1, 2
ROUND_HALF_UP, ROUND_HALF_EVEN, ROUND_HALF_DOWN = 0, 1, 2
KINDS = {"linear": 0, "conv": 1, "bn": 2, "relu": 3, "add": 4, "maxpool2": 5, "avgpool3": 6,
         "gap": 7, "concat": 8, "softmax_ce": 9, "maxpool3s2": 10}
MAX_INPUTS = 4


class XPipeError(RuntimeError):
    def __init__(self, status, msg):
        super().__init__(f"xpipe status {status}: {msg}")
        self.status = status


class LayerDesc(ctypes.Structure):
    _fields_ = [("kind", ctypes.c_int32), ("n_inputs", ctypes.c_int32),
                ("inputs", ctypes.c_int32 * MAX_INPUTS), ("cin", ctypes.c_int32),
                ("cout", ctypes.c_int32), ("k", ctypes.c_int32), ("has_bias", ctypes.c_int32),
                ("classes", ctypes.c_int32), ("stride", ctypes.c_int32), ("kw", ctypes.c_int32),
                ("pad", ctypes.c_int32)]


class HParams(ctypes.Structure):
    _fields_ = [("lr", ctypes.c_double), ("beta1", ctypes.c_double), ("beta2", ctypes.c_double),
                ("eps", ctypes.c_double), ("t", ctypes.c_int64), ("mode", ctypes.c_int32)]


class SchedEvent(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int32) for n in ("time", "kind", "micro", "mini", "bellwether",
                                             "update_after", "version", "s_eq", "s_excl", "s_incl")]


class RunIO(ctypes.Structure):
    _fields_ = [("n_micro", ctypes.c_int32), ("x", ctypes.c_void_p), ("dy", ctypes.c_void_p),
                ("labels", ctypes.c_void_p), ("y", ctypes.c_void_p), ("loss", ctypes.c_void_p),
                ("dx", ctypes.c_void_p)]


class RuleParams(ctypes.Structure):
    _fields_ = [("rule", ctypes.c_int32), ("lr", ctypes.c_double), ("momentum", ctypes.c_double),
                ("weight_decay", ctypes.c_double), ("alpha", ctypes.c_double), ("eps", ctypes.c_double)]


@dataclasses.dataclass
class Rule:
    """Update rule besides Adam (xpipe_rule_hparams)."""
    rule: int = RULE_MOMENTUM_SGD
    lr: float = 1e-2
    momentum: float = 0.9
    weight_decay: float = 0.0
    alpha: float = 0.99
    eps: float = 1e-8

    def c(self) -> RuleParams:
        return RuleParams(int(self.rule), self.lr, self.momentum, self.weight_decay, self.alpha, self.eps)


@dataclasses.dataclass
class Hyper:
    lr: float = 1e-3
    beta1: float = 0.9
    beta2: float = 0.999
    eps: float = 1e-8
    mode: int = PRED_EQ3

    def c(self, t: int) -> HParams:
        return HParams(self.lr, self.beta1, self.beta2, self.eps, int(t), int(self.mode))


_lib = None
_P = ctypes.c_void_p
_I32, _I64, _SZ = ctypes.c_int32, ctypes.c_int64, ctypes.c_size_t

_SIGS = {
    "xpipe_version_difference": [_I32, _I32, _I32, _I32, _I32, _I32, ctypes.POINTER(_I32)],
    "xpipe_stage_query": [_P, _I32, _I32, _I32, _I32, _I32, _I32, ctypes.POINTER(_I64),
                          ctypes.POINTER(_SZ)],
    "xpipe_stage_create": [_P, _I32, _I32, _I32, _I32, _I32, _I32, _I32, _P, _P, _P, _P, _P,
                           _P, _P, _P, _SZ, ctypes.POINTER(_P)],
    "xpipe_stage_create_static": [_P, _I32, _I32, _I32, _I32, _I32, _I32, _I32, _P, _P, _P, _P,
                                  _P, _P, _P, ctypes.POINTER(_P)],
    "xpipe_stage_num_param_tensors": [_P, ctypes.POINTER(_I32)],
    "xpipe_stage_param_layout": [_P, _I32, ctypes.POINTER(_I64), ctypes.POINTER(_I64)],
    "xpipe_stage_output_shape": [_P] + [ctypes.POINTER(_I32)] * 4,
    "xpipe_predict_weights": [_P, _I32, _I32, ctypes.POINTER(HParams)],
    "xpipe_stage_fwd": [_P, _P, _P, _P, _P],
    "xpipe_stage_bwd": [_P, _P, _P, _P, _P],
    "xpipe_adam_step": [_P, ctypes.POINTER(HParams), _I32, _I32, _I32],
    "xpipe_partition": [_P, _I32, _I32, ctypes.POINTER(_I32)],
    "xpipe_schedule": [_I32, _I32, _I32, _I32, _I32, _I32, _P, _I32, ctypes.POINTER(_I32)],
    "xpipe_stage_run": [_P, _P, _I32, ctypes.POINTER(RunIO), ctypes.POINTER(HParams), _P, _P, _P, _I32],
    "xpipe_rule_step": [_P, ctypes.POINTER(RuleParams), ctypes.POINTER(HParams), _P, _P, _I32, _I32,
                        _I32],
    "xpipe_rule_flat": [_P, _P, _P, _P, _P, _P, _I64, ctypes.POINTER(RuleParams),
                        ctypes.POINTER(HParams), _I32, _P, _I32, _P, _I32, _P],
    "xpipe_stage_destroy": [_P],
    "xpipe_predict_flat": [_P, _P, _P, _P, _P, _I64, _I32, ctypes.POINTER(HParams), _P],
    "xpipe_adam_flat": [_P, _P, _P, _P, _I64, ctypes.POINTER(HParams), _I32, _P, _I32, _P, _I32,
                        _P],
    "xpipe_probe_copy": [_P, _P, _I64, _P],
    "xpipe_probe_mfma": [_P, _I32, _I32, _P],
    "xpipe_probe_graph": [_P, _I32, _I32, _I32, _I32, ctypes.POINTER(ctypes.c_double), _P],
    "xpipe_probe_stream": [ctypes.POINTER(_P), _I32, ctypes.POINTER(_P), _I32, _I64, _P],
    "xpipe_stage_set_timing": [_P, _I32],
    "xpipe_stage_set_graphs": [_P, _I32],
    "xpipe_stage_set_fwd_stream": [_P, _P, ctypes.c_size_t, ctypes.POINTER(_P)],
    "xpipe_stage_timing_count": [_P, ctypes.POINTER(_I32)],
    "xpipe_stage_timing_entry": [_P, _I32, ctypes.POINTER(ctypes.c_char_p),
                                 ctypes.POINTER(ctypes.c_double), ctypes.POINTER(_I64),
                                 ctypes.POINTER(ctypes.c_double)],
}


def lib() -> ctypes.CDLL:
    """The loaded libxpipe.so; raises if it has not been built."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise ImportError(f"{LIB_PATH} is missing: build it with "
                              "`python -m paper_1911_04610_amd.build`")
        # The library and PyTorch must share one HIP runtime (the library
        # launches on torch's streams and into torch's allocations).  torch
        # ships its own copy of the runtime; loaded after the library, it would
        # come in as a second runtime with its own device contexts.  Importing
        # torch first makes the library bind to torch's copy.
        import torch  # noqa: F401
        L = ctypes.CDLL(LIB_PATH)
        for name, args in _SIGS.items():
            f = getattr(L, name)
            f.argtypes = args
            f.restype = ctypes.c_int
        L.xpipe_last_error.argtypes = []
        L.xpipe_last_error.restype = ctypes.c_char_p
        _lib = L
    return _lib


def _check(status: int):
    if status != OK:
        raise XPipeError(status, lib().xpipe_last_error().decode())


def layer_descs(layers: Sequence[dict]):
    """Layer dicts (kind, inputs, cin, cout, k, bias, classes) -> LayerDesc array."""
    arr = (LayerDesc * len(layers))()
    for i, L in enumerate(layers):
        d = arr[i]
        d.kind = KINDS[L["kind"]]
        ins = list(L["inputs"])
        d.n_inputs = len(ins)
        for j in range(MAX_INPUTS):
            d.inputs[j] = ins[j] if j < len(ins) else 0
        d.cin = int(L.get("cin", 0))
        d.cout = int(L.get("cout", 0))
        d.k = int(L.get("k", 1))
        d.has_bias = int(bool(L.get("bias", False)))
        d.classes = int(L.get("classes", 0))
        d.stride = int(L.get("stride", 1))
        d.kw = int(L.get("kw", d.k))
        d.pad = {"same": 0, "valid": 1}[L.get("pad", "same")]
    return arr


def xpipe_version_difference(size: int, T: int, rank: int, direction: int,
                             rounding: int = ROUND_HALF_UP, ceil_half_rank: bool = False) -> int:
    out = _I32(0)
    _check(lib().xpipe_version_difference(size, T, rank, direction, rounding,
                                          int(ceil_half_rank), ctypes.byref(out)))
    return out.value


def xpipe_stage_query(layers, micro_batch: int, in_shape, dtype: int):
    H, W, C = _hwc(in_shape)
    d = layer_descs(layers)
    P = _I64(0)
    ws = _SZ(0)
    _check(lib().xpipe_stage_query(d, len(layers), micro_batch, H, W, C, dtype, ctypes.byref(P),
                                   ctypes.byref(ws)))
    return P.value, ws.value


def _hwc(in_shape):
    if len(in_shape) == 1:
        return 1, 1, int(in_shape[0])
    return int(in_shape[0]), int(in_shape[1]), int(in_shape[2])


def _ptr(t) -> Optional[int]:
    return None if t is None else t.data_ptr()


def _stream_ptr(stream) -> Optional[int]:
    import torch
    s = stream if stream is not None else torch.cuda.current_stream()
    return s.cuda_stream


class Stage:
    """One stage on the current GPU: parameters, moments, gradient accumulator,
    prediction caches and workspace are torch tensors owned by this object."""

    def __init__(self, layers: List[dict], micro_batch: int, T: int, in_shape, dtype: int = F32,
                 device="cuda", stream=None, static_workspace: bool = False):
        """static_workspace=True creates the stage with xpipe_stage_create_static
        (the library's static device workspace; no workspace tensor here)."""
        import torch
        self.layers = layers
        self.micro_batch, self.T, self.dtype = micro_batch, T, dtype
        self.in_shape = tuple(in_shape)
        self.device = torch.device(device)
        self.stream = stream
        self.P, ws = xpipe_stage_query(layers, micro_batch, in_shape, dtype)
        self.ws_bytes = ws
        self.fwd_workspace = self.fwd_stream = None
        f32 = dict(dtype=torch.float32, device=self.device)
        self.W = torch.zeros(self.P, **f32)
        self.m = torch.zeros(self.P, **f32)
        self.v = torch.zeros(self.P, **f32)
        self.grad = torch.zeros(self.P, **f32)
        self.w_pred_fwd = torch.zeros(self.P, **f32)
        self.w_pred_bwd = torch.zeros(self.P, **f32)
        self._h = _P()
        H, W, C = _hwc(in_shape)
        self._descs = layer_descs(layers)
        if static_workspace:
            self.workspace = None
            _check(lib().xpipe_stage_create_static(self._descs, len(layers), micro_batch, T, H, W, C,
                                                   dtype, _stream_ptr(stream), _ptr(self.W),
                                                   _ptr(self.m), _ptr(self.v), _ptr(self.grad),
                                                   _ptr(self.w_pred_fwd), _ptr(self.w_pred_bwd),
                                                   ctypes.byref(self._h)))
        else:
            self.workspace = torch.empty(max(ws, 256) + 256, dtype=torch.uint8, device=self.device)
            base = self.workspace.data_ptr()
            ws_ptr = (base + 255) // 256 * 256
            _check(lib().xpipe_stage_create(self._descs, len(layers), micro_batch, T, H, W, C, dtype,
                                            _stream_ptr(stream), _ptr(self.W), _ptr(self.m),
                                            _ptr(self.v), _ptr(self.grad), _ptr(self.w_pred_fwd),
                                            _ptr(self.w_pred_bwd), ws_ptr, ws, ctypes.byref(self._h)))
        n = _I32(0)
        _check(lib().xpipe_stage_num_param_tensors(self._h, ctypes.byref(n)))
        self.layout = []
        for i in range(n.value):
            off, cnt = _I64(0), _I64(0)
            _check(lib().xpipe_stage_param_layout(self._h, i, ctypes.byref(off), ctypes.byref(cnt)))
            self.layout.append((off.value, cnt.value))
        dims = [_I32(0) for _ in range(4)]
        _check(lib().xpipe_stage_output_shape(self._h, *[ctypes.byref(d) for d in dims]))
        self.out_shape = tuple(d.value for d in dims)

    # ---- parameter marshalling (host <-> flat device buffers)
    def set_flat(self, buf, tensors):
        """Copy per-tensor host arrays into a flat device buffer (padding stays 0)."""
        import numpy as np
        import torch
        host = np.zeros(self.P, np.float32)
        for (off, cnt), a in zip(self.layout, tensors):
            host[off:off + cnt] = np.asarray(a, np.float32).ravel()
        buf.copy_(torch.from_numpy(host).to(self.device))

    def get_tensors(self, buf):
        """Split a flat device buffer into per-tensor host arrays (fp64 copies)."""
        import numpy as np
        host = buf.detach().cpu().numpy().astype(np.float64)
        return [host[off:off + cnt] for off, cnt in self.layout]

    # ---- the ABI calls
    def xpipe_predict_weights(self, which: int, s: int, hp: Hyper, t: int):
        c = hp.c(t)
        _check(lib().xpipe_predict_weights(self._h, which, s, ctypes.byref(c)))

    def xpipe_stage_fwd(self, x, y, labels=None, loss=None):
        _check(lib().xpipe_stage_fwd(self._h, _ptr(x), _ptr(y), _ptr(labels), _ptr(loss)))

    def xpipe_stage_set_fwd_stream(self, enable: bool):
        """Forwards on a stream of the stage's own, with a workspace of their
        own (allocated here), beside the backwards on the stage's stream.
        Returns that stream as a torch.cuda.ExternalStream (None when
        disabled), for ordering the forwards' inputs and outputs."""
        import torch
        if not enable:
            _check(lib().xpipe_stage_set_fwd_stream(self._h, None, 0, None))
            self.fwd_workspace = self.fwd_stream = None
            return None
        buf = torch.empty(max(self.ws_bytes, 256) + 256, dtype=torch.uint8, device=self.device)
        ptr = (buf.data_ptr() + 255) // 256 * 256
        s = _P()
        _check(lib().xpipe_stage_set_fwd_stream(self._h, ptr, self.ws_bytes, ctypes.byref(s)))
        self.fwd_workspace = buf
        self.fwd_stream = torch.cuda.ExternalStream(s.value, device=self.device)
        return self.fwd_stream

    def xpipe_stage_bwd(self, x, dy=None, labels=None, dx=None):
        _check(lib().xpipe_stage_bwd(self._h, _ptr(x), _ptr(dy), _ptr(labels), _ptr(dx)))

    def xpipe_adam_step(self, hp: Hyper, t: int, s_fwd_next: int = 0, s_bwd_next: int = 0,
                        emit_pred: bool = False):
        c = hp.c(t)
        _check(lib().xpipe_adam_step(self._h, ctypes.byref(c), s_fwd_next, s_bwd_next,
                                     int(emit_pred)))

    def xpipe_rule_step(self, rule: Rule, hp: Hyper, t: int, buf, sq=None, s_fwd_next: int = 0,
                        s_bwd_next: int = 0, emit_pred: bool = False):
        """Update with momentum SGD or RMSProp; buf / sq are fp32 device tensors
        of n_params elements carried between calls (zero before the first)."""
        r, c = rule.c(), hp.c(t)
        _check(lib().xpipe_rule_step(self._h, ctypes.byref(r), ctypes.byref(c), _ptr(buf), _ptr(sq),
                                     s_fwd_next, s_bwd_next, int(emit_pred)))

    def xpipe_stage_run(self, events, x, y, hp: Hyper, t: int, dy=None, labels=None, loss=None,
                        dx=None, rule: Optional[Rule] = None, buf=None, sq=None, draft=False):
        """Run schedule events (from xpipe_schedule) on this stage.  x, y, dy,
        labels, dx: lists of device tensors indexed by micro-batch - 1; loss: a
        device fp32 tensor [n_micro] or None."""
        n = len(x)
        arr = lambda ts: None if ts is None else (ctypes.c_void_p * n)(*[_ptr(a) for a in ts])
        keep = [arr(x), arr(dy), arr(labels), arr(y), arr(dx)]
        io = RunIO(n, *(ctypes.cast(a, ctypes.c_void_p) if a is not None else None for a in keep[:3]),
                   ctypes.cast(keep[3], ctypes.c_void_p), _ptr(loss),
                   ctypes.cast(keep[4], ctypes.c_void_p) if keep[4] is not None else None)
        ev = (SchedEvent * len(events))(*events)
        c = hp.c(t)
        r = rule.c() if rule is not None else None
        _check(lib().xpipe_stage_run(self._h, ctypes.cast(ev, ctypes.c_void_p), len(events),
                                     ctypes.byref(io), ctypes.byref(c),
                                     ctypes.cast(ctypes.pointer(r), ctypes.c_void_p) if r is not None else None,
                                     _ptr(buf), _ptr(sq), int(draft)))

    def set_timing(self, enable: bool):
        _check(lib().xpipe_stage_set_timing(self._h, int(enable)))

    def set_graphs(self, enable: bool):
        _check(lib().xpipe_stage_set_graphs(self._h, int(enable)))

    def timing(self):
        """{kernel name: (ms, launches, work)} over the launches since set_timing(True)."""
        n = _I32(0)
        _check(lib().xpipe_stage_timing_count(self._h, ctypes.byref(n)))
        out = {}
        for i in range(n.value):
            name, ms, cnt, work = ctypes.c_char_p(), ctypes.c_double(0), _I64(0), ctypes.c_double(0)
            _check(lib().xpipe_stage_timing_entry(self._h, i, ctypes.byref(name), ctypes.byref(ms),
                                                  ctypes.byref(cnt), ctypes.byref(work)))
            out[name.value.decode()] = (ms.value, cnt.value, work.value)
        return out

    def destroy(self):
        if self._h:
            lib().xpipe_stage_destroy(self._h)
            self._h = _P()

    def __del__(self):
        try:
            self.destroy()
        except Exception:
            pass


def xpipe_predict_flat(W, m, v, out, out_bf16, s: int, hp: Hyper, t: int, stream=None):
    c = hp.c(t)
    _check(lib().xpipe_predict_flat(_ptr(W), _ptr(m), _ptr(v), _ptr(out), _ptr(out_bf16),
                                    W.numel(), s, ctypes.byref(c), _stream_ptr(stream)))


def xpipe_partition(layers, stages: int) -> List[int]:
    """first layer index of each stage, and len(layers) (Sec. IV-B's partition)."""
    arr = layer_descs(layers)
    first = (_I32 * (stages + 1))()
    _check(lib().xpipe_partition(arr, len(layers), stages, first))
    return list(first)


def xpipe_schedule(size: int, T: int, rank: int, minibatches: int, rounding: int = 0,
                   ceil_half_rank: bool = False) -> List[SchedEvent]:
    """Events of GPU `rank` in the unit-time pipeline schedule (host only)."""
    n = _I32(0)
    _check(lib().xpipe_schedule(size, T, rank, minibatches, rounding, int(ceil_half_rank), None, 0,
                                ctypes.byref(n)))
    ev = (SchedEvent * max(n.value, 1))()
    _check(lib().xpipe_schedule(size, T, rank, minibatches, rounding, int(ceil_half_rank),
                                ctypes.cast(ev, ctypes.c_void_p), n.value, ctypes.byref(n)))
    return list(ev)[:n.value]


def xpipe_rule_flat(W, buf, sq, m, v, G, rule: Rule, hp: Hyper, t: int, zero_grad=True, pred_fwd=None,
                    s_fwd=0, pred_bwd=None, s_bwd=0, stream=None):
    r, c = rule.c(), hp.c(t)
    _check(lib().xpipe_rule_flat(_ptr(W), _ptr(buf), _ptr(sq), _ptr(m), _ptr(v), _ptr(G), W.numel(),
                                 ctypes.byref(r), ctypes.byref(c), int(zero_grad), _ptr(pred_fwd), s_fwd,
                                 _ptr(pred_bwd), s_bwd, _stream_ptr(stream)))


def xpipe_probe_copy(src, dst, stream=None):
    """dst[:] = src[:] (same byte size, multiple of 16) with the library's copy probe."""
    nbytes = src.numel() * src.element_size()
    if dst.numel() * dst.element_size() != nbytes:
        raise ValueError("src and dst must have the same byte size")
    _check(lib().xpipe_probe_copy(_ptr(src), _ptr(dst), nbytes, _stream_ptr(stream)))


def xpipe_probe_mfma(out, iters: int, stream=None):
    """One wave per element of the float32 tensor `out`, `iters` rounds of 8 MFMAs each."""
    _check(lib().xpipe_probe_mfma(_ptr(out), out.numel(), int(iters), _stream_ptr(stream)))


def xpipe_probe_graph(scratch, width: int, length: int, reps: int, spin: int, stream=None):
    """Recorded-graph fork/join probe: (us per diamond with `width` branches of
    `length` launches, us for the same launches as one chain).  scratch: a
    float32 device tensor of at least 2048 elements."""
    if scratch.numel() < 2048:
        raise ValueError("scratch needs at least 2048 floats")
    out = (ctypes.c_double * 2)()
    _check(lib().xpipe_probe_graph(_ptr(scratch), int(width), int(length), int(reps), int(spin),
                                   out, _stream_ptr(stream)))
    return out[0], out[1]


def xpipe_probe_stream(srcs, dsts, stream=None):
    """Bare stream: every float32 tensor in srcs read once, every one in dsts
    written once (all of one size, a multiple of 4 elements)."""
    n = dsts[0].numel()
    S = (_P * max(len(srcs), 1))(*[_ptr(t) for t in srcs])
    D = (_P * len(dsts))(*[_ptr(t) for t in dsts])
    _check(lib().xpipe_probe_stream(S, len(srcs), D, len(dsts), n, _stream_ptr(stream)))


def xpipe_adam_flat(W, m, v, G, hp: Hyper, t: int, zero_grad=True, pred_fwd=None, s_fwd=0,
                    pred_bwd=None, s_bwd=0, stream=None):
    c = hp.c(t)
    _check(lib().xpipe_adam_flat(_ptr(W), _ptr(m), _ptr(v), _ptr(G), W.numel(), ctypes.byref(c),
                                 int(zero_grad), _ptr(pred_fwd), s_fwd, _ptr(pred_bwd), s_bwd,
                                 _stream_ptr(stream)))
