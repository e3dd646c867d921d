"""Python binding of the LayUp C ABI (include/layup.h): ctypes marshalling only.

Every computation runs in the HIP library ``liblayup.so``; this module loads
it (and fails loudly when it is missing), mirrors the C structs and exposes
the entry points under the same names.  PyTorch is used only to allocate
device memory and to hand HIP streams to the library.
"""
from __future__ import annotations

import ctypes as C
import os
from typing import Dict, List, Optional

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "liblayup.so")

LAYUP_OK, LAYUP_ERR_INVALID_ARG, LAYUP_ERR_SHAPE, LAYUP_ERR_ALIGN, LAYUP_ERR_DTYPE, \
    LAYUP_ERR_STATE, LAYUP_ERR_HIP = range(7)
LAYUP_SGD_MOMENTUM, LAYUP_ADAMW = 0, 1
LAYUP_MODEL_MLP_F32, LAYUP_MODEL_GPT_BF16 = 0, 1
LAYUP_MAX_MLP_LAYERS = 8
LAYUP_MIX_PULL, LAYUP_MIX_PUSH = 0, 1
LAYUP_SCHEDULE_LAYERWISE, LAYUP_SCHEDULE_AFTER_BACKWARD, LAYUP_SCHEDULE_FUSED_DW = 0, 1, 2

STATUS_NAMES = {0: "OK", 1: "INVALID_ARG", 2: "SHAPE", 3: "ALIGN", 4: "DTYPE", 5: "STATE", 6: "HIP"}


class layup_hparams(C.Structure):
    _fields_ = [("kind", C.c_int32), ("lr", C.c_float), ("momentum", C.c_float),
                ("weight_decay", C.c_float), ("beta1", C.c_float), ("beta2", C.c_float),
                ("eps", C.c_float), ("step", C.c_int64)]


class layup_tensor(C.Structure):
    _fields_ = [("param", C.c_void_p), ("grad", C.c_void_p), ("state0", C.c_void_p),
                ("state1", C.c_void_p), ("peer", C.c_void_p), ("param_bf16", C.c_void_p),
                ("peer_bf16", C.c_void_p), ("numel", C.c_int64), ("decay", C.c_int32),
                ("reserved", C.c_int32)]


class layup_config(C.Structure):
    _fields_ = [("model", C.c_int32), ("n_mlp_layers", C.c_int32),
                ("mlp_dims", C.c_int32 * (LAYUP_MAX_MLP_LAYERS + 1)),
                ("n_layer", C.c_int32), ("d_model", C.c_int32), ("n_head", C.c_int32),
                ("d_ff", C.c_int32), ("seq", C.c_int32), ("vocab", C.c_int32),
                ("batch", C.c_int32), ("n_peers", C.c_int32)]


class layup_tensor_info(C.Structure):
    _fields_ = [("name", C.c_char * 32), ("offset", C.c_int64), ("numel", C.c_int64),
                ("rows", C.c_int32), ("cols", C.c_int32), ("padded_rows", C.c_int32),
                ("unit", C.c_int32), ("decay", C.c_int32), ("reserved", C.c_int32)]


class layup_buffers(C.Structure):
    _fields_ = [("params", C.c_void_p), ("grads", C.c_void_p), ("m", C.c_void_p),
                ("v", C.c_void_p), ("peers", C.c_void_p), ("params_bf16", C.c_void_p),
                ("trace", C.c_void_p), ("trace_counter", C.c_void_p),
                ("trace_capacity", C.c_int32), ("reserved", C.c_int32)]


class layup_step_args(C.Structure):
    _fields_ = [("tokens", C.c_void_p), ("x", C.c_void_p), ("hp", C.c_void_p), ("alpha", C.c_float),
                ("schedule", C.c_int32), ("mix_mode", C.c_int32), ("peer_slot", C.c_int32),
                ("push_params", C.c_void_p), ("push_params_bf16", C.c_void_p),
                ("loss_out", C.c_void_p), ("disagreement", C.c_void_p)]


class layup_gemm_desc(C.Structure):
    _fields_ = [("a_kmajor", C.c_int32), ("b_kmajor", C.c_int32),
                ("M", C.c_int64), ("N", C.c_int64), ("K", C.c_int64),
                ("A", C.c_void_p), ("lda", C.c_int64), ("B", C.c_void_p), ("ldb", C.c_int64),
                ("C", C.c_void_p), ("ldc", C.c_int64), ("c_f32", C.c_int32),
                ("batch", C.c_int32), ("inner", C.c_int32), ("reserved", C.c_int32),
                ("bias", C.c_void_p),
                ("a_outer", C.c_int64), ("a_inner", C.c_int64), ("b_outer", C.c_int64),
                ("b_inner", C.c_int64), ("c_outer", C.c_int64), ("c_inner", C.c_int64),
                ("workspace", C.c_void_p), ("workspace_bytes", C.c_size_t),
                ("a_rowsum", C.c_void_p)]


# exported names, in header order
EXPORTS = [
    "layup_param_layout", "layup_tensor_layout", "layup_workspace_size", "layup_init",
    "layup_destroy", "layup_last_error", "layup_global_error", "layup_synchronize",
    "layup_refresh_shadow", "layup_forward", "layup_layer_backward", "layup_unit_update_mix",
    "layup_layer_update_mix", "layup_layer_update_mix_static", "layup_units_update_mix",
    "layup_unit_update_push", "layup_step_ex", "layup_step",
    "layup_unit_timeline", "layup_gemm_timing", "layup_gemm_timing_read", "layup_push_sum_send", "layup_push_sum_receive", "layup_activation",
    "layup_gemm_bf16", "layup_gemm_f32",
]

_lib: Optional[C.CDLL] = None


def lib() -> C.CDLL:
    """Load liblayup.so.  There is no fallback: without the HIP library
    nothing in this package computes."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise RuntimeError(f"{LIB_PATH} is missing: build it with `python -m paper_2410_05985_amd.build`")
    L = C.CDLL(LIB_PATH)
    P = C.c_void_p
    sig = {
        "layup_param_layout": ([P, P, P, P], C.c_int),
        "layup_tensor_layout": ([P, C.c_int32, P], C.c_int),
        "layup_workspace_size": ([P, P], C.c_int),
        "layup_init": ([P, P, P, P, C.c_size_t, P, P], C.c_int),
        "layup_destroy": ([P], None),
        "layup_last_error": ([P], C.c_char_p),
        "layup_global_error": ([], C.c_char_p),
        "layup_synchronize": ([P], C.c_int),
        "layup_refresh_shadow": ([P], C.c_int),
        "layup_forward": ([P, P, P, P], C.c_int),
        "layup_layer_backward": ([P, C.c_int32], C.c_int),
        "layup_unit_update_mix": ([P, C.c_int32, P, C.c_float, C.c_int32, P], C.c_int),
        "layup_layer_update_mix": ([P, P, C.c_int32, P, C.c_float, C.c_int32, P, P], C.c_int),
        "layup_layer_update_mix_static": ([P, C.c_int32, P, C.c_float, C.c_int32, P, P], C.c_int),
        "layup_units_update_mix": ([P, P, C.c_int32, P, C.c_float, C.c_int32, P, P, C.c_int32, C.c_int32, P],
                                   C.c_int),
        "layup_unit_update_push": ([P, C.c_int32, P, C.c_float, P, P, P], C.c_int),
        "layup_step_ex": ([P, P], C.c_int),
        "layup_step": ([P, P, P, P, C.c_float, C.c_int32, P, P], C.c_int),
        "layup_unit_timeline": ([P, P, P, P], C.c_int),
        "layup_gemm_timing": ([P, C.c_int32], C.c_int),
        "layup_gemm_timing_read": ([P, P, P, P], C.c_int),
        "layup_push_sum_send": ([P, C.c_int32, C.c_int32, C.c_int32, P], C.c_int),
        "layup_push_sum_receive": ([P, C.c_int32, C.c_int32, C.c_int32], C.c_int),
        "layup_activation": ([P, C.c_int32, C.c_int32, P, P, P], C.c_int),
        "layup_gemm_bf16": ([P, P], C.c_int),
        "layup_gemm_f32": ([P, P], C.c_int),
    }
    for name, (args, res) in sig.items():
        f = getattr(L, name)
        f.argtypes = args
        f.restype = res
    _lib = L
    return L


class LayupError(RuntimeError):
    def __init__(self, status: int, msg: str):
        super().__init__(f"layup status {STATUS_NAMES.get(status, status)}: {msg}")
        self.status = status


def _check(st: int, ctx=None):
    if st != LAYUP_OK:
        L = lib()
        msg = (L.layup_last_error(ctx) if ctx else L.layup_global_error()) or b""
        raise LayupError(st, msg.decode())


def _ptr(t) -> Optional[int]:
    if t is None:
        return None
    if isinstance(t, int):
        return t
    return t.data_ptr()


def _stream(s) -> Optional[int]:
    if s is None:
        return None
    if isinstance(s, int):
        return s
    return s.cuda_stream


# ------------------------------------------------------------ configs


def mlp_config(dims, batch: int, n_peers: int = 1) -> layup_config:
    c = layup_config()
    c.model = LAYUP_MODEL_MLP_F32
    c.n_mlp_layers = len(dims) - 1
    for i, v in enumerate(dims):
        c.mlp_dims[i] = v
    c.batch = batch
    c.n_peers = n_peers
    return c


def gpt_config(n_layer, d_model, n_head, d_ff, seq, batch, vocab, n_peers: int = 1) -> layup_config:
    c = layup_config()
    c.model = LAYUP_MODEL_GPT_BF16
    c.n_layer, c.d_model, c.n_head, c.d_ff = n_layer, d_model, n_head, d_ff
    c.seq, c.batch, c.vocab, c.n_peers = seq, batch, vocab, n_peers
    return c


def hparams(kind: str, lr: float, momentum: float = 0.0, weight_decay: float = 0.0,
            beta1: float = 0.9, beta2: float = 0.999, eps: float = 1e-8, step: int = 1):
    h = layup_hparams()
    h.kind = LAYUP_ADAMW if kind == "adamw" else LAYUP_SGD_MOMENTUM
    h.lr, h.momentum, h.weight_decay = lr, momentum, weight_decay
    h.beta1, h.beta2, h.eps, h.step = beta1, beta2, eps, step
    return h


# ------------------------------------------------------- same-name calls


def layup_param_layout(cfg: layup_config):
    nt, nu, tot = C.c_int32(), C.c_int32(), C.c_int64()
    _check(lib().layup_param_layout(C.byref(cfg), C.byref(nt), C.byref(nu), C.byref(tot)))
    return nt.value, nu.value, tot.value


def layup_tensor_layout(cfg: layup_config, index: int) -> dict:
    info = layup_tensor_info()
    _check(lib().layup_tensor_layout(C.byref(cfg), index, C.byref(info)))
    return dict(name=info.name.decode(), offset=info.offset, numel=info.numel, rows=info.rows,
                cols=info.cols, padded_rows=info.padded_rows, unit=info.unit, decay=info.decay)


def layup_workspace_size(cfg: layup_config) -> int:
    n = C.c_size_t()
    _check(lib().layup_workspace_size(C.byref(cfg), C.byref(n)))
    return n.value


def layup_init(cfg: layup_config, bufs: layup_buffers, workspace, workspace_bytes: int,
               compute_stream, update_stream):
    ctx = C.c_void_p()
    _check(lib().layup_init(C.byref(ctx), C.byref(cfg), C.byref(bufs), _ptr(workspace),
                            workspace_bytes, _stream(compute_stream), _stream(update_stream)))
    return ctx


def layup_destroy(ctx):
    lib().layup_destroy(ctx)


def layup_synchronize(ctx):
    _check(lib().layup_synchronize(ctx), ctx)


def layup_refresh_shadow(ctx):
    _check(lib().layup_refresh_shadow(ctx), ctx)


def layup_forward(ctx, tokens, x=None, loss_out=None):
    _check(lib().layup_forward(ctx, _ptr(tokens), _ptr(x), _ptr(loss_out)), ctx)


def layup_layer_backward(ctx, unit: int):
    _check(lib().layup_layer_backward(ctx, unit), ctx)


def layup_unit_update_mix(ctx, unit: int, hp: layup_hparams, alpha: float, peer_slot: int = 0,
                          disagreement=None):
    _check(lib().layup_unit_update_mix(ctx, unit, C.byref(hp), alpha, peer_slot, _ptr(disagreement)), ctx)


def layup_layer_update_mix(ctx, tensors: List[layup_tensor], hp: layup_hparams, alpha: float,
                           disagreement=None, stream=None, mix_mode: int = LAYUP_MIX_PULL):
    arr = (layup_tensor * len(tensors))(*tensors)
    _check(lib().layup_layer_update_mix(ctx, arr, len(tensors), C.byref(hp), alpha, mix_mode,
                                        _ptr(disagreement), _stream(stream)), ctx)


def layup_layer_update_mix_static(tensors: List[layup_tensor], hp: layup_hparams, alpha: float,
                                  disagreement=None, stream=None, mix_mode: int = LAYUP_MIX_PULL):
    arr = (layup_tensor * len(tensors))(*tensors)
    _check(lib().layup_layer_update_mix_static(arr, len(tensors), C.byref(hp), alpha, mix_mode,
                                               _ptr(disagreement), _stream(stream)))


def layup_units_update_mix(tensors: List[layup_tensor], units: List[int], hp: layup_hparams, alpha: float,
                           mix_mode: int = LAYUP_MIX_PULL, trace=None, trace_counter=None,
                           trace_capacity: int = 0, trace_step: int = 0, stream=None):
    arr = (layup_tensor * len(tensors))(*tensors)
    uarr = (C.c_int32 * len(units))(*units)
    _check(lib().layup_units_update_mix(arr, uarr, len(tensors), C.byref(hp), alpha, mix_mode, _ptr(trace),
                                        _ptr(trace_counter), trace_capacity, trace_step, _stream(stream)))


def layup_unit_update_push(ctx, unit: int, hp: layup_hparams, alpha: float, peer_params,
                           peer_params_bf16=None, disagreement=None):
    _check(lib().layup_unit_update_push(ctx, unit, C.byref(hp), alpha, _ptr(peer_params),
                                        _ptr(peer_params_bf16), _ptr(disagreement)), ctx)


def layup_step_ex(ctx, tokens, x, hp: layup_hparams, alpha: float, schedule: int = LAYUP_SCHEDULE_LAYERWISE,
                  mix_mode: int = LAYUP_MIX_PULL, peer_slot: int = 0, push_params=None,
                  push_params_bf16=None, loss_out=None, disagreement=None):
    a = layup_step_args()
    a.tokens, a.x = _ptr(tokens), _ptr(x)
    a.hp = C.addressof(hp)
    a.alpha, a.schedule, a.mix_mode, a.peer_slot = alpha, schedule, mix_mode, peer_slot
    a.push_params, a.push_params_bf16 = _ptr(push_params), _ptr(push_params_bf16)
    a.loss_out, a.disagreement = _ptr(loss_out), _ptr(disagreement)
    _check(lib().layup_step_ex(ctx, C.byref(a)), ctx)


def layup_unit_timeline(ctx, n_units: int):
    """(forward_ms, ready_ms list, applied_ms list) of the last whole step."""
    f, r, a = C.c_float(), (C.c_float * n_units)(), (C.c_float * n_units)()
    _check(lib().layup_unit_timeline(ctx, C.byref(f), r, a), ctx)
    return f.value, list(r), list(a)


def layup_gemm_timing(ctx, enable: bool):
    _check(lib().layup_gemm_timing(ctx, int(enable)), ctx)


def layup_gemm_timing_read(ctx):
    """(total_ms, launches, flops) of the timed backward GEMMs."""
    ms, n, fl = C.c_float(), C.c_int32(), C.c_double()
    _check(lib().layup_gemm_timing_read(ctx, C.byref(ms), C.byref(n), C.byref(fl)), ctx)
    return ms.value, n.value, fl.value


def layup_push_sum_send(w, sender: int, receiver: int) -> float:
    """w: numpy float64 array of the workers' weights, updated in place."""
    assert w.dtype == np.float64 and w.flags.c_contiguous
    alpha = C.c_float()
    _check(lib().layup_push_sum_send(w.ctypes.data, len(w), sender, receiver, C.byref(alpha)))
    return alpha.value


def layup_push_sum_receive(w, sender: int, receiver: int):
    assert w.dtype == np.float64 and w.flags.c_contiguous
    _check(lib().layup_push_sum_receive(w.ctypes.data, len(w), sender, receiver))


def layup_step(ctx, tokens, x, hp: layup_hparams, alpha: float, peer_slot: int = 0, loss_out=None,
               disagreement=None):
    _check(lib().layup_step(ctx, _ptr(tokens), _ptr(x), C.byref(hp), alpha, peer_slot,
                            _ptr(loss_out), _ptr(disagreement)), ctx)


def layup_activation(ctx, which: int, layer: int = 0):
    p, n, dt = C.c_void_p(), C.c_int64(), C.c_int32()
    _check(lib().layup_activation(ctx, which, layer, C.byref(p), C.byref(n), C.byref(dt)), ctx)
    return p.value, n.value, dt.value


def gemm_desc(A, B, C_, M, N, K, lda, ldb, ldc, a_kmajor=True, b_kmajor=True, c_f32=True,
              bias=None, batch=1, inner=1, a_strides=(0, 0), b_strides=(0, 0), c_strides=(0, 0),
              workspace=None, workspace_bytes=0, a_rowsum=None) -> layup_gemm_desc:
    d = layup_gemm_desc()
    d.a_kmajor, d.b_kmajor = int(a_kmajor), int(b_kmajor)
    d.M, d.N, d.K = M, N, K
    d.A, d.lda, d.B, d.ldb, d.C, d.ldc = _ptr(A), lda, _ptr(B), ldb, _ptr(C_), ldc
    d.c_f32, d.batch, d.inner = int(c_f32), batch, inner
    d.bias = _ptr(bias)
    d.a_outer, d.a_inner = a_strides
    d.b_outer, d.b_inner = b_strides
    d.c_outer, d.c_inner = c_strides
    d.workspace, d.workspace_bytes = _ptr(workspace), workspace_bytes
    d.a_rowsum = _ptr(a_rowsum)
    return d


def layup_gemm_bf16(desc: layup_gemm_desc, stream=None):
    _check(lib().layup_gemm_bf16(C.byref(desc), _stream(stream)))


def layup_gemm_f32(desc: layup_gemm_desc, stream=None):
    _check(lib().layup_gemm_f32(C.byref(desc), _stream(stream)))


# ------------------------------------------------------------- harness


class Model:
    """Device buffers of one worker in the library's flat layout (caller
    owned, allocated with torch) plus a context.  Packing numpy dicts into
    the flat buffers and reading tensors back is plain memory plumbing."""

    def __init__(self, cfg: layup_config, optim: str, device="cuda", two_streams: bool = True,
                 trace_capacity: int = 4096, workspace=None, streams=None):
        import torch
        self.torch = torch
        self.cfg = cfg
        self.device = device
        self.n_tensors, self.n_units, self.total = layup_param_layout(cfg)
        self.infos = [layup_tensor_layout(cfg, i) for i in range(self.n_tensors)]
        self.by_name = {t["name"]: t for t in self.infos}
        f32 = dict(dtype=torch.float32, device=device)
        self.params = torch.zeros(self.total, **f32)
        self.grads = torch.zeros(self.total, **f32)
        self.m = torch.zeros(self.total, **f32)
        self.v = torch.zeros(self.total, **f32) if optim == "adamw" else None
        self.peers = torch.zeros(cfg.n_peers * self.total, **f32)
        self.gpt = cfg.model == LAYUP_MODEL_GPT_BF16
        self.params_bf16 = torch.zeros(self.total, dtype=torch.int16, device=device) if self.gpt else None
        self.trace = torch.zeros(2 * trace_capacity, dtype=torch.int32, device=device)
        self.trace_counter = torch.zeros(1, dtype=torch.int32, device=device)
        self.ws_bytes = layup_workspace_size(cfg)
        # a workspace may be shared by contexts whose steps never overlap
        self.workspace = workspace if workspace is not None else \
            torch.empty(self.ws_bytes, dtype=torch.uint8, device=device)
        if streams is not None:
            # contexts on one pair of streams run their steps in call order
            self.compute_stream, self.update_stream = streams
        else:
            self.compute_stream = torch.cuda.Stream(device=device)
            self.update_stream = torch.cuda.Stream(device=device) if two_streams else self.compute_stream
        b = layup_buffers()
        b.params, b.grads, b.m = _ptr(self.params), _ptr(self.grads), _ptr(self.m)
        b.v = _ptr(self.v)
        b.peers = _ptr(self.peers)
        b.params_bf16 = _ptr(self.params_bf16)
        b.trace, b.trace_counter, b.trace_capacity = _ptr(self.trace), _ptr(self.trace_counter), trace_capacity
        self.bufs = b
        self.ctx = layup_init(cfg, b, self.workspace, self.ws_bytes, self.compute_stream,
                              self.update_stream)

    # ---- packing
    def _view(self, flat, name, slot_total=0):
        t = self.by_name[name]
        return flat[slot_total + t["offset"]: slot_total + t["offset"] + t["numel"]]

    def load(self, which: str, tensors: Dict[str, np.ndarray], slot: int = 0):
        torch = self.torch
        flat = {"params": self.params, "m": self.m, "v": self.v, "grads": self.grads,
                "peers": self.peers}[which]
        base = slot * self.total if which == "peers" else 0
        host = torch.zeros(self.total, dtype=torch.float32)
        for name, arr in tensors.items():
            t = self.by_name[name]
            host[t["offset"]: t["offset"] + t["numel"]] = torch.from_numpy(
                np.ascontiguousarray(arr, dtype=np.float32).reshape(-1))
        self.synchronize()
        flat[base: base + self.total].copy_(host.to(self.device))
        torch.cuda.synchronize()
        if which == "params" and self.gpt:
            layup_refresh_shadow(self.ctx)
            self.synchronize()

    def read(self, which: str, slot: int = 0) -> Dict[str, np.ndarray]:
        flat = {"params": self.params, "m": self.m, "v": self.v, "grads": self.grads,
                "peers": self.peers}[which]
        base = slot * self.total if which == "peers" else 0
        self.synchronize()
        host = flat[base: base + self.total].cpu().numpy()
        out = {}
        for t in self.infos:
            a = host[t["offset"]: t["offset"] + t["numel"]]
            out[t["name"]] = a.reshape(t["rows"], t["cols"]) if t["cols"] > 1 else a.copy()
        return out

    def read_trace(self):
        self.synchronize()
        n = int(self.trace_counter.item())
        tr = self.trace[: 2 * n].cpu().numpy().reshape(-1, 2)
        return [tuple(map(int, r)) for r in tr]

    def activation(self, which: int, layer: int = 0):
        """Copy of a saved activation as a float32 numpy array."""
        torch = self.torch
        p, n, dt = layup_activation(self.ctx, which, layer)
        self.synchronize()
        dtype = torch.int16 if dt == 1 else torch.float32
        out = torch.empty(n, dtype=dtype, device=self.device)
        # device-to-device copy through the byte view of the workspace
        off = p - self.workspace.data_ptr()
        nbytes = n * (2 if dt == 1 else 4)
        out.view(torch.uint8).copy_(self.workspace[off: off + nbytes])
        if dt == 1:
            out = (out.to(torch.int32) << 16).view(torch.float32)
        return out.cpu().numpy()

    def synchronize(self):
        layup_synchronize(self.ctx)

    def close(self):
        if self.ctx:
            layup_destroy(self.ctx)
            self.ctx = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass
