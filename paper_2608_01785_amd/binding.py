"""ctypes binding of ``libhorizon.so``: argument marshalling only.

Every function here has the name of the C entry point it calls and only
converts arguments (torch tensors -> device pointers, Python sequences ->
host arrays, status codes -> exceptions).  All computation happens in the
library's HIP kernels.  Importing this module fails loudly when the library
has not been built.
"""
from __future__ import annotations

import ctypes
import os
from typing import Dict, List, Optional, Sequence, Tuple

import numpy as np

_LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libhorizon.so")

HS_OK, HS_ERR_INVALID_ARG, HS_ERR_UNSUPPORTED, HS_ERR_BUDGET, HS_ERR_WORKSPACE, HS_ERR_HIP, HS_ERR_INTERNAL = range(7)
HS_ROLE_SHARED, HS_ROLE_DOWN = 0, 1

SYMBOLS = (
    "hs_status_string", "hs_last_error", "hs_default_topology", "hs_cu_partition", "hs_plan_metadata",
    "hs_context_create", "hs_context_topology", "hs_context_stream", "hs_context_masks",
    "hs_context_destroy", "hs_workspace_size", "hs_workspace_size_paged", "hs_shared_stage_forward",
    "hs_shared_stage_forward_mrope", "hs_downstream_decode_step_mrope", "hs_downstream_decode_step",
    "hs_downstream_decode_step_noalloc", "hs_decode_graph_create", "hs_decode_graph_launch",
    "hs_decode_graph_destroy", "hs_dit_workspace_size", "hs_dit_forward",
    "hs_probe_hw_ids", "hs_timing_enable", "hs_timing_read", "hs_timing_read_clock", "hs_convert_weights_f16",
    "hs_controller_create", "hs_controller_step", "hs_controller_destroy", "hs_pressure_sample",
    "hs_temporal_create", "hs_temporal_step", "hs_temporal_destroy",
)
HS_WEIGHTS_BF16, HS_WEIGHTS_F16 = 0, 1

KERNEL_KINDS = {"rmsnorm": 0, "qkv": 1, "attention": 2, "decode_attn": 3, "o_proj": 4, "gate_up": 5,
                "down": 6, "rope_table": 7, "modulation": 8, "ln_mod": 9, "mlp_up": 10, "mlp_down": 11}


class LayerCfg(ctypes.Structure):
    _fields_ = [("hidden", ctypes.c_int32), ("n_q_heads", ctypes.c_int32), ("n_kv_heads", ctypes.c_int32),
                ("head_dim", ctypes.c_int32), ("ffn", ctypes.c_int32), ("rms_eps", ctypes.c_float),
                ("rope_base", ctypes.c_float), ("mrope_sections", ctypes.c_int32 * 3)]

    @classmethod
    def of(cls, s) -> "LayerCfg":
        sec = tuple(getattr(s, "mrope_sections", (0, 0, 0)))
        return cls(s.hidden, s.n_q_heads, s.n_kv_heads, s.head_dim, s.ffn, s.rms_eps, s.rope_base,
                   (ctypes.c_int32 * 3)(*sec))


MATRICES = ("w_qkv", "w_o", "w_gate_up", "w_down")
DIT_MATRICES = ("w_qkv", "w_o", "w_fc1", "w_fc2")   # the DiT projections fp16 preparation applies to
DIT_FIELDS = ("w_ada", "b_ada", "w_qkv", "b_qkv", "w_o", "b_o", "w_fc1", "b_fc1", "w_fc2", "b_fc2")


class DitCfg(ctypes.Structure):
    _fields_ = [("hidden", ctypes.c_int32), ("n_heads", ctypes.c_int32), ("head_dim", ctypes.c_int32),
                ("mlp", ctypes.c_int32), ("ln_eps", ctypes.c_float)]

    @classmethod
    def of(cls, s) -> "DitCfg":
        return cls(s.hidden, s.n_heads, s.head_dim, s.mlp, s.ln_eps)


class DitWeights(ctypes.Structure):
    _fields_ = [(n, ctypes.c_void_p) for n in DIT_FIELDS] + [("format", ctypes.c_int32)]


class LayerWeights(ctypes.Structure):
    _fields_ = [(n, ctypes.c_void_p) for n in ("ln1", "w_qkv", "w_o", "ln2", "w_gate_up", "w_down")] + \
               [("format", ctypes.c_int32), ("b_qkv", ctypes.c_void_p)]


class KvCache(ctypes.Structure):
    _fields_ = [("k", ctypes.POINTER(ctypes.c_void_p)), ("v", ctypes.POINTER(ctypes.c_void_p)),
                ("n_slots", ctypes.c_int32), ("max_ctx", ctypes.c_int32),
                ("block_table", ctypes.POINTER(ctypes.c_int32)), ("pages_per_seq", ctypes.c_int32)]


class Topology(ctypes.Structure):
    _fields_ = [("n_cus", ctypes.c_int32), ("n_xcc", ctypes.c_int32), ("xcc", ctypes.c_uint8 * 256),
                ("se", ctypes.c_uint8 * 256), ("cu", ctypes.c_uint8 * 256)]


class ControllerCfg(ctypes.Structure):
    _fields_ = [("total_cus", ctypes.c_int32), ("aggressive_cus", ctypes.c_int32),
                ("ladder", ctypes.POINTER(ctypes.c_int32)), ("n_ladder", ctypes.c_int32),
                ("ewma_weight", ctypes.c_double), ("saturation", ctypes.c_double),
                ("hysteresis_steps", ctypes.c_int32)]


HS_PATH_SHORT, HS_PATH_LONG = 0, 1
HS_WORK_PREFILL, HS_WORK_DECODE = 0, 1


class TemporalCfg(ctypes.Structure):
    _fields_ = [("n_min", ctypes.c_int32), ("n_max", ctypes.c_int32), ("m", ctypes.c_int32),
                ("u_guard", ctypes.c_double), ("long_cap", ctypes.c_int32)]


class RequestView(ctypes.Structure):
    _fields_ = [("path", ctypes.c_int32), ("work", ctypes.c_int32), ("deadline", ctypes.c_double),
                ("remaining", ctypes.c_double)]


class TemporalStepInfo(ctypes.Structure):
    _fields_ = [("step", ctypes.c_int64), ("n", ctypes.c_int32), ("phase", ctypes.c_int32),
                ("n_protected", ctypes.c_int32), ("n_hidden", ctypes.c_int32), ("n_capped", ctypes.c_int32)]


class Split(ctypes.Structure):
    _fields_ = [("shared_cus", ctypes.c_int32), ("down_cus", ctypes.c_int32), ("level", ctypes.c_int32),
                ("changed", ctypes.c_int32), ("pressure", ctypes.c_double), ("rho", ctypes.c_double)]


class HorizonError(RuntimeError):
    def __init__(self, status: int, msg: str):
        super().__init__(f"{_status_name(status)}: {msg}")
        self.status = status


_lib = None


def lib() -> ctypes.CDLL:
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB_PATH):
            raise ImportError(f"{_LIB_PATH} is missing: build it with python -m paper_2608_01785_amd.build")
        L = ctypes.CDLL(_LIB_PATH)
        vp, i32, u32p, i32p = ctypes.c_void_p, ctypes.c_int32, ctypes.POINTER(ctypes.c_uint32), ctypes.POINTER(ctypes.c_int32)
        L.hs_status_string.restype = ctypes.c_char_p
        L.hs_status_string.argtypes = [ctypes.c_int]
        L.hs_last_error.restype = ctypes.c_char_p
        L.hs_last_error.argtypes = []
        sigs = {
            "hs_default_topology": [i32, i32, ctypes.POINTER(Topology)],
            "hs_cu_partition": [ctypes.POINTER(Topology), i32, u32p, u32p],
            "hs_plan_metadata": [i32p, i32p, i32, i32p, i32p],
            "hs_context_create": [i32, i32p, i32, ctypes.POINTER(Topology), ctypes.POINTER(vp)],
            "hs_context_topology": [vp, ctypes.POINTER(Topology)],
            "hs_context_stream": [vp, i32, i32, ctypes.POINTER(vp)],
            "hs_context_masks": [vp, i32, u32p, u32p],
            "hs_context_destroy": [vp],
            "hs_workspace_size": [ctypes.POINTER(LayerCfg), i32, i32, i32, ctypes.POINTER(ctypes.c_size_t)],
            "hs_workspace_size_paged": [ctypes.POINTER(LayerCfg), i32, i32, i32, i32,
                                        ctypes.POINTER(ctypes.c_size_t)],
            "hs_shared_stage_forward": [vp, ctypes.POINTER(LayerCfg), ctypes.POINTER(LayerWeights), i32, vp, vp,
                                        i32p, i32p, i32, ctypes.POINTER(KvCache), i32, vp, vp, ctypes.c_size_t],
            "hs_shared_stage_forward_mrope": [vp, ctypes.POINTER(LayerCfg), ctypes.POINTER(LayerWeights), i32, vp,
                                              vp, i32p, i32p, i32, ctypes.POINTER(KvCache), i32p, i32, vp, vp,
                                              ctypes.c_size_t],
            "hs_downstream_decode_step_mrope": [vp, ctypes.POINTER(LayerCfg), ctypes.POINTER(LayerWeights), i32, vp,
                                                vp, ctypes.POINTER(KvCache), i32p, i32p, i32, i32, vp, vp,
                                                ctypes.c_size_t],
            "hs_downstream_decode_step": [vp, ctypes.POINTER(LayerCfg), ctypes.POINTER(LayerWeights), i32, vp, vp,
                                          ctypes.POINTER(KvCache), i32p, i32, i32, vp, vp, ctypes.c_size_t],
            "hs_downstream_decode_step_noalloc": [vp, ctypes.POINTER(LayerCfg), ctypes.POINTER(LayerWeights), i32,
                                                  vp, vp, ctypes.POINTER(KvCache), i32p, i32, i32, vp],
            "hs_decode_graph_create": [vp, ctypes.POINTER(LayerCfg), ctypes.POINTER(LayerWeights), i32, vp, vp,
                                       ctypes.POINTER(KvCache), i32, i32, vp, vp, ctypes.c_size_t,
                                       ctypes.POINTER(vp)],
            "hs_decode_graph_launch": [vp, i32p, i32p],
            "hs_dit_workspace_size": [ctypes.POINTER(DitCfg), i32, i32, ctypes.POINTER(ctypes.c_size_t)],
            "hs_dit_forward": [vp, ctypes.POINTER(DitCfg), ctypes.POINTER(DitWeights), i32, vp, vp, vp, i32p, i32,
                               i32, vp, vp, ctypes.c_size_t],
            "hs_decode_graph_destroy": [vp],
            "hs_probe_hw_ids": [vp, vp, i32, vp],
            "hs_timing_enable": [vp, i32],
            "hs_timing_read": [vp, i32, ctypes.POINTER(ctypes.c_double), i32p],
            "hs_timing_read_clock": [vp, i32, ctypes.POINTER(ctypes.c_double), i32p],
            "hs_convert_weights_f16": [vp, vp, vp, ctypes.c_int64, ctypes.c_int64, vp],
            "hs_controller_create": [ctypes.POINTER(ControllerCfg), ctypes.POINTER(vp)],
            "hs_controller_step": [vp, i32, ctypes.c_double, ctypes.POINTER(Split)],
            "hs_controller_destroy": [vp],
            "hs_pressure_sample": [i32, ctypes.POINTER(ctypes.c_double)],
            "hs_temporal_create": [ctypes.POINTER(TemporalCfg), ctypes.POINTER(vp)],
            "hs_temporal_step": [vp, ctypes.c_double, ctypes.POINTER(RequestView), i32,
                                 ctypes.POINTER(ctypes.c_uint8), ctypes.POINTER(TemporalStepInfo)],
            "hs_temporal_destroy": [vp],
        }
        for name, args in sigs.items():
            fn = getattr(L, name)
            fn.restype = ctypes.c_int
            fn.argtypes = args
        _lib = L
    return _lib


def _status_name(s: int) -> str:
    try:
        return lib().hs_status_string(s).decode()
    except Exception:  # pragma: no cover - library missing
        return str(s)


def _check(status: int) -> None:
    if status != HS_OK:
        raise HorizonError(status, lib().hs_last_error().decode())


def hs_last_error() -> str:
    return lib().hs_last_error().decode()


def _i32_array(values) -> Optional[ctypes.Array]:
    if values is None:
        return None
    a = np.ascontiguousarray(np.asarray(values, dtype=np.int32))
    return (ctypes.c_int32 * len(a))(*a.tolist())


def _ptr(t) -> Optional[int]:
    if t is None:
        return None
    if isinstance(t, int):
        return t
    return t.data_ptr()


# --------------------------------------------------------------------------- host-only calls

def hs_default_topology(n_cus: int = 256, n_xcc: int = 8) -> Topology:
    t = Topology()
    _check(lib().hs_default_topology(n_cus, n_xcc, ctypes.byref(t)))
    return t


def topology_from_lists(xcc, se, cu, n_xcc: int) -> Topology:
    t = Topology()
    t.n_cus, t.n_xcc = len(xcc), n_xcc
    for i in range(len(xcc)):
        t.xcc[i], t.se[i], t.cu[i] = int(xcc[i]), int(se[i]), int(cu[i])
    return t


def hs_cu_partition(topo: Topology, shared_cus: int) -> Tuple[List[int], List[int]]:
    sh = (ctypes.c_uint32 * 8)()
    dn = (ctypes.c_uint32 * 8)()
    _check(lib().hs_cu_partition(ctypes.byref(topo), shared_cus, sh, dn))
    return list(sh), list(dn)


def hs_plan_metadata(seq_offsets, ctx_lens=None) -> Tuple[np.ndarray, np.ndarray]:
    off = _i32_array(seq_offsets)
    T = int(off[len(off) - 1]) if len(off) else 0
    pos = (ctypes.c_int32 * max(T, 1))()
    sid = (ctypes.c_int32 * max(T, 1))()
    _check(lib().hs_plan_metadata(off, _i32_array(ctx_lens), len(off) - 1, pos, sid))
    return np.frombuffer(pos, dtype=np.int32)[:T].copy(), np.frombuffer(sid, dtype=np.int32)[:T].copy()


def hs_workspace_size(cfg, max_tokens: int, max_seqs: int, max_pos: int) -> int:
    n = ctypes.c_size_t(0)
    _check(lib().hs_workspace_size(ctypes.byref(LayerCfg.of(cfg)), max_tokens, max_seqs, max_pos, ctypes.byref(n)))
    return int(n.value)


def hs_workspace_size_paged(cfg, max_tokens: int, max_seqs: int, max_pos: int, page_positions: int) -> int:
    n = ctypes.c_size_t(0)
    _check(lib().hs_workspace_size_paged(ctypes.byref(LayerCfg.of(cfg)), max_tokens, max_seqs, max_pos,
                                         page_positions, ctypes.byref(n)))
    return int(n.value)


# --------------------------------------------------------------------------- spatial controller

class Controller:
    """Owns an hs_controller handle (the C object copies the configuration)."""

    def __init__(self, total_cus: int, aggressive_cus: int, ladder: Sequence[int], ewma_weight: float,
                 saturation: float, hysteresis_steps: int = 1):
        self._ladder = _i32_array(ladder)
        cfg = ControllerCfg(total_cus, aggressive_cus, self._ladder, len(ladder), ewma_weight, saturation,
                            hysteresis_steps)
        h = ctypes.c_void_p()
        _check(lib().hs_controller_create(ctypes.byref(cfg), ctypes.byref(h)))
        self.handle = h

    def close(self):
        if self.handle:
            lib().hs_controller_destroy(self.handle)
            self.handle = None

    def __del__(self):  # pragma: no cover
        try:
            self.close()
        except Exception:
            pass


def hs_controller_step(ctrl: Controller, downstream_active: bool, sample: float) -> Split:
    out = Split()
    _check(lib().hs_controller_step(ctrl.handle, 1 if downstream_active else 0, float(sample), ctypes.byref(out)))
    return out


class Temporal:
    """Owns an hs_temporal handle (shared-stage path rotation)."""

    def __init__(self, n_min: int = 2, n_max: int = 8, m: int = 2, u_guard: float = 1.0, long_cap: int = -1):
        cfg = TemporalCfg(n_min, n_max, m, u_guard, long_cap)
        h = ctypes.c_void_p()
        _check(lib().hs_temporal_create(ctypes.byref(cfg), ctypes.byref(h)))
        self.handle = h

    def close(self):
        if self.handle:
            lib().hs_temporal_destroy(self.handle)
            self.handle = None

    def __del__(self):  # pragma: no cover
        try:
            self.close()
        except Exception:
            pass


def hs_temporal_step(sched: Temporal, now: float, requests) -> Tuple[np.ndarray, TemporalStepInfo]:
    """requests: sequence of (path, work, deadline, remaining); returns (visible bool array, step info)."""
    n = len(requests)
    arr = (RequestView * max(n, 1))(*[RequestView(int(p), int(w), float(d), float(r)) for p, w, d, r in requests])
    vis = np.zeros(max(n, 1), np.uint8)
    info = TemporalStepInfo()
    _check(lib().hs_temporal_step(sched.handle, float(now), arr, n, vis.ctypes.data_as(ctypes.POINTER(ctypes.c_uint8)),
                                  ctypes.byref(info)))
    return vis[:n].astype(bool), info


def hs_pressure_sample(device: int = 0) -> float:
    v = ctypes.c_double(0.0)
    _check(lib().hs_pressure_sample(device, ctypes.byref(v)))
    return float(v.value)


# --------------------------------------------------------------------------- context

class Context:
    """Owns an ``hs_context`` (CU-masked stream ladder)."""

    def __init__(self, device: int = 0, budgets: Sequence[int] = (64, 128, 192, 256),
                 topo: Optional[Topology] = None):
        h = ctypes.c_void_p()
        b = _i32_array(list(budgets))
        _check(lib().hs_context_create(device, b, len(budgets), ctypes.byref(topo) if topo else None,
                                       ctypes.byref(h)))
        self.handle = h
        self.device = device

    def close(self):
        if self.handle:
            lib().hs_context_destroy(self.handle)
            self.handle = None

    def __del__(self):  # pragma: no cover
        try:
            self.close()
        except Exception:
            pass


def hs_context_create(device: int = 0, budgets=(64, 128, 192, 256), topo=None) -> Context:
    return Context(device, budgets, topo)


def hs_context_stream(ctx: Context, cu_budget: int, role: int = HS_ROLE_SHARED) -> int:
    s = ctypes.c_void_p()
    _check(lib().hs_context_stream(ctx.handle, cu_budget, role, ctypes.byref(s)))
    return int(s.value)


def hs_context_masks(ctx: Context, cu_budget: int) -> Tuple[List[int], List[int]]:
    sh = (ctypes.c_uint32 * 8)()
    dn = (ctypes.c_uint32 * 8)()
    _check(lib().hs_context_masks(ctx.handle, cu_budget, sh, dn))
    return list(sh), list(dn)


def hs_context_topology(ctx: Context) -> Topology:
    t = Topology()
    _check(lib().hs_context_topology(ctx.handle, ctypes.byref(t)))
    return t


def hs_context_destroy(ctx: Context) -> None:
    ctx.close()


# --------------------------------------------------------------------------- compute calls

def _weights_array(weights: List[Dict[str, object]]):
    arr = (LayerWeights * len(weights))()
    for i, w in enumerate(weights):
        for name in ("ln1", "w_qkv", "w_o", "ln2", "w_gate_up", "w_down"):
            setattr(arr[i], name, _ptr(w[name]))
        arr[i].format = int(w.get("format", HS_WEIGHTS_BF16))
        arr[i].b_qkv = _ptr(w.get("b_qkv"))
    return arr


def _kv_struct(kv) -> Optional[KvCache]:
    """kv: None, (k_list, v_list, n_slots, max_ctx) of device tensors / pointers, or the same
    plus a host block table [n_seqs, pages_per_seq] of slot indices (a paged cache)."""
    if kv is None:
        return None
    k_list, v_list, n_slots, max_ctx = kv[:4]
    table = kv[4] if len(kv) > 4 else None
    kp = (ctypes.c_void_p * len(k_list))(*[_ptr(t) for t in k_list])
    vp = (ctypes.c_void_p * len(v_list))(*[_ptr(t) for t in v_list])
    tp, pps = None, 0
    if table is not None:
        table = np.ascontiguousarray(table, dtype=np.int32)
        assert table.ndim == 2
        pps = table.shape[1]
        tp = table.ctypes.data_as(ctypes.POINTER(ctypes.c_int32))
    s = KvCache(ctypes.cast(kp, ctypes.POINTER(ctypes.c_void_p)), ctypes.cast(vp, ctypes.POINTER(ctypes.c_void_p)),
                n_slots, max_ctx, tp, pps)
    s._keep = (kp, vp, table)
    return s


def hs_shared_stage_forward(ctx: Context, cfg, weights, x_in, x_out, seq_offsets, ctx_lens=None, kv=None,
                            cu_budget: int = 256, stream=None, workspace=None, ws_bytes: Optional[int] = None) -> None:
    warr = _weights_array(weights)
    off = _i32_array(seq_offsets)
    kvs = _kv_struct(kv)
    if ws_bytes is None:
        ws_bytes = workspace.numel() * workspace.element_size()
    _check(lib().hs_shared_stage_forward(
        ctx.handle, ctypes.byref(LayerCfg.of(cfg)), warr, len(weights), _ptr(x_in), _ptr(x_out), off,
        _i32_array(ctx_lens), len(off) - 1, ctypes.byref(kvs) if kvs is not None else None, cu_budget,
        _ptr(stream), _ptr(workspace), ws_bytes))


def hs_shared_stage_forward_mrope(ctx: Context, cfg, weights, x_in, x_out, seq_offsets, positions3, ctx_lens=None,
                                  kv=None, cu_budget: int = 256, stream=None, workspace=None,
                                  ws_bytes: Optional[int] = None) -> None:
    """positions3: host int array [3, T] (temporal, height, width position of every packed row)."""
    warr = _weights_array(weights)
    off = _i32_array(seq_offsets)
    kvs = _kv_struct(kv)
    pos = np.ascontiguousarray(positions3, dtype=np.int32)
    n_rows = int(off[len(off) - 1])
    if pos.shape != (3, n_rows):
        raise ValueError(f"positions3 has shape {pos.shape}, expected (3, {n_rows})")
    if ws_bytes is None:
        ws_bytes = workspace.numel() * workspace.element_size()
    _check(lib().hs_shared_stage_forward_mrope(
        ctx.handle, ctypes.byref(LayerCfg.of(cfg)), warr, len(weights), _ptr(x_in), _ptr(x_out), off,
        _i32_array(ctx_lens), len(off) - 1, ctypes.byref(kvs) if kvs is not None else None,
        pos.ctypes.data_as(ctypes.POINTER(ctypes.c_int32)), cu_budget, _ptr(stream), _ptr(workspace), ws_bytes))


def hs_downstream_decode_step_mrope(ctx: Context, cfg, weights, x_in, x_out, kv, kv_lens, positions3, cu_budget: int,
                                    stream=None, workspace=None, ws_bytes: Optional[int] = None) -> None:
    """positions3: host int array [3, batch] (the new rows' temporal, height and width positions)."""
    warr = _weights_array(weights)
    kvs = _kv_struct(kv)
    lens = _i32_array(kv_lens)
    pos = np.ascontiguousarray(positions3, dtype=np.int32)
    if pos.shape != (3, len(lens)):
        raise ValueError(f"positions3 has shape {pos.shape}, expected (3, {len(lens)})")
    if ws_bytes is None:
        ws_bytes = workspace.numel() * workspace.element_size()
    _check(lib().hs_downstream_decode_step_mrope(
        ctx.handle, ctypes.byref(LayerCfg.of(cfg)), warr, len(weights), _ptr(x_in), _ptr(x_out), ctypes.byref(kvs),
        lens, pos.ctypes.data_as(ctypes.POINTER(ctypes.c_int32)), len(lens), cu_budget, _ptr(stream),
        _ptr(workspace), ws_bytes))


def hs_downstream_decode_step(ctx: Context, cfg, weights, x_in, x_out, kv, kv_lens, cu_budget: int,
                              stream=None, workspace=None, ws_bytes: Optional[int] = None) -> None:
    warr = _weights_array(weights)
    kvs = _kv_struct(kv)
    lens = _i32_array(kv_lens)
    if ws_bytes is None:
        ws_bytes = workspace.numel() * workspace.element_size()
    _check(lib().hs_downstream_decode_step(
        ctx.handle, ctypes.byref(LayerCfg.of(cfg)), warr, len(weights), _ptr(x_in), _ptr(x_out),
        ctypes.byref(kvs), lens, len(lens), cu_budget, _ptr(stream), _ptr(workspace), ws_bytes))


def hs_downstream_decode_step_noalloc(ctx: Context, cfg, weights, x_in, x_out, kv, kv_lens, cu_budget: int,
                                      stream=None) -> None:
    """The decode step on the library's static scratch (no workspace argument)."""
    warr = _weights_array(weights)
    kvs = _kv_struct(kv)
    lens = _i32_array(kv_lens)
    _check(lib().hs_downstream_decode_step_noalloc(
        ctx.handle, ctypes.byref(LayerCfg.of(cfg)), warr, len(weights), _ptr(x_in), _ptr(x_out),
        ctypes.byref(kvs) if kvs is not None else None, lens, len(lens), cu_budget, _ptr(stream)))


class DecodeGraph:
    """A captured decode step (hs_decode_graph_create); launch(kv_lens[, block_table]) replays it.

    kv as for hs_downstream_decode_step; with a block table there (any contents of the right
    shape [batch, pages_per_seq]) the graph addresses a paged cache and every launch takes
    that step's table."""

    def __init__(self, ctx: Context, cfg, weights, x_in, x_out, kv, batch: int, cu_budget: int,
                 stream=None, workspace=None, ws_bytes: Optional[int] = None):
        self.handle = None
        self._ctx = ctx
        warr = _weights_array(weights)
        kvs = _kv_struct(kv)
        if ws_bytes is None:
            ws_bytes = workspace.numel() * workspace.element_size()
        h = ctypes.c_void_p()
        _check(lib().hs_decode_graph_create(
            ctx.handle, ctypes.byref(LayerCfg.of(cfg)), warr, len(weights), _ptr(x_in), _ptr(x_out),
            ctypes.byref(kvs), batch, cu_budget, _ptr(stream), _ptr(workspace), ws_bytes, ctypes.byref(h)))
        self.handle = h
        self.batch = batch

    def launch(self, kv_lens, block_table=None) -> None:
        lens = _i32_array(kv_lens)
        assert len(lens) == self.batch, (len(lens), self.batch)
        tp = None
        if block_table is not None:
            table = np.ascontiguousarray(block_table, dtype=np.int32)
            assert table.ndim == 2 and table.shape[0] == self.batch
            tp = table.ctypes.data_as(ctypes.POINTER(ctypes.c_int32))
        _check(lib().hs_decode_graph_launch(self.handle, lens, tp))

    def close(self) -> None:
        if self.handle is not None:
            _check(lib().hs_decode_graph_destroy(self.handle))
            self.handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


def hs_dit_workspace_size(cfg, max_tokens: int, max_seqs: int) -> int:
    n = ctypes.c_size_t(0)
    _check(lib().hs_dit_workspace_size(ctypes.byref(DitCfg.of(cfg)), max_tokens, max_seqs, ctypes.byref(n)))
    return int(n.value)


def _dit_weights_array(weights):
    arr = (DitWeights * len(weights))()
    for i, w in enumerate(weights):
        for name in DIT_FIELDS:
            setattr(arr[i], name, _ptr(w[name]))
        arr[i].format = int(w.get("format", HS_WEIGHTS_BF16))
    return arr


def hs_dit_forward(ctx: Context, cfg, weights, x_in, x_out, cond, seq_offsets, cu_budget: int, stream=None,
                   workspace=None, ws_bytes: Optional[int] = None) -> None:
    """DiT blocks over a packed ragged batch on the downstream side (cu_budget = its CUs)."""
    warr = _dit_weights_array(weights)
    off = _i32_array(seq_offsets)
    if ws_bytes is None:
        ws_bytes = workspace.numel() * workspace.element_size()
    _check(lib().hs_dit_forward(ctx.handle, ctypes.byref(DitCfg.of(cfg)), warr, len(weights), _ptr(x_in),
                                _ptr(x_out), _ptr(cond), off, len(off) - 1, cu_budget, _ptr(stream),
                                _ptr(workspace), ws_bytes))


def hs_probe_hw_ids(ctx: Context, stream, n_groups: int, out_ids) -> None:
    _check(lib().hs_probe_hw_ids(ctx.handle, _ptr(stream), n_groups, _ptr(out_ids)))


def hs_timing_enable(ctx: Context, enable: bool = True) -> None:
    _check(lib().hs_timing_enable(ctx.handle, 1 if enable else 0))


def hs_timing_read_clock(ctx: Context, kind) -> Tuple[float, int]:
    """(average shader clock in MHz, launches with clock records) of one kernel kind."""
    k = KERNEL_KINDS[kind] if isinstance(kind, str) else int(kind)
    mhz = ctypes.c_double(0)
    n = ctypes.c_int32(0)
    _check(lib().hs_timing_read_clock(ctx.handle, k, ctypes.byref(mhz), ctypes.byref(n)))
    return float(mhz.value), int(n.value)


def hs_timing_read(ctx: Context, kind) -> Tuple[float, int]:
    """(summed milliseconds, launches) of one kernel kind since timing was enabled."""
    k = KERNEL_KINDS[kind] if isinstance(kind, str) else int(kind)
    ms = ctypes.c_double(0)
    n = ctypes.c_int32(0)
    _check(lib().hs_timing_read(ctx.handle, k, ctypes.byref(ms), ctypes.byref(n)))
    return float(ms.value), int(n.value)


def hs_convert_weights_f16(ctx: Context, src, dst, rows: Optional[int] = None, cols: Optional[int] = None,
                           stream=None) -> None:
    """bf16 [rows, cols] -> fp16 panel-major [cols / 32][rows][32] (shape taken from src if not given)."""
    if rows is None or cols is None:
        rows, cols = int(src.shape[0]), int(src.shape[1])
    _check(lib().hs_convert_weights_f16(ctx.handle, _ptr(src), _ptr(dst), int(rows), int(cols), _ptr(stream)))
