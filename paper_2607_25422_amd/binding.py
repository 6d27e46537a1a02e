"""Python binding of libskip.so (ctypes; argument marshalling only).

Every function here checks tensor placement/shape/dtype, reads raw device
pointers and the current HIP stream from torch, and calls the C entry point
of the same name.  All arithmetic happens in the library's HIP kernels; there
is no fallback path.  If the library is missing, importing this module raises.

Offsets arrays are given twice: as host numpy arrays (to fill the problem
description, which the C ABI takes by value on the host) and as device int32
tensors (which the kernels read).  ``Offsets.to_device`` makes the pair.
"""
from __future__ import annotations

import ctypes
import math
import os
from dataclasses import dataclass
from typing import Optional, Tuple

import numpy as np
import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "lib", "libskip.so")

SKIP_OK, SKIP_ERR_INVALID_ARG, SKIP_ERR_UNSUPPORTED, SKIP_ERR_WORKSPACE, SKIP_ERR_HIP = range(5)
SKIP_F32, SKIP_BF16 = 0, 1

ENTRY_POINTS = ("skip_abi_version", "skip_status_string", "skip_workspace_bytes",
                "skip_prune_topk", "skip_bipartite_xattn", "skip_route_fused",
                "skip_route_fused_profiled", "skip_workspace_bytes_mlp",
                "skip_prune_topk_mlp", "skip_workspace_bytes_gate", "skip_skv_gate",
                "skip_bipartite_xattn_masked", "skip_route_fused_gated",
                "skip_workspace_bytes_regions", "skip_region_kmeans",
                "skip_workspace_bytes_project", "skip_gather_project",
                "skip_bipartite_xattn_proj", "skip_pack_projection",
                "skip_gather_project_packed", "skip_route_fused_noalloc",
                "skip_workspace_bytes_project_keys", "skip_project_passage_keys")
FUSED_STAGES = ("pool", "score", "edge_cos", "edge_select", "attention")


class SkipError(RuntimeError):
    def __init__(self, status: int, where: str):
        self.status = status
        super().__init__(f"{where}: {status_string(status)}")


class SkipProblem(ctypes.Structure):
    _fields_ = [
        ("dtype", ctypes.c_int32), ("B", ctypes.c_int32), ("N", ctypes.c_int32),
        ("d", ctypes.c_int32), ("H", ctypes.c_int32), ("d_h", ctypes.c_int32),
        ("total_qtok", ctypes.c_int32), ("k_max", ctypes.c_int32),
        ("total_kept", ctypes.c_int32), ("P_max", ctypes.c_int32),
        ("total_passages", ctypes.c_int32), ("total_tokens", ctypes.c_int32),
        ("L_max", ctypes.c_int32), ("total_edges", ctypes.c_int32),
        ("avg_degree", ctypes.c_double), ("sm_scale", ctypes.c_float),
        ("o_f32", ctypes.c_int32), ("edge_rule", ctypes.c_int32),
        ("edge_metric", ctypes.c_int32), ("edge_beta", ctypes.c_double),
    ]


class SkipQvsMlp(ctypes.Structure):
    """skip_qvs_mlp_t: the main-text scorer's weights (device pointers)."""
    _fields_ = [
        ("hidden", ctypes.c_int32), ("reserved", ctypes.c_int32),
        ("W1", ctypes.c_void_p), ("b1", ctypes.c_void_p), ("w2", ctypes.c_void_p),
        ("b2", ctypes.c_double),
    ]


class SkipSkvGate(ctypes.Structure):
    """skip_skv_gate_t: the passage gate's weights (device pointers) and cuts."""
    _fields_ = [
        ("hidden", ctypes.c_int32), ("reserved", ctypes.c_int32),
        ("W", ctypes.c_void_p), ("b1", ctypes.c_void_p), ("w2", ctypes.c_void_p),
        ("b2", ctypes.c_double), ("tau", ctypes.c_double), ("rho", ctypes.c_double),
    ]


# skip_edge_rule_t and skip_edge_metric_t, by the names the oracle uses
EDGE_RULES = {"question": 0, "row": 1, "fraction": 2}
EDGE_METRICS = {"cosine": 0, "dot": 1}


def _load() -> ctypes.CDLL:
    if not os.path.exists(LIB_PATH):
        raise ImportError(
            f"{LIB_PATH} is missing: build it with `python -m paper_2607_25422_amd.build` "
            "(the routing core has no non-HIP implementation)")
    lib = ctypes.CDLL(LIB_PATH)
    P = ctypes.POINTER(SkipProblem)
    vp, i32p = ctypes.c_void_p, ctypes.c_void_p
    lib.skip_abi_version.restype = ctypes.c_int32
    lib.skip_abi_version.argtypes = []
    lib.skip_status_string.restype = ctypes.c_char_p
    lib.skip_status_string.argtypes = [ctypes.c_int]
    lib.skip_workspace_bytes.restype = ctypes.c_int
    lib.skip_workspace_bytes.argtypes = [P, ctypes.POINTER(ctypes.c_size_t)]
    lib.skip_prune_topk.restype = ctypes.c_int
    lib.skip_prune_topk.argtypes = [P, vp, vp, i32p, vp, i32p, i32p, vp, vp, vp,
                                    ctypes.c_size_t, vp]
    lib.skip_bipartite_xattn.restype = ctypes.c_int
    lib.skip_bipartite_xattn.argtypes = [P, vp, i32p, vp, vp, i32p, i32p, vp, i32p, i32p,
                                         vp, vp, i32p, i32p, vp, ctypes.c_size_t, vp]
    lib.skip_route_fused.restype = ctypes.c_int
    lib.skip_route_fused.argtypes = [P, vp, vp, i32p, vp, i32p, vp, vp, i32p, i32p, vp,
                                     i32p, vp, vp, vp, ctypes.c_size_t, vp]
    M = ctypes.POINTER(SkipQvsMlp)
    lib.skip_workspace_bytes_mlp.restype = ctypes.c_int
    lib.skip_workspace_bytes_mlp.argtypes = [P, ctypes.c_int32, ctypes.POINTER(ctypes.c_size_t)]
    lib.skip_prune_topk_mlp.restype = ctypes.c_int
    lib.skip_prune_topk_mlp.argtypes = [P, M, vp, vp, i32p, i32p, i32p, vp, vp, vp,
                                        ctypes.c_size_t, vp]
    G = ctypes.POINTER(SkipSkvGate)
    lib.skip_workspace_bytes_gate.restype = ctypes.c_int
    lib.skip_workspace_bytes_gate.argtypes = [P, ctypes.c_int32,
                                              ctypes.POINTER(ctypes.c_size_t)]
    lib.skip_skv_gate.restype = ctypes.c_int
    lib.skip_skv_gate.argtypes = [P, G, vp, i32p, vp, i32p, vp, i32p, i32p, vp, vp, vp, vp,
                                  ctypes.c_size_t, vp]
    lib.skip_bipartite_xattn_masked.restype = ctypes.c_int
    lib.skip_bipartite_xattn_masked.argtypes = [P, vp, i32p, vp, vp, i32p, i32p, vp, vp, vp,
                                                vp, i32p, i32p, vp, ctypes.c_size_t, vp]
    lib.skip_route_fused_gated.restype = ctypes.c_int
    lib.skip_route_fused_gated.argtypes = [P, G, vp, vp, i32p, vp, i32p, vp, vp, i32p, i32p,
                                           vp, i32p, vp, vp, vp, vp, vp, ctypes.c_size_t, vp]
    lib.skip_workspace_bytes_regions.restype = ctypes.c_int
    lib.skip_workspace_bytes_regions.argtypes = [P, ctypes.c_int32,
                                                 ctypes.POINTER(ctypes.c_size_t)]
    lib.skip_region_kmeans.restype = ctypes.c_int
    lib.skip_region_kmeans.argtypes = [P, vp, i32p, i32p, ctypes.c_int32, ctypes.c_int32, i32p,
                                       vp, i32p, vp, ctypes.c_size_t, vp]
    lib.skip_workspace_bytes_project.restype = ctypes.c_int
    lib.skip_workspace_bytes_project.argtypes = [P, ctypes.c_int32,
                                                 ctypes.POINTER(ctypes.c_size_t)]
    lib.skip_gather_project.restype = ctypes.c_int
    lib.skip_gather_project.argtypes = [P, vp, i32p, i32p, vp, ctypes.c_int32, vp,
                                        ctypes.c_int32, vp, ctypes.c_size_t, vp]
    lib.skip_workspace_bytes_project_keys.restype = ctypes.c_int
    lib.skip_workspace_bytes_project_keys.argtypes = [P, ctypes.c_int32,
                                                      ctypes.POINTER(ctypes.c_size_t)]
    lib.skip_project_passage_keys.restype = ctypes.c_int
    lib.skip_project_passage_keys.argtypes = [P, vp, i32p, vp, vp, ctypes.c_int32, vp, vp,
                                              ctypes.c_size_t, vp]
    lib.skip_pack_projection.restype = ctypes.c_int
    lib.skip_pack_projection.argtypes = [P, vp, ctypes.c_int32, vp, ctypes.c_size_t, vp]
    lib.skip_gather_project_packed.restype = ctypes.c_int
    lib.skip_gather_project_packed.argtypes = [P, vp, i32p, i32p, vp, ctypes.c_int32, vp,
                                               ctypes.c_int32, vp]
    lib.skip_bipartite_xattn_proj.restype = ctypes.c_int
    lib.skip_bipartite_xattn_proj.argtypes = [P, vp, vp, i32p, vp, vp, i32p, i32p, vp, vp, vp,
                                              vp, i32p, i32p, vp, ctypes.c_size_t, vp]
    lib.skip_route_fused_noalloc.restype = ctypes.c_int
    lib.skip_route_fused_noalloc.argtypes = [P, vp, vp, i32p, vp, i32p, vp, vp, i32p, i32p, vp,
                                             i32p, vp, vp, vp]
    lib.skip_route_fused_profiled.restype = ctypes.c_int
    lib.skip_route_fused_profiled.argtypes = [P, vp, vp, i32p, vp, i32p, vp, vp, i32p, i32p,
                                              vp, i32p, vp, vp, vp, ctypes.c_size_t, vp,
                                              ctypes.POINTER(ctypes.c_void_p), ctypes.c_int32]
    return lib


LIB = _load()


def status_string(status: int) -> str:
    return LIB.skip_status_string(status).decode()


def abi_version() -> int:
    return LIB.skip_abi_version()


def _check(status: int, where: str):
    if status != SKIP_OK:
        raise SkipError(status, where)


# ---------------------------------------------------------------------------
# Problem description

def _host_i32(x) -> np.ndarray:
    if isinstance(x, torch.Tensor):
        x = x.detach().cpu().numpy()
    return np.ascontiguousarray(np.asarray(x, dtype=np.int64))


def make_problem(dtype: str, *, B: int, N: int = 0, d: int, H: int = 0, d_h: int = 0,
                 q_offsets=None, kept_offsets=None, passage_offsets=None,
                 query_passages=None, avg_degree: float = 4.0,
                 sm_scale: Optional[float] = None, total_edges: int = 0,
                 o_f32: bool = False, edge_rule: str = "question",
                 edge_metric: str = "cosine", edge_beta: float = 0.1) -> SkipProblem:
    """Fill the host-side problem description from host copies of the offsets."""
    p = SkipProblem()
    p.dtype = SKIP_F32 if dtype in ("f32", torch.float32) else SKIP_BF16
    p.B, p.N, p.d, p.H, p.d_h = B, N, d, H, d_h
    if q_offsets is not None:
        qo = _host_i32(q_offsets)
        p.total_qtok = int(qo[-1])
    if kept_offsets is not None:
        ko = _host_i32(kept_offsets)
        p.total_kept = int(ko[-1])
        p.k_max = int(np.diff(ko).max()) if ko.size > 1 else 0
    if query_passages is not None:
        qp = _host_i32(query_passages)
        p.total_passages = int(qp[-1])
        p.P_max = int(np.diff(qp).max()) if qp.size > 1 else 0
    if passage_offsets is not None:
        po = _host_i32(passage_offsets)
        p.total_tokens = int(po[-1])
        p.L_max = int(np.diff(po).max()) if po.size > 1 else 0
    p.total_edges = int(total_edges)
    p.avg_degree = float(avg_degree)
    p.sm_scale = float(sm_scale if sm_scale is not None else (1.0 / math.sqrt(d_h) if d_h else 1.0))
    p.o_f32 = 1 if o_f32 else 0
    p.edge_rule = EDGE_RULES[edge_rule]
    p.edge_metric = EDGE_METRICS[edge_metric]
    p.edge_beta = float(edge_beta)
    return p


def workspace_bytes(p: SkipProblem) -> int:
    n = ctypes.c_size_t(0)
    _check(LIB.skip_workspace_bytes(ctypes.byref(p), ctypes.byref(n)), "skip_workspace_bytes")
    return int(n.value)


def new_workspace(p: SkipProblem, device="cuda") -> torch.Tensor:
    return torch.empty(max(workspace_bytes(p), 256), dtype=torch.uint8, device=device)


def workspace_bytes_mlp(p: SkipProblem, hidden: int) -> int:
    n = ctypes.c_size_t(0)
    _check(LIB.skip_workspace_bytes_mlp(ctypes.byref(p), int(hidden), ctypes.byref(n)),
           "skip_workspace_bytes_mlp")
    return int(n.value)


def workspace_bytes_gate(p: SkipProblem, hidden: int) -> int:
    n = ctypes.c_size_t(0)
    _check(LIB.skip_workspace_bytes_gate(ctypes.byref(p), int(hidden), ctypes.byref(n)),
           "skip_workspace_bytes_gate")
    return int(n.value)


def workspace_bytes_regions(p: SkipProblem, r_max: int) -> int:
    n = ctypes.c_size_t(0)
    _check(LIB.skip_workspace_bytes_regions(ctypes.byref(p), int(r_max), ctypes.byref(n)),
           "skip_workspace_bytes_regions")
    return int(n.value)


def workspace_bytes_project(p: SkipProblem, d_out: int) -> int:
    n = ctypes.c_size_t(0)
    _check(LIB.skip_workspace_bytes_project(ctypes.byref(p), int(d_out), ctypes.byref(n)),
           "skip_workspace_bytes_project")
    return int(n.value)


def workspace_bytes_project_keys(p: SkipProblem, d_out: int) -> int:
    n = ctypes.c_size_t(0)
    _check(LIB.skip_workspace_bytes_project_keys(ctypes.byref(p), int(d_out), ctypes.byref(n)),
           "skip_workspace_bytes_project_keys")
    return int(n.value)


# ---------------------------------------------------------------------------
# Pointer helpers

def _elem_dtype(p: SkipProblem) -> torch.dtype:
    return torch.float32 if p.dtype == SKIP_F32 else torch.bfloat16


def _out_dtype(p: SkipProblem) -> torch.dtype:
    return torch.float32 if (p.dtype == SKIP_F32 or p.o_f32) else torch.bfloat16


def _ptr(t: Optional[torch.Tensor], name: str, dtype=None, numel=None) -> Optional[int]:
    if t is None:
        return None
    if not t.is_cuda:
        raise ValueError(f"{name} must be a device tensor")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    if dtype is not None and t.dtype != dtype:
        raise ValueError(f"{name} must be {dtype}, got {t.dtype}")
    if numel is not None and t.numel() < numel:
        raise ValueError(f"{name} needs {numel} elements, has {t.numel()}")
    if t.numel() and t.data_ptr() % 16:
        raise ValueError(f"{name} must be 16-byte aligned")
    return t.data_ptr() if t.numel() else None


def _stream(stream) -> int:
    if stream is None:
        stream = torch.cuda.current_stream()
    return stream.cuda_stream if hasattr(stream, "cuda_stream") else int(stream)


def _torch_stream(stream):
    """The torch stream object of a stream argument (None: the current one)."""
    if stream is None:
        return torch.cuda.current_stream()
    if isinstance(stream, torch.cuda.Stream):
        return stream
    return torch.cuda.ExternalStream(int(stream))


def _fresh_workspace(nbytes: int, device, stream=None) -> torch.Tensor:
    """A workspace allocated for one call on ``stream`` (see _ws)."""
    ws = torch.empty(max(int(nbytes), 256), dtype=torch.uint8, device=device)
    s = _torch_stream(stream)
    if s != torch.cuda.current_stream():
        ws.record_stream(s)
    return ws


def _ws(p, workspace, stream=None):
    """The workspace of a call: the caller's, or a fresh one.  A fresh one is
    released when the call returns, while the kernels may still run on
    ``stream``; recording that stream on it keeps the caching allocator from
    handing the memory to other work before they finish."""
    if workspace is None:
        workspace = new_workspace(p)
        s = _torch_stream(stream)
        if s != torch.cuda.current_stream():
            workspace.record_stream(s)
    return workspace, workspace.data_ptr(), workspace.numel()


# ---------------------------------------------------------------------------
# Entry points (low level: caller-provided outputs)

def skip_prune_topk(p: SkipProblem, V, Qtok, q_offsets, w_bias, kept_offsets, kept_idx,
                    scores=None, V_kept=None, workspace=None, stream=None):
    et = _elem_dtype(p)
    ws, wsp, wsn = _ws(p, workspace, stream)
    st = LIB.skip_prune_topk(
        ctypes.byref(p), _ptr(V, "V", et, p.B * p.N * p.d), _ptr(Qtok, "Qtok", et, p.total_qtok * p.d),
        _ptr(q_offsets, "q_offsets", torch.int32, p.B + 1), _ptr(w_bias, "w_bias", et, p.d),
        _ptr(kept_offsets, "kept_offsets", torch.int32, p.B + 1),
        _ptr(kept_idx, "kept_idx", torch.int32, p.total_kept),
        _ptr(scores, "scores", torch.float32, p.B * p.N),
        _ptr(V_kept, "V_kept", et, p.total_kept * p.d), wsp, wsn, _stream(stream))
    _check(st, "skip_prune_topk")


def skip_prune_topk_mlp(p: SkipProblem, mlp: "QvsMlp", V, Qtok, q_offsets, kept_offsets,
                        kept_idx, scores=None, V_kept=None, workspace=None, stream=None):
    et = _elem_dtype(p)
    h = mlp.hidden
    if workspace is None:
        workspace = _fresh_workspace(workspace_bytes_mlp(p, h), V.device, stream)
    m = SkipQvsMlp(h, 0, _ptr(mlp.W1, "W1", et, h * 3 * p.d), _ptr(mlp.b1, "b1", torch.float32, h),
                   _ptr(mlp.w2, "w2", torch.float32, h), float(mlp.b2))
    st = LIB.skip_prune_topk_mlp(
        ctypes.byref(p), ctypes.byref(m), _ptr(V, "V", et, p.B * p.N * p.d),
        _ptr(Qtok, "Qtok", et, p.total_qtok * p.d),
        _ptr(q_offsets, "q_offsets", torch.int32, p.B + 1),
        _ptr(kept_offsets, "kept_offsets", torch.int32, p.B + 1),
        _ptr(kept_idx, "kept_idx", torch.int32, p.total_kept),
        _ptr(scores, "scores", torch.float32, p.B * p.N),
        _ptr(V_kept, "V_kept", et, p.total_kept * p.d), workspace.data_ptr(), workspace.numel(),
        _stream(stream))
    _check(st, "skip_prune_topk_mlp")


def skip_bipartite_xattn(p: SkipProblem, Qh, kept_offsets, Kh, Vh, passage_offsets,
                         query_passages, O, lse=None, passage_keys=None, edge_rowptr=None,
                         edge_col=None, edge_rowptr_out=None, edge_col_out=None,
                         workspace=None, stream=None):
    et = _elem_dtype(p)
    ws, wsp, wsn = _ws(p, workspace, stream)
    st = LIB.skip_bipartite_xattn(
        ctypes.byref(p), _ptr(Qh, "Qh", et, p.total_kept * p.d),
        _ptr(kept_offsets, "kept_offsets", torch.int32, p.B + 1),
        _ptr(Kh, "Kh", et, p.total_tokens * p.d), _ptr(Vh, "Vh", et, p.total_tokens * p.d),
        _ptr(passage_offsets, "passage_offsets", torch.int32, p.total_passages + 1),
        _ptr(query_passages, "query_passages", torch.int32, p.B + 1),
        _ptr(passage_keys, "passage_keys", torch.float32, p.total_passages * p.d),
        _ptr(edge_rowptr, "edge_rowptr", torch.int32, p.total_kept + 1),
        _ptr(edge_col, "edge_col", torch.int32, p.total_edges),
        _ptr(O, "O", _out_dtype(p), p.total_kept * p.d),
        _ptr(lse, "lse", torch.float32, p.total_kept * p.H),
        _ptr(edge_rowptr_out, "edge_rowptr_out", torch.int32, p.total_kept + 1),
        _ptr(edge_col_out, "edge_col_out", torch.int32, p.total_kept * p.P_max),
        wsp, wsn, _stream(stream))
    _check(st, "skip_bipartite_xattn")


def skip_skv_gate(p: SkipProblem, gate: "SkvGate", Qtok, q_offsets, V_kept, kept_offsets,
                  Kh, passage_offsets, query_passages, keep, logits=None, passage_keys=None,
                  workspace=None, stream=None):
    et = _elem_dtype(p)
    h = gate.hidden
    if workspace is None:
        workspace = _fresh_workspace(workspace_bytes_gate(p, h), Qtok.device, stream)
    g = _gate_struct(p, gate)
    st = LIB.skip_skv_gate(
        ctypes.byref(p), ctypes.byref(g), _ptr(Qtok, "Qtok", et, p.total_qtok * p.d),
        _ptr(q_offsets, "q_offsets", torch.int32, p.B + 1),
        _ptr(V_kept, "V_kept", et, p.total_kept * p.d),
        _ptr(kept_offsets, "kept_offsets", torch.int32, p.B + 1),
        _ptr(Kh, "Kh", et, p.total_tokens * p.d),
        _ptr(passage_offsets, "passage_offsets", torch.int32, p.total_passages + 1),
        _ptr(query_passages, "query_passages", torch.int32, p.B + 1),
        _ptr(passage_keys, "passage_keys", torch.float32, p.total_passages * p.d),
        _ptr(logits, "logits", torch.float32, p.total_passages),
        _ptr(keep, "keep", torch.uint8, p.total_passages), workspace.data_ptr(),
        workspace.numel(), _stream(stream))
    _check(st, "skip_skv_gate")


def skip_bipartite_xattn_masked(p: SkipProblem, Qh, kept_offsets, Kh, Vh, passage_offsets,
                                query_passages, passage_keep, O, lse=None, passage_keys=None,
                                edge_rowptr_out=None, edge_col_out=None, workspace=None,
                                stream=None):
    et = _elem_dtype(p)
    ws, wsp, wsn = _ws(p, workspace, stream)
    st = LIB.skip_bipartite_xattn_masked(
        ctypes.byref(p), _ptr(Qh, "Qh", et, p.total_kept * p.d),
        _ptr(kept_offsets, "kept_offsets", torch.int32, p.B + 1),
        _ptr(Kh, "Kh", et, p.total_tokens * p.d), _ptr(Vh, "Vh", et, p.total_tokens * p.d),
        _ptr(passage_offsets, "passage_offsets", torch.int32, p.total_passages + 1),
        _ptr(query_passages, "query_passages", torch.int32, p.B + 1),
        _ptr(passage_keys, "passage_keys", torch.float32, p.total_passages * p.d),
        _ptr(passage_keep, "passage_keep", torch.uint8, p.total_passages),
        _ptr(O, "O", _out_dtype(p), p.total_kept * p.d),
        _ptr(lse, "lse", torch.float32, p.total_kept * p.H),
        _ptr(edge_rowptr_out, "edge_rowptr_out", torch.int32, p.total_kept + 1),
        _ptr(edge_col_out, "edge_col_out", torch.int32, p.total_kept * p.P_max),
        wsp, wsn, _stream(stream))
    _check(st, "skip_bipartite_xattn_masked")


def _gate_struct(p: SkipProblem, gate: "SkvGate") -> SkipSkvGate:
    h = gate.hidden
    return SkipSkvGate(h, 0, _ptr(gate.W, "W", _elem_dtype(p), h * 5 * p.d),
                       _ptr(gate.b1, "b1", torch.float32, h), _ptr(gate.w2, "w2", torch.float32, h),
                       float(gate.b2), float(gate.tau), float(gate.rho))


def skip_route_fused_gated(p: SkipProblem, gate: "SkvGate", V, Qtok, q_offsets, w_bias,
                           kept_offsets, Kh, Vh, passage_offsets, query_passages, kept_idx,
                           passage_keep, O, lse=None, gate_logits=None, passage_keys=None,
                           workspace=None, stream=None):
    et = _elem_dtype(p)
    if workspace is None:
        workspace = _fresh_workspace(workspace_bytes_gate(p, gate.hidden), V.device, stream)
    g = _gate_struct(p, gate)
    st = LIB.skip_route_fused_gated(
        ctypes.byref(p), ctypes.byref(g), _ptr(V, "V", et, p.B * p.N * p.d),
        _ptr(Qtok, "Qtok", et, p.total_qtok * p.d),
        _ptr(q_offsets, "q_offsets", torch.int32, p.B + 1), _ptr(w_bias, "w_bias", et, p.d),
        _ptr(kept_offsets, "kept_offsets", torch.int32, p.B + 1),
        _ptr(Kh, "Kh", et, p.total_tokens * p.d), _ptr(Vh, "Vh", et, p.total_tokens * p.d),
        _ptr(passage_offsets, "passage_offsets", torch.int32, p.total_passages + 1),
        _ptr(query_passages, "query_passages", torch.int32, p.B + 1),
        _ptr(passage_keys, "passage_keys", torch.float32, p.total_passages * p.d),
        _ptr(kept_idx, "kept_idx", torch.int32, p.total_kept),
        _ptr(passage_keep, "passage_keep", torch.uint8, p.total_passages),
        _ptr(gate_logits, "gate_logits", torch.float32, p.total_passages),
        _ptr(O, "O", _out_dtype(p), p.total_kept * p.d),
        _ptr(lse, "lse", torch.float32, p.total_kept * p.H), workspace.data_ptr(),
        workspace.numel(), _stream(stream))
    _check(st, "skip_route_fused_gated")


def skip_region_kmeans(p: SkipProblem, rows, kept_offsets, kept_idx, r_max, n_iter, region,
                       centroids, sizes=None, workspace=None, stream=None):
    et = _elem_dtype(p)
    if workspace is None:
        workspace = _fresh_workspace(workspace_bytes_regions(p, r_max), centroids.device,
                                     stream)
    n_rows = p.B * p.N if kept_idx is not None else p.total_kept
    st = LIB.skip_region_kmeans(
        ctypes.byref(p), _ptr(rows, "rows", et, n_rows * p.d),
        _ptr(kept_offsets, "kept_offsets", torch.int32, p.B + 1),
        _ptr(kept_idx, "kept_idx", torch.int32, p.total_kept), int(r_max), int(n_iter),
        _ptr(region, "region", torch.int32, p.total_kept),
        _ptr(centroids, "centroids", torch.float32, p.B * r_max * p.d),
        _ptr(sizes, "sizes", torch.int32, p.B * r_max), workspace.data_ptr(), workspace.numel(),
        _stream(stream))
    _check(st, "skip_region_kmeans")


def skip_gather_project(p: SkipProblem, rows, kept_offsets, kept_idx, W, Y, out_f32=False,
                        workspace=None, stream=None):
    et = _elem_dtype(p)
    d_out = int(W.shape[0])
    if workspace is None:
        workspace = _fresh_workspace(workspace_bytes_project(p, d_out), W.device, stream)
    n_rows = p.B * p.N if kept_idx is not None else p.total_kept
    st = LIB.skip_gather_project(
        ctypes.byref(p), _ptr(rows, "rows", et, n_rows * p.d),
        _ptr(kept_offsets, "kept_offsets", torch.int32, p.B + 1),
        _ptr(kept_idx, "kept_idx", torch.int32, p.total_kept), _ptr(W, "W", et, d_out * p.d),
        d_out, _ptr(Y, "Y", torch.float32 if out_f32 else et, p.total_kept * d_out),
        1 if out_f32 else 0, workspace.data_ptr(), workspace.numel(), _stream(stream))
    _check(st, "skip_gather_project")


def skip_project_passage_keys(p: SkipProblem, Kh, passage_offsets, passage_keys, W, keys_out,
                              workspace=None, stream=None):
    et = _elem_dtype(p)
    d_out = int(W.shape[0])
    if workspace is None:
        workspace = _fresh_workspace(workspace_bytes_project_keys(p, d_out), W.device, stream)
    st = LIB.skip_project_passage_keys(
        ctypes.byref(p), _ptr(Kh, "Kh", et, p.total_tokens * p.d),
        _ptr(passage_offsets, "passage_offsets", torch.int32, p.total_passages + 1),
        _ptr(passage_keys, "passage_keys", torch.float32, p.total_passages * p.d),
        _ptr(W, "W", et, d_out * p.d),
        d_out, _ptr(keys_out, "keys_out", torch.float32, p.total_passages * d_out),
        workspace.data_ptr(), workspace.numel(), _stream(stream))
    _check(st, "skip_project_passage_keys")


def skip_pack_projection(p: SkipProblem, W, packed, stream=None):
    d_out = int(W.shape[0])
    st = LIB.skip_pack_projection(ctypes.byref(p), _ptr(W, "W", _elem_dtype(p), d_out * p.d),
                                  d_out, packed.data_ptr(), packed.numel(), _stream(stream))
    _check(st, "skip_pack_projection")


def skip_gather_project_packed(p: SkipProblem, rows, kept_offsets, kept_idx, packed, d_out, Y,
                               out_f32=False, stream=None):
    et = _elem_dtype(p)
    n_rows = p.B * p.N if kept_idx is not None else p.total_kept
    st = LIB.skip_gather_project_packed(
        ctypes.byref(p), _ptr(rows, "rows", et, n_rows * p.d),
        _ptr(kept_offsets, "kept_offsets", torch.int32, p.B + 1),
        _ptr(kept_idx, "kept_idx", torch.int32, p.total_kept), packed.data_ptr(), int(d_out),
        _ptr(Y, "Y", torch.float32 if out_f32 else et, p.total_kept * d_out),
        1 if out_f32 else 0, _stream(stream))
    _check(st, "skip_gather_project_packed")


def skip_bipartite_xattn_proj(p: SkipProblem, Qh, edge_rows, kept_offsets, Kh, Vh,
                              passage_offsets, query_passages, passage_keys, O, lse=None,
                              passage_keep=None, edge_rowptr_out=None, edge_col_out=None,
                              workspace=None, stream=None):
    et = _elem_dtype(p)
    ws, wsp, wsn = _ws(p, workspace, stream)
    st = LIB.skip_bipartite_xattn_proj(
        ctypes.byref(p), _ptr(Qh, "Qh", et, p.total_kept * p.d),
        _ptr(edge_rows, "edge_rows", et, p.total_kept * p.d),
        _ptr(kept_offsets, "kept_offsets", torch.int32, p.B + 1),
        _ptr(Kh, "Kh", et, p.total_tokens * p.d), _ptr(Vh, "Vh", et, p.total_tokens * p.d),
        _ptr(passage_offsets, "passage_offsets", torch.int32, p.total_passages + 1),
        _ptr(query_passages, "query_passages", torch.int32, p.B + 1),
        _ptr(passage_keys, "passage_keys", torch.float32, p.total_passages * p.d),
        _ptr(passage_keep, "passage_keep", torch.uint8, p.total_passages),
        _ptr(O, "O", _out_dtype(p), p.total_kept * p.d),
        _ptr(lse, "lse", torch.float32, p.total_kept * p.H),
        _ptr(edge_rowptr_out, "edge_rowptr_out", torch.int32, p.total_kept + 1),
        _ptr(edge_col_out, "edge_col_out", torch.int32, p.total_kept * p.P_max),
        wsp, wsn, _stream(stream))
    _check(st, "skip_bipartite_xattn_proj")


def skip_route_fused(p: SkipProblem, V, Qtok, q_offsets, w_bias, kept_offsets, Kh, Vh,
                     passage_offsets, query_passages, kept_idx, O, lse=None,
                     passage_keys=None, workspace=None, stream=None, stage_events=None):
    """``stage_events``: a StageEvents set to time each kernel stage (calls
    skip_route_fused_profiled)."""
    et = _elem_dtype(p)
    ws, wsp, wsn = _ws(p, workspace, stream)
    if stage_events is None:
        fn, extra = LIB.skip_route_fused, ()
    else:
        fn, extra = LIB.skip_route_fused_profiled, (stage_events.handles, len(stage_events))
    st = fn(
        ctypes.byref(p), _ptr(V, "V", et, p.B * p.N * p.d), _ptr(Qtok, "Qtok", et, p.total_qtok * p.d),
        _ptr(q_offsets, "q_offsets", torch.int32, p.B + 1), _ptr(w_bias, "w_bias", et, p.d),
        _ptr(kept_offsets, "kept_offsets", torch.int32, p.B + 1),
        _ptr(Kh, "Kh", et, p.total_tokens * p.d), _ptr(Vh, "Vh", et, p.total_tokens * p.d),
        _ptr(passage_offsets, "passage_offsets", torch.int32, p.total_passages + 1),
        _ptr(query_passages, "query_passages", torch.int32, p.B + 1),
        _ptr(passage_keys, "passage_keys", torch.float32, p.total_passages * p.d),
        _ptr(kept_idx, "kept_idx", torch.int32, p.total_kept),
        _ptr(O, "O", _out_dtype(p), p.total_kept * p.d),
        _ptr(lse, "lse", torch.float32, p.total_kept * p.H), wsp, wsn, _stream(stream), *extra)
    _check(st, "skip_route_fused")


NOALLOC_SCRATCH_BYTES = 16 << 20     # SKIP_NOALLOC_SCRATCH_BYTES


def skip_route_fused_noalloc(p: SkipProblem, V, Qtok, q_offsets, w_bias, kept_offsets, Kh, Vh,
                             passage_offsets, query_passages, kept_idx, O, lse=None,
                             passage_keys=None, stream=None):
    """skip_route_fused with the library's own device scratch (no workspace
    argument, nothing allocated by the call)."""
    et = _elem_dtype(p)
    st = LIB.skip_route_fused_noalloc(
        ctypes.byref(p), _ptr(V, "V", et, p.B * p.N * p.d), _ptr(Qtok, "Qtok", et, p.total_qtok * p.d),
        _ptr(q_offsets, "q_offsets", torch.int32, p.B + 1), _ptr(w_bias, "w_bias", et, p.d),
        _ptr(kept_offsets, "kept_offsets", torch.int32, p.B + 1),
        _ptr(Kh, "Kh", et, p.total_tokens * p.d), _ptr(Vh, "Vh", et, p.total_tokens * p.d),
        _ptr(passage_offsets, "passage_offsets", torch.int32, p.total_passages + 1),
        _ptr(query_passages, "query_passages", torch.int32, p.B + 1),
        _ptr(passage_keys, "passage_keys", torch.float32, p.total_passages * p.d),
        _ptr(kept_idx, "kept_idx", torch.int32, p.total_kept),
        _ptr(O, "O", _out_dtype(p), p.total_kept * p.d),
        _ptr(lse, "lse", torch.float32, p.total_kept * p.H), _stream(stream))
    _check(st, "skip_route_fused_noalloc")


class StageEvents:
    """SKIP_FUSED_STAGES + 1 timing events for skip_route_fused_profiled.
    torch events are created (by one record on the current stream) and their
    raw hipEvent_t handles handed to the library, which records them on the
    launch stream between its kernel stages."""

    def __init__(self):
        self.events = [torch.cuda.Event(enable_timing=True) for _ in range(len(FUSED_STAGES) + 1)]
        for e in self.events:
            e.record()
        arr = (ctypes.c_void_p * len(self.events))(*[e.cuda_event for e in self.events])
        self.handles = ctypes.cast(arr, ctypes.POINTER(ctypes.c_void_p))
        self._arr = arr

    def __len__(self):
        return len(self.events)

    def stage_ms(self):
        """Per-stage durations in ms (call after the stream has synchronised)."""
        return {name: self.events[i].elapsed_time(self.events[i + 1])
                for i, name in enumerate(FUSED_STAGES)}


# ---------------------------------------------------------------------------
# Convenience layer over a generated batch (allocates outputs)

@dataclass
class DeviceBatch:
    """A batch's tensors and offsets on the device, plus its problem."""
    p: SkipProblem
    V: torch.Tensor
    Qtok: torch.Tensor
    q_offsets: torch.Tensor
    kept_offsets: torch.Tensor
    Kh: torch.Tensor
    Vh: torch.Tensor
    passage_offsets: torch.Tensor
    query_passages: torch.Tensor
    w_bias: Optional[torch.Tensor]
    workspace: torch.Tensor


def to_device(batch, device="cuda", avg_degree: Optional[float] = None,
              sm_scale: Optional[float] = None, o_f32: bool = False,
              edge_rule: str = "question", edge_metric: str = "cosine",
              edge_beta: float = 0.1) -> DeviceBatch:
    """Move a generated batch (``workloads.Batch``) to the device."""
    wl = batch.wl
    B, N, d = batch.V.shape
    H, d_h = batch.Kh.shape[1], batch.Kh.shape[2]
    p = make_problem(wl.dtype, B=B, N=N, d=d, H=H, d_h=d_h, q_offsets=batch.q_offsets,
                     kept_offsets=batch.kept_offsets, passage_offsets=batch.passage_offsets,
                     query_passages=batch.query_passages,
                     avg_degree=wl.avg_degree if avg_degree is None else avg_degree,
                     sm_scale=wl.scale if sm_scale is None else sm_scale, o_f32=o_f32,
                     edge_rule=edge_rule, edge_metric=edge_metric, edge_beta=edge_beta)
    i32 = lambda a: torch.from_numpy(np.asarray(a, dtype=np.int32)).to(device)
    return DeviceBatch(
        p=p, V=batch.V.to(device), Qtok=batch.Qtok.to(device), q_offsets=i32(batch.q_offsets),
        kept_offsets=i32(batch.kept_offsets), Kh=batch.Kh.to(device), Vh=batch.Vh.to(device),
        passage_offsets=i32(batch.passage_offsets), query_passages=i32(batch.query_passages),
        w_bias=None if batch.w_bias is None else batch.w_bias.to(device),
        workspace=new_workspace(p, device))


def with_f32_output(db: DeviceBatch) -> DeviceBatch:
    """The same batch (shared tensors) with O written as float32."""
    q = SkipProblem.from_buffer_copy(db.p)
    q.o_f32 = 1
    return DeviceBatch(q, db.V, db.Qtok, db.q_offsets, db.kept_offsets, db.Kh, db.Vh,
                       db.passage_offsets, db.query_passages, db.w_bias, db.workspace)


def prune_topk(db: DeviceBatch, want_scores=True, want_rows=True):
    p = db.p
    kept_idx = torch.empty(max(p.total_kept, 1), dtype=torch.int32, device=db.V.device)
    scores = torch.empty(p.B * p.N, dtype=torch.float32, device=db.V.device) if want_scores else None
    V_kept = (torch.empty((max(p.total_kept, 1), p.d), dtype=db.V.dtype, device=db.V.device)
              if want_rows else None)
    skip_prune_topk(p, db.V, db.Qtok, db.q_offsets, db.w_bias, db.kept_offsets, kept_idx,
                    scores, V_kept, db.workspace)
    return (kept_idx[:p.total_kept], None if scores is None else scores.view(p.B, p.N),
            None if V_kept is None else V_kept[:p.total_kept])


@dataclass
class QvsMlp:
    """Device tensors of the main-text scorer: W1 [h, 3d] (element type of V),
    b1 [h] float32 or None, w2 [h] float32, and the scalar b2."""
    W1: torch.Tensor
    b1: Optional[torch.Tensor]
    w2: torch.Tensor
    b2: float

    @property
    def hidden(self) -> int:
        return int(self.W1.shape[0])


def prune_topk_mlp(db: DeviceBatch, mlp: QvsMlp, want_scores=True, want_rows=True,
                   workspace=None):
    """Stage 1 with the main-text scorer.  Returns (kept_idx, scores, V_kept)."""
    p = db.p
    dev = db.V.device
    kept_idx = torch.empty(max(p.total_kept, 1), dtype=torch.int32, device=dev)
    scores = torch.empty(p.B * p.N, dtype=torch.float32, device=dev) if want_scores else None
    V_kept = (torch.empty((max(p.total_kept, 1), p.d), dtype=db.V.dtype, device=dev)
              if want_rows else None)
    skip_prune_topk_mlp(p, mlp, db.V, db.Qtok, db.q_offsets, db.kept_offsets, kept_idx,
                        scores, V_kept, workspace)
    return (kept_idx[:p.total_kept], None if scores is None else scores.view(p.B, p.N),
            None if V_kept is None else V_kept[:p.total_kept])


def bipartite_xattn(db: DeviceBatch, Qh: torch.Tensor, passage_keys=None, edges=None,
                    want_edges=True) -> Tuple:
    """Qh: [total_kept, H, d_h].  ``edges`` = (rowptr, col) device int32 to
    use a given graph.  Returns (O, lse, rowptr, col)."""
    p = db.p
    dev = db.V.device
    O = torch.empty((max(p.total_kept, 1), p.H, p.d_h), dtype=_out_dtype(p), device=dev)
    lse = torch.empty((max(p.total_kept, 1), p.H), dtype=torch.float32, device=dev)
    rp = col = None
    q = p
    if edges is not None:
        q = SkipProblem.from_buffer_copy(p)
        q.total_edges = int(edges[1].numel())
    elif want_edges:
        rp = torch.empty(p.total_kept + 1, dtype=torch.int32, device=dev)
        col = torch.empty(max(p.total_kept * p.P_max, 1), dtype=torch.int32, device=dev)
    skip_bipartite_xattn(q, Qh if p.total_kept else None, db.kept_offsets, db.Kh, db.Vh,
                         db.passage_offsets, db.query_passages, O if p.total_kept else None,
                         lse if p.total_kept else None, passage_keys,
                         None if edges is None else edges[0],
                         None if edges is None else edges[1], rp, col, db.workspace)
    return O[:p.total_kept], lse[:p.total_kept], rp, col


@dataclass
class SkvGate:
    """Device tensors of the passage gate: W [h, 5d] (element type of V), b1
    [h] float32 or None, w2 [h] float32; scalars b2, tau (threshold on the
    gate probability) and rho (kept fraction of a question's passages)."""
    W: torch.Tensor
    b1: Optional[torch.Tensor]
    w2: torch.Tensor
    b2: float
    tau: float = 0.5
    rho: float = 0.5

    @property
    def hidden(self) -> int:
        return int(self.W.shape[0])


def skv_gate(db: DeviceBatch, gate: SkvGate, V_kept: torch.Tensor, passage_keys=None,
             workspace=None):
    """The passage gate on the kept rows V_kept [total_kept, d].  Returns
    (keep [total_passages] uint8, logits [total_passages] float32)."""
    p = db.p
    dev = db.V.device
    keep = torch.empty(max(p.total_passages, 1), dtype=torch.uint8, device=dev)
    logits = torch.empty(max(p.total_passages, 1), dtype=torch.float32, device=dev)
    skip_skv_gate(p, gate, db.Qtok, db.q_offsets, V_kept if p.total_kept else None,
                  db.kept_offsets, db.Kh, db.passage_offsets, db.query_passages, keep, logits,
                  passage_keys, workspace)
    return keep[:p.total_passages], logits[:p.total_passages]


def bipartite_xattn_masked(db: DeviceBatch, Qh: torch.Tensor, passage_keep: torch.Tensor,
                           passage_keys=None, want_edges=True) -> Tuple:
    """bipartite_xattn over the passages with passage_keep != 0.  Returns
    (O, lse, rowptr, col)."""
    p = db.p
    dev = db.V.device
    O = torch.empty((max(p.total_kept, 1), p.H, p.d_h), dtype=_out_dtype(p), device=dev)
    lse = torch.empty((max(p.total_kept, 1), p.H), dtype=torch.float32, device=dev)
    rp = col = None
    if want_edges:
        rp = torch.empty(p.total_kept + 1, dtype=torch.int32, device=dev)
        col = torch.empty(max(p.total_kept * p.P_max, 1), dtype=torch.int32, device=dev)
    skip_bipartite_xattn_masked(p, Qh if p.total_kept else None, db.kept_offsets, db.Kh, db.Vh,
                                db.passage_offsets, db.query_passages, passage_keep,
                                O if p.total_kept else None, lse if p.total_kept else None,
                                passage_keys, rp, col, db.workspace)
    return O[:p.total_kept], lse[:p.total_kept], rp, col


def route_fused_gated(db: DeviceBatch, gate: SkvGate, passage_keys=None, out=None,
                      workspace=None):
    """The fused route with the verification step.  Returns (kept_idx,
    passage_keep, gate_logits, O, lse).  ``out`` = preallocated tensors of
    the same five."""
    p = db.p
    dev = db.V.device
    if out is None:
        out = (torch.empty(max(p.total_kept, 1), dtype=torch.int32, device=dev),
               torch.empty(max(p.total_passages, 1), dtype=torch.uint8, device=dev),
               torch.empty(max(p.total_passages, 1), dtype=torch.float32, device=dev),
               torch.empty((max(p.total_kept, 1), p.H, p.d_h), dtype=_out_dtype(p), device=dev),
               torch.empty((max(p.total_kept, 1), p.H), dtype=torch.float32, device=dev))
    kept_idx, keep, logits, O, lse = out
    skip_route_fused_gated(p, gate, db.V, db.Qtok, db.q_offsets, db.w_bias, db.kept_offsets,
                           db.Kh, db.Vh, db.passage_offsets, db.query_passages, kept_idx, keep,
                           O, lse, logits, passage_keys, workspace)
    return (kept_idx[:p.total_kept], keep[:p.total_passages], logits[:p.total_passages],
            O[:p.total_kept], lse[:p.total_kept])


def region_kmeans(db: DeviceBatch, rows: torch.Tensor, kept_idx=None, r_max: int = 8,
                  n_iter: int = 10, workspace=None):
    """Regions of the kept tokens.  ``rows``: the kept rows [total_kept, d], or
    db.V with ``kept_idx``.  Returns (region [total_kept] int32, centroids
    [B, r_max, d] float32, sizes [B, r_max] int32)."""
    p = db.p
    dev = db.V.device
    region = torch.empty(max(p.total_kept, 1), dtype=torch.int32, device=dev)
    cent = torch.empty((p.B, r_max, p.d), dtype=torch.float32, device=dev)
    sizes = torch.empty((p.B, r_max), dtype=torch.int32, device=dev)
    skip_region_kmeans(p, rows if p.total_kept else None, db.kept_offsets, kept_idx, r_max,
                       n_iter, region if p.total_kept else None, cent, sizes, workspace)
    return region[:p.total_kept], cent, sizes


def gather_project(db: DeviceBatch, rows: torch.Tensor, W: torch.Tensor, kept_idx=None,
                   out_f32=False, workspace=None):
    """Y = W x_r for every kept row (``rows`` the kept rows, or db.V with
    ``kept_idx``).  Returns Y [total_kept, d_out] (bf16, or float32)."""
    p = db.p
    Y = torch.empty((max(p.total_kept, 1), int(W.shape[0])),
                    dtype=torch.float32 if out_f32 else db.V.dtype, device=db.V.device)
    skip_gather_project(p, rows if p.total_kept else None, db.kept_offsets, kept_idx, W,
                        Y if p.total_kept else None, out_f32, workspace)
    return Y[:p.total_kept]


def project_passage_keys(db: DeviceBatch, W: torch.Tensor, passage_keys=None):
    """h_k = W k~_j for every passage (k~ the bf16 rounding of the pooled key,
    or of ``passage_keys``).  Returns [total_passages, d_out] float32."""
    p = db.p
    out = torch.empty((max(p.total_passages, 1), int(W.shape[0])), dtype=torch.float32,
                      device=db.V.device)
    skip_project_passage_keys(p, db.Kh if p.total_tokens else None, db.passage_offsets,
                              passage_keys, W, out if p.total_passages else None)
    return out[:p.total_passages]


def pack_projection(db: DeviceBatch, W: torch.Tensor) -> torch.Tensor:
    """W [d_out, d] bf16 repacked for the matrix cores, for
    ``gather_project_packed`` (a uint8 tensor owned by the caller)."""
    packed = torch.empty(workspace_bytes_project(db.p, int(W.shape[0])), dtype=torch.uint8,
                         device=W.device)
    skip_pack_projection(db.p, W, packed)
    return packed


def gather_project_packed(db: DeviceBatch, rows: torch.Tensor, packed: torch.Tensor, d_out: int,
                          kept_idx=None, out_f32=False):
    """``gather_project`` with weights packed once by ``pack_projection``."""
    p = db.p
    Y = torch.empty((max(p.total_kept, 1), int(d_out)),
                    dtype=torch.float32 if out_f32 else db.V.dtype, device=db.V.device)
    skip_gather_project_packed(p, rows if p.total_kept else None, db.kept_offsets, kept_idx,
                               packed, d_out, Y if p.total_kept else None, out_f32)
    return Y[:p.total_kept]


def bipartite_xattn_proj(db: DeviceBatch, Qh: torch.Tensor, edge_rows: torch.Tensor,
                         passage_keys: torch.Tensor, passage_keep=None, want_edges=True):
    """Graph cut on ``edge_rows`` against ``passage_keys``, attention on Qh.
    Returns (O, lse, rowptr, col)."""
    p = db.p
    dev = db.V.device
    O = torch.empty((max(p.total_kept, 1), p.H, p.d_h), dtype=_out_dtype(p), device=dev)
    lse = torch.empty((max(p.total_kept, 1), p.H), dtype=torch.float32, device=dev)
    rp = col = None
    if want_edges:
        rp = torch.empty(p.total_kept + 1, dtype=torch.int32, device=dev)
        col = torch.empty(max(p.total_kept * p.P_max, 1), dtype=torch.int32, device=dev)
    skip_bipartite_xattn_proj(p, Qh if p.total_kept else None,
                              edge_rows if p.total_kept else None, db.kept_offsets, db.Kh,
                              db.Vh, db.passage_offsets, db.query_passages, passage_keys,
                              O if p.total_kept else None, lse if p.total_kept else None,
                              passage_keep, rp, col, db.workspace)
    return O[:p.total_kept], lse[:p.total_kept], rp, col


def route_fused(db: DeviceBatch, passage_keys=None, out=None, stage_events=None):
    """Returns (kept_idx, O, lse).  ``out`` = preallocated (kept_idx, O, lse)."""
    p = db.p
    dev = db.V.device
    if out is None:
        out = (torch.empty(max(p.total_kept, 1), dtype=torch.int32, device=dev),
               torch.empty((max(p.total_kept, 1), p.H, p.d_h), dtype=_out_dtype(p), device=dev),
               torch.empty((max(p.total_kept, 1), p.H), dtype=torch.float32, device=dev))
    kept_idx, O, lse = out
    skip_route_fused(p, db.V, db.Qtok, db.q_offsets, db.w_bias, db.kept_offsets, db.Kh, db.Vh,
                     db.passage_offsets, db.query_passages, kept_idx, O, lse, passage_keys,
                     db.workspace, stage_events=stage_events)
    return kept_idx[:p.total_kept], O[:p.total_kept], lse[:p.total_kept]
