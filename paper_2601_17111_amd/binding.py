"""Thin ctypes binding of libllep.so (include/llep.h).

Argument marshalling only: every step of the path runs in the library's HIP
kernels. Tensors are torch tensors on the GPU (torch supplies device memory
and streams); each function passes their data pointers and the current HIP
stream. The library must be built (``__graft_entry__.build()``); nothing
here falls back to another implementation when it is missing.
"""

from __future__ import annotations

import ctypes
import os
from typing import Optional

from ._build import LIB_PATH

LLEP_OK = 0
LLEP_E_ARG = -1
LLEP_E_WORKSPACE = -2
LLEP_E_DTYPE = -3
LLEP_E_HIP = -4
LLEP_F32 = 0
LLEP_BF16 = 1
LLEP_MODE_LLEP = 0
LLEP_MODE_EP = 1
LLEP_STATUS_BAD_EXPERT_ID = 1
LLEP_STATUS_FFN_WAIT = 2
LLEP_MAX_EXPERTS = 512
LLEP_MAX_DEVICES = 64
LLEP_MAX_FFN_DIM = 65536

EXPORTED = [
    "llep_plan", "llep_permute", "llep_grouped_ffn", "llep_combine",
    "llep_pack_weights", "llep_plan_max_chunks", "llep_plan_rank_base_elems",
    "llep_grouped_ffn_workspace_bytes", "llep_packed_gate_up_bytes",
    "llep_packed_down_bytes", "llep_last_error", "llep_combine_backward",
    "llep_pack_weights_backward", "llep_grouped_ffn_backward_workspace_bytes",
    "llep_grouped_ffn_backward", "llep_grouped_ffn_train", "llep_grouped_ffn_noalloc",
]
LLEP_NOALLOC_SCRATCH_BYTES = 64 << 20


class llep_plan_params(ctypes.Structure):
    _fields_ = [("T", ctypes.c_int64), ("K", ctypes.c_int32), ("E", ctypes.c_int32),
                ("P", ctypes.c_int32), ("min_chunk", ctypes.c_int32),
                ("capacity", ctypes.c_int64), ("lam", ctypes.c_double),
                ("mode", ctypes.c_int32), ("reserved", ctypes.c_int32)]


class llep_plan_info(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int32) for n in (
        "status", "n_chunks", "n_groups", "n_xfers", "bypassed", "forced",
        "max_device", "total_rows")]


_P = ctypes.c_void_p


class llep_plan_buffers(ctypes.Structure):
    _fields_ = [(n, _P) for n in (
        "loads", "chunks", "chunk_row", "expert_chunk_begin", "groups",
        "group_begin", "device_rows", "xfers", "rank_base", "info")]


class LLEPError(RuntimeError):
    def __init__(self, code: int, where: str, msg: str):
        super().__init__(f"{where} failed with code {code}: {msg}")
        self.code = code


_lib = None


def lib() -> ctypes.CDLL:
    """Load libllep.so (once). Raises if it has not been built."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(
                f"{LIB_PATH} is missing: build it with __graft_entry__.build()")
        L = ctypes.CDLL(LIB_PATH)
        pp = ctypes.POINTER(llep_plan_params)
        pb = ctypes.POINTER(llep_plan_buffers)
        i32, i64, sz = ctypes.c_int32, ctypes.c_int64, ctypes.c_size_t
        sigs = {
            "llep_plan_max_chunks": (i32, [pp]),
            "llep_plan_rank_base_elems": (i64, [pp]),
            "llep_plan": (ctypes.c_int, [pp, _P, pb, _P]),
            "llep_permute": (ctypes.c_int, [pp, pb, _P, _P, _P, i32, ctypes.c_int, _P, _P,
                                            _P, _P, _P]),
            "llep_packed_gate_up_bytes": (sz, [i32, i32, i32, ctypes.c_int]),
            "llep_packed_down_bytes": (sz, [i32, i32, i32, ctypes.c_int]),
            "llep_pack_weights": (ctypes.c_int, [i32, i32, i32, ctypes.c_int, _P, _P, _P, _P,
                                                 _P, _P]),
            "llep_grouped_ffn_workspace_bytes": (sz, [pp, i32, ctypes.c_int]),
            "llep_grouped_ffn": (ctypes.c_int, [pp, pb, i32, _P, _P, _P, i32, i32,
                                                ctypes.c_int, _P, _P, sz, _P]),
            "llep_grouped_ffn_train": (ctypes.c_int, [pp, pb, i32, _P, _P, _P, i32, i32,
                                                      ctypes.c_int, _P, _P, _P, sz, _P]),
            "llep_grouped_ffn_noalloc": (ctypes.c_int, [pp, pb, i32, _P, _P, _P, i32, i32,
                                                        ctypes.c_int, _P, _P]),
            "llep_combine": (ctypes.c_int, [pp, _P, _P, _P, i32, ctypes.c_int, _P, _P]),
            "llep_combine_backward": (ctypes.c_int, [pp, _P, _P, _P, _P, i32, ctypes.c_int, _P,
                                                     _P, _P]),
            "llep_pack_weights_backward": (ctypes.c_int, [i32, i32, i32, ctypes.c_int, _P, _P,
                                                          _P, _P, _P, _P]),
            "llep_grouped_ffn_backward_workspace_bytes": (sz, [pp, i32, i32, ctypes.c_int]),
            "llep_grouped_ffn_backward": (ctypes.c_int, [pp, pb, i32, _P, _P, _P, _P, _P, _P,
                                                         i32, i32, ctypes.c_int, _P, _P, _P, _P,
                                                         _P, sz, _P]),
            "llep_last_error": (ctypes.c_char_p, []),
        }
        for name, (res, args) in sigs.items():
            fn = getattr(L, name)
            fn.restype = res
            fn.argtypes = args
        _lib = L
    return _lib


def last_error() -> str:
    return lib().llep_last_error().decode()


def _check(rc: int, where: str):
    if rc != LLEP_OK:
        raise LLEPError(rc, where, last_error())


def _ptr(t) -> Optional[int]:
    return None if t is None else t.data_ptr()


def _stream(stream=None) -> int:
    import torch
    s = stream if stream is not None else torch.cuda.current_stream()
    return s.cuda_stream


def _dtype_code(t) -> int:
    import torch
    if t.dtype == torch.bfloat16:
        return LLEP_BF16
    if t.dtype == torch.float32:
        return LLEP_F32
    raise TypeError(f"unsupported dtype {t.dtype}")


def make_params(T: int, K: int, E: int, P: int, capacity: int, min_chunk: int = 1,
                lam: float = 0.0, mode: str = "llep") -> llep_plan_params:
    return llep_plan_params(T=T, K=K, E=E, P=P, min_chunk=min_chunk, capacity=capacity,
                            lam=lam, mode=LLEP_MODE_EP if mode == "ep" else LLEP_MODE_LLEP,
                            reserved=0)


# ---- size queries ----------------------------------------------------------

def llep_plan_max_chunks(params: llep_plan_params) -> int:
    n = lib().llep_plan_max_chunks(ctypes.byref(params))
    if n < 0:
        raise LLEPError(LLEP_E_ARG, "llep_plan_max_chunks", last_error())
    return n


def llep_plan_rank_base_elems(params: llep_plan_params) -> int:
    n = lib().llep_plan_rank_base_elems(ctypes.byref(params))
    if n < 0:
        raise LLEPError(LLEP_E_ARG, "llep_plan_rank_base_elems", last_error())
    return n


def llep_grouped_ffn_workspace_bytes(params: llep_plan_params, F: int, dtype_code: int) -> int:
    return lib().llep_grouped_ffn_workspace_bytes(ctypes.byref(params), F, dtype_code)


def llep_grouped_ffn_backward_workspace_bytes(params: llep_plan_params, D: int, F: int,
                                              dtype_code: int) -> int:
    return lib().llep_grouped_ffn_backward_workspace_bytes(ctypes.byref(params), D, F,
                                                           dtype_code)


# ---- plan buffers (device tensors) --------------------------------------------

class PlanBuffers:
    """Device tensors for llep_plan's tables, sized from the params."""

    def __init__(self, params: llep_plan_params, device="cuda"):
        import torch
        C = llep_plan_max_chunks(params)
        E, P = params.E, params.P
        i32 = dict(dtype=torch.int32, device=device)
        self.loads = torch.zeros(E, **i32)
        self.chunks = torch.zeros(C, 4, **i32)
        self.chunk_row = torch.zeros(C, **i32)
        self.expert_chunk_begin = torch.zeros(E + 1, **i32)
        self.groups = torch.zeros(C, 4, **i32)
        self.group_begin = torch.zeros(P + 1, **i32)
        self.device_rows = torch.zeros(P, **i32)
        self.xfers = torch.zeros(C, 3, **i32)
        self.rank_base = torch.zeros(max(1, llep_plan_rank_base_elems(params)), **i32)
        self.info = torch.zeros(8, **i32)
        self.struct = llep_plan_buffers(*[t.data_ptr() for t in (
            self.loads, self.chunks, self.chunk_row, self.expert_chunk_begin, self.groups,
            self.group_begin, self.device_rows, self.xfers, self.rank_base, self.info)])

    def info_dict(self) -> dict:
        v = self.info.cpu().tolist()
        return dict(zip(("status", "n_chunks", "n_groups", "n_xfers", "bypassed", "forced",
                         "max_device", "total_rows"), v))


# ---- the four steps and weight packing -----------------------------------------

def llep_plan(params: llep_plan_params, topk_ids, bufs: PlanBuffers, stream=None):
    _check(lib().llep_plan(ctypes.byref(params), _ptr(topk_ids), ctypes.byref(bufs.struct),
                           _stream(stream)), "llep_plan")


def llep_permute(params: llep_plan_params, bufs: PlanBuffers, topk_ids, topk_gates, x,
                 x_perm, gate_perm, row_pair, pair_row, stream=None):
    _check(lib().llep_permute(ctypes.byref(params), ctypes.byref(bufs.struct), _ptr(topk_ids),
                              _ptr(topk_gates), _ptr(x), x.shape[-1], _dtype_code(x),
                              _ptr(x_perm), _ptr(gate_perm), _ptr(row_pair), _ptr(pair_row),
                              _stream(stream)), "llep_permute")


def llep_pack_weights(w_gate, w_up, w_down, stream=None, out=None):
    """Packed copies of the expert weights (see llep.h); returns (gate_up, down).
    `out` = (gate_up, down) packs into those (contiguous) tensors instead, e.g.
    slices of a larger packed set filled a few experts at a time."""
    import torch
    E, D, F = w_gate.shape
    code = _dtype_code(w_gate)
    if out is None:
        gu = torch.empty((E, 2 * F, D), dtype=w_gate.dtype, device=w_gate.device)
        dn = torch.empty((E, D, F), dtype=w_gate.dtype, device=w_gate.device)
    else:
        gu, dn = out
        if (gu.numel() != E * 2 * F * D or dn.numel() != E * D * F or not gu.is_contiguous()
                or not dn.is_contiguous() or gu.dtype != w_gate.dtype or dn.dtype != w_gate.dtype):
            raise ValueError("out tensors do not match the weights")
    _check(lib().llep_pack_weights(E, D, F, code, _ptr(w_gate), _ptr(w_up), _ptr(w_down),
                                   _ptr(gu), _ptr(dn), _stream(stream)), "llep_pack_weights")
    return gu, dn


def llep_grouped_ffn(params: llep_plan_params, bufs: PlanBuffers, device: int, x_perm,
                     w_gate_up, w_down, out_perm, workspace, stream=None):
    D = x_perm.shape[-1]
    F = w_down.shape[-1]
    _check(lib().llep_grouped_ffn(ctypes.byref(params), ctypes.byref(bufs.struct), device,
                                  _ptr(x_perm), _ptr(w_gate_up), _ptr(w_down), D, F,
                                  _dtype_code(x_perm), _ptr(out_perm), _ptr(workspace),
                                  workspace.numel() * workspace.element_size(),
                                  _stream(stream)), "llep_grouped_ffn")


def llep_grouped_ffn_train(params: llep_plan_params, bufs: PlanBuffers, device: int, x_perm,
                           w_gate_up, w_down, out_perm, gate_up, workspace, stream=None):
    """llep_grouped_ffn that also keeps g and u ([T*K, 2F], interleaved per
    32 columns) for llep_grouped_ffn_backward."""
    D = x_perm.shape[-1]
    F = w_down.shape[-1]
    _check(lib().llep_grouped_ffn_train(ctypes.byref(params), ctypes.byref(bufs.struct), device,
                                        _ptr(x_perm), _ptr(w_gate_up), _ptr(w_down), D, F,
                                        _dtype_code(x_perm), _ptr(out_perm), _ptr(gate_up),
                                        _ptr(workspace),
                                        workspace.numel() * workspace.element_size(),
                                        _stream(stream)), "llep_grouped_ffn_train")


def llep_grouped_ffn_noalloc(params: llep_plan_params, bufs: PlanBuffers, device: int, x_perm,
                             w_gate_up, w_down, out_perm, stream=None):
    """llep_grouped_ffn with the library's own workspace array (no caller
    workspace; at most LLEP_NOALLOC_SCRATCH_BYTES)."""
    D = x_perm.shape[-1]
    F = w_down.shape[-1]
    _check(lib().llep_grouped_ffn_noalloc(ctypes.byref(params), ctypes.byref(bufs.struct),
                                          device, _ptr(x_perm), _ptr(w_gate_up), _ptr(w_down),
                                          D, F, _dtype_code(x_perm), _ptr(out_perm),
                                          _stream(stream)), "llep_grouped_ffn_noalloc")


def llep_combine(params: llep_plan_params, out_perm, pair_row, topk_gates, y, stream=None):
    _check(lib().llep_combine(ctypes.byref(params), _ptr(out_perm), _ptr(pair_row),
                              _ptr(topk_gates), out_perm.shape[-1], _dtype_code(out_perm),
                              _ptr(y), _stream(stream)), "llep_combine")


# ---- backward ------------------------------------------------------------------

def llep_combine_backward(params: llep_plan_params, out_perm, pair_row, topk_gates, dy,
                          d_out_perm, d_gates, stream=None):
    _check(lib().llep_combine_backward(ctypes.byref(params), _ptr(out_perm), _ptr(pair_row),
                                       _ptr(topk_gates), _ptr(dy), dy.shape[-1],
                                       _dtype_code(dy), _ptr(d_out_perm), _ptr(d_gates),
                                       _stream(stream)), "llep_combine_backward")


def llep_pack_weights_backward(w_gate, w_up, w_down, stream=None):
    """Packed weights of the backward GEMMs (see llep.h); returns
    (gate_up_t, down_t)."""
    import torch
    E, D, F = w_gate.shape
    gut = torch.empty((E, D, 2 * F), dtype=w_gate.dtype, device=w_gate.device)
    dnt = torch.empty((E, F, D), dtype=w_gate.dtype, device=w_gate.device)
    _check(lib().llep_pack_weights_backward(E, D, F, _dtype_code(w_gate), _ptr(w_gate),
                                            _ptr(w_up), _ptr(w_down), _ptr(gut), _ptr(dnt),
                                            _stream(stream)), "llep_pack_weights_backward")
    return gut, dnt


def llep_grouped_ffn_backward(params: llep_plan_params, bufs: PlanBuffers, device: int, x_perm,
                              d_out_perm, w_gate_up, w_gate_up_t, w_down_t, dx_perm, dw_gate,
                              dw_up, dw_down, workspace, stream=None, gate_up=None):
    """gate_up: the llep_grouped_ffn_train output (None: recompute g and u)."""
    D = x_perm.shape[-1]
    F = w_down_t.shape[-2]
    _check(lib().llep_grouped_ffn_backward(
        ctypes.byref(params), ctypes.byref(bufs.struct), device, _ptr(x_perm), _ptr(d_out_perm),
        _ptr(w_gate_up), _ptr(w_gate_up_t), _ptr(w_down_t), _ptr(gate_up), D, F,
        _dtype_code(x_perm),
        _ptr(dx_perm), _ptr(dw_gate), _ptr(dw_up), _ptr(dw_down), _ptr(workspace),
        workspace.numel() * workspace.element_size(), _stream(stream)),
        "llep_grouped_ffn_backward")
