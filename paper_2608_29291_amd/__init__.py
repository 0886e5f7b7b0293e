"""CE-Router routed block on MI355X (gfx950): thin Python binding of libce_router.so.

The five calls below have the names and arguments of the C ABI in
include/ce_router.h; this module only marshals torch tensors (device memory)
and the current HIP stream into pointers. Every step of the routed block runs
in the library's HIP kernels; there is no Python or CPU fallback. Importing
this package fails loudly when the library has not been built.

    ce_score             routing logits (Eq. 4) [+ sigmoid scores, Eq. 6]
    ce_topk_compact      per-sequence TopK (Eq. 6) + packed index maps [+ gather]
    ce_routed_ffn        SwiGLU FFN on the packed rows
    ce_scatter_residual  residual merge; dropped rows bypass
    ce_routed_block      all of the above, fused
    ce_drop_stability    drop-set Jaccard / RDA between two timesteps (Eq. 10-11)
    ce_ffn_down_colnorms, ce_ffn_saliency, ce_ffn_mask_channels
                         FFN-pruning saliency / leakage on the retained rows (Eq. 8-9)
    ce_layer_gap         layer-skipping redundancy gap of input/output cosines (Eq. 7)
    ce_routed_attention  attention over the packed retained tokens (compressed KV cache)
"""
from __future__ import annotations

import ctypes
import os
from dataclasses import dataclass
from typing import Optional, Sequence

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libce_router.so")

CE_OK, CE_ERR_INVALID_ARG, CE_ERR_UNSUPPORTED, CE_ERR_WORKSPACE, CE_ERR_HIP = 0, -1, -2, -3, -4
CE_F32, CE_BF16 = 0, 1
CE_TOK_GEN, CE_TOK_KEEP = 1, 2
CE_DEV_BAD_OFFSETS, CE_DEV_OVERFLOW = 1, 2
CE_WS_TOPK, CE_WS_FFN, CE_WS_BLOCK = 0, 1, 2

EXPORTED = [
    "ce_status_string", "ce_version", "ce_num_keep", "ce_kept_count_host", "ce_workspace_size",
    "ce_workspace_status", "ce_score", "ce_topk_compact", "ce_routed_ffn", "ce_ffn_gateup",
    "ce_ffn_down", "ce_scatter_residual", "ce_routed_block", "ce_drop_stability",
    "ce_ffn_down_colnorms", "ce_ffn_saliency", "ce_ffn_mask_channels", "ce_layer_gap",
    "ce_routed_attention", "ce_score_tiling",
]


class CERouterError(RuntimeError):
    def __init__(self, status: int, where: str):
        self.status = status
        super().__init__(f"{where}: {lib.ce_status_string(status).decode()} (status {status})")


if not os.path.exists(LIB_PATH):
    raise ImportError(
        f"{LIB_PATH} is missing: build it first with `python paper_2608_29291_amd/build.py` "
        "(hipcc, gfx950). There is no fallback path.")

# torch ships its own libamdhip64 (soname libamdhip64.so.7). Loading torch
# first makes this library bind to that same HIP runtime; loading it first
# would pull in a second runtime that cannot see torch's allocations.
import torch  # noqa: E402,F401

lib = ctypes.CDLL(LIB_PATH)

_p = ctypes.c_void_p
_i32 = ctypes.c_int32


class CEBatch(ctypes.Structure):
    _fields_ = [("B", _i32), ("T", _i32), ("seq_offsets", _p), ("flags", _p), ("t", _p),
                ("keep", ctypes.c_float), ("kept_capacity", _i32)]


class CEScorerW(ctypes.Structure):
    _fields_ = [("d", _i32), ("r_core", _i32), ("r_exp", _i32), ("n_seg", _i32), ("dtype", _i32),
                ("w1_core", _p), ("b1_core", _p), ("w2_core", _p), ("b2_core", ctypes.c_float),
                ("w1_exp", _p), ("b1_exp", _p), ("w2_exp", _p), ("b2_exp", _p)]


class CEFFNW(ctypes.Structure):
    _fields_ = [("d", _i32), ("d_ff", _i32), ("n_sets", _i32), ("dtype", _i32),
                ("w_gate", _p * 2), ("w_up", _p * 2), ("w_down", _p * 2)]


class CEAttn(ctypes.Structure):
    _fields_ = [("B", _i32), ("n_heads", _i32), ("n_kv_heads", _i32), ("head_dim", _i32),
                ("q_offsets", _p), ("kv_offsets", _p), ("q_capacity", _i32), ("kv_capacity", _i32),
                ("causal", _i32), ("scale", ctypes.c_float), ("dtype", _i32)]


def _sig(name, res, args):
    f = getattr(lib, name)
    f.restype = res
    f.argtypes = args
    return f


_sig("ce_status_string", ctypes.c_char_p, [ctypes.c_int])
_sig("ce_version", ctypes.c_char_p, [])
_sig("ce_num_keep", _i32, [ctypes.c_float, _i32])
_sig("ce_kept_count_host", ctypes.c_int64, [_i32, _i32, _p, _p, ctypes.c_float])
_sig("ce_workspace_size", ctypes.c_size_t, [ctypes.c_int, ctypes.POINTER(CEBatch), _i32, _i32, ctypes.c_int])
_sig("ce_workspace_status", ctypes.c_int, [_p, ctypes.POINTER(ctypes.c_uint32), _p])
_sig("ce_score", ctypes.c_int, [ctypes.POINTER(CEBatch), _p, ctypes.POINTER(CEScorerW), _p, _p, _p])
_sig("ce_topk_compact", ctypes.c_int, [ctypes.POINTER(CEBatch), _p, _p, ctypes.c_int, _i32, _p, _p, _p,
                                       _p, _p, ctypes.c_size_t, _p])
_sig("ce_routed_ffn", ctypes.c_int, [ctypes.POINTER(CEBatch), _p, _p, _p, ctypes.POINTER(CEFFNW), _p, _p,
                                     ctypes.c_size_t, _p])
_sig("ce_ffn_gateup", ctypes.c_int, [ctypes.POINTER(CEBatch), _p, _p, _p, ctypes.POINTER(CEFFNW), _p, _p,
                                     ctypes.c_size_t, _p])
_sig("ce_ffn_down", ctypes.c_int, [ctypes.POINTER(CEBatch), _p, _p, _p, ctypes.POINTER(CEFFNW), _p, _p,
                                   ctypes.c_size_t, _p])
_sig("ce_scatter_residual", ctypes.c_int, [ctypes.POINTER(CEBatch), _p, _p, _p, ctypes.c_int, _i32, _p,
                                           _p, _p])
_sig("ce_routed_block", ctypes.c_int, [ctypes.POINTER(CEBatch), _p, _p, ctypes.POINTER(CEScorerW),
                                       ctypes.POINTER(CEFFNW), _p, _p, _p, _p, ctypes.c_size_t, _p])
_sig("ce_drop_stability", ctypes.c_int, [ctypes.POINTER(CEBatch), _p, _p, _p, _p, _p, _p])
_sig("ce_ffn_down_colnorms", ctypes.c_int, [ctypes.POINTER(CEFFNW), _p, _p])
_sig("ce_ffn_saliency", ctypes.c_int, [ctypes.POINTER(CEBatch), _p, _p, _p, ctypes.POINTER(CEFFNW), _p, _p,
                                       ctypes.c_float, _p, _p, _p, _p, ctypes.c_size_t, _p])
_sig("ce_ffn_mask_channels", ctypes.c_int, [ctypes.POINTER(CEBatch), _p, _p, ctypes.c_int, _i32, _p, _p, _p])
_sig("ce_routed_attention", ctypes.c_int, [ctypes.POINTER(CEAttn), _p, _p, _p, _p, _p])
_sig("ce_score_tiling", ctypes.c_int, [ctypes.POINTER(CEBatch), ctypes.POINTER(CEScorerW), _p])
_sig("ce_layer_gap", ctypes.c_int, [ctypes.POINTER(CEBatch), _p, _p, ctypes.c_int, _i32, _p, ctypes.c_float,
                                    _p, _p, _p, _p, _p, _p])


# ----------------------------------------------------------------------------
# marshalling helpers
# ----------------------------------------------------------------------------

def _ptr(t) -> Optional[int]:
    if t is None:
        return None
    if not t.is_contiguous():
        raise ValueError("tensor must be contiguous")
    return t.data_ptr()


def _dev_ptr(t) -> Optional[int]:
    if t is None:
        return None
    if not t.is_cuda:
        raise ValueError("tensor must live in GPU memory")
    return _ptr(t)


def _dtype_code(t) -> int:
    import torch
    if t.dtype == torch.bfloat16:
        return CE_BF16
    if t.dtype == torch.float32:
        return CE_F32
    raise ValueError(f"unsupported dtype {t.dtype}")


def _stream(stream) -> Optional[int]:
    import torch
    if stream is None:
        stream = torch.cuda.current_stream()
    return stream.cuda_stream


def _check(status: int, where: str):
    if status != CE_OK:
        raise CERouterError(status, where)


@dataclass
class Batch:
    """A ragged batch on the device: seq_offsets int32 [B+1], flags uint8 [T], t float32 [B]."""
    seq_offsets: "object"
    flags: "object"
    t: "object"
    keep: float
    kept_capacity: int

    @property
    def B(self) -> int:
        return int(self.seq_offsets.numel() - 1)

    @property
    def T(self) -> int:
        return int(self.flags.numel())

    def c(self) -> CEBatch:
        return CEBatch(self.B, self.T, _dev_ptr(self.seq_offsets), _dev_ptr(self.flags),
                       _dev_ptr(self.t), float(self.keep), int(self.kept_capacity))


@dataclass
class Scorer:
    """Device tensors of one layer's router (core + n_seg expansions)."""
    w1_core: "object"
    w2_core: "object"
    w1_exp: "object"
    w2_exp: "object"
    b1_core: "object" = None
    b2_core: float = 0.0
    b1_exp: "object" = None
    b2_exp: "object" = None

    def c(self) -> CEScorerW:
        r_c, d = self.w1_core.shape
        n_seg, r_e = (self.w1_exp.shape[0], self.w1_exp.shape[1]) if self.w1_exp is not None else (1, 0)
        return CEScorerW(int(d), int(r_c), int(r_e), int(n_seg), _dtype_code(self.w1_core),
                         _dev_ptr(self.w1_core), _dev_ptr(self.b1_core), _dev_ptr(self.w2_core),
                         float(self.b2_core), _dev_ptr(self.w1_exp), _dev_ptr(self.b1_exp),
                         _dev_ptr(self.w2_exp), _dev_ptr(self.b2_exp))


@dataclass
class FFN:
    """SwiGLU weight sets (1, or 2 for MoT): gate/up [F, d], down [d, F] per set."""
    w_gate: Sequence
    w_up: Sequence
    w_down: Sequence

    def c(self) -> CEFFNW:
        n = len(self.w_gate)
        F, d = self.w_gate[0].shape
        s = CEFFNW(int(d), int(F), int(n), _dtype_code(self.w_gate[0]))
        for i in range(n):
            s.w_gate[i] = _dev_ptr(self.w_gate[i])
            s.w_up[i] = _dev_ptr(self.w_up[i])
            s.w_down[i] = _dev_ptr(self.w_down[i])
        return s


# ----------------------------------------------------------------------------
# C-ABI calls
# ----------------------------------------------------------------------------

def ce_version() -> str:
    return lib.ce_version().decode()


def ce_num_keep(keep: float, n_routable: int) -> int:
    return int(lib.ce_num_keep(ctypes.c_float(keep), int(n_routable)))


def ce_kept_count_host(seq_offsets, flags, keep: float) -> int:
    """Exact packed row count Kt from host (numpy) seq_offsets int32 [B+1] and flags uint8 [T]."""
    import numpy as np
    offs = np.ascontiguousarray(seq_offsets, dtype=np.int32)
    fl = np.ascontiguousarray(flags, dtype=np.uint8)
    return int(lib.ce_kept_count_host(len(offs) - 1, len(fl), offs.ctypes.data, fl.ctypes.data,
                                      ctypes.c_float(keep)))


def ce_workspace_size(which: int, batch: Batch, d: int, d_ff: int, dtype: int) -> int:
    cb = batch.c()
    return int(lib.ce_workspace_size(which, ctypes.byref(cb), int(d), int(d_ff), int(dtype)))


def alloc_workspace(which: int, batch: Batch, d: int, d_ff: int, dtype: int, device="cuda"):
    """Caller-owned workspace (uint8 device tensor, 256-byte aligned by torch's allocator)."""
    import torch
    n = ce_workspace_size(which, batch, d, d_ff, dtype)
    return torch.empty(max(n, 256), dtype=torch.uint8, device=device)


def ce_workspace_status(ws, stream=None) -> int:
    out = ctypes.c_uint32(0)
    _check(lib.ce_workspace_status(_dev_ptr(ws), ctypes.byref(out), _stream(stream)),
           "ce_workspace_status")
    return int(out.value)


def ce_score(batch: Batch, hidden, scorer: Scorer, logits, probs=None, stream=None):
    cb, sw = batch.c(), scorer.c()
    _check(lib.ce_score(ctypes.byref(cb), _dev_ptr(hidden), ctypes.byref(sw), _dev_ptr(logits),
                        _dev_ptr(probs), _stream(stream)), "ce_score")


def ce_topk_compact(batch: Batch, logits, kept_idx, kept_offsets, ws, token_pos=None,
                    hidden=None, compact=None, stream=None):
    cb = batch.c()
    dtype = _dtype_code(hidden) if hidden is not None else CE_F32
    d = int(hidden.shape[1]) if hidden is not None else 0
    _check(lib.ce_topk_compact(ctypes.byref(cb), _dev_ptr(logits), _dev_ptr(hidden), dtype, d,
                               _dev_ptr(kept_idx), _dev_ptr(kept_offsets), _dev_ptr(token_pos),
                               _dev_ptr(compact), _dev_ptr(ws), ws.numel(), _stream(stream)),
           "ce_topk_compact")


def ce_routed_ffn(batch: Batch, compact, kept_idx, kept_offsets, ffn: FFN, ffn_out, ws, stream=None):
    cb, fw = batch.c(), ffn.c()
    _check(lib.ce_routed_ffn(ctypes.byref(cb), _dev_ptr(compact), _dev_ptr(kept_idx),
                             _dev_ptr(kept_offsets), ctypes.byref(fw), _dev_ptr(ffn_out),
                             _dev_ptr(ws), ws.numel(), _stream(stream)), "ce_routed_ffn")


def ce_ffn_gateup(batch: Batch, compact, kept_idx, kept_offsets, ffn: FFN, act, ws, stream=None):
    cb, fw = batch.c(), ffn.c()
    _check(lib.ce_ffn_gateup(ctypes.byref(cb), _dev_ptr(compact), _dev_ptr(kept_idx),
                             _dev_ptr(kept_offsets), ctypes.byref(fw), _dev_ptr(act),
                             _dev_ptr(ws), ws.numel(), _stream(stream)), "ce_ffn_gateup")


def ce_ffn_down(batch: Batch, act, kept_idx, kept_offsets, ffn: FFN, ffn_out, ws, stream=None):
    cb, fw = batch.c(), ffn.c()
    _check(lib.ce_ffn_down(ctypes.byref(cb), _dev_ptr(act), _dev_ptr(kept_idx),
                           _dev_ptr(kept_offsets), ctypes.byref(fw), _dev_ptr(ffn_out),
                           _dev_ptr(ws), ws.numel(), _stream(stream)), "ce_ffn_down")


def ce_scatter_residual(batch: Batch, ffn_out, kept_idx, kept_offsets, hidden_in, hidden_out,
                        stream=None):
    cb = batch.c()
    _check(lib.ce_scatter_residual(ctypes.byref(cb), _dev_ptr(ffn_out), _dev_ptr(kept_idx),
                                   _dev_ptr(kept_offsets), _dtype_code(hidden_in),
                                   int(hidden_in.shape[1]), _dev_ptr(hidden_in),
                                   _dev_ptr(hidden_out), _stream(stream)), "ce_scatter_residual")


def ce_routed_block(batch: Batch, hidden_in, hidden_out, scorer: Scorer, ffn: FFN, ws,
                    logits_out=None, kept_idx_out=None, kept_offsets_out=None, stream=None):
    cb, sw, fw = batch.c(), scorer.c(), ffn.c()
    _check(lib.ce_routed_block(ctypes.byref(cb), _dev_ptr(hidden_in), _dev_ptr(hidden_out),
                               ctypes.byref(sw), ctypes.byref(fw), _dev_ptr(logits_out),
                               _dev_ptr(kept_idx_out), _dev_ptr(kept_offsets_out), _dev_ptr(ws),
                               ws.numel(), _stream(stream)), "ce_routed_block")


def ce_score_tiling(batch: Batch, scorer: Scorer):
    """(tm, tn) of the rank-tiled scorer ce_routed_block uses for this batch,
    or (token_tile, 0) for the single-launch scorer (host query, no GPU work)."""
    cb, sw = batch.c(), scorer.c()
    out = (ctypes.c_int32 * 2)()
    r = lib.ce_score_tiling(ctypes.byref(cb), ctypes.byref(sw), out)
    if r < 0:
        _check(r, "ce_score_tiling")
    return int(out[0]), int(out[1])


def ce_drop_stability(batch: Batch, token_pos_t, token_pos_ref, jaccard, j_rand=None, rda=None,
                      stream=None):
    cb = batch.c()
    _check(lib.ce_drop_stability(ctypes.byref(cb), _dev_ptr(token_pos_t), _dev_ptr(token_pos_ref),
                                 _dev_ptr(jaccard), _dev_ptr(j_rand), _dev_ptr(rda), _stream(stream)),
           "ce_drop_stability")


def ce_ffn_down_colnorms(ffn: FFN, norms, stream=None):
    fw = ffn.c()
    _check(lib.ce_ffn_down_colnorms(ctypes.byref(fw), _dev_ptr(norms), _stream(stream)), "ce_ffn_down_colnorms")


def ce_ffn_saliency(batch: Batch, act, kept_idx, kept_offsets, ffn: FFN, norms, prune_mask, delta,
                    saliency, leakage, ws, use_pruned=None, stream=None):
    cb, fw = batch.c(), ffn.c()
    _check(lib.ce_ffn_saliency(ctypes.byref(cb), _dev_ptr(act), _dev_ptr(kept_idx), _dev_ptr(kept_offsets),
                               ctypes.byref(fw), _dev_ptr(norms), _dev_ptr(prune_mask), float(delta),
                               _dev_ptr(saliency), _dev_ptr(leakage), _dev_ptr(use_pruned), _dev_ptr(ws),
                               ws.numel(), _stream(stream)), "ce_ffn_saliency")


def ce_ffn_mask_channels(batch: Batch, act, kept_offsets, prune_mask, use_pruned, stream=None):
    cb = batch.c()
    _check(lib.ce_ffn_mask_channels(ctypes.byref(cb), _dev_ptr(act), _dev_ptr(kept_offsets), _dtype_code(act),
                                    int(act.shape[1]), _dev_ptr(prune_mask), _dev_ptr(use_pruned),
                                    _stream(stream)), "ce_ffn_mask_channels")



def ce_layer_gap(batch: Batch, x_in, x_out, token_pos, delta, cos, rho_all, rho_ret, gap, skip=None,
                 stream=None):
    cb = batch.c()
    _check(lib.ce_layer_gap(ctypes.byref(cb), _dev_ptr(x_in), _dev_ptr(x_out), _dtype_code(x_in),
                            int(x_in.shape[1]), _dev_ptr(token_pos), float(delta), _dev_ptr(cos),
                            _dev_ptr(rho_all), _dev_ptr(rho_ret), _dev_ptr(gap), _dev_ptr(skip),
                            _stream(stream)), "ce_layer_gap")



def ce_routed_attention(q, k, v, o, q_offsets, kv_offsets, causal, scale, stream=None):
    """q, o [rows, H, head_dim], k, v [rows, H_kv, head_dim] bf16 device tensors;
    q_offsets / kv_offsets int32 device tensors [B+1]."""
    at = CEAttn(int(q_offsets.numel() - 1), int(q.shape[1]), int(k.shape[1]), int(q.shape[2]),
                _dev_ptr(q_offsets), _dev_ptr(kv_offsets), int(q.shape[0]), int(k.shape[0]),
                int(bool(causal)), float(scale), _dtype_code(q))
    _check(lib.ce_routed_attention(ctypes.byref(at), _dev_ptr(q), _dev_ptr(k), _dev_ptr(v), _dev_ptr(o),
                                   _stream(stream)), "ce_routed_attention")


__all__ = [
    "Batch", "Scorer", "FFN", "CERouterError", "lib", "alloc_workspace",
    "ce_version", "ce_num_keep", "ce_kept_count_host", "ce_workspace_size", "ce_workspace_status",
    "ce_score", "ce_topk_compact", "ce_routed_ffn", "ce_ffn_gateup", "ce_ffn_down",
    "ce_scatter_residual", "ce_routed_block", "ce_drop_stability",
    "ce_ffn_down_colnorms", "ce_ffn_saliency", "ce_ffn_mask_channels", "ce_layer_gap",
    "ce_routed_attention", "CEAttn",
    "CE_F32", "CE_BF16", "CE_TOK_GEN", "CE_TOK_KEEP", "CE_WS_TOPK", "CE_WS_FFN", "CE_WS_BLOCK",
    "CE_DEV_BAD_OFFSETS", "CE_DEV_OVERFLOW",
]
