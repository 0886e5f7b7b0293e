"""CE-Router routed block on MI355X (gfx950): thin Python binding of libce_router.so.

The calls below have the names and arguments of the C ABI in
include/ce_router.h; this module only checks and marshals torch tensors
(device memory) and the current HIP stream into pointers. Every step of the
routed block runs in the library's HIP kernels; there is no Python or CPU
fallback. Importing this package fails loudly when the library has not been
built.

    ce_score, ce_score_ws  routing logits (Eq. 4) [+ sigmoid scores, Eq. 6];
                           ce_score_ws with a workspace runs the fused block's scorer
    ce_topk_compact        per-sequence TopK (Eq. 6) + packed index maps [+ gather]
    ce_topk_compact_noalloc  the same without a workspace (a fixed device array)
    ce_routed_ffn          SwiGLU FFN on the packed rows (ce_ffn_gateup + ce_ffn_down)
    ce_routed_ffn_pruned   the FFN with the pruning choice (Eq. 8-9) fused in
    ce_scatter_residual    residual merge; dropped rows bypass
    ce_routed_block        all of the above, fused; ce_routed_block_gap adds the
                           layer-skipping gap (Eq. 7) from the down GEMM's epilogue
    ce_drop_stability      drop-set Jaccard / RDA between two timesteps (Eq. 10-11)
    ce_ffn_down_colnorms, ce_ffn_saliency, ce_ffn_mask_channels
                           FFN-pruning saliency / leakage on the retained rows (Eq. 8-9)
    ce_layer_gap           layer-skipping redundancy gap of input/output cosines (Eq. 7)
    ce_routed_attention    attention over the packed retained tokens (compressed KV cache)
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
CE_WS_TOPK, CE_WS_FFN, CE_WS_BLOCK, CE_WS_BLOCK_GAP, CE_WS_FFN_PRUNED, CE_WS_SCORE = 0, 1, 2, 3, 4, 5

EXPORTED = [
    "ce_status_string", "ce_version", "ce_num_keep", "ce_kept_count_host", "ce_workspace_size",
    "ce_workspace_status", "ce_score", "ce_topk_compact", "ce_routed_ffn", "ce_ffn_gateup",
    "ce_ffn_down", "ce_scatter_residual", "ce_routed_block", "ce_drop_stability",
    "ce_ffn_down_colnorms", "ce_ffn_saliency", "ce_ffn_mask_channels", "ce_layer_gap",
    "ce_routed_attention", "ce_score_tiling", "ce_topk_compact_noalloc", "ce_routed_block_gap",
    "ce_routed_ffn_pruned", "ce_score_ws",
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
_sig("ce_score_ws", ctypes.c_int, [ctypes.POINTER(CEBatch), _p, ctypes.POINTER(CEScorerW), _p, _p, _p,
                                   ctypes.c_size_t, _p])
_sig("ce_topk_compact", ctypes.c_int, [ctypes.POINTER(CEBatch), _p, _p, ctypes.c_int, _i32, _p, _p, _p,
                                       _p, _p, ctypes.c_size_t, _p])
_sig("ce_topk_compact_noalloc", ctypes.c_int, [ctypes.POINTER(CEBatch), _p, _p, ctypes.c_int, _i32, _p, _p,
                                               _p, _p, _p, _p])
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
_sig("ce_routed_block_gap", ctypes.c_int, [ctypes.POINTER(CEBatch), _p, _p, ctypes.POINTER(CEScorerW),
                                           ctypes.POINTER(CEFFNW), _p, _p, _p, ctypes.c_float, _p, _p, _p, _p, _p,
                                           _p, ctypes.c_size_t, _p])
_sig("ce_routed_ffn_pruned", ctypes.c_int, [ctypes.POINTER(CEBatch), _p, _p, _p, ctypes.POINTER(CEFFNW), _p, _i32,
                                            ctypes.c_float, _p, _p, _p, _p, _p, ctypes.c_size_t, _p])
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
#
# The library sees only pointers, so the binding checks what a pointer cannot
# carry before every call: dtype, shape or element count, contiguity, 16-byte
# alignment and the device. A wrong size or a sliced, misaligned tensor would
# otherwise become an out-of-bounds or misaligned access on the GPU. These are
# argument checks only; the routed block's arithmetic all runs in the library.

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


def _torch_dtype(code: int):
    import torch
    return {CE_BF16: torch.bfloat16, CE_F32: torch.float32}[code]


def _chk(t, name: str, dtype=None, numel: Optional[int] = None, shape=None, rows_min: Optional[int] = None,
         optional: bool = False):
    """Validate one device tensor argument; returns its pointer (None for an
    absent optional argument).

    dtype     required torch dtype
    numel     minimum element count
    shape     exact shape (a tuple; None entries match any size)
    rows_min  for matrices given by `shape` with a None row count: at least
              this many rows
    """
    import torch
    if t is None:
        if optional:
            return None
        raise ValueError(f"{name}: required tensor is missing")
    if not isinstance(t, torch.Tensor):
        raise ValueError(f"{name}: expected a torch.Tensor, got {type(t).__name__}")
    if not t.is_cuda:
        raise ValueError(f"{name}: tensor must live in GPU memory")
    if t.device.index != torch.cuda.current_device():
        raise ValueError(f"{name}: tensor is on {t.device}, the current device is "
                         f"cuda:{torch.cuda.current_device()}")
    if not t.is_contiguous():
        raise ValueError(f"{name}: tensor must be contiguous")
    if dtype is not None and t.dtype != dtype:
        raise ValueError(f"{name}: dtype {t.dtype}, expected {dtype}")
    if t.numel() > 0 and t.data_ptr() % 16 != 0:
        raise ValueError(f"{name}: data pointer is not 16-byte aligned")
    if numel is not None and t.numel() < numel:
        raise ValueError(f"{name}: {t.numel()} elements, need at least {numel}")
    if shape is not None:
        if t.dim() != len(shape) or any(s is not None and int(d) != int(s) for d, s in zip(t.shape, shape)):
            raise ValueError(f"{name}: shape {tuple(t.shape)}, expected {tuple(shape)}")
        if rows_min is not None and t.shape[0] < rows_min:
            raise ValueError(f"{name}: {t.shape[0]} rows, need at least {rows_min}")
    return t.data_ptr()


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
        import torch
        so = _chk(self.seq_offsets, "seq_offsets", torch.int32, numel=2)
        if self.seq_offsets.dim() != 1:
            raise ValueError("seq_offsets must be 1-D [B+1]")
        if self.flags is None or self.flags.dim() != 1:
            raise ValueError("flags must be a 1-D uint8 tensor [T]")
        fl = _chk(self.flags, "flags", torch.uint8)
        tp = _chk(self.t, "t", torch.float32, numel=self.B, optional=True)
        if int(self.kept_capacity) < 0:
            raise ValueError("kept_capacity must be >= 0")
        return CEBatch(self.B, self.T, so, fl, tp, float(self.keep), int(self.kept_capacity))


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

    @property
    def d(self) -> int:
        return int(self.w1_core.shape[1])

    @property
    def dtype(self) -> int:
        return _dtype_code(self.w1_core)

    def c(self) -> CEScorerW:
        import torch
        if self.w1_core is None or self.w1_core.dim() != 2:
            raise ValueError("w1_core must be a matrix [r_core, d]")
        r_c, d = (int(x) for x in self.w1_core.shape)
        tdt = self.w1_core.dtype
        _dtype_code(self.w1_core)
        if self.w1_exp is not None:
            if self.w1_exp.dim() != 3:
                raise ValueError("w1_exp must be [n_seg, r_exp, d]")
            n_seg, r_e = int(self.w1_exp.shape[0]), int(self.w1_exp.shape[1])
        else:
            n_seg, r_e = 1, 0
        f32 = torch.float32
        ptrs = (_chk(self.w1_core, "w1_core", tdt, shape=(r_c, d)),
                _chk(self.b1_core, "b1_core", f32, shape=(r_c,), optional=True),
                _chk(self.w2_core, "w2_core", f32, shape=(r_c,)),
                _chk(self.w1_exp, "w1_exp", tdt, shape=(n_seg, r_e, d), optional=r_e == 0),
                _chk(self.b1_exp, "b1_exp", f32, shape=(n_seg, r_e), optional=True),
                _chk(self.w2_exp, "w2_exp", f32, shape=(n_seg, r_e), optional=r_e == 0),
                _chk(self.b2_exp, "b2_exp", f32, shape=(n_seg,), optional=True))
        return CEScorerW(d, r_c, r_e, n_seg, _dtype_code(self.w1_core), ptrs[0], ptrs[1], ptrs[2],
                         float(self.b2_core), ptrs[3], ptrs[4], ptrs[5], ptrs[6])


@dataclass
class FFN:
    """SwiGLU weight sets (1, or 2 for MoT): gate/up [F, d], down [d, F] per set."""
    w_gate: Sequence
    w_up: Sequence
    w_down: Sequence

    @property
    def d(self) -> int:
        return int(self.w_gate[0].shape[1])

    @property
    def d_ff(self) -> int:
        return int(self.w_gate[0].shape[0])

    def c(self) -> CEFFNW:
        n = len(self.w_gate)
        if n not in (1, 2) or len(self.w_up) != n or len(self.w_down) != n:
            raise ValueError("an FFN has 1 or 2 weight sets, each with gate, up and down")
        if self.w_gate[0] is None or self.w_gate[0].dim() != 2:
            raise ValueError("w_gate must be a matrix [d_ff, d]")
        F, d = (int(x) for x in self.w_gate[0].shape)
        tdt = self.w_gate[0].dtype
        s = CEFFNW(d, F, n, _dtype_code(self.w_gate[0]))
        for i in range(n):
            s.w_gate[i] = _chk(self.w_gate[i], f"w_gate[{i}]", tdt, shape=(F, d))
            s.w_up[i] = _chk(self.w_up[i], f"w_up[{i}]", tdt, shape=(F, d))
            s.w_down[i] = _chk(self.w_down[i], f"w_down[{i}]", tdt, shape=(d, F))
        return s


def _ws_ptr(ws, need: int):
    """Workspace pointer and size in bytes (any dtype; the library checks the size)."""
    p = _chk(ws, "ws")
    nbytes = ws.numel() * ws.element_size()
    if nbytes < need:
        raise ValueError(f"ws: {nbytes} bytes, need {need}")
    return p, nbytes


def _hidden(h, name, T, d, tdt):
    return _chk(h, name, tdt, shape=(T, d))


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
    _check(lib.ce_workspace_status(_chk(ws, "ws", numel=4), ctypes.byref(out), _stream(stream)),
           "ce_workspace_status")
    return int(out.value)


def ce_score(batch: Batch, hidden, scorer: Scorer, logits, probs=None, stream=None):
    import torch
    cb, sw = batch.c(), scorer.c()
    T = batch.T
    h = _hidden(hidden, "hidden", T, sw.d, _torch_dtype(sw.dtype) if sw.dtype in (0, 1) else None)
    _check(lib.ce_score(ctypes.byref(cb), h, ctypes.byref(sw),
                        _chk(logits, "logits", torch.float32, numel=T),
                        _chk(probs, "probs", torch.float32, numel=T, optional=True), _stream(stream)),
           "ce_score")


def ce_score_ws(batch: Batch, hidden, scorer: Scorer, logits, ws, probs=None, stream=None):
    """ce_score with a workspace (CE_WS_SCORE): the fused block's scorer,
    rank-tiled where ce_score_tiling picks it."""
    import torch
    cb, sw = batch.c(), scorer.c()
    T = batch.T
    h = _hidden(hidden, "hidden", T, sw.d, _torch_dtype(sw.dtype) if sw.dtype in (0, 1) else None)
    wp, wn = _ws_ptr(ws, ce_workspace_size(CE_WS_SCORE, batch, sw.d, 0, sw.dtype))
    _check(lib.ce_score_ws(ctypes.byref(cb), h, ctypes.byref(sw),
                           _chk(logits, "logits", torch.float32, numel=T),
                           _chk(probs, "probs", torch.float32, numel=T, optional=True), wp, wn, _stream(stream)),
           "ce_score_ws")


def ce_topk_compact(batch: Batch, logits, kept_idx, kept_offsets, ws, token_pos=None,
                    hidden=None, compact=None, stream=None):
    import torch
    cb = batch.c()
    T, B, cap = batch.T, batch.B, int(batch.kept_capacity)
    dtype = _dtype_code(hidden) if hidden is not None else CE_F32
    d = int(hidden.shape[1]) if hidden is not None and hidden.dim() == 2 else 0
    hp = cp = None
    if compact is not None:
        if hidden is None:
            raise ValueError("compact needs hidden")
        hp = _hidden(hidden, "hidden", T, d, hidden.dtype)
        cp = _chk(compact, "compact", hidden.dtype, shape=(None, d), rows_min=cap)
    i32 = torch.int32
    wp, wn = _ws_ptr(ws, ce_workspace_size(CE_WS_TOPK, batch, d if compact is not None else 0, 0,
                                           dtype if compact is not None else CE_F32))
    _check(lib.ce_topk_compact(ctypes.byref(cb), _chk(logits, "logits", torch.float32, numel=T), hp, dtype, d,
                               _chk(kept_idx, "kept_idx", i32, numel=cap),
                               _chk(kept_offsets, "kept_offsets", i32, numel=B + 1),
                               _chk(token_pos, "token_pos", i32, numel=T, optional=True), cp,
                               wp, wn, _stream(stream)),
           "ce_topk_compact")


def ce_topk_compact_noalloc(batch: Batch, logits, kept_idx, kept_offsets, token_pos=None, hidden=None,
                            compact=None, status=None, stream=None):
    """ce_topk_compact without a workspace (the library's fixed per-GPU
    scratch holds the summaries; calls overlapping on one GPU race). status:
    optional uint32-sized device tensor (int32 is accepted) for the status word."""
    import torch
    cb = batch.c()
    T, B, cap = batch.T, batch.B, int(batch.kept_capacity)
    dtype = _dtype_code(hidden) if hidden is not None else CE_F32
    d = int(hidden.shape[1]) if hidden is not None and hidden.dim() == 2 else 0
    hp = cp = None
    if compact is not None:
        if hidden is None:
            raise ValueError("compact needs hidden")
        hp = _hidden(hidden, "hidden", T, d, hidden.dtype)
        cp = _chk(compact, "compact", hidden.dtype, shape=(None, d), rows_min=cap)
    if status is not None and status.dtype not in (torch.int32, torch.uint32):
        raise ValueError("status must be a 4-byte integer tensor")
    i32 = torch.int32
    _check(lib.ce_topk_compact_noalloc(ctypes.byref(cb), _chk(logits, "logits", torch.float32, numel=T), hp,
                                       dtype, d, _chk(kept_idx, "kept_idx", i32, numel=cap),
                                       _chk(kept_offsets, "kept_offsets", i32, numel=B + 1),
                                       _chk(token_pos, "token_pos", i32, numel=T, optional=True), cp,
                                       _chk(status, "status", numel=1, optional=True), _stream(stream)),
           "ce_topk_compact_noalloc")


def _ffn_common(batch: Batch, ffn: FFN, kept_idx, kept_offsets):
    import torch
    cb, fw = batch.c(), ffn.c()
    cap = int(batch.kept_capacity)
    ki = _chk(kept_idx, "kept_idx", torch.int32, numel=cap)
    ko = _chk(kept_offsets, "kept_offsets", torch.int32, numel=batch.B + 1)
    tdt = ffn.w_gate[0].dtype
    need = ce_workspace_size(CE_WS_FFN, batch, fw.d, fw.d_ff, fw.dtype)
    return cb, fw, cap, ki, ko, tdt, need


def ce_routed_ffn(batch: Batch, compact, kept_idx, kept_offsets, ffn: FFN, ffn_out, ws, stream=None):
    cb, fw, cap, ki, ko, tdt, need = _ffn_common(batch, ffn, kept_idx, kept_offsets)
    wp, wn = _ws_ptr(ws, need)
    _check(lib.ce_routed_ffn(ctypes.byref(cb), _chk(compact, "compact", tdt, shape=(None, fw.d), rows_min=cap),
                             ki, ko, ctypes.byref(fw),
                             _chk(ffn_out, "ffn_out", tdt, shape=(None, fw.d), rows_min=cap),
                             wp, wn, _stream(stream)), "ce_routed_ffn")


def ce_ffn_gateup(batch: Batch, compact, kept_idx, kept_offsets, ffn: FFN, act, ws, stream=None):
    cb, fw, cap, ki, ko, tdt, need = _ffn_common(batch, ffn, kept_idx, kept_offsets)
    wp, wn = _ws_ptr(ws, need)
    _check(lib.ce_ffn_gateup(ctypes.byref(cb), _chk(compact, "compact", tdt, shape=(None, fw.d), rows_min=cap),
                             ki, ko, ctypes.byref(fw),
                             _chk(act, "act", tdt, shape=(None, fw.d_ff), rows_min=cap),
                             wp, wn, _stream(stream)), "ce_ffn_gateup")


def ce_ffn_down(batch: Batch, act, kept_idx, kept_offsets, ffn: FFN, ffn_out, ws, stream=None):
    cb, fw, cap, ki, ko, tdt, need = _ffn_common(batch, ffn, kept_idx, kept_offsets)
    wp, wn = _ws_ptr(ws, need)
    _check(lib.ce_ffn_down(ctypes.byref(cb), _chk(act, "act", tdt, shape=(None, fw.d_ff), rows_min=cap),
                           ki, ko, ctypes.byref(fw),
                           _chk(ffn_out, "ffn_out", tdt, shape=(None, fw.d), rows_min=cap),
                           wp, wn, _stream(stream)), "ce_ffn_down")


def ce_routed_ffn_pruned(batch: Batch, compact, kept_idx, kept_offsets, ffn: FFN, norms, n_keep, delta, ffn_out,
                         saliency, leakage, use_pruned, ws, stream=None):
    """SwiGLU FFN on the packed rows with the FFN-pruning decision (Eq. 8-9)
    taken from the gate/up epilogue's |z| sums; P = channels [n_keep, d_ff).
    ws: ce_workspace_size(CE_WS_FFN_PRUNED, ...) bytes."""
    import torch
    cb = batch.c()
    fw = ffn.c()
    cap, B = int(batch.kept_capacity), batch.B
    tdt = ffn.w_gate[0].dtype
    f32 = torch.float32
    wp, wn = _ws_ptr(ws, ce_workspace_size(CE_WS_FFN_PRUNED, batch, fw.d, fw.d_ff, fw.dtype))
    _check(lib.ce_routed_ffn_pruned(ctypes.byref(cb), _chk(compact, "compact", tdt, shape=(None, fw.d), rows_min=cap),
                                    _chk(kept_idx, "kept_idx", torch.int32, numel=cap),
                                    _chk(kept_offsets, "kept_offsets", torch.int32, numel=B + 1), ctypes.byref(fw),
                                    _chk(norms, "norms", f32, numel=fw.n_sets * fw.d_ff), int(n_keep), float(delta),
                                    _chk(ffn_out, "ffn_out", tdt, shape=(None, fw.d), rows_min=cap),
                                    _chk(saliency, "saliency", f32, numel=B * fw.d_ff),
                                    _chk(leakage, "leakage", f32, numel=B),
                                    _chk(use_pruned, "use_pruned", torch.uint8, numel=B), wp, wn, _stream(stream)),
           "ce_routed_ffn_pruned")


def ce_scatter_residual(batch: Batch, ffn_out, kept_idx, kept_offsets, hidden_in, hidden_out,
                        stream=None):
    import torch
    cb = batch.c()
    cap, T = int(batch.kept_capacity), batch.T
    if hidden_in is None or hidden_in.dim() != 2:
        raise ValueError("hidden_in must be a matrix [T, d]")
    d, tdt = int(hidden_in.shape[1]), hidden_in.dtype
    _check(lib.ce_scatter_residual(ctypes.byref(cb), _chk(ffn_out, "ffn_out", tdt, shape=(None, d), rows_min=cap),
                                   _chk(kept_idx, "kept_idx", torch.int32, numel=cap),
                                   _chk(kept_offsets, "kept_offsets", torch.int32, numel=batch.B + 1),
                                   _dtype_code(hidden_in), d, _hidden(hidden_in, "hidden_in", T, d, tdt),
                                   _hidden(hidden_out, "hidden_out", T, d, tdt), _stream(stream)),
           "ce_scatter_residual")


def ce_routed_block(batch: Batch, hidden_in, hidden_out, scorer: Scorer, ffn: FFN, ws,
                    logits_out=None, kept_idx_out=None, kept_offsets_out=None, stream=None):
    import torch
    cb, sw, fw = batch.c(), scorer.c(), ffn.c()
    T, cap = batch.T, int(batch.kept_capacity)
    if sw.d != fw.d or sw.dtype != fw.dtype:
        raise ValueError("scorer and FFN must agree on d and dtype")
    tdt = ffn.w_gate[0].dtype
    wp, wn = _ws_ptr(ws, ce_workspace_size(CE_WS_BLOCK, batch, fw.d, fw.d_ff, fw.dtype))
    _check(lib.ce_routed_block(ctypes.byref(cb), _hidden(hidden_in, "hidden_in", T, fw.d, tdt),
                               _hidden(hidden_out, "hidden_out", T, fw.d, tdt),
                               ctypes.byref(sw), ctypes.byref(fw),
                               _chk(logits_out, "logits_out", torch.float32, numel=T, optional=True),
                               _chk(kept_idx_out, "kept_idx_out", torch.int32, numel=cap, optional=True),
                               _chk(kept_offsets_out, "kept_offsets_out", torch.int32, numel=batch.B + 1,
                                    optional=True),
                               wp, wn, _stream(stream)), "ce_routed_block")


def ce_routed_block_gap(batch: Batch, hidden_in, hidden_out, scorer: Scorer, ffn: FFN, ws, delta, cos, rho_all,
                        rho_ret, gap, skip=None, logits_out=None, kept_idx_out=None, kept_offsets_out=None,
                        stream=None):
    """ce_routed_block plus the block's layer-skipping gap (Eq. 7) from its
    down GEMM's epilogue; ws: ce_workspace_size(CE_WS_BLOCK_GAP, ...) bytes."""
    import torch
    cb, sw, fw = batch.c(), scorer.c(), ffn.c()
    T, B, cap = batch.T, batch.B, int(batch.kept_capacity)
    if sw.d != fw.d or sw.dtype != fw.dtype:
        raise ValueError("scorer and FFN must agree on d and dtype")
    tdt = ffn.w_gate[0].dtype
    f32 = torch.float32
    wp, wn = _ws_ptr(ws, ce_workspace_size(CE_WS_BLOCK_GAP, batch, fw.d, fw.d_ff, fw.dtype))
    _check(lib.ce_routed_block_gap(ctypes.byref(cb), _hidden(hidden_in, "hidden_in", T, fw.d, tdt),
                                   _hidden(hidden_out, "hidden_out", T, fw.d, tdt),
                                   ctypes.byref(sw), ctypes.byref(fw),
                                   _chk(logits_out, "logits_out", f32, numel=T, optional=True),
                                   _chk(kept_idx_out, "kept_idx_out", torch.int32, numel=cap, optional=True),
                                   _chk(kept_offsets_out, "kept_offsets_out", torch.int32, numel=B + 1,
                                        optional=True),
                                   float(delta), _chk(cos, "cos", f32, numel=T), _chk(rho_all, "rho_all", f32, numel=B),
                                   _chk(rho_ret, "rho_ret", f32, numel=B), _chk(gap, "gap", f32, numel=B),
                                   _chk(skip, "skip", torch.uint8, numel=B, optional=True), wp, wn, _stream(stream)),
           "ce_routed_block_gap")


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
    import torch
    cb = batch.c()
    T, B = batch.T, batch.B
    i32, f32 = torch.int32, torch.float32
    _check(lib.ce_drop_stability(ctypes.byref(cb), _chk(token_pos_t, "token_pos_t", i32, numel=T),
                                 _chk(token_pos_ref, "token_pos_ref", i32, numel=T),
                                 _chk(jaccard, "jaccard", f32, numel=B),
                                 _chk(j_rand, "j_rand", f32, numel=B, optional=True),
                                 _chk(rda, "rda", f32, numel=B, optional=True), _stream(stream)),
           "ce_drop_stability")


def ce_ffn_down_colnorms(ffn: FFN, norms, stream=None):
    import torch
    fw = ffn.c()
    _check(lib.ce_ffn_down_colnorms(ctypes.byref(fw),
                                    _chk(norms, "norms", torch.float32, numel=fw.n_sets * fw.d_ff),
                                    _stream(stream)), "ce_ffn_down_colnorms")


def ce_ffn_saliency(batch: Batch, act, kept_idx, kept_offsets, ffn: FFN, norms, prune_mask, delta,
                    saliency, leakage, ws, use_pruned=None, stream=None):
    import torch
    cb, fw, cap, ki, ko, tdt, need = _ffn_common(batch, ffn, kept_idx, kept_offsets)
    B, F = batch.B, fw.d_ff
    f32, u8 = torch.float32, torch.uint8
    wp, wn = _ws_ptr(ws, need)
    _check(lib.ce_ffn_saliency(ctypes.byref(cb), _chk(act, "act", tdt, shape=(None, F), rows_min=cap), ki, ko,
                               ctypes.byref(fw), _chk(norms, "norms", f32, numel=fw.n_sets * F),
                               _chk(prune_mask, "prune_mask", u8, numel=F), float(delta),
                               _chk(saliency, "saliency", f32, numel=B * F), _chk(leakage, "leakage", f32, numel=B),
                               _chk(use_pruned, "use_pruned", u8, numel=B, optional=True), wp, wn,
                               _stream(stream)), "ce_ffn_saliency")


def ce_ffn_mask_channels(batch: Batch, act, kept_offsets, prune_mask, use_pruned, stream=None):
    import torch
    cb = batch.c()
    cap, B = int(batch.kept_capacity), batch.B
    if act is None or act.dim() != 2:
        raise ValueError("act must be a matrix [kept_capacity, d_ff]")
    F = int(act.shape[1])
    _check(lib.ce_ffn_mask_channels(ctypes.byref(cb), _chk(act, "act", act.dtype, shape=(None, F), rows_min=cap),
                                    _chk(kept_offsets, "kept_offsets", torch.int32, numel=B + 1), _dtype_code(act),
                                    F, _chk(prune_mask, "prune_mask", torch.uint8, numel=F),
                                    _chk(use_pruned, "use_pruned", torch.uint8, numel=B), _stream(stream)),
           "ce_ffn_mask_channels")


def ce_layer_gap(batch: Batch, x_in, x_out, token_pos, delta, cos, rho_all, rho_ret, gap, skip=None,
                 stream=None):
    import torch
    cb = batch.c()
    T, B = batch.T, batch.B
    if x_in is None or x_in.dim() != 2:
        raise ValueError("x_in must be a matrix [T, d]")
    d, tdt = int(x_in.shape[1]), x_in.dtype
    f32 = torch.float32
    _check(lib.ce_layer_gap(ctypes.byref(cb), _hidden(x_in, "x_in", T, d, tdt), _hidden(x_out, "x_out", T, d, tdt),
                            _dtype_code(x_in), d, _chk(token_pos, "token_pos", torch.int32, numel=T), float(delta),
                            _chk(cos, "cos", f32, numel=T), _chk(rho_all, "rho_all", f32, numel=B),
                            _chk(rho_ret, "rho_ret", f32, numel=B), _chk(gap, "gap", f32, numel=B),
                            _chk(skip, "skip", torch.uint8, numel=B, optional=True), _stream(stream)),
           "ce_layer_gap")


def ce_routed_attention(q, k, v, o, q_offsets, kv_offsets, causal, scale, stream=None):
    """q, o [rows, H, head_dim], k, v [rows, H_kv, head_dim] bf16 device tensors;
    q_offsets / kv_offsets int32 device tensors [B+1]."""
    import torch
    for name, x in (("q", q), ("k", k)):
        if x is None or x.dim() != 3:
            raise ValueError(f"{name} must be [rows, heads, head_dim]")
    if q_offsets is None or q_offsets.dim() != 1 or kv_offsets is None or kv_offsets.numel() != q_offsets.numel():
        raise ValueError("q_offsets and kv_offsets must be 1-D [B+1] of equal length")
    tdt = q.dtype
    qs, ks = tuple(int(x) for x in q.shape), tuple(int(x) for x in k.shape)
    B = int(q_offsets.numel() - 1)
    ptrs = (_chk(q, "q", tdt, shape=qs), _chk(k, "k", tdt, shape=ks), _chk(v, "v", tdt, shape=ks),
            _chk(o, "o", tdt, shape=qs), _chk(q_offsets, "q_offsets", torch.int32, numel=2),
            _chk(kv_offsets, "kv_offsets", torch.int32, numel=2))
    at = CEAttn(B, qs[1], ks[1], qs[2], ptrs[4], ptrs[5], qs[0], ks[0], int(bool(causal)), float(scale),
                _dtype_code(q))
    _check(lib.ce_routed_attention(ctypes.byref(at), ptrs[0], ptrs[1], ptrs[2], ptrs[3], _stream(stream)),
           "ce_routed_attention")


__all__ = [
    "Batch", "Scorer", "FFN", "CERouterError", "lib", "alloc_workspace",
    "ce_version", "ce_num_keep", "ce_kept_count_host", "ce_workspace_size", "ce_workspace_status",
    "ce_score", "ce_score_ws", "ce_topk_compact", "ce_topk_compact_noalloc", "ce_routed_ffn",
    "ce_routed_ffn_pruned", "ce_ffn_gateup", "ce_ffn_down",
    "ce_scatter_residual", "ce_routed_block", "ce_routed_block_gap", "ce_drop_stability",
    "ce_ffn_down_colnorms", "ce_ffn_saliency", "ce_ffn_mask_channels", "ce_layer_gap",
    "ce_routed_attention", "CEAttn",
    "CE_F32", "CE_BF16", "CE_TOK_GEN", "CE_TOK_KEEP", "CE_WS_TOPK", "CE_WS_FFN", "CE_WS_BLOCK", "CE_WS_BLOCK_GAP",
    "CE_WS_FFN_PRUNED", "CE_WS_SCORE",
    "CE_DEV_BAD_OFFSETS", "CE_DEV_OVERFLOW",
]
