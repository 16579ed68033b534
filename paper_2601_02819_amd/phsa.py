"""Thin ctypes binding over libphsa (see include/phsa.h).

Argument marshalling only: every step of PHSA runs in the HIP kernels of
``libphsa.so``.  torch supplies device memory and the current HIP stream.
If the library has not been built this module raises; there is no fallback.
"""
from __future__ import annotations

import contextlib
import ctypes
import dataclasses
import os
from typing import Dict, List, Optional, Tuple

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libphsa.so")
PROF_LIB_PATH = os.path.join(_HERE, "libphsa_prof.so")   # profiling build (include/phsa_prof.h)

(OK, ERR_INVALID_ARG, ERR_SHAPE, ERR_DTYPE, ERR_NULL, ERR_WORKSPACE, ERR_UNSUPPORTED, ERR_HIP,
 ERR_SCRATCH_LIMIT) = range(9)
NOALLOC_SCRATCH_BYTES = 64 << 20
BF16, FP32 = 0, 1
OP_COMPRESS, OP_SELECT, OP_ATTN_FWD, OP_ATTN_BWD, OP_FORWARD, OP_DECODE = range(6)
FLAG_REUSE_INDEX = 1
FLAG_SELECT_SOFTMAX_SUM = 2

MAX_PUNCT_IDS = 16384

EXPORTS = (
    "phsa_ksel", "phsa_validate", "phsa_workspace_size", "phsa_status_string", "phsa_punct_mask", "phsa_compress",
    "phsa_select", "phsa_attn_fwd", "phsa_attn_bwd", "phsa_forward", "phsa_decode", "phsa_decode_varlen",
    "phsa_cache_append", "phsa_select_noalloc",
)
PROF_EXPORTS = ("phsa_prof_enable", "phsa_prof_durations", "phsa_prof_reset")


class Params(ctypes.Structure):
    _fields_ = [
        ("batch", ctypes.c_int32), ("seqlen_q", ctypes.c_int32), ("seqlen_k", ctypes.c_int32),
        ("n_heads_q", ctypes.c_int32), ("n_heads_kv", ctypes.c_int32), ("head_dim", ctypes.c_int32),
        ("block_size", ctypes.c_int32), ("top_k", ctypes.c_int32), ("n_init_blocks", ctypes.c_int32),
        ("window", ctypes.c_int32), ("lam", ctypes.c_float), ("softmax_scale", ctypes.c_float),
        ("dtype", ctypes.c_int32), ("flags", ctypes.c_int32),
    ]


class PHSAError(RuntimeError):
    def __init__(self, status: int, where: str):
        super().__init__(f"{where}: {status_string(status)} (status {status})")
        self.status = status


_libs: Dict[str, ctypes.CDLL] = {}
_active: Optional[ctypes.CDLL] = None   # the library the calls below go to (libphsa.so unless profiling)


def _load(path: str) -> ctypes.CDLL:
    if path not in _libs:
        if not os.path.exists(path):
            raise RuntimeError(f"{path} is missing: build it with `python -m paper_2601_02819_amd.build`")
        L = ctypes.CDLL(path)
        P, PP = ctypes.POINTER(Params), ctypes.c_void_p
        sig = {
            "phsa_ksel": (ctypes.c_int32, [P]),
            "phsa_validate": (ctypes.c_int, [P, ctypes.c_int32]),
            "phsa_workspace_size": (ctypes.c_size_t, [P, ctypes.c_int32]),
            "phsa_status_string": (ctypes.c_char_p, [ctypes.c_int]),
            "phsa_punct_mask": (ctypes.c_int, [PP, ctypes.c_int64, PP, ctypes.c_int32, PP, PP]),
            "phsa_compress": (ctypes.c_int, [P, PP, PP, PP, PP]),
            "phsa_select": (ctypes.c_int, [P, PP, PP, PP, PP, ctypes.c_size_t, PP]),
            "phsa_attn_fwd": (ctypes.c_int, [P, PP, PP, PP, PP, PP, PP, PP, ctypes.c_size_t, PP]),
            "phsa_attn_bwd": (ctypes.c_int, [P] + [PP] * 11 + [ctypes.c_size_t, PP]),
            "phsa_forward": (ctypes.c_int, [P] + [PP] * 9 + [ctypes.c_size_t, PP]),
            "phsa_decode": (ctypes.c_int, [P] + [PP] * 8 + [ctypes.c_size_t, PP]),
            "phsa_decode_varlen": (ctypes.c_int, [P] + [PP] * 9 + [ctypes.c_size_t, PP]),
            "phsa_cache_append": (ctypes.c_int, [P] + [PP] * 8 + [PP]),
            "phsa_select_noalloc": (ctypes.c_int, [P, PP, PP, PP, PP]),
        }
        if path == PROF_LIB_PATH:
            sig.update({
                "phsa_prof_enable": (ctypes.c_int, [ctypes.c_int32]),
                "phsa_prof_durations": (ctypes.c_int32, [ctypes.c_char_p, ctypes.POINTER(ctypes.c_float),
                                                         ctypes.c_int32]),
                "phsa_prof_reset": (None, []),
            })
        for name, (res, args) in sig.items():
            f = getattr(L, name)
            f.restype = res
            f.argtypes = args
        _libs[path] = L
    return _libs[path]


def lib() -> ctypes.CDLL:
    """The loaded libphsa.so (raises if it has not been built)."""
    global _active
    if _active is None:
        _active = _load(LIB_PATH)
    return _active


class KernelTimes:
    """Per-launch kernel durations read from the profiling build."""

    def __init__(self, L: ctypes.CDLL):
        self._L = L

    def durations(self, name: str) -> List[float]:
        """Milliseconds of every recorded launch of kernel `name`, in launch order."""
        n = self._L.phsa_prof_durations(name.encode(), None, 0)
        buf = (ctypes.c_float * max(n, 1))()
        n = self._L.phsa_prof_durations(name.encode(), buf, n)
        return [float(buf[i]) for i in range(n)]

    def reset(self) -> None:
        self._L.phsa_prof_reset()


@contextlib.contextmanager
def profiling():
    """Routes the calls of this module to libphsa_prof.so, which records a pair
    of HIP events around each kernel launch on its stream, and yields a
    KernelTimes to read them.  The kernels are those of libphsa.so."""
    global _active
    prev = lib()
    L = _load(PROF_LIB_PATH)
    L.phsa_prof_reset()
    L.phsa_prof_enable(1)
    _active = L
    try:
        yield KernelTimes(L)
    finally:
        L.phsa_prof_enable(0)
        _active = prev


def status_string(status: int) -> str:
    return lib().phsa_status_string(int(status)).decode()


@dataclasses.dataclass(frozen=True)
class Config:
    """Algorithm 1 hyperparameters (block size m, top-k, n_init, window w, gate lambda)."""
    block_size: int = 64
    top_k: int = 12
    n_init_blocks: int = 1
    window: int = 0
    lam: float = 0.5
    softmax_scale: float = 0.0   # <= 0: 1 / sqrt(head_dim)
    softmax_sum: bool = False    # rank blocks by summed per-head softmax (else by summed logits)

    @property
    def ksel(self) -> int:
        return self.n_init_blocks + self.window // self.block_size + 1 + self.top_k


def make_params(cfg: Config, batch: int, seqlen_q: int, seqlen_k: int, n_heads_q: int, n_heads_kv: int,
                head_dim: int, dtype, flags: int = 0) -> Params:
    code = BF16 if dtype in (torch.bfloat16, BF16) else FP32 if dtype in (torch.float32, FP32) else 99
    return Params(batch, seqlen_q, seqlen_k, n_heads_q, n_heads_kv, head_dim, cfg.block_size, cfg.top_k,
                  cfg.n_init_blocks, cfg.window, cfg.lam, cfg.softmax_scale, code,
                  flags | (FLAG_SELECT_SOFTMAX_SUM if cfg.softmax_sum else 0))


def workspace_size(p: Params, op: int) -> int:
    return int(lib().phsa_workspace_size(ctypes.byref(p), op))


def _ptr(t: Optional[torch.Tensor]):
    return ctypes.c_void_p(t.data_ptr()) if t is not None else None


def _stream():
    return ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)


def _check(st: int, where: str):
    if st != OK:
        raise PHSAError(st, where)


def _dev(*ts):
    for t in ts:
        if not t.is_cuda or not t.is_contiguous():
            raise ValueError("tensors must be contiguous device tensors")


def _workspace(p: Params, op: int, ws: Optional[torch.Tensor], device) -> Optional[torch.Tensor]:
    need = workspace_size(p, op)
    if need == 0:
        return ws
    if ws is not None and ws.numel() >= need:
        return ws
    return torch.empty(need, dtype=torch.uint8, device=device)


def punct_mask(ids: torch.Tensor, punct_ids) -> torch.Tensor:
    """Token ids (int32 device tensor, any shape) -> uint8 punctuation mask of the same shape.

    punct_ids: the punctuation id set, as a host sequence (sorted and uploaded
    here) or an int32 device tensor already sorted ascending."""
    _dev(ids)
    if ids.dtype != torch.int32:
        raise ValueError("ids must be int32")
    if isinstance(punct_ids, torch.Tensor) and punct_ids.is_cuda:
        pset = punct_ids.contiguous()
        if pset.dtype != torch.int32:
            raise ValueError("punct_ids must be int32")
    else:
        import numpy as np
        host = np.unique(np.asarray(list(punct_ids) if not isinstance(punct_ids, torch.Tensor) else punct_ids.numpy(),
                                    dtype=np.int64))
        if host.size and (host[0] < -2**31 or host[-1] >= 2**31):
            raise ValueError("punctuation ids must fit int32")
        pset = torch.from_numpy(host.astype(np.int32)).to(ids.device)
    mask = torch.empty(ids.shape, dtype=torch.uint8, device=ids.device)
    _check(lib().phsa_punct_mask(_ptr(ids), ids.numel(), _ptr(pset) if pset.numel() else None, pset.numel(),
                                 _ptr(mask), _stream()), "phsa_punct_mask")
    return mask


def compress(k: torch.Tensor, punct: torch.Tensor, cfg: Config) -> torch.Tensor:
    """K [B, Lk, Hkv, d], punct uint8 [B, Lk] -> K_comp float32 [B, Hkv, T, d]."""
    _dev(k, punct)
    B, Lk, Hkv, d = k.shape
    p = make_params(cfg, B, Lk, Lk, Hkv, Hkv, d, k.dtype)
    kc = torch.empty(B, Hkv, Lk // cfg.block_size, d, dtype=torch.float32, device=k.device)
    _check(lib().phsa_compress(ctypes.byref(p), _ptr(k), _ptr(punct), _ptr(kc), _stream()), "phsa_compress")
    return kc


def select(q: torch.Tensor, kc: torch.Tensor, seqlen_k: int, cfg: Config,
           ws: Optional[torch.Tensor] = None) -> torch.Tensor:
    """Q [B, Lq, Hq, d], K_comp [B, Hkv, T, d] -> sel int32 [B, Hkv, Lq, Ksel]."""
    _dev(q, kc)
    B, Lq, Hq, d = q.shape
    Hkv = kc.shape[1]
    p = make_params(cfg, B, Lq, seqlen_k, Hq, Hkv, d, q.dtype)
    sel = torch.empty(B, Hkv, Lq, cfg.ksel, dtype=torch.int32, device=q.device)
    w = _workspace(p, OP_SELECT, ws, q.device)
    _check(lib().phsa_select(ctypes.byref(p), _ptr(q), _ptr(kc), _ptr(sel), _ptr(w), w.numel() if w is not None else 0,
                             _stream()), "phsa_select")
    return sel


def select_noalloc(q: torch.Tensor, kc: torch.Tensor, seqlen_k: int, cfg: Config,
                   sel: Optional[torch.Tensor] = None) -> torch.Tensor:
    """phsa_select_noalloc: as select(), with the library's fixed scratch instead
    of a workspace.  Pass `sel` (int32 [B, Hkv, Lq, Ksel]) to make the call itself
    allocate nothing."""
    _dev(q, kc)
    B, Lq, Hq, d = q.shape
    Hkv = kc.shape[1]
    p = make_params(cfg, B, Lq, seqlen_k, Hq, Hkv, d, q.dtype)
    if sel is None:
        sel = torch.empty(B, Hkv, Lq, cfg.ksel, dtype=torch.int32, device=q.device)
    _dev(sel)
    if sel.dtype != torch.int32 or tuple(sel.shape) != (B, Hkv, Lq, cfg.ksel):
        raise ValueError(f"sel must be int32 {(B, Hkv, Lq, cfg.ksel)}")
    _check(lib().phsa_select_noalloc(ctypes.byref(p), _ptr(q), _ptr(kc), _ptr(sel), _stream()),
           "phsa_select_noalloc")
    return sel


def attn_fwd(q, k, v, sel, cfg: Config, ws: Optional[torch.Tensor] = None) -> Tuple[torch.Tensor, torch.Tensor]:
    """Sparse attention forward -> (O [B, Lq, Hq, d], LSE float32 [B, Hq, Lq])."""
    _dev(q, k, v, sel)
    B, Lq, Hq, d = q.shape
    Lk, Hkv = k.shape[1], k.shape[2]
    p = make_params(cfg, B, Lq, Lk, Hq, Hkv, d, q.dtype)
    o = torch.empty_like(q)
    lse = torch.empty(B, Hq, Lq, dtype=torch.float32, device=q.device)
    w = _workspace(p, OP_ATTN_FWD, ws, q.device)
    _check(lib().phsa_attn_fwd(ctypes.byref(p), _ptr(q), _ptr(k), _ptr(v), _ptr(sel), _ptr(o), _ptr(lse), _ptr(w),
                               w.numel() if w is not None else 0, _stream()), "phsa_attn_fwd")
    return o, lse


def attn_bwd(q, k, v, o, do, lse, sel, cfg: Config, ws: Optional[torch.Tensor] = None, reuse_index: bool = False):
    """Sparse attention backward (selection fixed) -> (dQ, dK, dV).

    reuse_index=True: `ws` is the workspace of the forward call that produced
    o/lse from the same sel, and its inverted index is reused."""
    _dev(q, k, v, o, do, lse, sel)
    B, Lq, Hq, d = q.shape
    Lk, Hkv = k.shape[1], k.shape[2]
    p = make_params(cfg, B, Lq, Lk, Hq, Hkv, d, q.dtype, FLAG_REUSE_INDEX if reuse_index else 0)
    if reuse_index and (ws is None or ws.numel() < workspace_size(p, OP_ATTN_BWD)):
        raise ValueError("reuse_index needs the forward's workspace, sized for the backward")
    dq, dk, dv = torch.empty_like(q), torch.empty_like(k), torch.empty_like(v)
    w = _workspace(p, OP_ATTN_BWD, ws, q.device)
    _check(lib().phsa_attn_bwd(ctypes.byref(p), _ptr(q), _ptr(k), _ptr(v), _ptr(o), _ptr(do), _ptr(lse), _ptr(sel),
                               _ptr(dq), _ptr(dk), _ptr(dv), _ptr(w), w.numel() if w is not None else 0, _stream()),
           "phsa_attn_bwd")
    return dq, dk, dv


def forward(q, k, v, punct, cfg: Config, ws: Optional[torch.Tensor] = None):
    """compress + select + sparse attention -> (K_comp, sel, O, LSE)."""
    _dev(q, k, v, punct)
    B, Lq, Hq, d = q.shape
    Lk, Hkv = k.shape[1], k.shape[2]
    p = make_params(cfg, B, Lq, Lk, Hq, Hkv, d, q.dtype)
    kc = torch.empty(B, Hkv, Lk // cfg.block_size, d, dtype=torch.float32, device=q.device)
    sel = torch.empty(B, Hkv, Lq, cfg.ksel, dtype=torch.int32, device=q.device)
    o = torch.empty_like(q)
    lse = torch.empty(B, Hq, Lq, dtype=torch.float32, device=q.device)
    w = _workspace(p, OP_FORWARD, ws, q.device)
    _check(lib().phsa_forward(ctypes.byref(p), _ptr(q), _ptr(k), _ptr(v), _ptr(punct), _ptr(kc), _ptr(sel), _ptr(o),
                              _ptr(lse), _ptr(w), w.numel() if w is not None else 0, _stream()), "phsa_forward")
    return kc, sel, o, lse


def decode(q, k_cache, v_cache, kc, cfg: Config, ws: Optional[torch.Tensor] = None):
    """One decode step: q [B, 1, Hq, d] at position Lk - 1 -> (sel, O, LSE)."""
    _dev(q, k_cache, v_cache, kc)
    B, Lq, Hq, d = q.shape
    Lk, Hkv = k_cache.shape[1], k_cache.shape[2]
    p = make_params(cfg, B, Lq, Lk, Hq, Hkv, d, q.dtype)
    sel = torch.empty(B, Hkv, Lq, cfg.ksel, dtype=torch.int32, device=q.device)
    o = torch.empty_like(q)
    lse = torch.empty(B, Hq, Lq, dtype=torch.float32, device=q.device)
    w = _workspace(p, OP_DECODE, ws, q.device)
    _check(lib().phsa_decode(ctypes.byref(p), _ptr(q), _ptr(k_cache), _ptr(v_cache), _ptr(kc), _ptr(sel), _ptr(o),
                             _ptr(lse), _ptr(w), w.numel() if w is not None else 0, _stream()), "phsa_decode")
    return sel, o, lse


def decode_varlen(q, k_cache, v_cache, kc, cache_len, cfg: Config):
    """Decode step with per-sequence cache lengths: q [B, 1, Hq, d], caches [B, Lk, Hkv, d]
    (capacity Lk), kc [B, Hkv, Lk/m, d], cache_len int32 [B] -> (sel, O, LSE)."""
    _dev(q, k_cache, v_cache, kc, cache_len)
    B, Lq, Hq, d = q.shape
    Lk, Hkv = k_cache.shape[1], k_cache.shape[2]
    p = make_params(cfg, B, Lq, Lk, Hq, Hkv, d, q.dtype)
    sel = torch.empty(B, Hkv, Lq, cfg.ksel, dtype=torch.int32, device=q.device)
    o = torch.empty_like(q)
    lse = torch.empty(B, Hq, Lq, dtype=torch.float32, device=q.device)
    w = _workspace(p, OP_DECODE, None, q.device)
    _check(lib().phsa_decode_varlen(ctypes.byref(p), _ptr(q), _ptr(k_cache), _ptr(v_cache), _ptr(kc), _ptr(cache_len),
                                    _ptr(sel), _ptr(o), _ptr(lse), _ptr(w), w.numel() if w is not None else 0,
                                    _stream()), "phsa_decode_varlen")
    return sel, o, lse


def cache_append(k_new, v_new, punct_new, k_cache, v_cache, punct_cache, cache_len, kc, cfg: Config) -> None:
    """Appends one token per sequence (k_new, v_new [B, Hkv, d], punct_new uint8 [B]) to the caches
    in place, growing cache_len and writing the representative of every block it completes."""
    _dev(k_new, v_new, punct_new, k_cache, v_cache, punct_cache, cache_len, kc)
    B, Lk, Hkv, d = k_cache.shape
    p = make_params(cfg, B, 1, Lk, Hkv, Hkv, d, k_cache.dtype)
    _check(lib().phsa_cache_append(ctypes.byref(p), _ptr(k_new), _ptr(v_new), _ptr(punct_new), _ptr(k_cache),
                                   _ptr(v_cache), _ptr(punct_cache), _ptr(cache_len), _ptr(kc), _stream()),
           "phsa_cache_append")


class SparseAttention(torch.autograd.Function):
    """Autograd wrapper: forward = phsa_attn_fwd, backward = phsa_attn_bwd (selection fixed).

    The forward's workspace, sized for both passes, is kept for the backward,
    which then reuses the inverted selection index instead of rebuilding it."""

    @staticmethod
    def forward(ctx, q, k, v, sel, cfg: Config):
        B, Lq, Hq, d = q.shape
        p = make_params(cfg, B, Lq, k.shape[1], Hq, k.shape[2], d, q.dtype)
        need = max(workspace_size(p, OP_ATTN_FWD), workspace_size(p, OP_ATTN_BWD))
        ws = torch.empty(need, dtype=torch.uint8, device=q.device) if need else None
        o, lse = attn_fwd(q, k, v, sel, cfg, ws)
        ctx.save_for_backward(q, k, v, o, lse, sel)
        ctx.cfg, ctx.ws = cfg, ws
        return o

    @staticmethod
    def backward(ctx, do):
        q, k, v, o, lse, sel = ctx.saved_tensors
        dq, dk, dv = attn_bwd(q, k, v, o, do.contiguous(), lse, sel, ctx.cfg, ctx.ws, reuse_index=ctx.ws is not None)
        ctx.ws = None
        return dq, dk, dv, None, None
