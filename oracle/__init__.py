"""PHSA oracle: plain fp64 CPU reference (TEST INFRASTRUCTURE ONLY).

Only ``tests/``, ``__graft_entry__.smoke()`` and the ``cpu_baseline`` leg of
``bench.py`` may import this package.  The product library never loads it and
shares no code with it.

Every function takes numpy arrays on the host.  Floating-point inputs are
passed as float32 (they hold the bf16 / fp32 test inputs exactly) and all
arithmetic inside the C library is IEEE double.  Citations refer to the paper
"Punctuation-aware Hybrid Trainable Sparse Attention for Large Language
Models" (arXiv 2601.02819):

* ``punct_mask`` - the indicator I(x_i in P) of Eq. 7 (token id in the
  punctuation set).
* ``compress``  - Eq. 3 (blocks), Eq. 6 (global mean), Eq. 7 (punctuation
  mean and its no-punctuation fallback), Eq. 8 (gated fusion).
* ``select``    - Eq. 8 relevance logits and Algorithm 1's block selection
  (forced init + local blocks, causal mask, top-k, Unique).
* ``attn_fwd``  - Eq. 10-11 sparse attention over the selected blocks.
* ``attn_bwd``  - gradient of Eq. 10-11 with the selection held fixed.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "phsa_oracle.c")
_LIB_PATH = os.path.join(_HERE, "libphsa_oracle.so")
_lib = None


def build(force: bool = False) -> str:
    """Compile the oracle with gcc (-O2, OpenMP, no fast-math)."""
    if force or not os.path.exists(_LIB_PATH) or os.path.getmtime(_LIB_PATH) < os.path.getmtime(_SRC):
        tmp = _LIB_PATH + ".tmp%d" % os.getpid()
        subprocess.check_call(
            ["gcc", "-O2", "-std=c11", "-fopenmp", "-fPIC", "-shared", "-Wall", "-Wno-unused-function",
             _SRC, "-o", tmp, "-lm"])
        os.replace(tmp, _LIB_PATH)
    return _LIB_PATH


def _load():
    global _lib
    if _lib is None:
        # PHSA_ORACLE_LIB: a prebuilt copy of this library to load instead (the
        # host-sanitizer test builds one with AddressSanitizer and UBSan)
        path = os.environ.get("PHSA_ORACLE_LIB")
        if not path:
            path = build()
        _lib = ctypes.CDLL(path)
        I, D, L, P = ctypes.c_int, ctypes.c_double, ctypes.c_int64, ctypes.c_void_p
        _lib.oracle_compress.argtypes = [I, I, I, I, I, D, P, P, P]
        _lib.oracle_punct_mask.argtypes = [L, P, ctypes.c_int32, P, P]
        _lib.oracle_select.argtypes = [I] * 12 + [D, P, P, L, P, P, P, P]
        _lib.oracle_score_row.argtypes = [I] * 7 + [D, P, P, I, I, I, I, I, P]
        _lib.oracle_attn_fwd.argtypes = [I] * 9 + [D, P, P, P, P, L, P, P, P]
        _lib.oracle_attn_bwd.argtypes = [I] * 9 + [D, P, P, P, P, P, L, P, P, L, P, P, P]
        _lib.oracle_num_threads.argtypes = []
        _lib.oracle_num_threads.restype = ctypes.c_int
        for f in ("oracle_compress", "oracle_select", "oracle_score_row", "oracle_attn_fwd", "oracle_attn_bwd",
                  "oracle_punct_mask"):
            getattr(_lib, f).restype = None
    return _lib


def _f32(x) -> np.ndarray:
    a = np.asarray(x)
    if a.dtype != np.float32:
        a = a.astype(np.float32)
    return np.ascontiguousarray(a)


def _ptr(a: np.ndarray):
    return a.ctypes.data_as(ctypes.c_void_p) if a is not None else None


def _rows_arg(rows, total):
    if rows is None:
        return total, None
    r = np.ascontiguousarray(np.asarray(rows, dtype=np.int64))
    return int(r.size), r


def num_threads() -> int:
    """Threads the oracle's OpenMP loops run on."""
    return int(_load().oracle_num_threads())


def ksel(block_size: int, top_k: int, n_init: int, window: int) -> int:
    """Number of index slots per row: init + local (w/m + 1) + top-k."""
    return n_init + window // block_size + 1 + top_k


def punct_mask(ids, punct_ids) -> np.ndarray:
    """Token ids (any shape, int32) and the punctuation id set -> uint8 mask of the same shape."""
    ids = np.ascontiguousarray(np.asarray(ids, dtype=np.int32))
    pid = np.ascontiguousarray(np.asarray(punct_ids, dtype=np.int32).reshape(-1))
    out = np.empty(ids.shape, dtype=np.uint8)
    _load().oracle_punct_mask(ids.size, _ptr(ids), int(pid.size), _ptr(pid), _ptr(out))
    return out


def compress(K, punct, block_size: int, lam: float) -> np.ndarray:
    """K [B, Lk, Hkv, d], punct [B, Lk] -> Kc [B, Hkv, T, d] (float64)."""
    K = _f32(K)
    punct = np.ascontiguousarray(np.asarray(punct, dtype=np.uint8))
    B, Lk, Hkv, d = K.shape
    T = Lk // block_size
    out = np.empty((B, Hkv, T, d), dtype=np.float64)
    _load().oracle_compress(B, Lk, Hkv, d, block_size, float(lam), _ptr(K), _ptr(punct), _ptr(out))
    return out


SUM_LOGITS, SOFTMAX_SUM = 0, 1   # group aggregation of the per-head Eq. 8 scores


def select(Q, Kc, block_size: int, top_k: int, n_init: int, window: int, scale: float,
           seqlen_k: int, rows=None, q_pos0=None, mode: int = SUM_LOGITS):
    """Q [B, Lq, Hq, d], Kc [B, Hkv, T, d] float64.  Query row i sits at position
    q_pos0 + i (default seqlen_k - Lq); seqlen_k must cover whole blocks up to
    the last query's own block.  mode SUM_LOGITS ranks blocks on the group's
    summed scaled logits; SOFTMAX_SUM on log sum_h softmax_h(t), each head's
    softmax taken over the complete causal blocks 0 .. cur-1.

    Returns (sel, kth, gap).  With rows=None: sel [B, Hkv, Lq, Ksel] and
    kth/gap [B, Hkv, Lq].  With rows (flat b*Lq + i): sel [n, Hkv, Ksel],
    kth/gap [n, Hkv].
    """
    Q = _f32(Q)
    Kc = np.ascontiguousarray(np.asarray(Kc, dtype=np.float64))
    B, Lq, Hq, d = Q.shape
    Hkv = Kc.shape[1]
    ks = ksel(block_size, top_k, n_init, window)
    n, r = _rows_arg(rows, B * Lq)
    sel = np.empty((n, Hkv, ks), dtype=np.int32)
    kth = np.empty((n, Hkv), dtype=np.float64)
    gap = np.empty((n, Hkv), dtype=np.float64)
    pos0 = seqlen_k - Lq if q_pos0 is None else int(q_pos0)
    assert mode in (SUM_LOGITS, SOFTMAX_SUM) and Hq // Hkv <= 64
    _load().oracle_select(B, Lq, seqlen_k, Hq, Hkv, d, block_size, top_k, n_init, window,
                          pos0, int(mode), float(scale), _ptr(Q), _ptr(Kc), n, _ptr(r), _ptr(sel),
                          _ptr(kth), _ptr(gap))
    if rows is None:
        sel = sel.reshape(B, Lq, Hkv, ks).transpose(0, 2, 1, 3).copy()
        kth = kth.reshape(B, Lq, Hkv).transpose(0, 2, 1).copy()
        gap = gap.reshape(B, Lq, Hkv).transpose(0, 2, 1).copy()
    return sel, kth, gap


def score_row(Q, Kc, block_size: int, scale: float, seqlen_k: int, b: int, i: int, g: int,
              q_pos0=None, mode: int = SUM_LOGITS) -> np.ndarray:
    """Group relevance scores of every block for one (b, i, g) in the given
    mode: float64 [T] (SOFTMAX_SUM gives -inf outside blocks 0 .. cur-1)."""
    Q = _f32(Q)
    Kc = np.ascontiguousarray(np.asarray(Kc, dtype=np.float64))
    B, Lq, Hq, d = Q.shape
    Hkv, T = Kc.shape[1], Kc.shape[2]
    out = np.empty(T, dtype=np.float64)
    pos0 = seqlen_k - Lq if q_pos0 is None else int(q_pos0)
    assert mode in (SUM_LOGITS, SOFTMAX_SUM) and Hq // Hkv <= 64
    _load().oracle_score_row(B, Lq, seqlen_k, Hq, Hkv, d, block_size, float(scale), _ptr(Q), _ptr(Kc),
                             b, i, g, pos0, int(mode), _ptr(out))
    return out


def attn_fwd(Q, K, V, sel, block_size: int, scale: float, rows=None, q_pos0=None):
    """Sparse attention forward.  sel [B, Hkv, Lq, Ksel] int32.

    Returns (O, LSE): with rows=None O [B, Lq, Hq, d], LSE [B, Hq, Lq];
    with rows (flat b*Lq + i) O [n, Hq, d], LSE [n, Hq].  Query row i sits at
    position q_pos0 + i (default Lk - Lq); keys past it are never read.
    """
    Q, K, V = _f32(Q), _f32(K), _f32(V)
    sel = np.ascontiguousarray(np.asarray(sel, dtype=np.int32))
    B, Lq, Hq, d = Q.shape
    Lk, Hkv = K.shape[1], K.shape[2]
    ks = sel.shape[-1]
    n, r = _rows_arg(rows, B * Lq)
    O = np.empty((n, Hq, d), dtype=np.float64)
    LSE = np.empty((n, Hq), dtype=np.float64)
    pos0 = Lk - Lq if q_pos0 is None else int(q_pos0)
    _load().oracle_attn_fwd(B, Lq, Lk, Hq, Hkv, d, block_size, ks, pos0, float(scale), _ptr(Q), _ptr(K),
                            _ptr(V), _ptr(sel), n, _ptr(r), _ptr(O), _ptr(LSE))
    if rows is None:
        O = O.reshape(B, Lq, Hq, d)
        LSE = LSE.reshape(B, Lq, Hq).transpose(0, 2, 1).copy()
    return O, LSE


def attn_bwd(Q, K, V, dO, sel, block_size: int, scale: float, rows=None, blocks=None,
             want_dq: bool = True, want_dkv: bool = True):
    """Sparse attention backward with the selection fixed.

    With rows=None/blocks=None returns full dQ [B, Lq, Hq, d] and
    dK, dV [B, Lk, Hkv, d].  With rows (flat b*Lq + i): dQ [n, Hq, d].  With
    blocks (flat b*Hkv*T + g*T + t): dK, dV [nb, m, d].
    """
    Q, K, V, dO = _f32(Q), _f32(K), _f32(V), _f32(dO)
    sel = np.ascontiguousarray(np.asarray(sel, dtype=np.int32))
    B, Lq, Hq, d = Q.shape
    Lk, Hkv = K.shape[1], K.shape[2]
    m = block_size
    T = Lk // m
    ks = sel.shape[-1]
    n, r = _rows_arg(rows, B * Lq) if want_dq else (0, None)
    nb, bl = _rows_arg(blocks, B * Hkv * T) if want_dkv else (0, None)
    dQ = np.empty((max(n, 1), Hq, d), dtype=np.float64)
    dK = np.empty((max(nb, 1), m, d), dtype=np.float64)
    dV = np.empty((max(nb, 1), m, d), dtype=np.float64)
    _load().oracle_attn_bwd(B, Lq, Lk, Hq, Hkv, d, m, ks, Lk - Lq, float(scale), _ptr(Q), _ptr(K), _ptr(V),
                            _ptr(dO), _ptr(sel), n, _ptr(r), _ptr(dQ), nb, _ptr(bl), _ptr(dK), _ptr(dV))
    dQ, dK, dV = dQ[:n], dK[:nb], dV[:nb]
    if want_dq and rows is None:
        dQ = dQ.reshape(B, Lq, Hq, d)
    if want_dkv and blocks is None:
        # compact order is (b, g, t, row-in-block, d) -> [B, Lk, Hkv, d]
        dK = dK.reshape(B, Hkv, T, m, d).transpose(0, 2, 3, 1, 4).reshape(B, Lk, Hkv, d)
        dV = dV.reshape(B, Hkv, T, m, d).transpose(0, 2, 3, 1, 4).reshape(B, Lk, Hkv, d)
    return (dQ if want_dq else None), (dK if want_dkv else None), (dV if want_dkv else None)
