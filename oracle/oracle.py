"""ctypes wrapper of the C oracle (oracle.c): exact top-k sparse decode attention
in float64 on the CPU.

Test infrastructure only: the tests, the package smoke check and the
benchmark's CPU-baseline leg may call it; the product path never does.
It imports nothing from the HIP package.  Inputs are duck-typed: any object
with the attributes of a decode-step description (B, Hq, Hkv, d, dtype, q, k,
v, seq_lens, layout, ncap, ratio, rounding, group_shared, page_size,
block_table) works.  bfloat16 arrays are uint16 arrays of bfloat16 bits.
"""
from __future__ import annotations

import ctypes as C
import math
import os

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_LIB_PATH = os.path.join(_HERE, "liboracle.so")
# Test hook: the mutation tests point this at a deliberately broken copy.
_LIB_OVERRIDE = os.environ.get("ORACLE_LIB_OVERRIDE")


class _Cache(C.Structure):
    _fields_ = [("data", C.c_void_p), ("dtype", C.c_int32), ("paged", C.c_int32),
                ("ncap", C.c_int64), ("num_pages", C.c_int64), ("page_size", C.c_int32),
                ("max_pages", C.c_int32), ("block_table", C.c_void_p)]


_lib = None


def lib() -> C.CDLL:
    """Load liboracle.so, compiling it first if it has not been built."""
    global _lib
    if _lib is None:
        path = _LIB_OVERRIDE or _LIB_PATH
        if not _LIB_OVERRIDE and not os.path.exists(_LIB_PATH):
            from . import build
            build.build()
        L = C.CDLL(path)
        L.oracle_budget.restype = C.c_int64
        L.oracle_budget.argtypes = [C.c_int64, C.c_double, C.c_int32]
        L.oracle_select_row.restype = C.c_int32
        L.oracle_select_row.argtypes = [C.c_void_p, C.c_int64, C.c_int64, C.c_int64,
                                        C.c_void_p, C.c_void_p]
        L.oracle_scores.restype = C.c_int32
        L.oracle_scores.argtypes = [C.c_int, C.c_int, C.c_int, C.c_int, C.c_void_p, C.c_int32,
                                    C.POINTER(_Cache), C.c_void_p, C.c_int32, C.c_int64,
                                    C.c_void_p, C.c_int]
        L.oracle_select_f32.restype = C.c_int32
        L.oracle_select_f32.argtypes = [C.c_int, C.c_int, C.c_int64, C.c_void_p, C.c_void_p,
                                        C.c_double, C.c_int32, C.c_void_p, C.c_int64,
                                        C.c_int64, C.c_int64, C.c_void_p, C.c_void_p, C.c_int]
        L.oracle_select_forced.restype = C.c_int32
        L.oracle_select_forced.argtypes = [C.c_void_p, C.c_int64, C.c_int64, C.c_int64,
                                           C.c_int64, C.c_int64, C.c_void_p, C.c_void_p]
        L.oracle_attend.restype = C.c_int32
        L.oracle_attend.argtypes = [C.c_int, C.c_int, C.c_int, C.c_int, C.c_void_p, C.c_int32,
                                    C.POINTER(_Cache), C.POINTER(_Cache), C.c_void_p, C.c_int32,
                                    C.c_double, C.c_int64, C.c_void_p, C.c_void_p, C.c_void_p,
                                    C.c_int]
        L.oracle_sparse_attention.restype = C.c_int32
        L.oracle_attend_weighted.restype = C.c_int32
        L.oracle_attend_weighted.argtypes = [C.c_int, C.c_int, C.c_int, C.c_int, C.c_void_p,
                                             C.c_int32, C.c_void_p, C.c_void_p, C.c_void_p,
                                             C.c_int32, C.c_double, C.c_int64, C.c_void_p,
                                             C.c_void_p, C.c_void_p, C.c_void_p, C.c_int]
        L.oracle_sparse_attention.argtypes = [
            C.c_int, C.c_int, C.c_int, C.c_int, C.c_void_p, C.c_int32, C.POINTER(_Cache),
            C.POINTER(_Cache), C.c_void_p, C.c_double, C.c_int32, C.c_int32, C.c_double,
            C.c_void_p, C.c_int64, C.c_int64, C.c_int64, C.c_void_p, C.c_void_p, C.c_void_p,
            C.c_void_p, C.c_int]
        L.oracle_label_scores.restype = C.c_int32
        L.oracle_label_scores.argtypes = [C.c_int, C.c_int, C.c_int, C.c_int, C.c_void_p,
                                          C.c_int32, C.POINTER(_Cache), C.c_int, C.c_void_p,
                                          C.c_void_p, C.c_int32, C.c_int64, C.c_void_p, C.c_int]
        L.oracle_label_attention.restype = C.c_int32
        L.oracle_label_attention.argtypes = [
            C.c_int, C.c_int, C.c_int, C.c_int, C.c_void_p, C.c_int32, C.POINTER(_Cache),
            C.POINTER(_Cache), C.POINTER(_Cache), C.c_int, C.c_void_p, C.c_void_p, C.c_double,
            C.c_int32, C.c_int32, C.c_double, C.c_void_p, C.c_int64, C.c_int64, C.c_int64,
            C.c_void_p, C.c_void_p, C.c_void_p, C.c_void_p, C.c_int]
        L.oracle_max_threads.restype = C.c_int32
        L.oracle_max_threads.argtypes = [C.c_int]
        _lib = L
    return _lib


class OracleError(RuntimeError):
    pass


def _check(rc: int, what: str) -> None:
    if rc != 0:
        raise OracleError(f"{what} failed with code {rc}")


def _ptr(a) -> int | None:
    return None if a is None else a.ctypes.data


def _dtype_code(dtype: str) -> int:
    return {"f32": 0, "bf16": 1}[dtype]


def _cache(inp, arr: np.ndarray, keep: list) -> _Cache:
    c = _Cache()
    arr = np.ascontiguousarray(arr)
    keep.append(arr)
    c.data = arr.ctypes.data
    c.dtype = _dtype_code(inp.dtype)
    if inp.layout == "paged":
        bt = np.ascontiguousarray(inp.block_table, dtype=np.int32)
        keep.append(bt)
        c.paged = 1
        c.ncap = 0
        c.num_pages = arr.shape[0]
        c.page_size = inp.page_size
        c.max_pages = bt.shape[1]
        c.block_table = bt.ctypes.data
    else:
        c.paged = 0
        c.ncap = arr.shape[2]
        c.num_pages = 0
        c.page_size = 0
        c.max_pages = 0
        c.block_table = None
    return c


def budget(L: int, ratio: float, rounding: int = 0) -> int:
    """k for a sequence of L positions at sparsity ``ratio`` (0 nearest, 1 ceil)."""
    return int(lib().oracle_budget(int(L), float(ratio), int(rounding)))


def max_threads(nthreads: int = 0) -> int:
    return int(lib().oracle_max_threads(int(nthreads)))


def select_row(scores: np.ndarray, k: int, k_max: int | None = None):
    """Exact top-k of one row of float64 scores; returns (ascending idx padded
    with -1 to k_max, tau = k-th largest score)."""
    s = np.ascontiguousarray(scores, dtype=np.float64)
    k_max = k if k_max is None else k_max
    idx = np.empty(max(k_max, 1), dtype=np.int32)
    tau = np.empty(1, dtype=np.float64)
    _check(lib().oracle_select_row(s.ctypes.data, len(s), int(k), int(k_max),
                                   idx.ctypes.data, tau.ctypes.data), "select_row")
    return idx[:k_max], float(tau[0])


def scores(inp, nthreads: int = 0) -> np.ndarray:
    """float64 selection scores [B, R, ncap] (NaN at j >= L_b)."""
    keep: list = []
    K = _cache(inp, inp.k, keep)
    q = np.ascontiguousarray(inp.q)
    lens = np.ascontiguousarray(inp.seq_lens, dtype=np.int32)
    out = np.empty((inp.B, inp.rows, inp.ncap), dtype=np.float64)
    _check(lib().oracle_scores(inp.B, inp.Hq, inp.Hkv, inp.d, q.ctypes.data,
                               _dtype_code(inp.dtype), C.byref(K), lens.ctypes.data,
                               int(inp.group_shared), inp.ncap, out.ctypes.data, nthreads),
           "scores")
    return out


def forced_of(inp) -> tuple:
    """(n_sink, n_local) of a decode step (0, 0 unless the step sets them)."""
    return int(getattr(inp, "n_sink", 0) or 0), int(getattr(inp, "n_local", 0) or 0)


def select_forced(scores: np.ndarray, n_sink: int, n_local: int, kh: int,
                  k_max: int | None = None):
    """Kept set of one float64 score row with forced positions: the first
    n_sink and last n_local positions, plus the exact top-kh in between;
    returns (ascending idx padded with -1 to k_max, tau)."""
    s = np.ascontiguousarray(scores, dtype=np.float64)
    L = len(s)
    ns = min(n_sink, L)
    nl = min(n_local, L - ns)
    k_max = ns + nl + kh if k_max is None else k_max
    idx = np.empty(max(k_max, 1), dtype=np.int32)
    tau = np.empty(1, dtype=np.float64)
    _check(lib().oracle_select_forced(s.ctypes.data, L, int(n_sink), int(n_local), int(kh),
                                      int(k_max), idx.ctypes.data, tau.ctypes.data),
           "select_forced")
    return idx[:k_max], float(tau[0])


def k_max_for(inp) -> int:
    """Largest budget any sequence of this cache capacity can need (forced
    positions included)."""
    ns, nl = forced_of(inp)
    n = int(inp.ncap)
    fs = min(ns, n)
    fl = min(nl, n - fs)
    return fs + fl + min(budget(n, inp.ratio, inp.rounding), n - fs - fl)


def select_f32(scores_f32: np.ndarray, seq_lens, ratio: float, rounding: int, k_max: int,
               k_override=None, nthreads: int = 0, n_sink: int = 0, n_local: int = 0):
    """Exact top-k over given float32 scores [B, R, ncap] (with forced
    positions when n_sink or n_local is set); returns (idx, tau)."""
    s = np.ascontiguousarray(scores_f32, dtype=np.float32)
    B, R, ncap = s.shape
    lens = np.ascontiguousarray(seq_lens, dtype=np.int32)
    ko = None if k_override is None else np.ascontiguousarray(k_override, dtype=np.int32)
    idx = np.empty((B, R, k_max), dtype=np.int32)
    tau = np.empty((B, R), dtype=np.float64)
    _check(lib().oracle_select_f32(B, R, ncap, s.ctypes.data, lens.ctypes.data, float(ratio),
                                   int(rounding), _ptr(ko), int(n_sink), int(n_local),
                                   int(k_max), idx.ctypes.data, tau.ctypes.data, nthreads),
           "select_f32")
    return idx, tau


def attend(inp, idx: np.ndarray, scale: float = 0.0, nthreads: int = 0):
    """Softmax attention over given index sets idx [B, R, k_max]; returns
    (out [B,Hq,d], absw [B,Hq,d]) in float64."""
    keep: list = []
    K = _cache(inp, inp.k, keep)
    V = _cache(inp, inp.v, keep)
    q = np.ascontiguousarray(inp.q)
    lens = np.ascontiguousarray(inp.seq_lens, dtype=np.int32)
    ix = np.ascontiguousarray(idx, dtype=np.int32)
    out = np.empty((inp.B, inp.Hq, inp.d), dtype=np.float64)
    absw = np.empty_like(out)
    _check(lib().oracle_attend(inp.B, inp.Hq, inp.Hkv, inp.d, q.ctypes.data,
                               _dtype_code(inp.dtype), C.byref(K), C.byref(V), lens.ctypes.data,
                               int(inp.group_shared), float(scale), ix.shape[2], ix.ctypes.data,
                               out.ctypes.data, absw.ctypes.data, nthreads), "attend")
    return out, absw


def attend_weighted(inp, idx: np.ndarray, weights: np.ndarray, scale: float = 0.0,
                    nthreads: int = 0):
    """Weighted softmax attention over given index sets: weights [B, R, k_max]
    (float32, >= 0) aligned with idx; returns (out, absw) in float64."""
    keep: list = []
    K = _cache(inp, inp.k, keep)
    V = _cache(inp, inp.v, keep)
    q = np.ascontiguousarray(inp.q)
    lens = np.ascontiguousarray(inp.seq_lens, dtype=np.int32)
    ix = np.ascontiguousarray(idx, dtype=np.int32)
    wt = np.ascontiguousarray(weights, dtype=np.float32)
    if wt.shape != ix.shape:
        raise ValueError("weights must have the shape of idx")
    out = np.empty((inp.B, inp.Hq, inp.d), dtype=np.float64)
    absw = np.empty_like(out)
    _check(lib().oracle_attend_weighted(inp.B, inp.Hq, inp.Hkv, inp.d, q.ctypes.data,
                                        _dtype_code(inp.dtype), C.byref(K), C.byref(V),
                                        lens.ctypes.data, int(inp.group_shared), float(scale),
                                        ix.shape[2], ix.ctypes.data, wt.ctypes.data,
                                        out.ctypes.data, absw.ctypes.data, nthreads),
           "attend_weighted")
    return out, absw


def dense_attention(inp, scale: float = 0.0, nthreads: int = 0, batch=None):
    """Dense decode attention over every position j < L_b (Table 1's
    full-attention baseline): attention over the index set of all positions.
    batch: optional list of sequences to compute (others are left as NaN).
    Returns out [B, Hq, d] float64."""
    out = np.full((inp.B, inp.Hq, inp.d), np.nan)
    for b in (range(inp.B) if batch is None else batch):
        sub = _one_sequence(inp, b)
        L = int(inp.seq_lens[b])
        idx = np.broadcast_to(np.arange(max(L, 1), dtype=np.int32) if L else
                              np.full(1, -1, np.int32), (1, sub.rows, max(L, 1)))
        out[b], _ = attend(sub, np.ascontiguousarray(idx), scale, nthreads)
    return out


def _one_sequence(inp, b: int):
    """Sequence b of a decode step as a batch of one (views, no copies of the cache)."""
    import copy
    one = copy.copy(inp)
    one.B = 1
    one.q = inp.q[b:b + 1]
    one.seq_lens = np.asarray(inp.seq_lens)[b:b + 1]
    if inp.layout == "paged":
        one.block_table = inp.block_table[b:b + 1]
    else:
        one.k, one.v = inp.k[b:b + 1], inp.v[b:b + 1]
    return one


def sparse_attention(inp, k_max: int | None = None, k_override=None, scale: float = 0.0,
                     nthreads: int = 0) -> dict:
    """The whole method: returns dict(idx, tau, out, absw).  Forced positions
    come from the step's n_sink / n_local attributes when it has them."""
    keep: list = []
    K = _cache(inp, inp.k, keep)
    V = _cache(inp, inp.v, keep)
    q = np.ascontiguousarray(inp.q)
    lens = np.ascontiguousarray(inp.seq_lens, dtype=np.int32)
    k_max = k_max_for(inp) if k_max is None else k_max
    ko = None if k_override is None else np.ascontiguousarray(k_override, dtype=np.int32)
    idx = np.empty((inp.B, inp.rows, k_max), dtype=np.int32)
    tau = np.empty((inp.B, inp.rows), dtype=np.float64)
    out = np.empty((inp.B, inp.Hq, inp.d), dtype=np.float64)
    absw = np.empty_like(out)
    _check(lib().oracle_sparse_attention(
        inp.B, inp.Hq, inp.Hkv, inp.d, q.ctypes.data, _dtype_code(inp.dtype), C.byref(K),
        C.byref(V), lens.ctypes.data, float(inp.ratio), int(inp.rounding),
        int(inp.group_shared), float(scale), _ptr(ko), *forced_of(inp), int(k_max),
        idx.ctypes.data, tau.ctypes.data, out.ctypes.data, absw.ctypes.data, nthreads),
        "sparse_attention")
    return {"idx": idx, "tau": tau, "out": out, "absw": absw}


def label_scores(inp, labels: np.ndarray, channels: np.ndarray, nthreads: int = 0) -> np.ndarray:
    """float64 approximate scores [B, R, ncap] of the low-channel indexer
    (NaN at j >= L_b).  labels: the label cache in the step's layout with
    nlab channels per key; channels: int32 [Hkv, nlab], the query channel
    each label column multiplies."""
    keep: list = []
    lab = _cache(inp, labels, keep)
    ch = np.ascontiguousarray(channels, dtype=np.int32)
    q = np.ascontiguousarray(inp.q)
    lens = np.ascontiguousarray(inp.seq_lens, dtype=np.int32)
    out = np.empty((inp.B, inp.rows, inp.ncap), dtype=np.float64)
    _check(lib().oracle_label_scores(inp.B, inp.Hq, inp.Hkv, inp.d, q.ctypes.data,
                                     _dtype_code(inp.dtype), C.byref(lab), ch.shape[1],
                                     ch.ctypes.data, lens.ctypes.data, int(inp.group_shared),
                                     inp.ncap, out.ctypes.data, nthreads), "label_scores")
    return out


def label_attention(inp, labels: np.ndarray, channels: np.ndarray, k_max: int | None = None,
                    k_override=None, scale: float = 0.0, nthreads: int = 0) -> dict:
    """The method with the low-channel indexer choosing the positions:
    returns dict(idx, tau, out, absw)."""
    keep: list = []
    K = _cache(inp, inp.k, keep)
    V = _cache(inp, inp.v, keep)
    lab = _cache(inp, labels, keep)
    ch = np.ascontiguousarray(channels, dtype=np.int32)
    q = np.ascontiguousarray(inp.q)
    lens = np.ascontiguousarray(inp.seq_lens, dtype=np.int32)
    k_max = k_max_for(inp) if k_max is None else k_max
    ko = None if k_override is None else np.ascontiguousarray(k_override, dtype=np.int32)
    idx = np.empty((inp.B, inp.rows, k_max), dtype=np.int32)
    tau = np.empty((inp.B, inp.rows), dtype=np.float64)
    out = np.empty((inp.B, inp.Hq, inp.d), dtype=np.float64)
    absw = np.empty_like(out)
    _check(lib().oracle_label_attention(
        inp.B, inp.Hq, inp.Hkv, inp.d, q.ctypes.data, _dtype_code(inp.dtype), C.byref(K),
        C.byref(V), C.byref(lab), ch.shape[1], ch.ctypes.data, lens.ctypes.data,
        float(inp.ratio), int(inp.rounding), int(inp.group_shared), float(scale), _ptr(ko),
        *forced_of(inp), int(k_max), idx.ctypes.data, tau.ctypes.data, out.ctypes.data,
        absw.ctypes.data, nthreads), "label_attention")
    return {"idx": idx, "tau": tau, "out": out, "absw": absw}


def default_scale(d: int) -> float:
    return 1.0 / math.sqrt(d)


# ---------------------------------------------------------------------------
# Stochastic index selection with importance weights (the paper's vAttention
# runs, Section 4 and the RULER-HARD figure).  The paper names the method
# but does not define it; this is the reading built here: the exact top-k
# set S of a row (with its forced positions), plus s positions drawn
# uniformly, with replacement, from the rest C = [0, L) \ S, each drawn
# entry weighted |C| / s, so that the weighted sums over the draws estimate
# the sums over C without bias; the attention is the self-normalised
# weighted softmax over S and the draws.  The random numbers are inputs:
# draw i of a row is a uint32 u, and it picks the floor(u |C| / 2^32)-th
# position of C in ascending order.
# ---------------------------------------------------------------------------
def sampled_lists(idx: np.ndarray, seq_lens, draws: np.ndarray):
    """Index lists and weights of the sampled selection, from the exact
    selection's lists idx [B, R, k_max] (ascending, -1 padded) and the draws
    [B, R, s] (uint32): per row its kept positions (weight 1), then its s
    drawn positions (weight |C| / s, float32), then -1 (weight 0).  Rows
    whose kept set is the whole sequence draw nothing."""
    B, R, k_max = idx.shape
    s = draws.shape[2]
    out_idx = np.full((B, R, k_max + s), -1, dtype=np.int32)
    out_w = np.zeros((B, R, k_max + s), dtype=np.float32)
    for b in range(B):
        L = int(seq_lens[b])
        for r in range(R):
            kept = idx[b, r][idx[b, r] >= 0]
            n = len(kept)
            out_idx[b, r, :n] = kept
            out_w[b, r, :n] = 1.0
            c = L - n
            if c <= 0 or s == 0:
                continue
            rest = np.setdiff1d(np.arange(L, dtype=np.int64), kept.astype(np.int64))
            ranks = (draws[b, r].astype(np.uint64) * np.uint64(c)) >> np.uint64(32)
            out_idx[b, r, n:n + s] = rest[ranks.astype(np.int64)]
            out_w[b, r, n:n + s] = np.float32(c) / np.float32(s)
    return out_idx, out_w


def sampled_attention(inp, draws: np.ndarray, k_max: int | None = None, k_override=None,
                      scale: float = 0.0, nthreads: int = 0) -> dict:
    """The sampled selection's attention: exact top-k (sparse_attention's
    selection), the draws of the rest, weighted softmax.  Returns dict(idx,
    weights, out, absw, topk_idx)."""
    base = sparse_attention(inp, k_max=k_max, k_override=k_override, scale=scale,
                            nthreads=nthreads)
    idx, w = sampled_lists(base["idx"], inp.seq_lens, np.asarray(draws, dtype=np.uint32))
    out, absw = attend_weighted(inp, idx, w, scale=scale, nthreads=nthreads)
    return {"idx": idx, "weights": w, "out": out, "absw": absw, "topk_idx": base["idx"]}
