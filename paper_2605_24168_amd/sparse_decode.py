"""Python binding of libsparse_decode.so (exact top-k context-sparse decode
attention on MI355X).

Argument marshalling only: every step of the method runs in the library's HIP
kernels.  PyTorch supplies device memory and the current HIP stream.  The
names follow the C ABI in include/sparse_decode.h:

    sparse_decode_score(q, cache, seq_lens, sparsity)        -> scores
    sparse_decode_topk(scores, seq_lens, sparsity, k_max)    -> idx (, vals)
    sparse_decode_attend(q, cache, seq_lens, idx, sparsity)  -> out
    sparse_decode_attention(q, cache, seq_lens, sparsity)    -> (out, idx)
    sparse_decode_attend_weighted(q, cache, seq_lens, idx, weights, sparsity) -> out
    sparse_decode_dense_attention(q, cache, seq_lens)        -> out
    sparse_decode_label_attention(q, cache, labels, seq_lens, sparsity) -> (out, idx)
    sparse_decode_label_score(q, cache, labels, seq_lens, sparsity)     -> scores

Importing this module raises if the library has not been built; nothing here
falls back to another implementation.
"""
from __future__ import annotations

import ctypes as C
import dataclasses
import os
from typing import Optional

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libsparse_decode.so")
HEADER_PATH = os.path.join(os.path.dirname(_HERE), "include", "sparse_decode.h")

SD_OK, SD_ERR_INVALID_ARG, SD_ERR_UNSUPPORTED, SD_ERR_WORKSPACE, SD_ERR_HIP = 0, -1, -2, -3, -4
SD_F32, SD_BF16, SD_I32 = 0, 1, 2
SD_KV_BHND, SD_KV_PAGED_NHD = 0, 1

if not os.path.exists(LIB_PATH):
    raise ImportError(
        f"{LIB_PATH} is missing: build it with `python -m paper_2605_24168_amd.build` "
        "(the HIP path has no fallback)")


class SdTensor(C.Structure):
    _fields_ = [("data", C.c_void_p), ("dtype", C.c_int32), ("ndim", C.c_int32),
                ("shape", C.c_int64 * 4)]


class SdKv(C.Structure):
    _fields_ = [("t", SdTensor), ("layout", C.c_int32), ("page_size", C.c_int32),
                ("block_table", C.c_void_p), ("max_pages_per_seq", C.c_int32)]


class SdSparsity(C.Structure):
    _fields_ = [("ratio", C.c_double), ("k_rounding", C.c_int32), ("group_shared", C.c_int32),
                ("softmax_scale", C.c_float), ("k_override", C.c_void_p),
                ("n_sink", C.c_int32), ("n_local", C.c_int32)]


class SdLabels(C.Structure):
    _fields_ = [("t", SdTensor), ("channels", C.c_void_p)]


class SdProfile(C.Structure):
    _fields_ = [("pilot_ms", C.c_float), ("score_ms", C.c_float), ("select_ms", C.c_float),
                ("repair_ms", C.c_float), ("attend_ms", C.c_float), ("total_ms", C.c_float),
                ("repaired_rows", C.c_int32), ("valid", C.c_int32)]


_P = C.POINTER
lib = C.CDLL(LIB_PATH)
lib.sparse_decode_score.restype = C.c_int
lib.sparse_decode_score.argtypes = [_P(SdTensor), _P(SdKv), C.c_void_p, _P(SdSparsity),
                                    _P(SdTensor), C.c_void_p]
lib.sparse_decode_topk.restype = C.c_int
lib.sparse_decode_topk.argtypes = [_P(SdTensor), C.c_void_p, _P(SdSparsity), _P(SdTensor),
                                   _P(SdTensor), C.c_void_p]
lib.sparse_decode_attend.restype = C.c_int
lib.sparse_decode_attend.argtypes = [_P(SdTensor), _P(SdKv), _P(SdKv), C.c_void_p, _P(SdTensor),
                                     _P(SdSparsity), _P(SdTensor), C.c_void_p]
lib.sparse_decode_attend_weighted.restype = C.c_int
lib.sparse_decode_attend_weighted.argtypes = [_P(SdTensor), _P(SdKv), _P(SdKv), C.c_void_p,
                                              _P(SdTensor), _P(SdTensor), _P(SdSparsity),
                                              _P(SdTensor), C.c_void_p]
lib.sparse_decode_dense_attention.restype = C.c_int
lib.sparse_decode_dense_attention.argtypes = [_P(SdTensor), _P(SdKv), _P(SdKv), C.c_void_p,
                                              C.c_float, _P(SdTensor), C.c_void_p]
lib.sparse_decode_dense_workspace_size.restype = C.c_int
lib.sparse_decode_dense_workspace_size.argtypes = [_P(SdTensor), _P(SdKv), _P(C.c_size_t)]
lib.sparse_decode_label_attention.restype = C.c_int
lib.sparse_decode_label_attention.argtypes = [_P(SdTensor), _P(SdKv), _P(SdKv), _P(SdLabels),
                                              C.c_void_p, _P(SdSparsity), _P(SdTensor),
                                              _P(SdTensor), C.c_void_p]
lib.sparse_decode_label_score.restype = C.c_int
lib.sparse_decode_label_score.argtypes = [_P(SdTensor), _P(SdKv), _P(SdLabels), C.c_void_p,
                                          _P(SdSparsity), _P(SdTensor), C.c_void_p]
lib.sparse_decode_attention.restype = C.c_int
lib.sparse_decode_attention.argtypes = [_P(SdTensor), _P(SdKv), _P(SdKv), C.c_void_p,
                                        _P(SdSparsity), _P(SdTensor), _P(SdTensor), C.c_void_p]
lib.sparse_decode_attention_noalloc.restype = C.c_int
lib.sparse_decode_attention_noalloc.argtypes = [_P(SdTensor), _P(SdKv), _P(SdKv), C.c_void_p,
                                                _P(SdSparsity), _P(SdTensor), _P(SdTensor),
                                                C.c_void_p]
lib.sparse_decode_workspace_size.restype = C.c_int
lib.sparse_decode_workspace_size.argtypes = [_P(SdTensor), _P(SdKv), _P(SdSparsity), _P(SdTensor),
                                             _P(C.c_size_t)]
lib.sparse_decode_set_workspace.restype = C.c_int
lib.sparse_decode_set_workspace.argtypes = [C.c_void_p, C.c_size_t]
lib.sparse_decode_budget.restype = C.c_int64
lib.sparse_decode_budget.argtypes = [C.c_int64, _P(SdSparsity)]
lib.sparse_decode_set_profiling.restype = C.c_int
lib.sparse_decode_set_profiling.argtypes = [C.c_int32]
lib.sparse_decode_last_profile.restype = C.c_int
lib.sparse_decode_last_profile.argtypes = [_P(SdProfile)]
lib.sparse_decode_profile_mean.restype = C.c_int
lib.sparse_decode_profile_mean.argtypes = [_P(SdProfile), _P(C.c_int32)]
lib.sparse_decode_set_debug.restype = C.c_int
lib.sparse_decode_set_debug.argtypes = [C.c_int32]
lib.sparse_decode_sampled_attention.restype = C.c_int
lib.sparse_decode_sampled_attention.argtypes = [_P(SdTensor), _P(SdKv), _P(SdKv), C.c_void_p,
                                                _P(SdSparsity), _P(SdTensor), _P(SdTensor),
                                                _P(SdTensor), _P(SdTensor), C.c_void_p]
lib.sparse_decode_read_probe.restype = C.c_int
lib.sparse_decode_read_probe.argtypes = [C.c_void_p, C.c_size_t, C.c_void_p, C.c_void_p]
lib.sparse_decode_status_string.restype = C.c_char_p
lib.sparse_decode_status_string.argtypes = [C.c_int]


class SparseDecodeError(RuntimeError):
    def __init__(self, status: int, what: str):
        msg = lib.sparse_decode_status_string(status).decode()
        super().__init__(f"{what}: {msg} ({status})")
        self.status = status


def _check(status: int, what: str) -> None:
    if status != SD_OK:
        raise SparseDecodeError(status, what)


@dataclasses.dataclass
class Sparsity:
    """k = clamp(round(L / ratio), 1, L) per row (rounding 0 = nearest, 1 = ceil)."""
    ratio: float
    rounding: int = 0
    group_shared: bool = False
    softmax_scale: float = 0.0          # <= 0: 1/sqrt(128)
    k_override: Optional[torch.Tensor] = None   # int32 [B] on the device
    n_sink: int = 0                     # first positions always kept
    n_local: int = 0                    # last positions always kept

    def c(self) -> SdSparsity:
        ko = self.k_override
        if ko is not None:
            _need_device(ko, "k_override", torch.int32)
        return SdSparsity(float(self.ratio), int(self.rounding), int(bool(self.group_shared)),
                          float(self.softmax_scale), ko.data_ptr() if ko is not None else None,
                          int(self.n_sink), int(self.n_local))


@dataclasses.dataclass
class KVCache:
    """Key and value caches: "bhnd" [B, Hkv, Ncap, 128] or "paged"
    [pages, 16, Hkv, 128] with an int32 block table [B, max_pages]."""
    k: torch.Tensor
    v: torch.Tensor
    layout: str = "bhnd"
    block_table: Optional[torch.Tensor] = None
    page_size: int = 16

    @property
    def capacity(self) -> int:
        if self.layout == "paged":
            return int(self.block_table.shape[1]) * self.page_size
        return int(self.k.shape[2])

    @property
    def num_kv_heads(self) -> int:
        return int(self.k.shape[2] if self.layout == "paged" else self.k.shape[1])

    def c(self, which: str) -> SdKv:
        t = self.k if which == "k" else self.v
        kv = SdKv()
        kv.t = _tensor(t, which)
        if self.layout == "paged":
            _need_device(self.block_table, "block_table", torch.int32)
            kv.layout = SD_KV_PAGED_NHD
            kv.page_size = self.page_size
            kv.block_table = self.block_table.data_ptr()
            kv.max_pages_per_seq = int(self.block_table.shape[1])
        elif self.layout == "bhnd":
            kv.layout = SD_KV_BHND
            kv.page_size = 0
            kv.block_table = None
            kv.max_pages_per_seq = 0
        else:
            raise ValueError(f"unknown layout {self.layout!r}")
        return kv


_DTYPES = {torch.float32: SD_F32, torch.bfloat16: SD_BF16, torch.int32: SD_I32}


@dataclasses.dataclass
class Labels:
    """Label cache of the low-channel indexer: `t` holds 8 bf16 channels per
    key, [B, Hkv, Ncap, 8] beside a contiguous cache or [pages, Hkv, 16, 8]
    beside a paged one; `channels` (int32 [Hkv, 8], device) names the key
    channel of each column."""
    t: torch.Tensor
    channels: torch.Tensor

    def c(self) -> SdLabels:
        _need_device(self.channels, "channels", torch.int32)
        lab = SdLabels()
        lab.t = _tensor(self.t, "labels")
        lab.channels = self.channels.data_ptr()
        return lab


def _need_device(t: torch.Tensor, name: str, dtype=None) -> None:
    if not isinstance(t, torch.Tensor) or not t.is_cuda:
        raise ValueError(f"{name} must be a device tensor")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    if dtype is not None and t.dtype != dtype:
        raise ValueError(f"{name} must be {dtype}, got {t.dtype}")


def _tensor(t: torch.Tensor, name: str) -> SdTensor:
    _need_device(t, name)
    if t.dtype not in _DTYPES:
        raise ValueError(f"{name}: unsupported dtype {t.dtype}")
    if t.dim() > 4:
        raise ValueError(f"{name}: at most 4 dimensions")
    st = SdTensor()
    st.data = t.data_ptr() if t.numel() else None
    st.dtype = _DTYPES[t.dtype]
    st.ndim = t.dim()
    for i, n in enumerate(t.shape):
        st.shape[i] = int(n)
    return st


def _stream(stream) -> Optional[int]:
    if stream is None:
        stream = torch.cuda.current_stream()
    return stream.cuda_stream if hasattr(stream, "cuda_stream") else int(stream)


def budget(L: int, sparsity: Sparsity) -> int:
    """k for a sequence of L positions under the ratio rule."""
    return int(lib.sparse_decode_budget(int(L), C.byref(sparsity.c())))


def rows_of(q: torch.Tensor, cache: KVCache, sparsity: Sparsity) -> int:
    return cache.num_kv_heads if sparsity.group_shared else int(q.shape[1])


def k_max_of(cache: KVCache, sparsity: Sparsity) -> int:
    return budget(cache.capacity, sparsity)


def sparse_decode_score(q, cache: KVCache, seq_lens, sparsity: Sparsity, scores=None, stream=None):
    """float32 scores [B, R, capacity] (-inf beyond each sequence)."""
    _need_device(seq_lens, "seq_lens", torch.int32)
    if scores is None:
        scores = torch.empty((q.shape[0], rows_of(q, cache, sparsity), cache.capacity),
                             dtype=torch.float32, device=q.device)
    sp, kq, kk, ks = sparsity.c(), _tensor(q, "q"), cache.c("k"), _tensor(scores, "scores")
    _check(lib.sparse_decode_score(C.byref(kq), C.byref(kk), seq_lens.data_ptr(), C.byref(sp),
                                   C.byref(ks), _stream(stream)), "sparse_decode_score")
    return scores


def sparse_decode_topk(scores, seq_lens, sparsity: Sparsity, k_max: Optional[int] = None,
                       idx=None, vals=None, with_vals: bool = False, stream=None):
    """Exact top-k positions (ascending, -1 padded) of each score row."""
    _need_device(seq_lens, "seq_lens", torch.int32)
    if k_max is None:
        k_max = budget(scores.shape[2], sparsity)
    if idx is None:
        idx = torch.empty((scores.shape[0], scores.shape[1], k_max), dtype=torch.int32,
                          device=scores.device)
    if with_vals and vals is None:
        vals = torch.empty(idx.shape, dtype=torch.float32, device=scores.device)
    sp, cs, ci = sparsity.c(), _tensor(scores, "scores"), _tensor(idx, "idx")
    cv = _tensor(vals, "vals") if vals is not None else None
    _check(lib.sparse_decode_topk(C.byref(cs), seq_lens.data_ptr(), C.byref(sp), C.byref(ci),
                                  C.byref(cv) if cv is not None else None, _stream(stream)),
           "sparse_decode_topk")
    return (idx, vals) if vals is not None else idx


def sparse_decode_attend(q, cache: KVCache, seq_lens, idx, sparsity: Sparsity, out=None,
                         stream=None):
    """Softmax attention of each query head over its listed positions."""
    _need_device(seq_lens, "seq_lens", torch.int32)
    if out is None:
        out = torch.empty_like(q)
    sp = sparsity.c()
    cq, kk, kv = _tensor(q, "q"), cache.c("k"), cache.c("v")
    ci, co = _tensor(idx, "idx"), _tensor(out, "out")
    _check(lib.sparse_decode_attend(C.byref(cq), C.byref(kk), C.byref(kv), seq_lens.data_ptr(),
                                    C.byref(ci), C.byref(sp), C.byref(co), _stream(stream)),
           "sparse_decode_attend")
    return out


def sparse_decode_attend_weighted(q, cache: KVCache, seq_lens, idx, weights, sparsity: Sparsity,
                                  out=None, stream=None):
    """Attention of each query head over its listed positions, entry t of a
    row weighted by weights[b, r, t] (float32, the shape of idx)."""
    _need_device(seq_lens, "seq_lens", torch.int32)
    _need_device(weights, "weights", torch.float32)
    if out is None:
        out = torch.empty_like(q)
    sp = sparsity.c()
    cq, kk, kv = _tensor(q, "q"), cache.c("k"), cache.c("v")
    ci, cw, co = _tensor(idx, "idx"), _tensor(weights, "weights"), _tensor(out, "out")
    _check(lib.sparse_decode_attend_weighted(C.byref(cq), C.byref(kk), C.byref(kv),
                                             seq_lens.data_ptr(), C.byref(ci), C.byref(cw),
                                             C.byref(sp), C.byref(co), _stream(stream)),
           "sparse_decode_attend_weighted")
    return out


def sparse_decode_dense_attention(q, cache: KVCache, seq_lens, softmax_scale: float = 0.0,
                                  out=None, stream=None):
    """Dense decode attention over every cached position (bfloat16)."""
    _need_device(seq_lens, "seq_lens", torch.int32)
    if out is None:
        out = torch.empty_like(q)
    cq, kk, kv, co = _tensor(q, "q"), cache.c("k"), cache.c("v"), _tensor(out, "out")
    _check(lib.sparse_decode_dense_attention(C.byref(cq), C.byref(kk), C.byref(kv),
                                             seq_lens.data_ptr(), float(softmax_scale),
                                             C.byref(co), _stream(stream)),
           "sparse_decode_dense_attention")
    return out


def dense_workspace_size(q, cache: KVCache) -> int:
    n = C.c_size_t(0)
    cq, kk = _tensor(q, "q"), cache.c("k")
    _check(lib.sparse_decode_dense_workspace_size(C.byref(cq), C.byref(kk), C.byref(n)),
           "sparse_decode_dense_workspace_size")
    return int(n.value)


def sparse_decode_attention(q, cache: KVCache, seq_lens, sparsity: Sparsity, out=None, idx=None,
                            k_max: Optional[int] = None, stream=None):
    """The fused method: returns (out [B, Hq, 128], idx [B, R, k_max])."""
    _need_device(seq_lens, "seq_lens", torch.int32)
    if out is None:
        out = torch.empty_like(q)
    if idx is None:
        if k_max is None:
            k_max = k_max_of(cache, sparsity)
        idx = torch.empty((q.shape[0], rows_of(q, cache, sparsity), k_max), dtype=torch.int32,
                          device=q.device)
    sp = sparsity.c()
    cq, kk, kv = _tensor(q, "q"), cache.c("k"), cache.c("v")
    co, ci = _tensor(out, "out"), _tensor(idx, "idx")
    _check(lib.sparse_decode_attention(C.byref(cq), C.byref(kk), C.byref(kv), seq_lens.data_ptr(),
                                       C.byref(sp), C.byref(co), C.byref(ci), _stream(stream)),
           "sparse_decode_attention")
    return out, idx


NOALLOC_SCRATCH_BYTES = 64 << 20  # SD_NOALLOC_SCRATCH_BYTES


def sparse_decode_attention_noalloc(q, cache: KVCache, seq_lens, sparsity: Sparsity, out,
                                    idx, stream=None):
    """The fused method with the library's static scratch instead of its
    workspace (no device allocation); out and idx are the caller's."""
    _need_device(seq_lens, "seq_lens", torch.int32)
    sp = sparsity.c()
    cq, kk, kv = _tensor(q, "q"), cache.c("k"), cache.c("v")
    co, ci = _tensor(out, "out"), _tensor(idx, "idx")
    _check(lib.sparse_decode_attention_noalloc(C.byref(cq), C.byref(kk), C.byref(kv),
                                               seq_lens.data_ptr(), C.byref(sp), C.byref(co),
                                               C.byref(ci), _stream(stream)),
           "sparse_decode_attention_noalloc")
    return out, idx


def sparse_decode_label_attention(q, cache: KVCache, labels: Labels, seq_lens, sparsity: Sparsity,
                                  out=None, idx=None, k_max: Optional[int] = None, stream=None):
    """The method with the low-channel indexer choosing the positions:
    returns (out [B, Hq, 128], idx [B, R, k_max])."""
    _need_device(seq_lens, "seq_lens", torch.int32)
    if out is None:
        out = torch.empty_like(q)
    if idx is None:
        if k_max is None:
            k_max = k_max_of(cache, sparsity)
        idx = torch.empty((q.shape[0], rows_of(q, cache, sparsity), k_max), dtype=torch.int32,
                          device=q.device)
    sp, lab = sparsity.c(), labels.c()
    cq, kk, kv = _tensor(q, "q"), cache.c("k"), cache.c("v")
    co, ci = _tensor(out, "out"), _tensor(idx, "idx")
    _check(lib.sparse_decode_label_attention(C.byref(cq), C.byref(kk), C.byref(kv), C.byref(lab),
                                             seq_lens.data_ptr(), C.byref(sp), C.byref(co),
                                             C.byref(ci), _stream(stream)),
           "sparse_decode_label_attention")
    return out, idx


def sparse_decode_label_score(q, cache: KVCache, labels: Labels, seq_lens, sparsity: Sparsity,
                              scores=None, stream=None):
    """float32 approximate label scores [B, R, capacity] (-inf beyond each sequence)."""
    _need_device(seq_lens, "seq_lens", torch.int32)
    if scores is None:
        scores = torch.empty((q.shape[0], rows_of(q, cache, sparsity), cache.capacity),
                             dtype=torch.float32, device=q.device)
    sp, lab = sparsity.c(), labels.c()
    cq, kk, ks = _tensor(q, "q"), cache.c("k"), _tensor(scores, "scores")
    _check(lib.sparse_decode_label_score(C.byref(cq), C.byref(kk), C.byref(lab),
                                         seq_lens.data_ptr(), C.byref(sp), C.byref(ks),
                                         _stream(stream)), "sparse_decode_label_score")
    return scores


def workspace_size(q, cache: KVCache, sparsity: Sparsity, idx) -> int:
    n = C.c_size_t(0)
    sp, cq, kk, ci = sparsity.c(), _tensor(q, "q"), cache.c("k"), _tensor(idx, "idx")
    _check(lib.sparse_decode_workspace_size(C.byref(cq), C.byref(kk), C.byref(sp), C.byref(ci),
                                            C.byref(n)), "sparse_decode_workspace_size")
    return int(n.value)


_workspace_ref = None


def set_workspace(buf: Optional[torch.Tensor]) -> None:
    """Use a caller tensor (device, any dtype) as the library workspace, or
    None to let the library allocate its own."""
    global _workspace_ref
    if buf is None:
        _check(lib.sparse_decode_set_workspace(None, 0), "sparse_decode_set_workspace")
    else:
        _need_device(buf, "workspace")
        _check(lib.sparse_decode_set_workspace(buf.data_ptr(), buf.numel() * buf.element_size()),
               "sparse_decode_set_workspace")
    _workspace_ref = buf


def set_profiling(enable) -> None:
    """True/1: events between every stage; 2: only around the scoring stream."""
    level = 2 if enable == 2 else int(bool(enable))
    _check(lib.sparse_decode_set_profiling(level), "sparse_decode_set_profiling")


def last_profile() -> dict:
    p = SdProfile()
    _check(lib.sparse_decode_last_profile(C.byref(p)), "sparse_decode_last_profile")
    return {f: getattr(p, f) for f, _ in SdProfile._fields_}


def profile_mean() -> dict:
    """Mean stage times (ms) over the profiled calls since set_profiling(True)."""
    p, n = SdProfile(), C.c_int32(0)
    _check(lib.sparse_decode_profile_mean(C.byref(p), C.byref(n)), "sparse_decode_profile_mean")
    d = {f: getattr(p, f) for f, _ in SdProfile._fields_}
    d["calls"] = int(n.value)
    return d


def sparse_decode_sampled_attention(q, cache: KVCache, seq_lens, sparsity: Sparsity, draws,
                                    out=None, idx=None, weights=None, k_max: Optional[int] = None,
                                    stream=None):
    """Exact top-k plus s importance-weighted uniform draws of the rest of
    each row (draws: int32 [B, R, s], read as uint32 bits).  Returns (out,
    idx [B, R, k_max + s], weights, same shape)."""
    _need_device(seq_lens, "seq_lens", torch.int32)
    _need_device(draws, "draws", torch.int32)
    s = int(draws.shape[2])
    if idx is None:
        km = k_max_of(cache, sparsity) if k_max is None else k_max
        idx = torch.empty((q.shape[0], rows_of(q, cache, sparsity), km + s), dtype=torch.int32,
                          device=q.device)
    if weights is None:
        weights = torch.empty(idx.shape, dtype=torch.float32, device=q.device)
    if out is None:
        out = torch.empty_like(q)
    sp = sparsity.c()
    cq, kk, kv = _tensor(q, "q"), cache.c("k"), cache.c("v")
    cd, co, ci, cw = _tensor(draws, "draws"), _tensor(out, "out"), _tensor(idx, "idx"), \
        _tensor(weights, "weights")
    _check(lib.sparse_decode_sampled_attention(C.byref(cq), C.byref(kk), C.byref(kv),
                                               seq_lens.data_ptr(), C.byref(sp), C.byref(cd),
                                               C.byref(co), C.byref(ci), C.byref(cw),
                                               _stream(stream)),
           "sparse_decode_sampled_attention")
    return out, idx, weights


def read_probe(buf: torch.Tensor, sink: torch.Tensor, stream=None) -> None:
    """One plain streaming read of buf (device, contiguous, 16-byte aligned):
    the device's reference read rate when timed.  sink: a device int32/uint32
    scalar the kernel may write."""
    _need_device(buf, "buf")
    _need_device(sink, "sink")
    if not buf.is_contiguous():
        raise ValueError("buf must be contiguous")
    nbytes = buf.numel() * buf.element_size()
    _check(lib.sparse_decode_read_probe(buf.data_ptr(), nbytes, sink.data_ptr(), _stream(stream)),
           "sparse_decode_read_probe")


def set_debug(flags: int) -> None:
    _check(lib.sparse_decode_set_debug(int(flags)), "sparse_decode_set_debug")


def cache_from_inputs(inp, device="cuda") -> tuple:
    """Copy a host decode-step description (uint16 bfloat16 bits or float32
    arrays) to the device: returns (q, KVCache, seq_lens)."""
    def dev(a):
        t = torch.from_numpy(a)
        if a.dtype.name == "uint16":
            t = t.view(torch.bfloat16)
        return t.to(device)
    q = dev(inp.q)
    cache = KVCache(k=dev(inp.k), v=dev(inp.v), layout=inp.layout,
                    block_table=(torch.from_numpy(inp.block_table).to(device)
                                 if inp.block_table is not None else None),
                    page_size=inp.page_size)
    seq_lens = torch.from_numpy(inp.seq_lens.astype("int32")).to(device)
    return q, cache, seq_lens


def sparsity_from_inputs(inp, **kw) -> Sparsity:
    kw.setdefault("n_sink", int(getattr(inp, "n_sink", 0) or 0))
    kw.setdefault("n_local", int(getattr(inp, "n_local", 0) or 0))
    return Sparsity(ratio=inp.ratio, rounding=inp.rounding, group_shared=inp.group_shared, **kw)
