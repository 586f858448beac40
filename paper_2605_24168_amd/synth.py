"""Seeded synthetic decode-step inputs for exact top-k sparse decode attention.

This module only draws inputs: random values, planted high-similarity keys,
bfloat16 rounding, page tables.  It holds none of the method's arithmetic
(no scoring, selection or softmax), so both the HIP path and the CPU oracle
can consume its arrays.

Five workloads, shaped like the paper's kernel benchmarks (Table 1 and
Table 2: head dimension 128, GQA with 8 KV heads, page size 16 in NHD
layout, 128K context, 10x-100x sparsity):

  1  one sequence, 1 query head / 1 KV head, N = 4096, float32, 10x;
     K, V ~ N(0,1), q ~ N(0,1)/sqrt(d), 16 planted keys with cosine 0.9 to q.
  2  batch 4, 32 query / 8 KV heads, N = 32768, bfloat16 [B,Hkv,N,d], 20x;
     entries N(0,1) times a per-KV-head scale U[0.5, 2]; 1% planted keys.
  3  batch 16, 64 query / 8 KV heads, N = 131072, bfloat16, 100x; as 2, plus
     a 64-token prefix whose keys have 4x the norm ("sink" tokens).
  4  32 ragged sequences, lengths U{8192..131072}, paged KV cache (page 16,
     NHD, random physical page permutation), 32 / 8 heads, bfloat16, 50x with
     k = ceil(L/50).
  5  one sequence, 40 query / 8 KV heads, N = 1048576, bfloat16, 100x, one
     index set per KV head chosen on the group-summed score; keys drawn from
     a 256-centroid Gaussian mixture so that scores are clustered.

Every (workload, seed, sequence, KV head, tensor) slab has its own numpy
PCG64 stream, so slabs are generated in parallel and any slab can be
regenerated alone.
"""
from __future__ import annotations

import concurrent.futures as cf
import dataclasses
import math
import os
from typing import Optional

import numpy as np

HEAD_DIM = 128
PAGE_SIZE = 16
ROOT_SEED = 260524168
POISON = 64.0  # written to allocated-but-unused positions (never a valid key)

(TAG_Q, TAG_K, TAG_V, TAG_PLANT, TAG_SCALE, TAG_LENS, TAG_PAGES, TAG_CENTROID, TAG_SETS,
 TAG_WEIGHTS, TAG_CHANNELS) = range(11)


@dataclasses.dataclass
class DecodeInputs:
    """One decode step.  bf16 tensors are uint16 arrays of bfloat16 bits."""
    name: str
    B: int
    Hq: int
    Hkv: int
    d: int
    dtype: str                 # "bf16" or "f32"
    q: np.ndarray              # [B, Hq, d]
    k: np.ndarray              # bhnd: [B, Hkv, ncap, d]; paged: [P, page, Hkv, d]
    v: np.ndarray
    seq_lens: np.ndarray       # int32 [B]
    layout: str                # "bhnd" or "paged"
    ncap: int                  # positions addressable per sequence
    ratio: float               # sparsity S (k = L / S rounded)
    rounding: int              # 0: nearest (half up), 1: ceil
    group_shared: bool
    page_size: int = PAGE_SIZE
    block_table: Optional[np.ndarray] = None   # int32 [B, max_pages] (paged)
    planted: Optional[dict] = None             # (b, g) -> (positions, heads)
    n_sink: int = 0                            # forced first positions (0 = none)
    n_local: int = 0                           # forced last positions (0 = none)

    @property
    def G(self) -> int:
        return self.Hq // self.Hkv

    @property
    def rows(self) -> int:
        return self.Hkv if self.group_shared else self.Hq

    @property
    def max_pages(self) -> int:
        return 0 if self.block_table is None else int(self.block_table.shape[1])

    @property
    def num_pages(self) -> int:
        return int(self.k.shape[0]) if self.layout == "paged" else 0


def _rng(*key: int) -> np.random.Generator:
    return np.random.Generator(np.random.PCG64(np.random.SeedSequence([ROOT_SEED, *key])))


def bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round float32 values to bfloat16 (round to nearest, ties to even)."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    r = (u + (((u >> 16) & np.uint32(1)) + np.uint32(0x7FFF))) >> np.uint32(16)
    return r.astype(np.uint16)


def bf16_to_f32(bits: np.ndarray) -> np.ndarray:
    """Exact widening of bfloat16 bits to float32."""
    return (bits.astype(np.uint32) << np.uint32(16)).view(np.float32)


def _store(x: np.ndarray, dtype: str) -> np.ndarray:
    return bf16_bits(x) if dtype == "bf16" else np.ascontiguousarray(x, dtype=np.float32)


def _as_f32(x: np.ndarray, dtype: str) -> np.ndarray:
    return bf16_to_f32(x) if dtype == "bf16" else x.astype(np.float32)


def _workers(threads: Optional[int]) -> int:
    if threads:
        return threads
    try:
        n = len(os.sched_getaffinity(0))
    except AttributeError:  # pragma: no cover
        n = os.cpu_count() or 1
    return max(1, min(n, 16))


def _unit_perp(rng: np.random.Generator, qhat: np.ndarray) -> np.ndarray:
    """A random unit vector orthogonal to the unit vector qhat."""
    u = rng.standard_normal(qhat.shape[0])
    u -= u.dot(qhat) * qhat
    return u / np.linalg.norm(u)


def _plant(rng: np.random.Generator, keys: np.ndarray, L: int, n: int,
           qf: np.ndarray, scale: float) -> tuple[np.ndarray, np.ndarray]:
    """Overwrite n random positions of keys[:L] with keys of cosine 0.9 to one
    query head (chosen uniformly among the rows of qf) and norm scale*sqrt(d)."""
    if n == 0:
        return np.zeros(0, np.int64), np.zeros(0, np.int64)
    d = keys.shape[1]
    pos = np.sort(rng.choice(L, size=n, replace=False))
    heads = rng.integers(0, qf.shape[0], size=n)
    for p, h in zip(pos, heads):
        qhat = qf[h] / np.linalg.norm(qf[h])
        u = _unit_perp(rng, qhat)
        keys[p] = math.sqrt(d) * scale * (0.9 * qhat + math.sqrt(1 - 0.81) * u)
    return pos, heads


@dataclasses.dataclass
class _Spec:
    cfg: int
    B: int
    Hq: int
    Hkv: int
    N: int
    dtype: str
    ratio: float
    rounding: int
    group_shared: bool
    layout: str
    lmin: int = 0
    lmax: int = 0
    plant_frac: float = 0.0
    n_plant_fixed: int = 0
    sink: int = 0
    head_scale: bool = False
    mixture: int = 0


DEFAULTS = {
    1: _Spec(1, 1, 1, 1, 4096, "f32", 10.0, 0, False, "bhnd", n_plant_fixed=16),
    2: _Spec(2, 4, 32, 8, 32768, "bf16", 20.0, 0, False, "bhnd", plant_frac=0.01, head_scale=True),
    3: _Spec(3, 16, 64, 8, 131072, "bf16", 100.0, 0, False, "bhnd", plant_frac=0.01,
             head_scale=True, sink=64),
    4: _Spec(4, 32, 32, 8, 131072, "bf16", 50.0, 1, False, "paged", lmin=8192, lmax=131072,
             plant_frac=0.01, head_scale=True),
    5: _Spec(5, 1, 40, 8, 1048576, "bf16", 100.0, 0, True, "bhnd", mixture=256),
}

NAMES = {
    1: "single-seq 1q/1kv N=4096 f32 10x",
    2: "B=4 GQA 32q/8kv N=32768 bf16 20x",
    3: "B=16 GQA 64q/8kv N=131072 bf16 100x +64 sink",
    4: "32 ragged seqs L~U[8K,128K] paged16 GQA 32q/8kv bf16 50x ceil",
    5: "B=1 GQA 40q/8kv N=1048576 bf16 100x group-shared mixture keys",
}


def make_inputs(cfg: int, seed: int = 0, *, B: Optional[int] = None, N: Optional[int] = None,
                Hq: Optional[int] = None, Hkv: Optional[int] = None,
                lmin: Optional[int] = None, lmax: Optional[int] = None,
                seq_lens: Optional[list] = None, ncap: Optional[int] = None,
                layout: Optional[str] = None, dtype: Optional[str] = None,
                ratio: Optional[float] = None, group_shared: Optional[bool] = None,
                threads: Optional[int] = None, n_sink: int = 0,
                n_local: int = 0) -> DecodeInputs:
    """Draw the inputs of workload ``cfg`` (1..5).  Keyword overrides shrink or
    reshape a workload for tests (e.g. a ragged batch with ``seq_lens``)."""
    s = dataclasses.replace(DEFAULTS[cfg])
    if B is not None: s.B = B
    if N is not None: s.N = N
    if Hq is not None: s.Hq = Hq
    if Hkv is not None: s.Hkv = Hkv
    if lmin is not None: s.lmin = lmin
    if lmax is not None: s.lmax = lmax
    if layout is not None: s.layout = layout
    if dtype is not None: s.dtype = dtype
    if ratio is not None: s.ratio = ratio
    if group_shared is not None: s.group_shared = group_shared
    if s.Hq % s.Hkv:
        raise ValueError("Hq must be a multiple of Hkv")
    d = HEAD_DIM
    G = s.Hq // s.Hkv

    # Sequence lengths.
    if seq_lens is not None:
        lens = np.asarray(seq_lens, dtype=np.int32)
        s.B = len(lens)
    elif s.lmax:
        lens = _rng(cfg, seed, 0, 0, TAG_LENS).integers(s.lmin, s.lmax + 1, size=s.B).astype(np.int32)
    else:
        lens = np.full(s.B, s.N, dtype=np.int32)
    if ncap is None:
        ncap = max(s.N if not s.lmax else s.lmax, int(lens.max(initial=0)))
    if s.layout == "paged":
        ncap = -(-ncap // PAGE_SIZE) * PAGE_SIZE
    if int(lens.max(initial=0)) > ncap:
        raise ValueError("a sequence is longer than the cache capacity")

    # Queries: N(0,1)/sqrt(d), one stream per sequence.
    qf = np.stack([_rng(cfg, seed, b, 0, TAG_Q).standard_normal((s.Hq, d), dtype=np.float32)
                   for b in range(s.B)]) / np.float32(math.sqrt(d)) if s.B else \
        np.zeros((0, s.Hq, d), np.float32)
    q = _store(qf, s.dtype)
    q_seen = _as_f32(q, s.dtype)  # what the kernels see; planted keys align with it

    head_scale = (_rng(cfg, seed, 0, 0, TAG_SCALE).uniform(0.5, 2.0, size=s.Hkv)
                  if s.head_scale else np.ones(s.Hkv))
    store_dt = np.uint16 if s.dtype == "bf16" else np.float32
    poison = _store(np.array([POISON], np.float32), s.dtype)[0]

    # Cache storage.
    if s.layout == "paged":
        pages_per = [-(-int(L) // PAGE_SIZE) for L in lens]
        total_pages = int(sum(pages_per))
        perm = _rng(cfg, seed, 0, 0, TAG_PAGES).permutation(total_pages).astype(np.int32)
        max_pages = ncap // PAGE_SIZE
        block_table = np.full((s.B, max_pages), -1, dtype=np.int32)
        start = 0
        for b, n in enumerate(pages_per):
            block_table[b, :n] = perm[start:start + n]
            start += n
        k = np.full((total_pages, PAGE_SIZE, s.Hkv, d), poison, dtype=store_dt)
        v = np.full((total_pages, PAGE_SIZE, s.Hkv, d), poison, dtype=store_dt)
    else:
        block_table = None
        k = np.empty((s.B, s.Hkv, ncap, d), dtype=store_dt)
        v = np.empty((s.B, s.Hkv, ncap, d), dtype=store_dt)

    planted: dict = {}

    def slab(b: int, g: int) -> None:
        L = int(lens[b])
        c = float(head_scale[g])
        if s.mixture:
            mu = _rng(cfg, seed, b, g, TAG_CENTROID).standard_normal((s.mixture, d), dtype=np.float32)
            r = _rng(cfg, seed, b, g, TAG_K)
            z = r.integers(0, s.mixture, size=L)
            kf = mu[z] + np.float32(0.25) * r.standard_normal((L, d), dtype=np.float32)
        else:
            kf = _rng(cfg, seed, b, g, TAG_K).standard_normal((L, d), dtype=np.float32)
            if c != 1.0:
                kf *= np.float32(c)
        n_plant = s.n_plant_fixed if s.n_plant_fixed else int(round(s.plant_frac * L))
        n_plant = min(n_plant, L)
        if n_plant:
            pos, heads = _plant(_rng(cfg, seed, b, g, TAG_PLANT), kf, L, n_plant,
                                q_seen[b, g * G:(g + 1) * G].astype(np.float64), c)
            planted[(b, g)] = (pos, heads)
        if s.sink:
            kf[:min(s.sink, L)] *= np.float32(4.0)
        vf = _rng(cfg, seed, b, g, TAG_V).standard_normal((L, d), dtype=np.float32)
        if c != 1.0 and not s.mixture:
            vf *= np.float32(c)
        kb, vb = _store(kf, s.dtype), _store(vf, s.dtype)
        if s.layout == "paged":
            n = -(-L // PAGE_SIZE)
            pages = block_table[b, :n]
            full = L // PAGE_SIZE
            if full:
                k[pages[:full], :, g, :] = kb[:full * PAGE_SIZE].reshape(full, PAGE_SIZE, d)
                v[pages[:full], :, g, :] = vb[:full * PAGE_SIZE].reshape(full, PAGE_SIZE, d)
            rem = L - full * PAGE_SIZE
            if rem:
                k[pages[full], :rem, g, :] = kb[full * PAGE_SIZE:]
                v[pages[full], :rem, g, :] = vb[full * PAGE_SIZE:]
        else:
            k[b, g, :L] = kb
            v[b, g, :L] = vb
            k[b, g, L:] = poison
            v[b, g, L:] = poison

    jobs = [(b, g) for b in range(s.B) for g in range(s.Hkv)]
    with cf.ThreadPoolExecutor(max_workers=_workers(threads)) as ex:
        for f in [ex.submit(slab, b, g) for b, g in jobs]:
            f.result()

    return DecodeInputs(
        name=NAMES[cfg], B=s.B, Hq=s.Hq, Hkv=s.Hkv, d=d, dtype=s.dtype, q=q, k=k, v=v,
        seq_lens=lens, layout=s.layout, ncap=int(ncap), ratio=float(s.ratio),
        rounding=s.rounding, group_shared=bool(s.group_shared), page_size=PAGE_SIZE,
        block_table=block_table, planted=planted, n_sink=int(n_sink), n_local=int(n_local))


def index_sets(inp: DecodeInputs, k: int, seed: int = 0, k_max: Optional[int] = None,
               extra_invalid: int = 0) -> np.ndarray:
    """Irregular index lists for the attend-only backend (Table 1 imposes no
    block structure): row (b, r) holds min(k, L_b) distinct positions drawn
    uniformly from [0, L_b), ascending, then -1 padding up to k_max.  With
    extra_invalid > 0 that many entries of each row (within k_max) are
    replaced by positions the attention must skip (-1 or >= L_b)."""
    k_max = k if k_max is None else k_max
    idx = np.full((inp.B, inp.rows, k_max), -1, dtype=np.int32)
    for b in range(inp.B):
        L = int(inp.seq_lens[b])
        n = min(k, L, k_max)
        rng = _rng(0, seed, b, 0, TAG_SETS)
        for r in range(inp.rows):
            if n:
                idx[b, r, :n] = np.sort(rng.choice(L, size=n, replace=False))
            if extra_invalid and k_max:
                at = rng.choice(k_max, size=min(extra_invalid, k_max), replace=False)
                idx[b, r, at] = np.where(rng.random(at.size) < 0.5, -1, L + rng.integers(0, 64, at.size))
    return idx


def index_weights(shape, seed: int = 0, zero_frac: float = 0.0) -> np.ndarray:
    """Per-entry weights for index lists: U[0.05, 3), a fraction zero_frac of
    them exactly 0."""
    rng = _rng(0, seed, 0, 0, TAG_WEIGHTS)
    w = rng.uniform(0.05, 3.0, size=shape).astype(np.float32)
    if zero_frac:
        w[rng.random(shape) < zero_frac] = 0.0
    return w


def backend_sweep_inputs(B: int = 16, N: int = 131072, Hq: int = 32, Hkv: int = 8,
                         seed: int = 0, device="cuda"):
    """The kernel-benchmark shape of Table 1 drawn directly on the GPU (host
    generation of 8.6 GB would dominate a sweep): B sequences of N positions
    in a paged NHD cache (page 16) with a random physical page order, bfloat16
    K, V ~ N(0, 1) and q ~ N(0, 1) / sqrt(d).  Returns a dict of device
    tensors: q [B, Hq, d], k and v [pages, 16, Hkv, d], block_table
    [B, N / 16] int32, seq_lens [B] int32."""
    import torch
    gen = torch.Generator(device=device)
    gen.manual_seed(ROOT_SEED * 1000 + seed)
    per = -(-N // PAGE_SIZE)
    pages = B * per
    perm = torch.randperm(pages, generator=gen, device=device).to(torch.int32)
    shape = (pages, PAGE_SIZE, Hkv, HEAD_DIM)
    k = torch.randn(shape, generator=gen, device=device, dtype=torch.float32).to(torch.bfloat16)
    v = torch.randn(shape, generator=gen, device=device, dtype=torch.float32).to(torch.bfloat16)
    q = (torch.randn((B, Hq, HEAD_DIM), generator=gen, device=device) /
         math.sqrt(HEAD_DIM)).to(torch.bfloat16)
    return {"q": q, "k": k, "v": v, "block_table": perm.view(B, per).contiguous(),
            "seq_lens": torch.full((B,), N, dtype=torch.int32, device=device)}


def backend_sweep_sets(rows: int, N: int, k: int, seed: int = 0, device="cuda"):
    """Irregular index lists on the GPU for the backend sweep: each of `rows`
    rows holds k distinct positions of [0, N), uniform, ascending (no block
    structure), with weights U[0.05, 3).  Returns (idx int32, weights f32)."""
    import torch
    gen = torch.Generator(device=device)
    gen.manual_seed(ROOT_SEED * 1000 + 7919 * seed + k)
    idx = torch.empty((rows, k), dtype=torch.int32, device=device)
    for r0 in range(0, rows, 64):  # bounded temporary: 64 rows of N keys at a time
        r1 = min(rows, r0 + 64)
        keys = torch.rand((r1 - r0, N), generator=gen, device=device)
        idx[r0:r1] = torch.sort(torch.topk(keys, k, dim=1, sorted=False).indices, dim=1).values
    w = torch.rand((rows, k), generator=gen, device=device) * 2.95 + 0.05
    return idx, w


N_LABELS = 8


def label_channels(Hkv: int, seed: int = 0, n: int = N_LABELS) -> np.ndarray:
    """Label channels of the low-channel indexer, uncalibrated (Table 2's
    indexer is untuned): n distinct channels per KV head drawn uniformly,
    ascending.  int32 [Hkv, n]."""
    rng = _rng(0, seed, 0, 0, TAG_CHANNELS)
    return np.stack([np.sort(rng.choice(HEAD_DIM, size=n, replace=False))
                     for _ in range(Hkv)]).astype(np.int32)


def label_cache(inp: DecodeInputs, channels: np.ndarray) -> np.ndarray:
    """The label cache of a decode step: each key's label channels (copied
    bits, so 16-bit for bfloat16 caches), in the key cache's layout with
    rows of len(channels[g]) elements."""
    n = channels.shape[1]
    if inp.layout == "paged":
        out = np.empty(inp.k.shape[:3] + (n,), dtype=inp.k.dtype)
        for g in range(inp.Hkv):
            out[:, :, g, :] = inp.k[:, :, g, :][:, :, channels[g]]
    else:
        out = np.empty(inp.k.shape[:3] + (n,), dtype=inp.k.dtype)
        for g in range(inp.Hkv):
            out[:, g] = inp.k[:, g][:, :, channels[g]]
    return out


def label_cache_device_layout(inp: DecodeInputs, labels: np.ndarray) -> np.ndarray:
    """The label cache in the library's layout: unchanged beside a
    contiguous cache; [pages, Hkv, 16, n] (head-major inside a page) beside a
    paged one, where label_cache gives the key cache's [pages, 16, Hkv, n]."""
    if inp.layout == "paged":
        return np.ascontiguousarray(labels.transpose(0, 2, 1, 3))
    return labels
