"""Comparison rules between the HIP path and the CPU oracle.

Index sets: bit-exact outside a near-tie band.  With tau the oracle's k-th
largest selection score (float64) and band = {j : |s_j - tau| <= 1e-3 *
max(1, |tau|)}, the GPU set minus the band must equal the oracle set minus
the band; swaps inside the band are counted, not failed.

Outputs: float32 caches must match element by element within 1e-4 relative,
|gpu_i - ref_i| <= 1e-4 |ref_i| + 1e-6 (the absolute floor covers elements
near zero); bfloat16 within 2e-2 absolute.  When the band swapped positions, the reference output is the
oracle's attention over the GPU's own index set, so that a legitimate swap
does not count as an output error.
"""
from __future__ import annotations

import dataclasses
import math
import sys

import numpy as np

from oracle import oracle as O

BAND_REL = 1e-3
F32_OUT_REL = 1e-4
F32_OUT_ABS = 1e-6
BF16_OUT_ABS = 2e-2


def log(msg: str) -> None:
    print(msg, flush=True)
    sys.stdout.flush()


@dataclasses.dataclass
class IdxReport:
    rows: int = 0
    band_swaps: int = 0
    strict_mismatch_rows: int = 0
    first_failure: str = ""


def check_idx_rows(gpu_idx: np.ndarray, ora_idx: np.ndarray, ora_scores: np.ndarray,
                   tau: np.ndarray, seq_lens: np.ndarray, ks: np.ndarray,
                   rows=None) -> IdxReport:
    """gpu_idx, ora_idx: [B, R, k_max]; ora_scores: [B, R, ncap] float64 (or a
    callable (b, r) -> row); ks: [B] budgets.  rows: iterable of (b, r)."""
    rep = IdxReport()
    B, R, k_max = gpu_idx.shape
    rows = rows if rows is not None else [(b, r) for b in range(B) for r in range(R)]
    for b, r in rows:
        rep.rows += 1
        k = int(ks[b])
        L = int(seq_lens[b])
        g = gpu_idx[b, r]
        o = ora_idx[b, r]
        # Structure of a GPU row: k ascending valid positions, then -1.
        gk = g[:k]
        ok = (g[k:] == -1).all() and (gk >= 0).all() and (gk < L).all() and \
            (np.diff(gk) > 0).all()
        if not ok:
            rep.strict_mismatch_rows += 1
            rep.first_failure = rep.first_failure or f"row {(b, r)} malformed: {g[:8]}..."
            continue
        gs, os_ = set(gk.tolist()), set(o[:k].tolist())
        if gs == os_:
            continue
        srow = ora_scores(b, r) if callable(ora_scores) else ora_scores[b, r]
        t = tau[b, r]
        width = BAND_REL * max(1.0, abs(t))
        in_band = lambda j: abs(srow[j] - t) <= width
        d1 = {j for j in gs - os_ if not in_band(j)}
        d2 = {j for j in os_ - gs if not in_band(j)}
        if d1 or d2:
            rep.strict_mismatch_rows += 1
            rep.first_failure = rep.first_failure or (
                f"row {(b, r)}: gpu-only {sorted(d1)[:5]} oracle-only {sorted(d2)[:5]} "
                f"tau={t}")
        rep.band_swaps += len(gs - os_)
    return rep


def out_errors(gpu_out: np.ndarray, ref_out: np.ndarray, dtype: str):
    """Return (ok, worst_ratio, rel_l2): worst_ratio = max over elements of the
    error divided by its allowance (<= 1 passes)."""
    g = gpu_out.astype(np.float64)
    r = ref_out.astype(np.float64)
    err = np.abs(g - r)
    if dtype == "f32":
        allow = F32_OUT_REL * np.abs(r) + F32_OUT_ABS
    else:
        allow = np.full_like(err, BF16_OUT_ABS)
    ratio = float((err / allow).max()) if err.size else 0.0
    den = np.linalg.norm(r)
    rel_l2 = float(np.linalg.norm(g - r) / den) if den > 0 else float(np.linalg.norm(g - r))
    return ratio <= 1.0, ratio, rel_l2


def score_allowance(q: np.ndarray, K: np.ndarray) -> np.ndarray:
    """Bound on |float32 score - exact score| for one query row q [d] against
    keys K [n, d]: float32 accumulation of d exact products has error at most
    gamma_d * sum_i |q_i K_ji|, gamma_d = d u / (1 - d u), u = 2^-24; doubled
    to leave room for the matrix unit's internal summation order."""
    d = q.shape[-1]
    u = 2.0 ** -24
    gamma = d * u / (1 - d * u)
    return 2.0 * gamma * (np.abs(K.astype(np.float64)) @ np.abs(q.astype(np.float64))) + 1e-30


def budgets(inp) -> np.ndarray:
    return np.array([O.budget(int(L), inp.ratio, inp.rounding) for L in inp.seq_lens], np.int64)


def to_host(t) -> np.ndarray:
    import torch
    t = t.detach()
    if t.dtype == torch.bfloat16:
        t = t.float()
    return t.cpu().numpy()


def fmt_s(x: float) -> str:
    return "nan" if math.isnan(x) else f"{x:.3g}"


def slice_batch(inp, bs):
    """Sequences bs of a decode step as a smaller step (views of the cache;
    a paged step keeps its page pool and slices its block table)."""
    import dataclasses
    bs = list(bs)
    if inp.layout == "paged":
        return dataclasses.replace(inp, B=len(bs), q=inp.q[bs], seq_lens=inp.seq_lens[bs],
                                   block_table=inp.block_table[bs])
    return dataclasses.replace(inp, B=len(bs), q=inp.q[bs], k=inp.k[bs], v=inp.v[bs],
                               seq_lens=inp.seq_lens[bs])
