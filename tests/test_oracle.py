"""Pins of the CPU oracle against things other than itself.

Each test ties the oracle to a fact the paper or mathematics fixes: the k
values the workloads print, closed forms, brute-force enumeration of every
k-subset, a library attention routine, invariants of softmax averaging, and
hand-derived worked examples (tests/golden/).  A dropped term, a wrong sign
or index, a reversed tie-break or a transposed operand in the oracle fails
at least one of them (tests/test_oracle_mutants.py checks exactly that).
"""
import itertools
import json
import math
import os
import types

import numpy as np
import pytest
import torch

from oracle import oracle as O
from paper_2605_24168_amd import synth

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "hand_examples.json")


def problem(q, k, v, seq_lens=None, ratio=2.0, rounding=0, group_shared=False,
            dtype="f32", Hkv=1):
    """A tiny decode step in the contiguous [B, Hkv, N, d] layout (float32)."""
    q = np.asarray(q, np.float32)
    k = np.asarray(k, np.float32)
    v = np.asarray(v, np.float32)
    if q.ndim == 2:
        q = q[None]
    if k.ndim == 2:
        k, v = k[None, None], v[None, None]
    B, Hq, d = q.shape
    ncap = k.shape[2]
    lens = np.full(B, ncap, np.int32) if seq_lens is None else np.asarray(seq_lens, np.int32)
    return types.SimpleNamespace(B=B, Hq=Hq, Hkv=k.shape[1], d=d, dtype=dtype, q=q, k=k, v=v,
                                 seq_lens=lens, layout="bhnd", ncap=ncap, ratio=ratio,
                                 rounding=rounding, group_shared=group_shared, page_size=0,
                                 block_table=None,
                                 rows=(k.shape[1] if group_shared else Hq))


def to_paged(p, page_size, seed=0):
    """Same decode step in the paged [pages, page, Hkv, d] layout with a random
    physical page order."""
    rng = np.random.default_rng(seed)
    B, Hkv, ncap, d = p.k.shape
    per = -(-ncap // page_size)
    total = B * per
    perm = rng.permutation(total).astype(np.int32)
    bt = perm.reshape(B, per)
    kp = np.full((total, page_size, Hkv, d), 1e6, np.float32)
    vp = np.full_like(kp, -1e6)
    for b in range(B):
        for t in range(per):
            n = min(page_size, ncap - t * page_size)
            kp[bt[b, t], :n] = p.k[b, :, t * page_size:t * page_size + n].transpose(1, 0, 2)
            vp[bt[b, t], :n] = p.v[b, :, t * page_size:t * page_size + n].transpose(1, 0, 2)
    return types.SimpleNamespace(**{**vars(p), "k": kp, "v": vp, "layout": "paged",
                                    "page_size": page_size, "block_table": bt,
                                    "ncap": per * page_size})


# --------------------------------------------------------------------------
# k = N / S (Table 1 caption); printed values of the five workloads.
# --------------------------------------------------------------------------

def test_budget_printed_values():
    assert O.budget(4096, 10) == 410           # workload 1: k = 410
    assert O.budget(32768, 20) == 1638         # workload 2: k = 1638
    assert O.budget(131072, 100) == 1311       # workload 3: k = 1311
    assert O.budget(1048576, 100) == 10486     # workload 5
    assert O.budget(8192, 50, 1) == 164        # workload 4: k = ceil(L/50)
    assert O.budget(131072, 50, 1) == 2622


def test_budget_integer_forms_and_clamps():
    for s in (1, 2, 3, 7, 10, 20, 50, 100, 500):
        for L in list(range(0, 300)) + [4095, 4096, 4097, 131071, 131072]:
            near = O.budget(L, s, 0)
            ceil_ = O.budget(L, s, 1)
            if L == 0:
                assert near == 0 and ceil_ == 0
                continue
            assert near == min(L, max(1, (2 * L + s) // (2 * s)))   # nearest, halves up
            assert ceil_ == min(L, max(1, (L + s - 1) // s))
    assert O.budget(5, 100) == 1          # at least one kept position
    assert O.budget(10, 0.5) == 10        # never more than L
    assert O.budget(5, 2) == 3            # 2.5 rounds up
    assert O.budget(7, 2) == 4            # 3.5 rounds up


# --------------------------------------------------------------------------
# Scores: closed forms.
# --------------------------------------------------------------------------

def test_bf16_decoding_exact():
    # bfloat16 bit patterns and their exact values (upper half of a float32).
    bits = np.array([0x3F80, 0xC000, 0x0001, 0x7F7F, 0x8080, 0x3EAB, 0x0000, 0x4040], np.uint16)
    want = np.array([1.0, -2.0, 2.0 ** -133, (2 - 2 ** -7) * 2.0 ** 127, -(2.0 ** -126),
                     0.333984375, 0.0, 3.0])
    d, N = 8, len(bits)
    for i in range(d):
        q = np.zeros((1, 1, d), np.uint16)
        q[0, 0, i] = 0x3F80  # one-hot query: score_j = K[j, i]
        K = np.zeros((1, 1, N, d), np.uint16)
        K[0, 0, :, i] = bits
        p = problem(np.zeros((1, d)), np.zeros((N, d)), np.zeros((N, d)))
        p.q, p.k, p.v, p.dtype = q, K, K.copy(), "bf16"
        s = O.scores(p)[0, 0]
        np.testing.assert_array_equal(s, want)


def test_scores_match_exact_integer_products():
    rng = np.random.default_rng(1)
    B, Hq, Hkv, N, d = 2, 6, 3, 37, 16
    q = rng.integers(-8, 9, (B, Hq, d))
    K = rng.integers(-8, 9, (B, Hkv, N, d))
    p = problem(q, K, K, seq_lens=[N, 29], Hkv=Hkv)
    s = O.scores(p)
    G = Hq // Hkv
    for b in range(B):
        for h in range(Hq):
            L = p.seq_lens[b]
            exact = K[b, h // G, :L] @ q[b, h]          # integer arithmetic, exact
            np.testing.assert_array_equal(s[b, h, :L], exact.astype(np.float64))
            assert np.isnan(s[b, h, L:]).all()
    # Group-shared scores: the group's summed query dotted with each key.
    pg = problem(q, K, K, seq_lens=[N, 29], group_shared=True, Hkv=Hkv)
    sg = O.scores(pg)
    for b in range(B):
        for g in range(Hkv):
            L = p.seq_lens[b]
            qsum = q[b, g * G:(g + 1) * G].sum(0)
            np.testing.assert_array_equal(sg[b, g, :L], (K[b, g, :L] @ qsum).astype(np.float64))


# --------------------------------------------------------------------------
# Selection: brute force over every k-subset.
# --------------------------------------------------------------------------

def _beats(si, i, sj, j):
    return si > sj or (si == sj and i < j)


def brute_force_topk(s, k):
    """The unique k-subset whose every member beats every non-member under
    (score descending, position ascending), found by enumerating all subsets."""
    n = len(s)
    hits = []
    for S in itertools.combinations(range(n), k):
        Sset = set(S)
        if all(_beats(s[i], i, s[j], j) for i in S for j in range(n) if j not in Sset):
            hits.append(S)
    assert len(hits) == 1
    return list(hits[0])


def test_select_matches_subset_enumeration():
    rng = np.random.default_rng(2)
    for trial in range(60):
        n = int(rng.integers(1, 11))
        s = rng.integers(-3, 4, n).astype(np.float64)   # small range: many ties
        if trial % 3 == 0:
            s = s + rng.standard_normal(n) * 1e-3
        for k in range(0, n + 1):
            idx, tau = O.select_row(s, k, k_max=n + 2)
            want = brute_force_topk(list(s), k)
            assert list(idx[:k]) == want
            assert (idx[k:] == -1).all()
            if k:
                assert tau == min(s[j] for j in want)
            else:
                assert math.isnan(tau)


def test_select_matches_library_lexsort():
    rng = np.random.default_rng(3)
    for n in (1, 2, 17, 64, 257, 1000):
        s = np.round(rng.standard_normal(n), 1)           # rounded: ties
        order = np.lexsort((np.arange(n), -s))             # key: -score, then position
        for k in sorted({1, n // 3, n // 2, n}):
            if k == 0:
                continue
            idx, _ = O.select_row(s, k)
            np.testing.assert_array_equal(idx, np.sort(order[:k]))


def test_select_degenerate_rows():
    idx, tau = O.select_row(np.full(9, 0.25), 4)
    assert list(idx) == [0, 1, 2, 3] and tau == 0.25     # all equal -> lowest positions
    s = np.array([1.0, 5.0, 3.0, 5.0, 5.0])
    idx, tau = O.select_row(s, 2)                        # duplicate maxima: lower ones
    assert list(idx) == [1, 3] and tau == 5.0
    idx, tau = O.select_row(np.array([-1.0, -2.0]), 2)   # k = L keeps everything
    assert list(idx) == [0, 1] and tau == -2.0
    with pytest.raises(O.OracleError):
        O.select_row(np.array([1.0, np.nan]), 1)         # non-finite scores rejected


def test_select_f32_uses_float32_values_exactly():
    # Two float32 scores one ulp apart must be ordered, not tied.
    a = np.float32(1.0)
    b = np.nextafter(a, np.float32(2.0))
    s = np.array([[[a, b, a]]], np.float32)
    idx, tau = O.select_f32(s, [3], ratio=3.0, rounding=0, k_max=2)
    assert list(idx[0, 0]) == [1, -1] and tau[0, 0] == float(b)


# --------------------------------------------------------------------------
# Selection with forced sink and local positions.
# --------------------------------------------------------------------------

def test_forced_selection_matches_enumeration_of_the_middle():
    rng = np.random.default_rng(31)
    for trial in range(80):
        L = int(rng.integers(0, 12))
        ns, nl = int(rng.integers(0, 5)), int(rng.integers(0, 5))
        s = rng.integers(-3, 4, L).astype(np.float64)
        fs = min(ns, L)
        fl = min(nl, L - fs)
        mid = list(range(fs, L - fl))
        for kh in range(0, len(mid) + 1):
            idx, tau = O.select_forced(s, ns, nl, kh, k_max=L + 3)
            # the exact top-kh of the middle positions alone, then the union
            heavy = [mid[i] for i in brute_force_topk([s[j] for j in mid], kh)]
            want = sorted(set(range(fs)) | set(heavy) | set(range(L - fl, L)))
            assert list(idx[:len(want)]) == want, (L, ns, nl, kh)
            assert (idx[len(want):] == -1).all()
            if kh:
                assert tau == min(s[j] for j in heavy)
            else:
                assert math.isnan(tau)


def test_forced_selection_special_cases():
    rng = np.random.default_rng(32)
    s = rng.standard_normal(40)
    for k in (0, 1, 7, 40):
        a, ta = O.select_forced(s, 0, 0, k, k_max=45)   # nothing forced: plain top-k
        b, tb = O.select_row(s, k, k_max=45)
        np.testing.assert_array_equal(a, b)
        assert (math.isnan(ta) and math.isnan(tb)) or ta == tb
    # Forced positions are kept whatever their scores, and never use budget.
    s = np.array([9.0, -5.0, 1.0, 2.0, 3.0, 8.0, -9.0, -7.0])
    idx, _ = O.select_forced(s, 2, 2, 1)
    assert list(idx) == [0, 1, 5, 6, 7]                  # middle top-1 is position 5
    idx, _ = O.select_forced(s, 2, 2, 0)
    assert list(idx) == [0, 1, 6, 7]
    # Forced windows covering the sequence keep every position once.
    idx, _ = O.select_forced(s, 5, 5, 0, k_max=9)
    assert list(idx) == list(range(8)) + [-1]
    idx, _ = O.select_forced(s, 20, 3, 0)
    assert list(idx) == list(range(8))
    with pytest.raises(O.OracleError):
        O.select_forced(s, 2, 2, 5)                      # more heavy than the middle holds


def test_forced_positions_in_the_whole_method():
    rng = np.random.default_rng(33)
    B, Hq, N, d = 2, 3, 50, 16
    q = rng.standard_normal((B, Hq, d)).astype(np.float32)
    K = rng.standard_normal((B, 1, N, d)).astype(np.float32)
    V = rng.standard_normal((B, 1, N, d)).astype(np.float32)
    p = problem(q, K, V, seq_lens=[50, 9], ratio=10.0)     # heavy k = 5 and 1
    p.n_sink, p.n_local = 4, 3
    r = O.sparse_attention(p)
    assert r["idx"].shape[2] == O.k_max_for(p) == 4 + 3 + 5
    sc = O.scores(p)
    for b, (L, kh) in enumerate(((50, 5), (9, 1))):
        for h in range(Hq):
            want, _ = O.select_forced(sc[b, h, :L], 4, 3, kh, k_max=12)
            np.testing.assert_array_equal(r["idx"][b, h], want)
    # The same sets through the plain attention give the same output.
    out, _ = O.attend(p, r["idx"])
    np.testing.assert_array_equal(out, r["out"])
    # Forced windows plus budget covering everything: dense attention.
    p.n_sink, p.n_local = 25, 25
    full = O.sparse_attention(p)
    np.testing.assert_allclose(full["out"], O.dense_attention(p), rtol=0, atol=1e-12)
    # The float32 selection entry point agrees.
    p.n_sink, p.n_local = 4, 3
    s32 = np.nan_to_num(sc, nan=-np.inf).astype(np.float32)
    idx32, _ = O.select_f32(s32, p.seq_lens, 10.0, 0, 12, n_sink=4, n_local=3)
    ref32 = np.array([[O.select_forced(s32[b, h, :L].astype(np.float64), 4, 3, kh, k_max=12)[0]
                       for h in range(Hq)] for b, (L, kh) in enumerate(((50, 5), (9, 1)))])
    np.testing.assert_array_equal(idx32, ref32)


# --------------------------------------------------------------------------
# Low-channel indexer (label cache of a few channels per key).
# --------------------------------------------------------------------------

def _labels_from(K, channels):
    """Label cache [B, Hkv, N, nlab] holding each KV head's label channels."""
    B, Hkv, N, d = K.shape
    return np.stack([K[:, g][:, :, channels[g]] for g in range(Hkv)], axis=1)


def test_label_scores_are_integer_exact():
    rng = np.random.default_rng(41)
    B, Hq, Hkv, N, d, nl = 2, 6, 3, 19, 16, 4
    q = rng.integers(-4, 5, (B, Hq, d)).astype(np.float32)
    K = rng.integers(-4, 5, (B, Hkv, N, d)).astype(np.float32)
    ch = np.stack([rng.choice(d, nl, replace=False) for _ in range(Hkv)]).astype(np.int32)
    lab = rng.integers(-4, 5, (B, Hkv, N, nl)).astype(np.float32)   # independent of K
    p = problem(q, K, K, Hkv=Hkv)
    got = O.label_scores(p, lab, ch)
    G = Hq // Hkv
    qi, li = q.astype(np.int64), lab.astype(np.int64)
    for b in range(B):
        for h in range(Hq):
            g = h // G
            want = li[b, g] @ qi[b, h, ch[g]]
            np.testing.assert_array_equal(got[b, h], want.astype(np.float64))
    # Group-shared rows sum their heads; permuting label columns together
    # with their channels changes nothing.
    pg = problem(q, K, K, Hkv=Hkv, group_shared=True)
    gs = O.label_scores(pg, lab, ch)
    for b in range(B):
        for g in range(Hkv):
            np.testing.assert_array_equal(gs[b, g], got[b, g * G:(g + 1) * G].sum(axis=0))
    perm = rng.permutation(nl)
    np.testing.assert_array_equal(O.label_scores(p, lab[..., perm], ch[:, perm]), got)


def test_label_indexer_with_the_channels_q_uses_is_the_exact_method():
    # When q is zero outside the label channels and the labels are those
    # channels of K, the approximate scores are the exact ones: the same
    # sets and outputs as the exact method (channels ascending keep the
    # summation order, so bit for bit).
    rng = np.random.default_rng(42)
    B, Hq, Hkv, N, d, nl = 2, 4, 2, 64, 32, 8
    ch = np.stack([np.sort(rng.choice(d, nl, replace=False)) for _ in range(Hkv)]).astype(np.int32)
    q = rng.standard_normal((B, Hq, d)).astype(np.float32)
    G = Hq // Hkv
    for h in range(Hq):
        mask = np.zeros(d, bool)
        mask[ch[h // G]] = True
        q[:, h, ~mask] = 0.0
    K = rng.standard_normal((B, Hkv, N, d)).astype(np.float32)
    V = rng.standard_normal((B, Hkv, N, d)).astype(np.float32)
    p = problem(q, K, V, Hkv=Hkv, ratio=8.0, seq_lens=[64, 37])
    lab = _labels_from(K, ch)
    np.testing.assert_array_equal(O.label_scores(p, lab, ch), O.scores(p))
    a, e = O.label_attention(p, lab, ch), O.sparse_attention(p)
    np.testing.assert_array_equal(a["idx"], e["idx"])
    np.testing.assert_array_equal(a["out"], e["out"])


def test_label_indexer_selects_on_labels_and_attends_on_full_keys():
    rng = np.random.default_rng(43)
    B, Hq, Hkv, N, d, nl = 1, 2, 1, 40, 16, 2
    q = rng.standard_normal((B, Hq, d)).astype(np.float32)
    K = rng.standard_normal((B, Hkv, N, d)).astype(np.float32)
    V = rng.standard_normal((B, Hkv, N, d)).astype(np.float32)
    ch = np.array([[3, 11]], np.int32)
    lab = rng.standard_normal((B, Hkv, N, nl)).astype(np.float32)
    p = problem(q, K, V, Hkv=Hkv, ratio=8.0)                    # k = 5
    r = O.label_attention(p, lab, ch)
    ls = O.label_scores(p, lab, ch)
    for h in range(Hq):
        want, tau = O.select_row(ls[0, h], 5)
        np.testing.assert_array_equal(r["idx"][0, h], want)     # chosen by label scores
        assert r["tau"][0, h] == tau
    out, _ = O.attend(p, r["idx"])                              # attended with full K, V
    np.testing.assert_array_equal(r["out"], out)
    # The paged layout gives the same result; forced positions apply too.
    pp = to_paged(p, 4, seed=1)
    lab_p = np.full((pp.k.shape[0], 4, Hkv, nl), 99.0, np.float32)
    for j in range(N):
        page = pp.block_table[0, j // 4]
        lab_p[page, j % 4] = lab[0, :, j]
    np.testing.assert_array_equal(O.label_attention(pp, lab_p, ch)["idx"], r["idx"])
    p.n_sink, p.n_local = 2, 3
    f = O.label_attention(p, lab, ch)
    for h in range(Hq):
        want, _ = O.select_forced(ls[0, h], 2, 3, 5)
        np.testing.assert_array_equal(f["idx"][0, h], want)


# --------------------------------------------------------------------------
# Attention: dense limit, special cases, invariants.
# --------------------------------------------------------------------------

def test_k_equals_L_is_dense_sdpa():
    rng = np.random.default_rng(4)
    B, Hq, Hkv, N, d = 2, 4, 2, 23, 32
    q = rng.standard_normal((B, Hq, d)).astype(np.float32)
    K = rng.standard_normal((B, Hkv, N, d)).astype(np.float32)
    V = rng.standard_normal((B, Hkv, N, d)).astype(np.float32)
    p = problem(q, K, V, Hkv=Hkv, ratio=1.0)
    r = O.sparse_attention(p)
    assert (r["idx"] == np.arange(N)).all()
    G = Hq // Hkv
    kt = torch.from_numpy(K.astype(np.float64)).repeat_interleave(G, dim=1)
    vt = torch.from_numpy(V.astype(np.float64)).repeat_interleave(G, dim=1)
    qt = torch.from_numpy(q.astype(np.float64))[:, :, None, :]
    ref = torch.nn.functional.scaled_dot_product_attention(qt, kt, vt)[:, :, 0, :].numpy()
    np.testing.assert_allclose(r["out"], ref, rtol=0, atol=1e-12)


def test_k_one_returns_the_argmax_value_row():
    rng = np.random.default_rng(5)
    N, d = 50, 8
    q = rng.standard_normal((1, d))
    K = rng.standard_normal((N, d))
    V = rng.standard_normal((N, d))
    p = problem(q, K, V, ratio=float(N))                 # k = 1
    r = O.sparse_attention(p)
    j = int(np.argmax(K.astype(np.float32).astype(np.float64) @ q[0].astype(np.float32)))
    assert list(r["idx"][0, 0]) == [j] + [-1] * (r["idx"].shape[2] - 1)
    np.testing.assert_array_equal(r["out"][0, 0], V.astype(np.float32)[j].astype(np.float64))


def test_equal_logits_give_the_mean_of_selected_values():
    rng = np.random.default_rng(6)
    N, d = 12, 8
    q = np.zeros((1, d)); q[0, 0] = 1.0
    K = np.zeros((N, d)); K[:, 0] = 3.0                  # every score equal
    V = rng.standard_normal((N, d))
    r = O.sparse_attention(problem(q, K, V, ratio=3.0))  # k = 4: positions 0..3
    assert list(r["idx"][0, 0][:4]) == [0, 1, 2, 3]
    np.testing.assert_allclose(r["out"][0, 0], V.astype(np.float32)[:4].astype(np.float64).mean(0),
                               rtol=0, atol=1e-15)


def test_softmax_weights_sum_to_one_and_output_in_hull():
    rng = np.random.default_rng(7)
    B, Hq, Hkv, N, d = 2, 4, 2, 40, 16
    q = rng.standard_normal((B, Hq, d)) * 2
    K = rng.standard_normal((B, Hkv, N, d))
    p1 = problem(q, K, np.ones((B, Hkv, N, d)), Hkv=Hkv, ratio=4.0)
    r1 = O.sparse_attention(p1)
    np.testing.assert_allclose(r1["out"], 1.0, rtol=0, atol=1e-14)   # sum of weights = 1
    V = rng.standard_normal((B, Hkv, N, d)).astype(np.float32)
    p2 = problem(q, K, V, Hkv=Hkv, ratio=4.0)
    r2 = O.sparse_attention(p2)
    G = Hq // Hkv
    for b in range(B):
        for h in range(Hq):
            S = [j for j in r2["idx"][b, h] if j >= 0]
            rows = V[b, h // G, S].astype(np.float64)
            assert (r2["out"][b, h] >= rows.min(0) - 1e-12).all()
            assert (r2["out"][b, h] <= rows.max(0) + 1e-12).all()
            assert (r2["absw"][b, h] >= np.abs(r2["out"][b, h]) - 1e-12).all()


# --------------------------------------------------------------------------
# Weighted attention over given sets (Section 4: the sparse backend attends
# given the index set and associated weights; reading: w_j proportional to
# omega_j exp(z_j)).  Pinned to a library routine: scaled dot-product
# attention with the additive mask log(omega).
# --------------------------------------------------------------------------

def _random_sets(rng, B, R, N, k):
    idx = np.stack([np.stack([np.sort(rng.choice(N, size=k, replace=False)) for _ in range(R)])
                    for _ in range(B)]).astype(np.int32)
    return idx


def test_weighted_attention_is_sdpa_with_log_weight_mask():
    rng = np.random.default_rng(21)
    B, Hq, Hkv, N, d, k = 2, 4, 2, 40, 16, 9
    q = rng.standard_normal((B, Hq, d)).astype(np.float32)
    K = rng.standard_normal((B, Hkv, N, d)).astype(np.float32)
    V = rng.standard_normal((B, Hkv, N, d)).astype(np.float32)
    p = problem(q, K, V, Hkv=Hkv)
    idx = _random_sets(rng, B, Hq, N, k)
    w = rng.uniform(0.05, 3.0, size=idx.shape).astype(np.float32)
    out, _ = O.attend_weighted(p, idx, w)
    G = Hq // Hkv
    for b in range(B):
        for h in range(Hq):
            S = idx[b, h]
            kt = torch.from_numpy(K[b, h // G, S].astype(np.float64))[None, None]
            vt = torch.from_numpy(V[b, h // G, S].astype(np.float64))[None, None]
            qt = torch.from_numpy(q[b, h].astype(np.float64))[None, None, None]
            mask = torch.from_numpy(np.log(w[b, h].astype(np.float64)))[None, None, None]
            ref = torch.nn.functional.scaled_dot_product_attention(qt, kt, vt, attn_mask=mask)
            np.testing.assert_allclose(out[b, h], ref[0, 0, 0].numpy(), rtol=0, atol=1e-12)


def test_weighted_attention_special_cases():
    rng = np.random.default_rng(22)
    B, Hq, N, d, k = 1, 3, 30, 8, 6
    q = rng.standard_normal((B, Hq, d)).astype(np.float32)
    K = rng.standard_normal((N, d)).astype(np.float32)
    V = rng.standard_normal((N, d)).astype(np.float32)
    p = problem(q, np.broadcast_to(K, (1, 1, N, d)), np.broadcast_to(V, (1, 1, N, d)))
    idx = _random_sets(rng, B, Hq, N, k)
    plain, _ = O.attend(p, idx)
    ones, _ = O.attend_weighted(p, idx, np.ones(idx.shape, np.float32))
    np.testing.assert_array_equal(ones, plain)                       # weights 1: unweighted
    const, _ = O.attend_weighted(p, idx, np.full(idx.shape, 7.5, np.float32))
    np.testing.assert_allclose(const, plain, rtol=0, atol=1e-13)     # scale invariant
    hot = np.zeros(idx.shape, np.float32)
    hot[..., 2] = 1.0                                                # one position kept
    one, _ = O.attend_weighted(p, idx, hot)
    for h in range(Hq):
        np.testing.assert_array_equal(one[0, h], V[idx[0, h, 2]].astype(np.float64))
    zero, _ = O.attend_weighted(p, idx, np.zeros(idx.shape, np.float32))
    assert (zero == 0).all()                                         # no weight: zero output
    with pytest.raises(RuntimeError):
        O.attend_weighted(p, idx, -hot)                              # negative weights rejected


def test_dense_attention_is_plain_sdpa_over_each_sequence():
    rng = np.random.default_rng(23)
    B, Hq, Hkv, N, d = 3, 6, 2, 37, 16
    q = rng.standard_normal((B, Hq, d)).astype(np.float32)
    K = rng.standard_normal((B, Hkv, N, d)).astype(np.float32)
    V = rng.standard_normal((B, Hkv, N, d)).astype(np.float32)
    lens = [37, 0, 5]
    p = problem(q, K, V, seq_lens=lens, Hkv=Hkv)
    out = O.dense_attention(p)
    G = Hq // Hkv
    for b in range(B):
        for h in range(Hq):
            L = lens[b]
            if L == 0:
                assert (out[b, h] == 0).all()
                continue
            kt = torch.from_numpy(K[b, h // G, :L].astype(np.float64))[None, None]
            vt = torch.from_numpy(V[b, h // G, :L].astype(np.float64))[None, None]
            qt = torch.from_numpy(q[b, h].astype(np.float64))[None, None, None]
            ref = torch.nn.functional.scaled_dot_product_attention(qt, kt, vt)
            np.testing.assert_allclose(out[b, h], ref[0, 0, 0].numpy(), rtol=0, atol=1e-12)
    # The same step in the paged layout, and a subset of the batch.
    pp = to_paged(p, 4, seed=3)
    np.testing.assert_array_equal(O.dense_attention(pp), out)
    part = O.dense_attention(p, batch=[2])
    np.testing.assert_array_equal(part[2], out[2])
    assert np.isnan(part[0]).all()


def test_empty_sequence_gives_zero_output_and_no_indices():
    rng = np.random.default_rng(8)
    q = rng.standard_normal((2, 2, 8))
    K = rng.standard_normal((2, 1, 10, 8))
    p = problem(q, K, K, seq_lens=[0, 10], ratio=5.0)
    r = O.sparse_attention(p)
    assert (r["idx"][0] == -1).all() and (r["out"][0] == 0).all()
    assert math.isnan(r["tau"][0, 0])
    assert (r["idx"][1, :, :2] >= 0).all()


def test_selection_uses_raw_scores_and_scale_only_in_softmax():
    # A larger softmax scale sharpens the weights but never changes the set.
    rng = np.random.default_rng(9)
    q = rng.standard_normal((1, 16)); K = rng.standard_normal((64, 16)); V = rng.standard_normal((64, 16))
    p = problem(q, K, V, ratio=8.0)
    a = O.sparse_attention(p, scale=0.01)
    b = O.sparse_attention(p, scale=10.0)
    np.testing.assert_array_equal(a["idx"], b["idx"])
    assert not np.allclose(a["out"], b["out"])


def test_gqa_head_mapping_consecutive_heads_share_a_kv_head():
    # Head h must read KV head h // G: give each KV head a distinct constant V.
    rng = np.random.default_rng(10)
    B, Hq, Hkv, N, d = 1, 6, 3, 10, 4
    q = rng.standard_normal((B, Hq, d))
    K = rng.standard_normal((B, Hkv, N, d))
    V = np.stack([np.full((N, d), float(g + 1)) for g in range(Hkv)])[None]
    r = O.sparse_attention(problem(q, K, V, Hkv=Hkv, ratio=2.0))
    for h in range(Hq):
        np.testing.assert_allclose(r["out"][0, h], h // 2 + 1.0, rtol=0, atol=1e-14)


# --------------------------------------------------------------------------
# Paged layout: any physical page order gives the same result.
# --------------------------------------------------------------------------

def test_paged_layout_equals_contiguous():
    rng = np.random.default_rng(11)
    B, Hq, Hkv, N, d = 3, 4, 2, 45, 8
    q = rng.standard_normal((B, Hq, d))
    K = rng.standard_normal((B, Hkv, N, d))
    V = rng.standard_normal((B, Hkv, N, d))
    p = problem(q, K, V, seq_lens=[45, 17, 1], Hkv=Hkv, ratio=3.0)
    a = O.sparse_attention(p)
    for ps, seed in ((4, 0), (16, 1), (1, 2)):
        pp = to_paged(p, ps, seed)
        b = O.sparse_attention(pp, k_max=a["idx"].shape[2])
        np.testing.assert_array_equal(a["idx"], b["idx"])
        np.testing.assert_array_equal(a["out"], b["out"])


# --------------------------------------------------------------------------
# Hand-worked examples (tests/golden/hand_examples.json).
# --------------------------------------------------------------------------

@pytest.mark.parametrize("name", ["per_head_tie_at_cut", "gqa_per_head_sets", "gqa_group_shared"])
def test_hand_worked_examples(name):
    ex = json.load(open(GOLDEN))[name]
    q = np.array(ex["q"], np.float32)[None]
    K = np.array(ex["k"], np.float32)[None, None]
    V = np.array(ex["v"], np.float32)[None, None]
    p = problem(q, K, V, ratio=ex["ratio"], rounding=ex["rounding"],
                group_shared=ex["group_shared"])
    r = O.sparse_attention(p)
    k = len(ex["expect_idx"][0])
    np.testing.assert_array_equal(r["idx"][0, :, :k], np.array(ex["expect_idx"]))
    np.testing.assert_array_equal(r["tau"][0], np.array(ex["expect_tau"]))
    e = math.e
    closed = np.array([[eval(t, {"e": e}) for t in row] for row in ex["expect_out"]], float)
    np.testing.assert_allclose(closed, ex["expect_out_values"], rtol=0, atol=1e-15)
    np.testing.assert_allclose(r["out"][0], closed, rtol=0, atol=1e-15)
    # The same example through the paged layout.
    b = O.sparse_attention(to_paged(p, 2, 3), k_max=r["idx"].shape[2])
    np.testing.assert_array_equal(b["out"], r["out"])


def test_stage_functions_compose_to_the_fused_oracle():
    rng = np.random.default_rng(12)
    B, Hq, Hkv, N, d = 2, 4, 2, 33, 8
    q = rng.standard_normal((B, Hq, d)); K = rng.standard_normal((B, Hkv, N, d))
    V = rng.standard_normal((B, Hkv, N, d))
    for gs in (False, True):
        p = problem(q, K, V, seq_lens=[33, 20], Hkv=Hkv, ratio=4.0, group_shared=gs)
        fused = O.sparse_attention(p)
        s = O.scores(p)
        kmax = fused["idx"].shape[2]
        # Scores of these float32 inputs at d = 8 are exact in float32 too? Not in
        # general, so select on the float64 rows directly.
        for b in range(B):
            for r in range(p.rows):
                L = p.seq_lens[b]
                idx, tau = O.select_row(s[b, r, :L], O.budget(L, 4.0), kmax)
                np.testing.assert_array_equal(idx, fused["idx"][b, r])
                assert tau == fused["tau"][b, r]
        out, _ = O.attend(p, fused["idx"])
        np.testing.assert_array_equal(out, fused["out"])


# ---------------------------------------------------------------------------
# Sampled selection (the stochastic index selection reading): pinned to dense
# attention, which the oracle computes separately over every position.
# ---------------------------------------------------------------------------

def _enumerating_draws(c: int, rows: int) -> np.ndarray:
    """Draws whose ranks are 0, 1, ..., c-1: draw i = ceil(i 2^32 / c)."""
    i = np.arange(c, dtype=np.uint64)
    d = ((i << np.uint64(32)) + np.uint64(c - 1)) // np.uint64(c)
    return np.broadcast_to(d.astype(np.uint32), (1, rows, c)).copy()


def test_sampled_selection_enumerating_the_rest_is_dense_attention():
    # s = |C| draws of ranks 0..|C|-1 list every position outside the top-k
    # once, with weight |C| / s = 1: the attention is dense attention.
    inp = synth.make_inputs(2, seed=3, B=1, N=2000, Hq=8, Hkv=2)
    k = O.budget(2000, inp.ratio, inp.rounding)
    r = O.sampled_attention(inp, _enumerating_draws(2000 - k, inp.rows))
    for row in range(inp.rows):
        got = np.sort(r["idx"][0, row][r["idx"][0, row] >= 0])
        np.testing.assert_array_equal(got, np.arange(2000))
    assert (r["weights"][0][r["idx"][0] >= 0] == 1.0).all()
    dense = O.dense_attention(inp)
    np.testing.assert_allclose(r["out"], dense, rtol=0, atol=1e-12)


def test_sampled_selection_enumerating_the_rest_twice_is_dense_attention():
    # s = 2 |C| draws listing every position outside the top-k twice, each
    # with weight |C| / s = 1/2: again exactly dense attention (a weight of 1,
    # or s / |C|, would count the rest twice or four times).
    inp = synth.make_inputs(2, seed=7, B=1, N=900, Hq=4, Hkv=1, ratio=10.0)
    c = 900 - O.budget(900, inp.ratio, inp.rounding)
    d = _enumerating_draws(c, inp.rows)
    r = O.sampled_attention(inp, np.concatenate([d, d], axis=2), scale=1.0)
    assert (r["weights"][0][:, -2 * c:] == np.float32(0.5)).all()
    np.testing.assert_allclose(r["out"], O.dense_attention(inp, scale=1.0), rtol=0, atol=1e-12)


def test_sampled_selection_converges_to_dense_attention():
    # Many random draws with weight |C| / s: the weighted sums over the draws
    # estimate the sums over the rest without bias, so the output nears dense
    # attention, while the top-k part alone stays far from it (softmax scale
    # 1, so the attention is peaked enough to tell weights apart: with a
    # weight of 1 or s / |C| the error is as large as the top-k part's).
    inp = synth.make_inputs(2, seed=4, B=1, N=1500, Hq=4, Hkv=1, ratio=20.0)
    rng = np.random.default_rng(5)
    draws = rng.integers(0, 2**32, size=(1, inp.rows, 60000), dtype=np.uint64).astype(np.uint32)
    r = O.sampled_attention(inp, draws, scale=1.0)
    dense = O.dense_attention(inp, scale=1.0)
    topk_only = O.sparse_attention(inp, scale=1.0)["out"]
    err_s = np.abs(r["out"] - dense).max()
    err_k = np.abs(topk_only - dense).max()
    assert err_s < 0.05 * err_k, (err_s, err_k)


def test_sampled_selection_zero_draws_pick_the_first_position_outside_the_set():
    inp = synth.make_inputs(2, seed=6, B=1, N=700, Hq=4, Hkv=1, ratio=10.0)
    r = O.sampled_attention(inp, np.zeros((1, inp.rows, 5), np.uint32))
    for row in range(inp.rows):
        kept = r["topk_idx"][0, row][r["topk_idx"][0, row] >= 0]
        first = min(set(range(700)) - set(kept.tolist()))
        n = len(kept)
        assert (r["idx"][0, row, n:n + 5] == first).all()
        assert r["weights"][0, row, n] == np.float32(700 - n) / np.float32(5)
