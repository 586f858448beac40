"""Parity of the HIP path (through the C ABI) with the CPU oracle.

Sizes here let the oracle finish in seconds while spanning several scoring
workgroups (8192 keys each), several 16-key tiles and a ragged tail; the
full-size workloads are checked on sampled sequences at the end.
"""
import dataclasses

import numpy as np
import pytest
import torch

from oracle import oracle as O
from paper_2605_24168_amd import synth
from tests import parity as P

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def sd():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2605_24168_amd import sparse_decode
    sparse_decode.set_debug(0)
    return sparse_decode


# Small versions of the five workloads (same structure, oracle-sized).
SMALL = {
    "w1": dict(cfg=1),
    "w2": dict(cfg=2, B=2, N=20007),
    "w3": dict(cfg=3, B=2, N=24003),
    "w4": dict(cfg=4, B=5, lmin=1000, lmax=30000, N=30000),
    "w5": dict(cfg=5, N=65536 + 77),
}


def make(name, seed=0, **over):
    kw = dict(SMALL[name])
    cfg = kw.pop("cfg")
    kw.update(over)
    return synth.make_inputs(cfg, seed=seed, **kw)


def gpu_fused(sd, inp, **sp_kw):
    q, cache, lens = sd.cache_from_inputs(inp)
    sp = sd.sparsity_from_inputs(inp, **sp_kw)
    out, idx = sd.sparse_decode_attention(q, cache, lens, sp, k_max=O.k_max_for(inp))
    torch.cuda.synchronize()
    return P.to_host(out), idx.cpu().numpy(), (q, cache, lens, sp)


def check_fused(inp, gpu_out, gpu_idx, ora=None, ora_scores=None, rows=None, label=""):
    ora = ora or O.sparse_attention(inp)
    if ora_scores is None:
        ora_scores = O.scores(inp)
    ks = P.budgets(inp)
    rep = P.check_idx_rows(gpu_idx, ora["idx"], ora_scores, ora["tau"], inp.seq_lens, ks, rows)
    assert rep.strict_mismatch_rows == 0, f"{label}: {rep.first_failure}"
    ref = ora["out"]
    if rep.band_swaps:
        ref, _ = O.attend(inp, gpu_idx)
    ok, ratio, rel = P.out_errors(gpu_out, ref, inp.dtype)
    P.log(f"  {label}: rows={rep.rows} band_swaps={rep.band_swaps} out worst/allow={ratio:.3g} "
          f"relL2={rel:.2e}")
    assert ok, f"{label}: output error {ratio:.3g} x allowance"
    return rep


# ---------------------------------------------------------------------------
# Stage parity.
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("name", list(SMALL))
def test_stage_scores_within_float32_bound(sd, name):
    inp = make(name)
    q, cache, lens = sd.cache_from_inputs(inp)
    sp = sd.sparsity_from_inputs(inp)
    s = sd.sparse_decode_score(q, cache, lens, sp).cpu().numpy()
    ref = O.scores(inp)
    qf = synth.bf16_to_f32(inp.q) if inp.dtype == "bf16" else inp.q
    G = inp.G
    worst = 0.0
    for b in range(inp.B):
        L = int(inp.seq_lens[b])
        assert np.isneginf(s[b, :, L:]).all()
        # Logical key rows of this sequence (contiguous or through the page table).
        if inp.layout == "paged":
            pages = inp.block_table[b, :-(-L // 16)]
            kk = inp.k[pages].reshape(-1, inp.Hkv, 128)[:L].transpose(1, 0, 2)
        else:
            kk = inp.k[b, :, :L]
        kf = synth.bf16_to_f32(kk) if inp.dtype == "bf16" else kk
        for r in range(inp.rows):
            if inp.group_shared:
                allow = sum(P.score_allowance(qf[b, h], kf[r]) for h in range(r * G, (r + 1) * G))
                allow = allow * 2  # plus the float32 sum over the group's heads
            else:
                allow = P.score_allowance(qf[b, r], kf[r // G])
            err = np.abs(s[b, r, :L].astype(np.float64) - ref[b, r, :L])
            worst = max(worst, float((err / allow).max()))
    P.log(f"  {name}: worst score error / bound = {worst:.3g}")
    assert worst <= 1.0


@pytest.mark.parametrize("name", list(SMALL))
def test_stage_topk_bit_exact_on_identical_scores(sd, name):
    inp = make(name)
    q, cache, lens = sd.cache_from_inputs(inp)
    sp = sd.sparsity_from_inputs(inp)
    k_max = O.k_max_for(inp)
    scores = sd.sparse_decode_score(q, cache, lens, sp)
    idx, vals = sd.sparse_decode_topk(scores, lens, sp, k_max=k_max, with_vals=True)
    s_host = scores.cpu().numpy()
    ora_idx, _ = O.select_f32(s_host, inp.seq_lens, inp.ratio, inp.rounding, k_max)
    np.testing.assert_array_equal(idx.cpu().numpy(), ora_idx)
    v = vals.cpu().numpy()
    for b in range(inp.B):
        for r in range(inp.rows):
            sel = ora_idx[b, r][ora_idx[b, r] >= 0]
            np.testing.assert_array_equal(v[b, r, :len(sel)], s_host[b, r, sel])
            assert np.isneginf(v[b, r, len(sel):]).all()


def test_stage_topk_ties_go_to_the_lower_position(sd):
    # Rows of many exactly equal scores: the selection must keep the lowest
    # positions among the tied ones, bit-exactly like the oracle.
    rng = np.random.default_rng(5)
    B, R, N = 3, 4, 5000
    s = np.round(rng.standard_normal((B, R, N)), 1).astype(np.float32)  # ~60 distinct values
    s[1] = 0.5
    s[2, :, ::2] = -0.0
    s[2, :, 1::2] = 0.0
    lens = np.array([5000, 4999, 4097], np.int32)
    sp = sd.Sparsity(ratio=7.0)
    k_max = O.budget(N, 7.0)
    idx = sd.sparse_decode_topk(torch.from_numpy(s).cuda(), torch.from_numpy(lens).cuda(), sp,
                                k_max=k_max).cpu().numpy()
    ora, _ = O.select_f32(s, lens, 7.0, 0, k_max)
    np.testing.assert_array_equal(idx, ora)


@pytest.mark.parametrize("name", list(SMALL))
def test_stage_attend_on_oracle_sets(sd, name):
    inp = make(name)
    ora = O.sparse_attention(inp)
    q, cache, lens = sd.cache_from_inputs(inp)
    sp = sd.sparsity_from_inputs(inp)
    out = sd.sparse_decode_attend(q, cache, lens, torch.from_numpy(ora["idx"]).cuda(), sp)
    ok, ratio, rel = P.out_errors(P.to_host(out), ora["out"], inp.dtype)
    P.log(f"  {name}: attend worst/allow={ratio:.3g} relL2={rel:.2e}")
    assert ok


# ---------------------------------------------------------------------------
# The fused path.
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("name", list(SMALL))
def test_fused_matches_oracle(sd, name):
    inp = make(name)
    out, idx, (q, cache, lens, sp) = gpu_fused(sd, inp)
    check_fused(inp, out, idx, label=name)
    # The fused selection equals score -> topk on the same float32 scores.
    scores = sd.sparse_decode_score(q, cache, lens, sp)
    idx2 = sd.sparse_decode_topk(scores, lens, sp, k_max=idx.shape[2]).cpu().numpy()
    np.testing.assert_array_equal(idx, idx2)


@pytest.mark.parametrize("name", list(SMALL))
def test_fused_exact_fallback_path_gives_identical_results(sd, name):
    inp = make(name, seed=3)
    out_a, idx_a, _ = gpu_fused(sd, inp)
    sd.set_debug(1)
    try:
        sd.set_profiling(True)
        out_b, idx_b, _ = gpu_fused(sd, inp)
        prof = sd.last_profile()
    finally:
        sd.set_debug(0)
        sd.set_profiling(False)
    rows_with_k = sum(inp.rows for L in inp.seq_lens if L > 0)
    assert prof["valid"] == 1 and prof["repaired_rows"] == rows_with_k
    np.testing.assert_array_equal(idx_a, idx_b)
    np.testing.assert_array_equal(out_a, out_b)


@pytest.mark.parametrize("debug", [0, 1])
def test_fused_ties_at_the_threshold_go_to_the_lower_position(sd, debug):
    # Keys repeat with period 50, so each head's scores take 50 values and
    # the k-th is shared by about 400 positions: both the candidate path and
    # the fallback (its selection cut into pieces over several workgroups,
    # whose tied keys straddle the pieces) must keep the lowest positions
    # among the tied ones, exactly as the oracle does.
    inp = make("w2", seed=12)
    period = np.arange(inp.ncap) % 50
    inp = dataclasses.replace(inp, k=np.ascontiguousarray(inp.k[:, :, period]),
                              v=np.ascontiguousarray(inp.v[:, :, period]))
    sd.set_debug(debug)
    try:
        sd.set_profiling(True)
        out, idx, _ = gpu_fused(sd, inp)
        prof = sd.last_profile()
    finally:
        sd.set_debug(0)
        sd.set_profiling(False)
    if debug:
        assert prof["repaired_rows"] == inp.B * inp.rows
    ora = O.sparse_attention(inp)
    np.testing.assert_array_equal(idx, ora["idx"])
    ok, ratio, _ = P.out_errors(out, ora["out"], inp.dtype)
    assert ok, f"output error {ratio:.3g} x allowance"


def test_fused_crowded_k_th_bucket_takes_the_radix_passes(sd):
    # Twenty sampled keys far above the rest stretch the selection's first
    # histogram (its range runs up to the largest pilot sample), and 700
    # nearly equal keys above every other key hold the k-th largest (40
    # distinct bf16 values among them), so the k-th bucket holds hundreds of
    # keys and the selection falls back to radix passes over the key bits.
    inp = make("w5", seed=33)
    G = inp.Hq // inp.Hkv
    L = int(inp.seq_lens[0])
    qs = synth.bf16_to_f32(inp.q[0, :G]).astype(np.float64).sum(axis=0)
    u = qs / np.linalg.norm(qs)
    k = inp.k.copy()
    top = float((synth.bf16_to_f32(k[0, 0]).astype(np.float64) @ qs).max())
    sampled = (np.arange(100, 120) * L) // min(L, 2048)  # pilot sample positions
    far = (u * 4.0 * top / np.linalg.norm(qs)).astype(np.float32)
    k[0, 0, sampled] = synth.bf16_bits(np.repeat(far[None, :], len(sampled), axis=0))
    c = 1.5 * top / np.linalg.norm(qs) * (1.0 + 2e-3 * np.arange(700) / 700.0)
    k[0, 0, 30000:30700] = synth.bf16_bits((c[:, None] * u[None, :]).astype(np.float32))
    inp = dataclasses.replace(inp, k=k)
    out, idx, _ = gpu_fused(sd, inp)
    ora = O.sparse_attention(inp)
    np.testing.assert_array_equal(idx, ora["idx"])
    ok, ratio, _ = P.out_errors(out, ora["out"], inp.dtype)
    assert ok, f"output error {ratio:.3g} x allowance"
    k0 = int(P.budgets(inp)[0])
    assert set(idx[0, 0, :k0]) <= set(range(30000, 30700)) | set(sampled.tolist())


def test_fused_low_sparsity_takes_the_fallback_for_every_row(sd):
    # At 2x with 4 heads per KV head a scoring wave's expected candidates
    # would overfill the staging areas, so the call scores every row in full
    # and selects over several workgroups per row.
    inp = make("w2", seed=13, ratio=2.0)
    sd.set_profiling(True)
    try:
        out, idx, _ = gpu_fused(sd, inp)
        prof = sd.last_profile()
    finally:
        sd.set_profiling(False)
    assert prof["repaired_rows"] == inp.B * inp.rows
    check_fused(inp, out, idx, label="2x, every row on the fallback")


def test_fused_is_deterministic(sd):
    inp = make("w3", seed=4)
    a = gpu_fused(sd, inp)
    b = gpu_fused(sd, inp)
    np.testing.assert_array_equal(a[0], b[0])
    np.testing.assert_array_equal(a[1], b[1])


def test_paged_page_order_does_not_matter(sd):
    inp = make("w4", seed=5)
    out_a, idx_a, _ = gpu_fused(sd, inp)
    # Same logical cache with another physical page order.
    rng = np.random.default_rng(9)
    P_ = inp.k.shape[0]
    perm = rng.permutation(P_).astype(np.int32)          # old page p -> new page perm[p]
    k2 = np.empty_like(inp.k); v2 = np.empty_like(inp.v)
    k2[perm] = inp.k; v2[perm] = inp.v
    bt2 = np.where(inp.block_table >= 0, perm[np.maximum(inp.block_table, 0)], -1).astype(np.int32)
    inp2 = dataclasses.replace(inp, k=k2, v=v2, block_table=bt2)
    out_b, idx_b, _ = gpu_fused(sd, inp2)
    np.testing.assert_array_equal(idx_a, idx_b)
    np.testing.assert_array_equal(out_a, out_b)


def test_contiguous_and_paged_layouts_agree(sd):
    inp = make("w2", seed=6, B=3, N=5000)
    out_a, idx_a, _ = gpu_fused(sd, inp)
    # The same sequences laid out in pages of 16 (identity page order, padded).
    per = -(-inp.ncap // 16)
    kp = np.full((inp.B * per, 16, inp.Hkv, 128), synth.bf16_bits(np.float32([64.0]))[0], np.uint16)
    vp = kp.copy()
    for b in range(inp.B):
        for t in range(per):
            n = min(16, inp.ncap - 16 * t)
            kp[b * per + t, :n] = inp.k[b, :, 16 * t:16 * t + n].transpose(1, 0, 2)
            vp[b * per + t, :n] = inp.v[b, :, 16 * t:16 * t + n].transpose(1, 0, 2)
    bt = np.arange(inp.B * per, dtype=np.int32).reshape(inp.B, per)
    inp2 = dataclasses.replace(inp, k=kp, v=vp, layout="paged", block_table=bt, ncap=per * 16)
    out_b, idx_b, _ = gpu_fused(sd, inp2)
    np.testing.assert_array_equal(idx_a, idx_b[:, :, :idx_a.shape[2]])
    np.testing.assert_array_equal(out_a, out_b)


# ---------------------------------------------------------------------------
# Edge cases.
# ---------------------------------------------------------------------------

def test_ragged_contiguous_batch_with_empty_and_tiny_sequences(sd):
    # Lengths 0, 1, 15, 17, full tile multiples, ones at and across the
    # scoring-wave (2048) and scoring-workgroup (8192) boundaries, and a
    # capacity that is not a tile multiple; positions beyond each length
    # hold poison.
    inp = synth.make_inputs(2, seq_lens=[0, 1, 15, 17, 2047, 2048, 2049, 4096, 8191, 8192, 8193,
                                         12000], ncap=12011)
    out, idx, _ = gpu_fused(sd, inp)
    check_fused(inp, out, idx, label="ragged bhnd")
    assert (idx[0] == -1).all() and (out[0] == 0).all()


@pytest.mark.parametrize("ratio", [1.0, 2.0, 3.0, 1000.0])
def test_extreme_sparsity_ratios(sd, ratio):
    inp = make("w2", seed=7, B=2, N=3001, ratio=ratio)
    out, idx, _ = gpu_fused(sd, inp)
    check_fused(inp, out, idx, label=f"ratio {ratio}")


@pytest.mark.parametrize("Hq,Hkv", [(8, 8), (8, 1), (16, 1), (40, 8), (12, 4)])
def test_head_groupings(sd, Hq, Hkv):
    inp = make("w2", seed=8, B=2, N=9000, Hq=Hq, Hkv=Hkv)
    out, idx, _ = gpu_fused(sd, inp)
    check_fused(inp, out, idx, label=f"{Hq}q/{Hkv}kv")


@pytest.mark.parametrize("Hq,Hkv,shared", [(8, 1, False), (8, 2, False), (16, 4, False),
                                            (24, 12, False), (8, 2, True), (16, 4, True)])
def test_paged_head_counts(sd, Hq, Hkv, shared):
    # Paged caches are scored one KV head per wave, four heads per workgroup,
    # when Hkv is a multiple of 4, else one head per workgroup; both paths.
    inp = make("w4", seed=17, B=3, lmin=2000, lmax=20000, N=20000, Hq=Hq, Hkv=Hkv,
               group_shared=shared)
    out, idx, _ = gpu_fused(sd, inp)
    check_fused(inp, out, idx, label=f"paged {Hq}q/{Hkv}kv shared={shared}")


@pytest.mark.parametrize("G", [1, 4, 16])
def test_group_shared_mode_group_sizes(sd, G):
    inp = make("w5", seed=9, N=20000, Hq=2 * G, Hkv=2)
    out, idx, _ = gpu_fused(sd, inp)
    check_fused(inp, out, idx, label=f"group-shared G={G}")


@pytest.mark.parametrize("name,ratio", [("w3", 4.0), ("w2", 6.0), ("w5", 5.0), ("w4", 8.0)])
def test_long_candidate_lists(sd, name, ratio):
    # Low sparsity: hundreds of candidates per row and wave, so the scoring
    # waves shrink, and rows too dense for the staging areas are sent to the
    # exact fallback by the pilot.
    kw = {"w4": dict(B=2, lmin=6000, lmax=9000, N=9000)}.get(name, dict(B=1, N=12000))
    inp = make(name, seed=14, ratio=ratio, **kw)
    out, idx, _ = gpu_fused(sd, inp)
    check_fused(inp, out, idx, label=f"{name} ratio {ratio}")


@pytest.mark.parametrize("name,kw", [
    ("w3", dict(B=1, N=65536, Hq=8, Hkv=8, ratio=4.0)),
    ("w3", dict(B=2, N=65536, Hq=8, Hkv=8, ratio=3.0, seq_lens=[65536, 50001])),
    ("w5", dict(N=65536 + 77, ratio=4.0)),
])
def test_candidates_beyond_the_lds_select_from_global_scratch(sd, name, kw):
    # k of 12K-22K: the ~2.5 k candidates of a row exceed the ~36K keys a
    # selection workgroup stages in LDS, so a row that does not take the
    # exact fallback copies its candidates into its unused fallback score row
    # and selects there.
    inp = make(name, seed=21, **kw)
    sd.set_profiling(True)
    try:
        out, idx, _ = gpu_fused(sd, inp)
        prof = sd.last_profile()
    finally:
        sd.set_profiling(False)
    rows_with_k = sum(inp.rows for L in inp.seq_lens if L > 0)
    assert prof["repaired_rows"] < rows_with_k
    check_fused(inp, out, idx, label=f"{name} ratio {inp.ratio} from global scratch")


def test_clustered_candidates_overflow_to_the_exact_fallback(sd):
    # 400 consecutive keys close to head 0's query direction: with 8 heads
    # per group a row's staging area holds 128 keys per scoring wave (of at
    # least 256 keys), and the cluster puts more than that into one wave, so
    # the row must take the exact fallback.
    inp = make("w2", seed=15, B=1, N=12000, ratio=50.0, Hq=64, Hkv=8)
    rng = np.random.default_rng(15)
    q0 = synth.bf16_to_f32(inp.q[0, 0]).astype(np.float64)
    base = 3.0 * q0 / np.linalg.norm(q0) * np.sqrt(inp.d)
    clus = base[None, :] + 0.3 * rng.standard_normal((400, inp.d))
    k = inp.k.copy()
    k[0, 0, 100:500] = synth.bf16_bits(clus.astype(np.float32))
    inp = dataclasses.replace(inp, k=k)
    sd.set_profiling(True)
    out, idx, _ = gpu_fused(sd, inp)
    prof = sd.last_profile()
    sd.set_profiling(False)
    assert prof["repaired_rows"] >= 1
    check_fused(inp, out, idx, label="clustered overflow")
    k0 = int(P.budgets(inp)[0])
    assert set(idx[0, 0, :k0]) <= set(range(100, 500))


def test_profiling_levels(sd):
    # Level 1 times every stage; level 2 only the scoring kernel (events
    # attached to its dispatch).  Both leave the results unchanged, and level
    # 2 still works when no scoring kernel runs (every row forced to the
    # exact fallback).
    inp = make("w3", seed=16)
    q, cache, lens = sd.cache_from_inputs(inp)
    sp = sd.sparsity_from_inputs(inp)
    k_max = O.k_max_for(inp)
    out0, idx0 = sd.sparse_decode_attention(q, cache, lens, sp, k_max=k_max)
    profs = {}
    for level in (1, 2):
        sd.set_profiling(level)
        for _ in range(3):
            out, idx = sd.sparse_decode_attention(q, cache, lens, sp, k_max=k_max)
        torch.cuda.synchronize()
        sd.set_profiling(False)
        profs[level] = sd.profile_mean()
        assert torch.equal(out, out0) and torch.equal(idx, idx0)
    assert profs[1]["valid"] == 1 and profs[1]["calls"] == 3 and profs[1]["total_ms"] > 0
    assert profs[2]["valid"] == 1 and profs[2]["score_ms"] > 0 and profs[2]["total_ms"] == 0
    sd.set_debug(1)
    try:
        sd.set_profiling(2)
        out, idx = sd.sparse_decode_attention(q, cache, lens, sp, k_max=k_max)
        torch.cuda.synchronize()
        sd.set_profiling(False)
        prof = sd.profile_mean()
    finally:
        sd.set_debug(0)
    assert prof["valid"] == 1 and prof["score_ms"] >= 0
    assert torch.equal(out, out0) and torch.equal(idx, idx0)


def test_float32_gqa_and_paged(sd):
    inp = make("w4", seed=10, B=3, lmin=3000, lmax=9000, N=9000, dtype="f32")
    out, idx, _ = gpu_fused(sd, inp)
    check_fused(inp, out, idx, label="f32 paged")


def test_float32_rows_selected_in_pieces(sd):
    # float32 caches take the full-score path for every row; rows of 16K
    # positions and more are selected over several workgroups each.
    inp = make("w4", seed=14, B=3, lmin=16000, lmax=24000, N=24000, dtype="f32")
    out, idx, _ = gpu_fused(sd, inp)
    check_fused(inp, out, idx, label="f32 paged, pieces")


def test_k_override(sd):
    inp = make("w2", seed=11, B=4, N=3000)
    ko = np.array([0, 1, 3000, 77], np.int32)
    q, cache, lens = sd.cache_from_inputs(inp)
    sp = sd.sparsity_from_inputs(inp, k_override=torch.from_numpy(ko).cuda())
    out, idx = sd.sparse_decode_attention(q, cache, lens, sp, k_max=3000)
    torch.cuda.synchronize()
    ora = O.sparse_attention(inp, k_max=3000, k_override=ko)
    rep = P.check_idx_rows(idx.cpu().numpy(), ora["idx"], O.scores(inp), ora["tau"],
                           inp.seq_lens, ko)
    assert rep.strict_mismatch_rows == 0, rep.first_failure
    ok, ratio, _ = P.out_errors(P.to_host(out), ora["out"] if not rep.band_swaps
                                else O.attend(inp, idx.cpu().numpy())[0], "bf16")
    assert ok
    assert (idx.cpu().numpy()[0] == -1).all()


def test_fallback_pieces_at_extreme_budgets(sd):
    # Every row forced onto the fallback with rows long enough to be cut
    # into pieces: budgets of 0, 1, the whole row and one in between, so
    # that the kept positions sit in one piece, in all pieces, or in none.
    N = 20007
    inp = make("w2", seed=16, B=4, N=N)
    ko = np.array([0, 1, N, 4099], np.int32)
    q, cache, lens = sd.cache_from_inputs(inp)
    sp = sd.sparsity_from_inputs(inp, k_override=torch.from_numpy(ko).cuda())
    sd.set_debug(1)
    try:
        out, idx = sd.sparse_decode_attention(q, cache, lens, sp, k_max=N)
        torch.cuda.synchronize()
    finally:
        sd.set_debug(0)
    idx = idx.cpu().numpy()
    ora = O.sparse_attention(inp, k_max=N, k_override=ko)
    rep = P.check_idx_rows(idx, ora["idx"], O.scores(inp), ora["tau"], inp.seq_lens, ko)
    assert rep.strict_mismatch_rows == 0, rep.first_failure
    assert (idx[0] == -1).all()
    np.testing.assert_array_equal(idx[2], np.broadcast_to(np.arange(N), idx[2].shape))
    ok, ratio, _ = P.out_errors(P.to_host(out), ora["out"] if not rep.band_swaps
                                else O.attend(inp, idx)[0], "bf16")
    assert ok, f"{ratio:.3g} x allowance"


def test_workspace_from_caller(sd):
    inp = make("w2", seed=12, B=2, N=7000)
    q, cache, lens = sd.cache_from_inputs(inp)
    sp = sd.sparsity_from_inputs(inp)
    idx = torch.empty((inp.B, inp.rows, O.k_max_for(inp)), dtype=torch.int32, device="cuda")
    n = sd.workspace_size(q, cache, sp, idx)
    ws = torch.empty(n, dtype=torch.uint8, device="cuda")
    sd.set_workspace(ws)
    try:
        out, _ = sd.sparse_decode_attention(q, cache, lens, sp, idx=idx)
        torch.cuda.synchronize()
        sd.set_workspace(ws[: n // 2 // 256 * 256])
        with pytest.raises(sd.SparseDecodeError):
            sd.sparse_decode_attention(q, cache, lens, sp, idx=idx)
    finally:
        sd.set_workspace(None)
    check_fused(inp, P.to_host(out), idx.cpu().numpy(), label="caller workspace")


def test_invalid_arguments_are_rejected_before_launch(sd):
    inp = make("w2", seed=13, B=1, N=1000)
    q, cache, lens = sd.cache_from_inputs(inp)
    sp = sd.sparsity_from_inputs(inp)
    small_idx = torch.empty((1, inp.rows, 3), dtype=torch.int32, device="cuda")
    with pytest.raises(sd.SparseDecodeError) as e:
        sd.sparse_decode_attention(q, cache, lens, sp, idx=small_idx)
    assert e.value.status == sd.SD_ERR_INVALID_ARG
    bad_q = torch.zeros((1, inp.Hq, 64), dtype=torch.bfloat16, device="cuda")
    with pytest.raises(sd.SparseDecodeError) as e:
        sd.sparse_decode_attention(bad_q, cache, lens, sp)
    assert e.value.status == sd.SD_ERR_UNSUPPORTED


# ---------------------------------------------------------------------------
# Full-size workloads, as the benchmark runs them: every sequence of the
# 128K batch and of the ragged paged batch, a sampled one of the others.
# ---------------------------------------------------------------------------

slice_batch = P.slice_batch


@pytest.mark.parametrize("cfg,sample", [(1, [0]), (2, [1]), (3, list(range(16))),
                                        (4, list(range(32))), (5, [0])])
def test_full_size_workloads_on_sampled_sequences(sd, cfg, sample):
    P.log(f"  generating workload {cfg} at full size")
    inp = synth.make_inputs(cfg, seed=0)
    q, cache, lens = sd.cache_from_inputs(inp)
    sp = sd.sparsity_from_inputs(inp)
    sd.set_profiling(True)
    out, idx = sd.sparse_decode_attention(q, cache, lens, sp, k_max=O.k_max_for(inp))
    torch.cuda.synchronize()
    prof = sd.last_profile()
    sd.set_profiling(False)
    P.log(f"  workload {cfg}: stages {prof}")
    out_h, idx_h = P.to_host(out), idx.cpu().numpy()
    del q, cache, lens, out, idx
    torch.cuda.empty_cache()
    sub = slice_batch(inp, sample)
    P.log(f"  oracle on sequences {sample}")
    check_fused(sub, out_h[sample], idx_h[sample], label=f"full workload {cfg}")
    # Every row of every sequence: well-formed, and the budget respected.
    ks = P.budgets(inp)
    for b in range(inp.B):
        k = int(ks[b])
        row = idx_h[b]
        assert (row[:, k:] == -1).all() and (row[:, :k] >= 0).all()
        assert (row[:, :k] < inp.seq_lens[b]).all()
        assert (np.diff(row[:, :k], axis=1) > 0).all()


def test_read_probe_reads_buffers_of_any_length(sd):
    # The bandwidth reference the bench reports: any multiple of 16 bytes,
    # from one 16-byte word to more than the grid covers in one sweep.
    sink = torch.zeros(1, dtype=torch.int32, device="cuda")
    for n in (16, 16 * 255, 1 << 20, (64 << 20) + 48):
        buf = torch.zeros(n, dtype=torch.uint8, device="cuda")
        sd.read_probe(buf, sink)
    torch.cuda.synchronize()
    assert int(sink.item()) == 0   # zeros XOR to 0, never the store's value
