"""Parity of the sampled selection (exact top-k plus importance-weighted
uniform draws of the rest of each row; the stochastic index selection of
Section 4, in the reading the oracle states) with the CPU oracle, through
the C ABI.  The random numbers are inputs: both sides get the same draws.
"""
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


SMALL = {
    "w2": dict(cfg=2, B=2, N=20007),
    "w3": dict(cfg=3, B=2, N=24003),
    "w4": dict(cfg=4, B=5, lmin=1000, lmax=30000, N=30000),
}


def make(name, seed=0, **over):
    kw = dict(SMALL[name])
    cfg = kw.pop("cfg")
    kw.update(over)
    return synth.make_inputs(cfg, seed=seed, **kw)


def random_draws(inp, s, seed):
    rng = np.random.default_rng(seed)
    return rng.integers(0, 2**32, size=(inp.B, inp.rows, s), dtype=np.uint64).astype(np.uint32)


def run(sd, inp, draws):
    q, cache, lens = sd.cache_from_inputs(inp)
    sp = sd.sparsity_from_inputs(inp)
    d = torch.from_numpy(draws.view(np.int32)).cuda()
    out, idx, w = sd.sparse_decode_sampled_attention(q, cache, lens, sp, d,
                                                     k_max=O.k_max_for(inp))
    torch.cuda.synchronize()
    return P.to_host(out), idx.cpu().numpy(), w.cpu().numpy()


def check(inp, draws, out, idx, w, label):
    ora = O.sampled_attention(inp, draws, k_max=O.k_max_for(inp))
    # The kept part: exact up to near-ties at the k-th score (the float32
    # scores may order them differently); the draws then follow the GPU's
    # own kept set, and the weights are exact.
    km = O.k_max_for(inp)
    kept = np.where(w == 1.0, idx, -1)
    top = np.full((inp.B, inp.rows, km), -1, np.int32)
    for b in range(inp.B):
        for r in range(inp.rows):
            k = kept[b, r][kept[b, r] >= 0]
            top[b, r, :len(k)] = k
    ks = []
    for L in inp.seq_lens:
        L = int(L)
        ns = min(inp.n_sink, L)
        nl = min(inp.n_local, L - ns)
        ks.append(ns + nl + min(O.budget(L, inp.ratio, inp.rounding), L - ns - nl))
    base = O.sparse_attention(inp, k_max=km)
    rep = P.check_idx_rows(top, base["idx"], O.scores(inp), base["tau"], inp.seq_lens,
                           np.array(ks))
    assert rep.strict_mismatch_rows == 0, f"{label}: {rep.first_failure}"
    ref_idx, ref_w = O.sampled_lists(top, inp.seq_lens, draws)
    np.testing.assert_array_equal(idx, ref_idx)
    np.testing.assert_array_equal(w, ref_w)
    ref, _ = O.attend_weighted(inp, ref_idx, ref_w)
    ok, ratio, rel = P.out_errors(out, ref, inp.dtype)
    P.log(f"  {label}: band_swaps={rep.band_swaps} worst/allow={ratio:.3g} relL2={rel:.2e}")
    assert ok, f"{label}: output error {ratio:.3g} x allowance"
    if rep.band_swaps == 0:
        np.testing.assert_array_equal(idx, ora["idx"])


@pytest.mark.parametrize("name,s", [("w2", 64), ("w3", 300), ("w4", 32)])
def test_sampled_matches_oracle(sd, name, s):
    inp = make(name, seed=1)
    draws = random_draws(inp, s, seed=2)
    out, idx, w = run(sd, inp, draws)
    check(inp, draws, out, idx, w, f"{name} s={s}")


def test_sampled_with_forced_windows_and_short_sequences(sd):
    # Sink/local windows join the kept set; sequences no longer than their
    # kept set draw nothing (weights 0, entries -1), an empty one gives 0.
    inp = make("w4", seed=3, n_sink=16, n_local=16, seq_lens=[0, 1, 20, 33, 5000, 30000],
               N=30000)
    draws = random_draws(inp, 40, seed=4)
    out, idx, w = run(sd, inp, draws)
    assert (idx[0] == -1).all() and (out[0] == 0).all()
    assert (w[1][:, 1:] == 0).all() and (idx[1][:, 1:] == -1).all()
    check(inp, draws, out, idx, w, "forced + short")


def test_sampled_enumerating_draws_give_dense_attention(sd):
    # Draws with ranks 0..|C|-1 list every position outside the top-k once
    # with weight 1: the GPU's output is dense attention.
    inp = make("w2", seed=5, B=1, N=4000)
    c = 4000 - O.budget(4000, inp.ratio, inp.rounding)
    i = np.arange(c, dtype=np.uint64)
    d = (((i << np.uint64(32)) + np.uint64(c - 1)) // np.uint64(c)).astype(np.uint32)
    draws = np.broadcast_to(d, (1, inp.rows, c)).copy()
    out, idx, w = run(sd, inp, draws)
    for r in range(inp.rows):
        np.testing.assert_array_equal(np.sort(idx[0, r][idx[0, r] >= 0]), np.arange(4000))
    assert (w[0][idx[0] >= 0] == 1.0).all()
    ok, ratio, rel = P.out_errors(out, O.dense_attention(inp), inp.dtype)
    P.log(f"  enumerating draws: worst/allow={ratio:.3g} relL2={rel:.2e}")
    assert ok


def test_sampled_without_draws_is_the_top_k_attention(sd):
    inp = make("w3", seed=6)
    out, idx, w = run(sd, inp, np.zeros((inp.B, inp.rows, 0), np.uint32))
    q, cache, lens = sd.cache_from_inputs(inp)
    sp = sd.sparsity_from_inputs(inp)
    out2, idx2 = sd.sparse_decode_attention(q, cache, lens, sp, k_max=O.k_max_for(inp))
    np.testing.assert_array_equal(idx, idx2.cpu().numpy())
    assert ((w == 1.0) == (idx >= 0)).all()
    ok, ratio, _ = P.out_errors(out, P.to_host(out2), inp.dtype)
    assert ok, f"{ratio:.3g} x allowance"


def test_sampled_at_low_sparsity_through_the_fallback(sd):
    # At 2x with 4 heads per KV head every row takes the exact fallback, its
    # selection cut into pieces over several workgroups, with the draws'
    # slots after each kept list.
    inp = make("w2", seed=7, ratio=2.0)
    draws = random_draws(inp, 96, seed=8)
    out, idx, w = run(sd, inp, draws)
    check(inp, draws, out, idx, w, "sampled 2x")


def test_sampled_full_size_on_sampled_sequences(sd):
    # Workload 3 at full size with the bench's first sampled line (top-k
    # 1/200 plus 1311 draws per row), two sequences checked by the oracle.
    P.log("  generating workload 3 at full size")
    inp = synth.make_inputs(3, seed=0, ratio=200.0)
    draws = random_draws(inp, 1311, seed=9)
    out, idx, w = run(sd, inp, draws)
    sample = [0, 15]
    check(P.slice_batch(inp, sample), draws[sample], out[sample], idx[sample], w[sample],
          "sampled full workload 3")


def test_sampled_selection_with_the_exact_part_in_pieces(sd):
    # Few rows: the exact part selected over several workgroups per row
    # (debug flag 32) gives the lists, weights and output of one workgroup
    # per row (flag 16) bit for bit, and the oracle's.
    inp = make("w2", seed=9)
    draws = random_draws(inp, 64, seed=9)
    sd.set_debug(32)
    try:
        out, idx, w = run(sd, inp, draws)
    finally:
        sd.set_debug(0)
    sd.set_debug(16)
    try:
        out2, idx2, w2 = run(sd, inp, draws)
    finally:
        sd.set_debug(0)
    np.testing.assert_array_equal(idx, idx2)
    np.testing.assert_array_equal(w, w2)
    np.testing.assert_array_equal(out, out2)
    check(inp, draws, out, idx, w, "sampled, exact part in pieces")
