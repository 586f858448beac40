"""Parity of forced sink and local positions beside the exact top-k (the
scaffolding of the paper's long-context runs: Sink(128) + Local(128) +
OracleTopK with a heavy fraction; K retrieved tokens with 64 sinks) with
the CPU oracle, through the C ABI."""
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
    "w1": dict(cfg=1),
    "w2": dict(cfg=2, B=2, N=20007),
    "w3": dict(cfg=3, B=2, N=24003),
    "w4": dict(cfg=4, B=5, lmin=1000, lmax=30000, N=30000),
    "w5": dict(cfg=5, N=65536 + 77),
}


def make(name, n_sink, n_local, seed=0, **over):
    kw = dict(SMALL[name])
    cfg = kw.pop("cfg")
    kw.update(over)
    return synth.make_inputs(cfg, seed=seed, n_sink=n_sink, n_local=n_local, **kw)


def totals(inp, k_override=None):
    """Entries of each sequence's list: forced positions plus the heavy budget."""
    out = []
    for b, L in enumerate(inp.seq_lens):
        L = int(L)
        ns = min(inp.n_sink, L)
        nl = min(inp.n_local, L - ns)
        kh = (min(int(k_override[b]), L) if k_override is not None
              else O.budget(L, inp.ratio, inp.rounding))
        out.append(ns + nl + min(kh, L - ns - nl))
    return np.array(out, np.int64)


def run_fused(sd, inp, k_override=None):
    q, cache, lens = sd.cache_from_inputs(inp)
    ko = None if k_override is None else torch.tensor(k_override, dtype=torch.int32).cuda()
    sp = sd.sparsity_from_inputs(inp, k_override=ko)
    k_max = O.k_max_for(inp) if k_override is None else int(max(totals(inp, k_override)))
    out, idx = sd.sparse_decode_attention(q, cache, lens, sp, k_max=k_max)
    torch.cuda.synchronize()
    return P.to_host(out), idx.cpu().numpy()


def check(inp, out, idx, label, k_override=None):
    ko = None if k_override is None else np.asarray(k_override, np.int32)
    ora = O.sparse_attention(inp, k_max=idx.shape[2], k_override=ko)
    ks = totals(inp, k_override)
    rep = P.check_idx_rows(idx, ora["idx"], O.scores(inp), ora["tau"], inp.seq_lens, ks)
    assert rep.strict_mismatch_rows == 0, f"{label}: {rep.first_failure}"
    # Every forced position is listed in every row.
    for b, L in enumerate(inp.seq_lens):
        L = int(L)
        ns = min(inp.n_sink, L)
        nl = min(inp.n_local, L - ns)
        forced = set(range(ns)) | set(range(L - nl, L))
        for r in range(idx.shape[1]):
            assert forced <= set(idx[b, r, :ks[b]].tolist()), (label, b, r)
    ref = ora["out"] if rep.band_swaps == 0 else O.attend(inp, idx)[0]
    ok, ratio, rel = P.out_errors(out, ref, inp.dtype)
    P.log(f"  {label}: rows={rep.rows} band_swaps={rep.band_swaps} worst/allow={ratio:.3g} "
          f"relL2={rel:.2e}")
    assert ok, f"{label}: output error {ratio:.3g} x allowance"


@pytest.mark.parametrize("name", list(SMALL))
def test_sink_and_local_windows_match_oracle(sd, name):
    inp = make(name, 128, 128)
    out, idx = run_fused(sd, inp)
    check(inp, out, idx, f"{name} sink128+local128")


@pytest.mark.parametrize("ratio", [5.0, 50.0])
def test_heavy_fractions_of_the_swe_runs(sd, ratio):
    # Heavy fraction 0.20 and 0.02 of the context beside 128 + 128 forced.
    inp = make("w2", 128, 128, ratio=ratio)
    out, idx = run_fused(sd, inp)
    check(inp, out, idx, f"heavy 1/{ratio:g}")


@pytest.mark.parametrize("K", [1, 4, 16, 64, 128])
def test_fixed_k_with_64_sinks(sd, K):
    inp = make("w4", 64, 0)
    ko = [K] * inp.B
    out, idx = run_fused(sd, inp, k_override=ko)
    check(inp, out, idx, f"K={K} + 64 sinks", k_override=ko)


def test_forced_windows_at_low_sparsity(sd):
    # Heavy fraction 1/3 of 65K positions: the candidates of a row exceed
    # what a selection workgroup stages in LDS.
    inp = make("w3", 64, 200, B=2, N=65536, Hq=8, Hkv=8, ratio=3.0, seq_lens=[65536, 50001])
    out, idx = run_fused(sd, inp)
    check(inp, out, idx, "sink 64 + local 200, heavy 1/3")


def test_ragged_sequences_shorter_than_the_windows(sd):
    inp = make("w4", 100, 60, seq_lens=[0, 1, 50, 100, 160, 161, 300, 5000, 17001], N=17001)
    out, idx = run_fused(sd, inp)
    assert (idx[0] == -1).all() and (out[0] == 0).all()
    check(inp, out, idx, "short sequences")


def test_forced_rows_through_the_exact_fallback_are_identical(sd):
    inp = make("w3", 64, 32)
    a_out, a_idx = run_fused(sd, inp)
    sd.set_debug(1)
    try:
        b_out, b_idx = run_fused(sd, inp)
    finally:
        sd.set_debug(0)
    np.testing.assert_array_equal(a_idx, b_idx)
    np.testing.assert_array_equal(a_out, b_out)


def test_stage_topk_with_forced_positions_is_bit_exact(sd):
    inp = make("w4", 128, 128)
    q, cache, lens = sd.cache_from_inputs(inp)
    sp = sd.sparsity_from_inputs(inp)
    scores = sd.sparse_decode_score(q, cache, lens, sp)
    k_max = O.k_max_for(inp)
    idx, vals = sd.sparse_decode_topk(scores, lens, sp, k_max=k_max, with_vals=True)
    s_host = scores.cpu().numpy()
    ora, _ = O.select_f32(s_host, inp.seq_lens, inp.ratio, inp.rounding, k_max,
                          n_sink=128, n_local=128)
    gi = idx.cpu().numpy()
    np.testing.assert_array_equal(gi, ora)
    v = vals.cpu().numpy()
    for b in range(inp.B):
        for r in range(0, inp.rows, 7):
            n = int((gi[b, r] >= 0).sum())
            np.testing.assert_array_equal(v[b, r, :n], s_host[b, r, gi[b, r, :n]])


@pytest.mark.parametrize("Hq,Hkv,flags", [(32, 8, 0), (32, 2, 8), (16, 4, 8)])
def test_forced_windows_union_attention(sd, Hq, Hkv, flags):
    # Sink and local windows beside a heavy 1/3 (the cost rule picks the
    # group-deduplicated attention), or forced on (flag 8) at the workload's
    # sparsity; a 16-head group takes two passes over the heads.
    ratio = 3.0 if flags == 0 else None
    kw = dict(B=3, N=40000, Hq=Hq, Hkv=Hkv, seq_lens=[40000, 333, 25000])
    if ratio:
        kw["ratio"] = ratio
    inp = make("w4", 64, 200, **kw)
    sd.set_debug(flags)
    try:
        out, idx = run_fused(sd, inp)
    finally:
        sd.set_debug(0)
    check(inp, out, idx, f"union {Hq}/{Hkv} flags {flags}")
