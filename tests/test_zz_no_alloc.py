"""The allocation-free fused call (sparse_decode_attention_noalloc) against
the fused call with the library workspace, through the C ABI: two calls in
a row, the second on a smaller problem (its static scratch keeps the first
call's contents), and a problem beyond the scratch refused before any
launch."""
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


def run_both(sd, inp):
    q, cache, lens = sd.cache_from_inputs(inp)
    sp = sd.sparsity_from_inputs(inp)
    k_max = O.k_max_for(inp)
    out_ref, idx_ref = sd.sparse_decode_attention(q, cache, lens, sp, k_max=k_max)
    out = torch.full_like(q, 7.0)
    idx = torch.full_like(idx_ref, -7)
    sd.sparse_decode_attention_noalloc(q, cache, lens, sp, out, idx)
    torch.cuda.synchronize()
    return (P.to_host(out_ref), idx_ref.cpu().numpy()), (P.to_host(out), idx.cpu().numpy())


@pytest.mark.parametrize("cfg,first,second", [
    (2, dict(B=3, N=20007), dict(B=2, N=9001)),
    (4, dict(B=6, lmin=3000, lmax=24000, N=24000), dict(B=3, lmin=1000, lmax=9000, N=9000)),
    (5, dict(N=65536 + 77), dict(N=20001)),
])
def test_noalloc_equals_the_workspace_call_twice(sd, cfg, first, second):
    for i, kw in enumerate((first, second)):
        inp = synth.make_inputs(cfg, seed=40 + i, **kw)
        (out_ref, idx_ref), (out, idx) = run_both(sd, inp)
        np.testing.assert_array_equal(idx, idx_ref)
        np.testing.assert_array_equal(out, out_ref)
        # and the oracle, to the usual bar
        ora = O.sparse_attention(inp)
        rep = P.check_idx_rows(idx, ora["idx"], O.scores(inp), ora["tau"], inp.seq_lens,
                               P.budgets(inp))
        assert rep.strict_mismatch_rows == 0, rep.first_failure
        ref = ora["out"] if not rep.band_swaps else O.attend(inp, idx)[0]
        ok, ratio, _ = P.out_errors(out, ref, inp.dtype)
        assert ok, f"call {i}: output error {ratio:.3g} x allowance"


def test_noalloc_refuses_a_problem_beyond_its_scratch(sd):
    # 16 sequences of 128K positions, 64 query heads: the fallback scores
    # alone need 537 MB, beyond the 64 MiB scratch.
    B, Hq, Hkv, N = 16, 64, 8, 131072
    q = torch.zeros((B, Hq, 128), dtype=torch.bfloat16, device="cuda")
    kc = torch.zeros((B, Hkv, N, 128), dtype=torch.bfloat16, device="cuda")
    cache = sd.KVCache(k=kc, v=kc, layout="bhnd")
    lens = torch.full((B,), N, dtype=torch.int32, device="cuda")
    sp = sd.Sparsity(ratio=100.0)
    out = torch.full_like(q, 3.0)
    idx = torch.full((B, Hq, sd.k_max_of(cache, sp)), -5, dtype=torch.int32, device="cuda")
    with pytest.raises(sd.SparseDecodeError) as err:
        sd.sparse_decode_attention_noalloc(q, cache, lens, sp, out, idx)
    assert err.value.status == sd.SD_ERR_WORKSPACE
    torch.cuda.synchronize()
    assert bool((out == 3.0).all()) and bool((idx == -5).all())  # nothing launched
