"""Parity of the attend-only weighted sparse backend and of the dense decode
baseline (the two kernels Table 1 compares) with the CPU oracle, through the
C ABI.

Index lists are irregular (uniform random positions, no block structure, as
in Table 1), with padding and out-of-range entries the backend must skip;
weights are U[0.05, 3) with some exact zeros.
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


# (workload, overrides): float32 contiguous, bf16 contiguous GQA, bf16 with
# 8 heads per group, ragged paged, and group-shared rows.
CASES = {
    "w1": (1, {}),
    "w2": (2, dict(B=2, N=20007)),
    "w3": (3, dict(B=2, N=9001)),
    "w4": (4, dict(B=5, lmin=1000, lmax=30000, N=30000)),
    "w5": (5, dict(N=40000)),
}


def make(name, seed=0, **over):
    cfg, kw = CASES[name]
    kw = dict(kw)
    kw.update(over)
    return synth.make_inputs(cfg, seed=seed, **kw)


def to_dev(a, dtype=None):
    t = torch.from_numpy(np.ascontiguousarray(a)).cuda()
    return t if dtype is None else t.to(dtype)


def usable(idx, w, seq_lens):
    """The oracle's index-set form of lists the library skips entries of:
    per row the entries in [0, L_b) in their order (with their weights),
    then -1 padding (weight 0)."""
    ci = np.full_like(idx, -1)
    cw = np.zeros_like(w)
    for b in range(idx.shape[0]):
        L = int(seq_lens[b])
        for r in range(idx.shape[1]):
            keep = (idx[b, r] >= 0) & (idx[b, r] < L)
            n = int(keep.sum())
            ci[b, r, :n] = idx[b, r][keep]
            cw[b, r, :n] = w[b, r][keep]
    return ci, cw


def check_out(gpu, ref, dtype, label):
    ok, ratio, rel = P.out_errors(gpu, ref, dtype)
    P.log(f"  {label}: worst/allow={ratio:.3g} relL2={rel:.2e}")
    assert ok, f"{label}: output error {ratio:.3g} x allowance"
    return rel


# ---------------------------------------------------------------------------
# Weighted sparse backend.
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("name", list(CASES))
def test_weighted_attend_matches_oracle(sd, name):
    inp = make(name)
    k = max(O.budget(int(inp.ncap), inp.ratio, inp.rounding), 1)
    idx = synth.index_sets(inp, k, seed=1, k_max=k + 8, extra_invalid=3)
    w = synth.index_weights(idx.shape, seed=2, zero_frac=0.1)
    q, cache, lens = sd.cache_from_inputs(inp)
    sp = sd.sparsity_from_inputs(inp)
    out = sd.sparse_decode_attend_weighted(q, cache, lens, to_dev(idx), to_dev(w), sp)
    torch.cuda.synchronize()
    ref, _ = O.attend_weighted(inp, *usable(idx, w, inp.seq_lens))
    check_out(P.to_host(out), ref, inp.dtype, f"{name} weighted")


@pytest.mark.parametrize("name", ["w1", "w4", "w5"])
def test_unit_weights_reproduce_the_unweighted_attend_bit_for_bit(sd, name):
    inp = make(name)
    k = O.budget(int(inp.ncap), inp.ratio, inp.rounding)
    idx = to_dev(synth.index_sets(inp, k, seed=3, extra_invalid=2))
    q, cache, lens = sd.cache_from_inputs(inp)
    sp = sd.sparsity_from_inputs(inp)
    plain = sd.sparse_decode_attend(q, cache, lens, idx, sp)
    ones = sd.sparse_decode_attend_weighted(q, cache, lens, idx,
                                            torch.ones(idx.shape, device="cuda"), sp)
    torch.cuda.synchronize()
    assert torch.equal(plain, ones)


def test_weighted_special_rows(sd):
    """One row keeps a single entry (output = that value row), one has all
    weights 0 (zeros), one has constant weights (= unweighted)."""
    inp = make("w2")
    k = 300
    idx_h = synth.index_sets(inp, k, seed=5)
    w = np.ones(idx_h.shape, np.float32)
    w[0, 0, :] = 0.0
    w[0, 0, 17] = 1.0
    w[0, 1, :] = 0.0
    w[1, 3, :] = 7.25
    q, cache, lens = sd.cache_from_inputs(inp)
    sp = sd.sparsity_from_inputs(inp)
    idx = to_dev(idx_h)
    out = P.to_host(sd.sparse_decode_attend_weighted(q, cache, lens, idx, to_dev(w), sp))
    plain = P.to_host(sd.sparse_decode_attend(q, cache, lens, idx, sp))
    j = int(idx_h[0, 0, 17])
    vrow = synth.bf16_to_f32(inp.v[0, 0, j])          # head 0 reads KV head 0
    np.testing.assert_array_equal(out[0, 0], vrow)
    assert (out[0, 1] == 0).all()
    np.testing.assert_allclose(out[1, 3], plain[1, 3], rtol=0, atol=2e-2)
    ref, _ = O.attend_weighted(inp, idx_h, w)
    check_out(out, ref, inp.dtype, "special rows")


def test_weighted_long_lists_split_over_workgroups(sd):
    # k = 8000 of 20007 positions: every row is split and merged.
    inp = make("w2")
    idx = synth.index_sets(inp, 8000, seed=6)
    w = synth.index_weights(idx.shape, seed=7, zero_frac=0.3)
    q, cache, lens = sd.cache_from_inputs(inp)
    sp = sd.sparsity_from_inputs(inp)
    out = sd.sparse_decode_attend_weighted(q, cache, lens, to_dev(idx), to_dev(w), sp)
    ref, _ = O.attend_weighted(inp, idx, w)
    check_out(P.to_host(out), ref, inp.dtype, "long weighted lists")


# ---------------------------------------------------------------------------
# Dense decode baseline.
# ---------------------------------------------------------------------------

def gpu_dense(sd, inp):
    q, cache, lens = sd.cache_from_inputs(inp)
    out = sd.sparse_decode_dense_attention(q, cache, lens)
    torch.cuda.synchronize()
    return P.to_host(out)


@pytest.mark.parametrize("name", ["w2", "w3", "w4", "w5"])
def test_dense_matches_oracle(sd, name):
    inp = make(name)
    rel = check_out(gpu_dense(sd, inp), O.dense_attention(inp), inp.dtype, f"{name} dense")
    assert rel < 5e-3


@pytest.mark.parametrize("Hq,Hkv,layout", [(32, 32, "paged"), (8, 4, "paged"), (12, 4, "bhnd"),
                                           (16, 2, "bhnd"), (24, 8, "paged"), (6, 3, "bhnd"),
                                           (10, 2, "paged"), (3, 3, "paged")])
def test_dense_head_groupings(sd, Hq, Hkv, layout):
    inp = synth.make_inputs(4, seed=2, Hq=Hq, Hkv=Hkv, layout=layout,
                            seq_lens=[5000, 1, 16, 4097], N=5000)
    check_out(gpu_dense(sd, inp), O.dense_attention(inp), inp.dtype, f"dense {Hq}/{Hkv} {layout}")


def test_dense_ragged_lengths_at_tile_and_range_boundaries(sd):
    lens = [0, 1, 15, 16, 17, 255, 256, 257, 1023, 1024, 1025, 4095, 4096, 4097, 12289]
    for layout in ("bhnd", "paged"):
        inp = synth.make_inputs(4, seed=3, layout=layout, seq_lens=lens, N=12289)
        out = gpu_dense(sd, inp)
        assert (out[0] == 0).all()
        check_out(out, O.dense_attention(inp), inp.dtype, f"dense ragged {layout}")


def test_dense_single_sequence_split_finely(sd):
    # One sequence with few KV heads: the key ranges shrink to 256 keys, so
    # a long sequence is merged from many partials.
    inp = synth.make_inputs(2, seed=4, B=1, N=65536 + 33, Hq=8, Hkv=2)
    check_out(gpu_dense(sd, inp), O.dense_attention(inp), inp.dtype, "dense one sequence")


def test_dense_paged_page_order_does_not_matter(sd):
    inp = make("w4", seed=5)
    a = gpu_dense(sd, inp)
    perm = np.random.default_rng(0).permutation(inp.k.shape[0]).astype(np.int32)
    inv = np.empty_like(perm)
    inv[perm] = np.arange(perm.size, dtype=np.int32)
    import dataclasses
    moved = dataclasses.replace(inp, k=inp.k[inv], v=inp.v[inv],
                                block_table=np.where(inp.block_table >= 0,
                                                     perm[np.maximum(inp.block_table, 0)], -1))
    np.testing.assert_array_equal(gpu_dense(sd, moved), a)


def test_dense_is_deterministic_and_matches_full_index_attend(sd):
    inp = make("w2", seed=6)
    a, b = gpu_dense(sd, inp), gpu_dense(sd, inp)
    np.testing.assert_array_equal(a, b)
    # The sparse backend with every position listed computes the same thing.
    q, cache, lens = sd.cache_from_inputs(inp)
    idx = torch.arange(inp.ncap, dtype=torch.int32, device="cuda").expand(inp.B, inp.rows, -1)
    full = sd.sparse_decode_attend(q, cache, lens, idx.contiguous(), sd.sparsity_from_inputs(inp))
    np.testing.assert_allclose(P.to_host(full), a, rtol=0, atol=2e-2)


def test_dense_rejects_float32(sd):
    inp = make("w1")
    q, cache, lens = sd.cache_from_inputs(inp)
    with pytest.raises(sd.SparseDecodeError) as e:
        sd.sparse_decode_dense_attention(q, cache, lens)
    assert e.value.status == sd.SD_ERR_UNSUPPORTED
