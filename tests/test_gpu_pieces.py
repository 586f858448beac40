"""Candidate selection of few rows over several workgroups each.

Calls with fewer rows than the 1024-thread selection needs to fill the GPU
select each row's candidates in pieces of consecutive chunks: one kernel
takes every piece's value-bucket counts and a bucket-ordered copy of its
keys, then each piece finds the k-th bucket from the counts, ranks that
bucket's keys across pieces and writes its own kept candidates.  The lists
and outputs must equal, bit for bit, those of one workgroup per row (debug
flags 32 / 16 turn the pieces on / off whatever the row's candidates), and
match the oracle: few rows with one to
several chunks per piece, ragged paged batches, group-shared rows, forced
windows, exactly tied keys straddling the pieces (a k-th bucket within the
workgroup's width, ranked by an exact count, and one beyond it, ranked by
radix passes over its keys), low sparsity, and a row on the exact fallback
beside rows in pieces.
"""
import dataclasses

import numpy as np
import pytest
import torch

from oracle import oracle as O
from paper_2605_24168_amd import synth
from tests import parity as P

pytestmark = pytest.mark.gpu

PIECES_OFF, PIECES_ON = 16, 32


@pytest.fixture(scope="module")
def sd():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2605_24168_amd import sparse_decode
    sparse_decode.set_debug(0)
    return sparse_decode


def run(sd, inp, flags=0):
    q, cache, lens = sd.cache_from_inputs(inp)
    sp = sd.sparsity_from_inputs(inp)
    sd.set_debug(flags)
    try:
        out, idx = sd.sparse_decode_attention(q, cache, lens, sp, k_max=O.k_max_for(inp))
        torch.cuda.synchronize()
    finally:
        sd.set_debug(0)
    return P.to_host(out), idx.cpu().numpy()


def list_lengths(inp):
    """Entries of each sequence's list: forced positions plus the top-k budget."""
    out = []
    for L in inp.seq_lens:
        L = int(L)
        ns = min(inp.n_sink, L)
        nl = min(inp.n_local, L - ns)
        out.append(ns + nl + min(O.budget(L, inp.ratio, inp.rounding), L - ns - nl))
    return np.array(out, np.int64)


def check_oracle(inp, out, idx, label):
    ora = O.sparse_attention(inp, k_max=idx.shape[2])
    rep = P.check_idx_rows(idx, ora["idx"], O.scores(inp), ora["tau"], inp.seq_lens,
                           list_lengths(inp))
    assert rep.strict_mismatch_rows == 0, f"{label}: {rep.first_failure}"
    ref = ora["out"] if not rep.band_swaps else O.attend(inp, idx)[0]
    ok, ratio, _ = P.out_errors(out, ref, inp.dtype)
    assert ok, f"{label}: output error {ratio:.3g} x allowance"


def tied(inp, period):
    """The same inputs with keys and values repeating every `period` positions
    along each sequence (contiguous layout): each head's scores then take
    `period` values, so the k-th largest is shared by many positions."""
    rep = np.arange(inp.ncap) % period
    return dataclasses.replace(inp, k=np.ascontiguousarray(inp.k[:, :, rep]),
                               v=np.ascontiguousarray(inp.v[:, :, rep]))


CASES = {
    # 64 per-head rows, three chunks: a piece per chunk.
    "gqa 64 rows": lambda: synth.make_inputs(2, seed=4, B=2, N=20007),
    # 8 group-shared rows over 9 chunks.
    "group-shared 8 rows": lambda: synth.make_inputs(5, seed=4, N=65536 + 77),
    # 8 group-shared rows over 37 chunks: 32 pieces of one or two chunks.
    "group-shared 37 chunks": lambda: synth.make_inputs(5, seed=5, N=300001),
    # A ragged paged batch (64 rows, lengths 1K-60K).
    "paged ragged": lambda: synth.make_inputs(4, seed=4, B=2, lmin=1000, lmax=60000, N=60000),
    # Sink and local windows beside the top-k.
    "forced windows": lambda: synth.make_inputs(3, seed=4, B=2, N=24003, n_sink=64, n_local=200),
    # Low sparsity: pieces of many candidates.
    "gqa 4x": lambda: synth.make_inputs(2, seed=6, B=2, N=20007, ratio=4.0),
}


@pytest.mark.parametrize("name", list(CASES))
def test_pieces_equal_one_workgroup_per_row(sd, name):
    inp = CASES[name]()
    out_a, idx_a = run(sd, inp, PIECES_ON)
    out_b, idx_b = run(sd, inp, PIECES_OFF)
    np.testing.assert_array_equal(idx_a, idx_b)
    np.testing.assert_array_equal(out_a, out_b)
    if name != "group-shared 37 chunks":  # (the oracle's time: the others)
        check_oracle(inp, out_a, idx_a, name)


@pytest.mark.parametrize("period", [50, 7])
def test_pieces_with_tied_keys_across_pieces(sd, period):
    # Period 50: about 400 positions share the k-th key, the bucket's keys
    # are ranked across pieces.  Period 7: about 2900 do, more than the
    # workgroup's width: radix passes over the bucket's keys rank them.
    inp = tied(synth.make_inputs(2, seed=12, B=2, N=20007), period)
    out_a, idx_a = run(sd, inp, PIECES_ON)
    out_b, idx_b = run(sd, inp, PIECES_OFF)
    np.testing.assert_array_equal(idx_a, idx_b)
    np.testing.assert_array_equal(out_a, out_b)
    ora = O.sparse_attention(inp)
    np.testing.assert_array_equal(idx_a, ora["idx"])
    ok, ratio, _ = P.out_errors(out_a, ora["out"], inp.dtype)
    assert ok, f"output error {ratio:.3g} x allowance"


def test_pieces_repeat_calls_of_different_shapes(sd):
    # The piece records and copies live in the workspace: a call with more
    # chunks, then one with fewer, each equal to the one-workgroup result.
    for N in (120001, 30011):
        inp = synth.make_inputs(5, seed=N, N=N)
        out_a, idx_a = run(sd, inp, PIECES_ON)
        out_b, idx_b = run(sd, inp, PIECES_OFF)
        np.testing.assert_array_equal(idx_a, idx_b)
        np.testing.assert_array_equal(out_a, out_b)


def test_pieces_beside_rows_on_the_exact_fallback(sd):
    # A cluster of 400 keys close to head 0's query overflows that row's
    # staging area, so it takes the exact fallback (its first piece selects
    # it from full scores) while the call's other rows are selected in
    # pieces; lists and outputs equal the one-workgroup call's and the
    # oracle's.
    inp = synth.make_inputs(2, seed=15, B=1, N=12000, ratio=50.0, Hq=64, Hkv=8)
    rng = np.random.default_rng(15)
    q0 = synth.bf16_to_f32(inp.q[0, 0]).astype(np.float64)
    base = 3.0 * q0 / np.linalg.norm(q0) * np.sqrt(inp.d)
    clus = base[None, :] + 0.3 * rng.standard_normal((400, inp.d))
    k = inp.k.copy()
    k[0, 0, 100:500] = synth.bf16_bits(clus.astype(np.float32))
    inp = dataclasses.replace(inp, k=k)
    sd.set_profiling(True)
    try:
        out_a, idx_a = run(sd, inp, PIECES_ON)
        prof = sd.last_profile()
    finally:
        sd.set_profiling(False)
    assert prof["repaired_rows"] >= 1
    out_b, idx_b = run(sd, inp, PIECES_OFF)
    np.testing.assert_array_equal(idx_a, idx_b)
    np.testing.assert_array_equal(out_a, out_b)
    check_oracle(inp, out_a, idx_a, "fallback row beside pieces")
