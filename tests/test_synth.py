"""The seeded input generator: determinism, shapes and planted structure."""
import math

import numpy as np
import torch

from paper_2605_24168_amd import synth
from oracle import oracle as O


def test_bf16_rounding_matches_torch_round_to_nearest_even():
    rng = np.random.default_rng(0)
    x = np.concatenate([rng.standard_normal(100000).astype(np.float32) * 10,
                        np.array([1.00390625, 1.01171875, -1.00390625, 3.0, 0.0, -0.0,
                                  1e-40, 65504.0], np.float32)])
    ours = synth.bf16_bits(x)
    ref = torch.from_numpy(x).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    np.testing.assert_array_equal(ours, ref)
    np.testing.assert_array_equal(synth.bf16_to_f32(ours),
                                  torch.from_numpy(x).to(torch.bfloat16).float().numpy())


def test_deterministic_per_seed_and_distinct_across_seeds():
    a = synth.make_inputs(2, seed=0, B=2, N=512)
    b = synth.make_inputs(2, seed=0, B=2, N=512)
    c = synth.make_inputs(2, seed=1, B=2, N=512)
    for f in ("q", "k", "v"):
        np.testing.assert_array_equal(getattr(a, f), getattr(b, f))
    assert not np.array_equal(a.k, c.k)


def test_shapes_and_budgets_of_the_five_workloads():
    # Small versions keep every structural feature of the full workloads.
    w1 = synth.make_inputs(1)
    assert w1.k.shape == (1, 1, 4096, 128) and w1.dtype == "f32"
    assert O.budget(4096, w1.ratio, w1.rounding) == 410
    w2 = synth.make_inputs(2, B=1, N=2048)
    assert w2.k.shape == (1, 8, 2048, 128) and w2.q.shape == (1, 32, 128) and w2.dtype == "bf16"
    assert O.budget(32768, synth.DEFAULTS[2].ratio, 0) == 1638
    assert O.budget(131072, synth.DEFAULTS[3].ratio, 0) == 1311
    w4 = synth.make_inputs(4, B=3, lmin=100, lmax=300, N=300)
    assert w4.layout == "paged" and w4.block_table.shape == (3, 304 // 16)
    assert w4.rounding == 1 and O.budget(8192, w4.ratio, w4.rounding) == 164
    w5 = synth.make_inputs(5, N=4096)
    assert w5.group_shared and w5.rows == 8 and w5.q.shape == (1, 40, 128)


def test_planted_keys_have_cosine_0_9_with_their_head():
    w = synth.make_inputs(1)
    qf = w.q[0, 0].astype(np.float64)
    pos, _ = w.planted[(0, 0)]
    assert len(pos) == 16
    for p in pos:
        kv = w.k[0, 0, p].astype(np.float64)
        cos = kv.dot(qf) / np.linalg.norm(kv) / np.linalg.norm(qf)
        assert abs(cos - 0.9) < 1e-6
        assert abs(np.linalg.norm(kv) - math.sqrt(128)) < 1e-3
    w2 = synth.make_inputs(2, B=1, N=4000)
    q = synth.bf16_to_f32(w2.q[0]).astype(np.float64)
    for g in range(8):
        pos, heads = w2.planted[(0, g)]
        assert len(pos) == 40   # 1% of the positions
        for p, h in zip(pos[:5], heads[:5]):
            kv = synth.bf16_to_f32(w2.k[0, g, p]).astype(np.float64)
            qh = q[g * 4 + h]
            cos = kv.dot(qh) / np.linalg.norm(kv) / np.linalg.norm(qh)
            assert abs(cos - 0.9) < 0.02     # bf16 rounding of the key


def test_sink_prefix_has_four_times_the_key_norm():
    w = synth.make_inputs(3, B=1, N=1024, Hq=16)
    kf = synth.bf16_to_f32(w.k[0, 0]).astype(np.float64)
    planted = set(w.planted[(0, 0)][0].tolist())
    sink = [np.linalg.norm(kf[j]) for j in range(64) if j not in planted]
    rest = [np.linalg.norm(kf[j]) for j in range(64, 1024) if j not in planted]
    assert 3.5 < np.mean(sink) / np.mean(rest) < 4.5


def test_paged_cache_is_a_permutation_and_poisons_the_unused_tail():
    w = synth.make_inputs(4, B=4, lmin=20, lmax=70, N=70)
    used = np.concatenate([w.block_table[b, :-(-int(L) // 16)] for b, L in enumerate(w.seq_lens)])
    assert sorted(used.tolist()) == list(range(w.k.shape[0]))    # a bijection onto the pool
    poison = synth.bf16_bits(np.array([synth.POISON], np.float32))[0]
    for b, L in enumerate(w.seq_lens):
        L = int(L)
        if L % 16:
            last = w.block_table[b, L // 16]
            assert (w.k[last, L % 16:] == poison).all()
        assert (w.block_table[b, -(-L // 16):] == -1).all()


def test_mixture_keys_are_clustered():
    w = synth.make_inputs(5, N=2048, Hq=8, Hkv=2)
    kf = synth.bf16_to_f32(w.k[0, 0]).astype(np.float64)
    # 256 centroids with within-cluster spread 0.25: nearest-neighbour distances
    # are far below those of independent Gaussian vectors (~16).
    sample = kf[:200]
    d2 = ((sample[:, None, :] - kf[None, :, :]) ** 2).sum(-1)
    d2[np.arange(200), np.arange(200)] = np.inf
    assert np.median(np.sqrt(d2.min(1))) < 6.0


def test_index_sets_and_weights_for_the_attend_only_backend():
    inp = synth.make_inputs(4, seed=0, B=3, seq_lens=[0, 20, 500], N=512)
    a = synth.index_sets(inp, 50, seed=4, k_max=64)
    b = synth.index_sets(inp, 50, seed=4, k_max=64)
    np.testing.assert_array_equal(a, b)
    assert a.shape == (3, inp.rows, 64)
    assert (a[0] == -1).all()                       # empty sequence: all padding
    for bb, n in ((1, 20), (2, 50)):
        L = int(inp.seq_lens[bb])
        row = a[bb]
        assert (row[:, n:] == -1).all()
        live = row[:, :n]
        assert ((live >= 0) & (live < L)).all()
        assert (np.diff(live, axis=1) > 0).all()   # distinct, ascending
    c = synth.index_sets(inp, 50, seed=4, k_max=64, extra_invalid=5)
    for r in range(inp.rows):
        bad = (c[2, r] < 0) | (c[2, r] >= 500)
        assert bad.sum() >= 5
    w = synth.index_weights(a.shape, seed=1, zero_frac=0.25)
    assert w.dtype == np.float32 and w.shape == a.shape
    assert (w >= 0).all() and (w < 3.0).all()
    assert 0.15 < (w == 0).mean() < 0.35
    np.testing.assert_array_equal(w, synth.index_weights(a.shape, seed=1, zero_frac=0.25))
