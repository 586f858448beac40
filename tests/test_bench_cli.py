"""bench.py's command line, without a GPU: one GPU only, and a clean refusal
of more (before anything touches a device)."""
import os
import subprocess
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _bench(*args):
    return subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), *args],
                          capture_output=True, text=True, timeout=120)


def test_more_than_one_gpu_is_refused_with_a_message():
    r = _bench("--gpus", "2")
    assert r.returncode == 2
    assert "one GPU" in r.stderr


def test_help_lists_the_contract_flags():
    r = _bench("--help")
    assert r.returncode == 0
    for flag in ("--gpus", "--steps", "--warmup", "--workload", "--cpu-sample"):
        assert flag in r.stdout


def test_cpu_baseline_repeats_the_oracle_sample_for_a_bounded_time():
    import bench
    from oracle import oracle as O
    from paper_2605_24168_amd import synth
    inp = synth.make_inputs(1, seed=0)
    rec = bench.cpu_baseline(inp, 1, O.k_max_for(inp), min_s=0.3)
    assert rec["kind"] == "oracle" and rec["unit"] == "queries/s"
    assert rec["value"] > 0 and rec["cores"] >= 1
    assert "passes in" in rec["sample"]
    one = bench.cpu_baseline(inp, 1, O.k_max_for(inp), min_s=0.1, threads=1)
    assert one["cores"] == 1


def test_union_gather_rows_counts_distinct_positions_per_kv_head():
    import types
    import torch
    import bench
    # 2 sequences, 2 KV heads of 2 query heads each; -1 is padding.
    idx = torch.tensor([[[0, 5, 9], [5, 9, -1], [1, 2, 3], [4, 5, 6]],
                        [[7, -1, -1], [7, -1, -1], [0, 1, -1], [1, 0, -1]]], dtype=torch.int32)
    inp = types.SimpleNamespace(B=2, Hkv=2, G=2, group_shared=False)
    # (b0,g0): {0,5,9}; (b0,g1): {1..6}; (b1,g0): {7}; (b1,g1): {0,1}
    assert bench.union_gather_rows(torch, idx, inp) == 3 + 6 + 1 + 2
