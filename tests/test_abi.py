"""The C ABI on the CPU: the library loads, exports every symbol the header
declares, and rejects invalid arguments before touching the GPU.

No call here reaches a kernel launch: every case carries exactly one defect
that the host-side checks catch (device pointers are never dereferenced by
those checks, so placeholders stand in for them).
"""
import ctypes as C
import math
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
LIB = os.path.join(ROOT, "paper_2605_24168_amd", "libsparse_decode.so")
HEADER = os.path.join(ROOT, "include", "sparse_decode.h")


@pytest.fixture(scope="module")
def sd():
    if not os.path.exists(LIB):
        from paper_2605_24168_amd import build
        build.build()
    from paper_2605_24168_amd import sparse_decode
    return sparse_decode


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(sparse_decode_\w+)\s*\(", text)))


def test_library_exports_every_declared_function(sd):
    names = declared_functions()
    assert len(names) >= 11
    lib = C.CDLL(LIB)
    for n in names:
        assert hasattr(lib, n), f"{n} declared in the header but not exported"
    assert os.path.samefile(sd.LIB_PATH, LIB)


FAKE = 0x100000  # placeholder device address (never dereferenced by the checks)


def tensor(sd, shape, dtype=None, data=FAKE):
    t = sd.SdTensor()
    t.data = data
    t.dtype = sd.SD_BF16 if dtype is None else dtype
    t.ndim = len(shape)
    for i, n in enumerate(shape):
        t.shape[i] = n
    return t


def bhnd(sd, B=2, Hkv=8, N=4096, d=128, dtype=None):
    kv = sd.SdKv()
    kv.t = tensor(sd, (B, Hkv, N, d), dtype)
    kv.layout = sd.SD_KV_BHND
    return kv


def paged(sd, P=100, Hkv=8, d=128, page=16, max_pages=64, dtype=None):
    kv = sd.SdKv()
    kv.t = tensor(sd, (P, page, Hkv, d), dtype)
    kv.layout = sd.SD_KV_PAGED_NHD
    kv.page_size = page
    kv.block_table = FAKE
    kv.max_pages_per_seq = max_pages
    return kv


def sparsity(sd, ratio=20.0, rounding=0, group=0, scale=0.0, sink=0, local=0):
    return sd.SdSparsity(ratio, rounding, group, scale, None, sink, local)


def call_attention(sd, q, K, V, lens, sp, out, idx):
    return sd.lib.sparse_decode_attention(C.byref(q), C.byref(K), C.byref(V), lens, C.byref(sp),
                                          C.byref(out), C.byref(idx), None)


def valid_parts(sd, B=2, Hq=32, Hkv=8, N=4096):
    q = tensor(sd, (B, Hq, 128))
    K, V = bhnd(sd, B, Hkv, N), bhnd(sd, B, Hkv, N)
    sp = sparsity(sd, 20.0)
    out = tensor(sd, (B, Hq, 128))
    idx = tensor(sd, (B, Hq, 205), sd.SD_I32)   # budget(4096, 20) = 205
    return q, K, V, FAKE, sp, out, idx


@pytest.mark.parametrize("defect,code", [
    ("q_null", -1), ("q_ndim", -1), ("head_dim_64", -2), ("hq_not_multiple", -1),
    ("group_too_large", -2), ("kv_dtype_mismatch", -1), ("idx_too_small", -1),
    ("idx_wrong_dtype", -1), ("ratio_zero", -1), ("ratio_nan", -1), ("rounding_2", -1),
    ("out_wrong_shape", -1), ("v_layout_differs", -1), ("seq_lens_null", -1),
    ("page_size_32", -2), ("batch_mismatch", -1), ("scale_nan", -1),
])
def test_attention_rejects_invalid_arguments(sd, defect, code):
    q, K, V, lens, sp, out, idx = valid_parts(sd)
    if defect == "q_null":
        q.data = None
    elif defect == "q_ndim":
        q.ndim = 2
    elif defect == "head_dim_64":
        q.shape[2] = 64
        K.t.shape[3] = V.t.shape[3] = 64
        out.shape[2] = 64
    elif defect == "hq_not_multiple":
        q.shape[1] = 30
        out.shape[1] = 30
        idx.shape[1] = 30
    elif defect == "group_too_large":
        q, K, V, lens, sp, out, idx = valid_parts(sd, Hq=64, Hkv=2)
    elif defect == "kv_dtype_mismatch":
        K.t.dtype = sd.SD_F32
    elif defect == "idx_too_small":
        idx.shape[2] = 204
    elif defect == "idx_wrong_dtype":
        idx.dtype = sd.SD_F32
    elif defect == "ratio_zero":
        sp.ratio = 0.0
    elif defect == "ratio_nan":
        sp.ratio = math.nan
    elif defect == "rounding_2":
        sp.k_rounding = 2
    elif defect == "out_wrong_shape":
        out.shape[1] = 31
    elif defect == "v_layout_differs":
        V = paged(sd)
    elif defect == "seq_lens_null":
        lens = None
    elif defect == "page_size_32":
        K, V = paged(sd, page=32), paged(sd, page=32)
    elif defect == "batch_mismatch":
        K.t.shape[0] = 3
    elif defect == "scale_nan":
        sp.softmax_scale = math.nan
    assert call_attention(sd, q, K, V, lens, sp, out, idx) == code


def test_stage_entry_points_reject_invalid_arguments(sd):
    q, K, V, lens, sp, out, idx = valid_parts(sd)
    bad_scores = tensor(sd, (2, 32, 4095), sd.SD_F32)
    assert sd.lib.sparse_decode_score(C.byref(q), C.byref(K), lens, C.byref(sp),
                                      C.byref(bad_scores), None) == -1
    scores = tensor(sd, (2, 32, 4096), sd.SD_F32)
    scores_bf16 = tensor(sd, (2, 32, 4096), sd.SD_BF16)
    assert sd.lib.sparse_decode_topk(C.byref(scores_bf16), lens, C.byref(sp), C.byref(idx), None,
                                     None) == -1
    bad_vals = tensor(sd, (2, 32, 204), sd.SD_F32)
    assert sd.lib.sparse_decode_topk(C.byref(scores), lens, C.byref(sp), C.byref(idx),
                                     C.byref(bad_vals), None) == -1
    small_idx = tensor(sd, (2, 32, 10), sd.SD_I32)
    assert sd.lib.sparse_decode_topk(C.byref(scores), lens, C.byref(sp), C.byref(small_idx), None,
                                     None) == -1
    wrong_rows = tensor(sd, (2, 8, 205), sd.SD_I32)   # group_shared is off: rows = Hq
    assert sd.lib.sparse_decode_attend(C.byref(q), C.byref(K), C.byref(V), lens,
                                       C.byref(wrong_rows), C.byref(sp), C.byref(out), None) == -1


def test_weighted_attend_rejects_invalid_weights(sd):
    q, K, V, lens, sp, out, idx = valid_parts(sd)

    def call(w):
        return sd.lib.sparse_decode_attend_weighted(C.byref(q), C.byref(K), C.byref(V), lens,
                                                    C.byref(idx), w, C.byref(sp), C.byref(out),
                                                    None)
    assert call(None) == -1
    assert call(C.byref(tensor(sd, (2, 32, 204), sd.SD_F32))) == -1   # shape differs from idx
    assert call(C.byref(tensor(sd, (2, 32, 205), sd.SD_BF16))) == -1  # not float32
    assert call(C.byref(tensor(sd, (2, 8, 205), sd.SD_F32))) == -1
    w = tensor(sd, (2, 32, 205), sd.SD_F32, data=None)                # k_max > 0, no data
    assert call(C.byref(w)) == -1


@pytest.mark.parametrize("defect,code", [
    ("f32", -2), ("group_16", -2), ("seq_lens_null", -1), ("out_wrong_shape", -1),
    ("scale_nan", -1), ("v_missing", -1), ("out_dtype", -1),
])
def test_dense_attention_rejects_invalid_arguments(sd, defect, code):
    q, K, V, lens, sp, out, idx = valid_parts(sd)
    scale = 0.0
    if defect == "f32":
        q.dtype = K.t.dtype = V.t.dtype = out.dtype = sd.SD_F32
    elif defect == "group_16":
        q, K, V, lens, sp, out, idx = valid_parts(sd, Hq=64, Hkv=4)
    elif defect == "seq_lens_null":
        lens = None
    elif defect == "out_wrong_shape":
        out.shape[1] = 16
    elif defect == "scale_nan":
        scale = math.nan
    elif defect == "out_dtype":
        out.dtype = sd.SD_F32
    vref = None if defect == "v_missing" else C.byref(V)
    assert sd.lib.sparse_decode_dense_attention(C.byref(q), C.byref(K), vref, lens, scale,
                                                C.byref(out), None) == code


def test_dense_workspace_grows_with_the_cache(sd):
    sizes = []
    for N in (4096, 65536, 131072):
        q, K, *_ = valid_parts(sd, B=4, N=N)
        n = C.c_size_t(0)
        assert sd.lib.sparse_decode_dense_workspace_size(C.byref(q), C.byref(K), C.byref(n)) == 0
        sizes.append(n.value)
    assert 0 < sizes[0] <= sizes[1] <= sizes[2]
    q, K, *_ = valid_parts(sd)
    K.t.dtype = q.dtype = sd.SD_F32
    n = C.c_size_t(0)
    assert sd.lib.sparse_decode_dense_workspace_size(C.byref(q), C.byref(K), C.byref(n)) == -2


def test_label_arguments_are_checked_on_the_host(sd):
    q, K, V, lens, sp, out, idx = valid_parts(sd)

    def labels(shape, dtype=None, channels=FAKE):
        lab = sd.SdLabels()
        lab.t = tensor(sd, shape, dtype)
        lab.channels = channels
        return lab

    def call(lab):
        return sd.lib.sparse_decode_label_attention(C.byref(q), C.byref(K), C.byref(V),
                                                    C.byref(lab) if lab is not None else None,
                                                    lens, C.byref(sp), C.byref(out),
                                                    C.byref(idx), None)
    assert call(None) == -1
    assert call(labels((2, 8, 4096, 8), channels=None)) == -1
    assert call(labels((2, 8, 4095, 8))) == -1                 # capacity differs from K
    assert call(labels((2, 4, 4096, 8))) == -1                 # KV heads differ
    assert call(labels((2, 8, 4096, 4))) == -2                 # only 8 label channels
    assert call(labels((2, 8, 4096, 8), sd.SD_F32)) == -2      # 16-bit labels only
    scores = tensor(sd, (2, 32, 4096), sd.SD_F32)
    assert sd.lib.sparse_decode_label_score(C.byref(q), C.byref(K),
                                            C.byref(labels((2, 8, 4096, 8))), None,
                                            C.byref(sp), C.byref(scores), None) == -1  # seq_lens


def test_empty_batch_is_a_no_op(sd):
    q = tensor(sd, (0, 32, 128))
    K, V = bhnd(sd, 0, 8, 4096), bhnd(sd, 0, 8, 4096)
    out = tensor(sd, (0, 32, 128))
    idx = tensor(sd, (0, 32, 205), sd.SD_I32)
    assert call_attention(sd, q, K, V, None, sparsity(sd), out, idx) == 0


def test_budget_rule_matches_the_printed_k_values(sd):
    f = lambda L, s, r=0: sd.lib.sparse_decode_budget(L, C.byref(sparsity(sd, s, r)))
    assert f(4096, 10) == 410 and f(32768, 20) == 1638 and f(131072, 100) == 1311
    assert f(1048576, 100) == 10486 and f(8192, 50, 1) == 164 and f(131072, 50, 1) == 2622
    assert f(0, 10) == 0 and f(3, 100) == 1 and f(10, 0.5) == 10
    assert f(10, 0.0) == -1


def test_forced_positions_in_the_budget_and_checks(sd):
    f = lambda L, s, ns, nl: sd.lib.sparse_decode_budget(L, C.byref(sparsity(sd, s, 0, 0, 0.0,
                                                                              ns, nl)))
    assert f(4096, 20, 128, 128) == 128 + 128 + 205
    assert f(4096, 20, 64, 0) == 64 + 205
    assert f(100, 10, 64, 64) == 100          # windows cover the sequence: no heavy budget
    assert f(300, 10, 64, 64) == 64 + 64 + 30
    assert f(0, 10, 64, 64) == 0
    assert f(4096, 20, -1, 0) == -1
    q, K, V, lens, sp, out, idx = valid_parts(sd)
    sp.n_sink, sp.n_local = 128, 128
    assert call_attention(sd, q, K, V, lens, sp, out, idx) == -1   # idx too short now
    idx.shape[2] = 461
    out.data = None
    assert call_attention(sd, q, K, V, lens, sp, out, idx) == -1   # only out's pointer is wrong
    out.data = FAKE
    sp.n_local = -1
    assert call_attention(sd, q, K, V, lens, sp, out, idx) == -1


def test_workspace_size_and_status_strings(sd):
    q, K, V, lens, sp, out, idx = valid_parts(sd)
    n1 = C.c_size_t(0)
    assert sd.lib.sparse_decode_workspace_size(C.byref(q), C.byref(K), C.byref(sp), C.byref(idx),
                                               C.byref(n1)) == 0
    q2, K2, V2, _, _, _, idx2 = valid_parts(sd, N=65536)
    idx2.shape[2] = 3277
    n2 = C.c_size_t(0)
    assert sd.lib.sparse_decode_workspace_size(C.byref(q2), C.byref(K2), C.byref(sp),
                                               C.byref(idx2), C.byref(n2)) == 0
    assert 0 < n1.value < n2.value
    assert sd.lib.sparse_decode_set_workspace(FAKE + 3, 1024) == -1   # misaligned
    for code, text in [(0, "ok"), (-1, "invalid argument"), (-2, "unsupported configuration"),
                       (-3, "workspace"), (-4, "HIP")]:
        assert text in sd.lib.sparse_decode_status_string(code).decode()


def test_binding_refuses_host_tensors(sd):
    import torch
    q = torch.zeros((1, 8, 128), dtype=torch.bfloat16)
    cache = sd.KVCache(k=torch.zeros((1, 8, 64, 128), dtype=torch.bfloat16),
                       v=torch.zeros((1, 8, 64, 128), dtype=torch.bfloat16))
    with pytest.raises(ValueError):
        sd.sparse_decode_attention(q, cache, torch.zeros(1, dtype=torch.int32), sd.Sparsity(10.0))


def test_read_probe_checks_its_buffer_on_the_host(sd):
    probe = sd.lib.sparse_decode_read_probe
    sink = FAKE
    assert probe(None, 1024, sink, None) == -1          # no buffer
    assert probe(FAKE + 8, 1024, sink, None) == -1      # misaligned
    assert probe(FAKE, 1000, sink, None) == -1          # not a multiple of 16 bytes
    assert probe(FAKE, 0, sink, None) == -1             # empty
    assert probe(FAKE, 1024, None, None) == -1          # no sink
    assert probe(FAKE, 1024, FAKE + 2, None) == -1      # misaligned sink


@pytest.mark.parametrize("defect,code", [
    ("draws_null", -1), ("draws_dtype", -1), ("draws_rows", -1), ("weights_shape", -1),
    ("weights_dtype", -1), ("idx_short_of_draws", -1), ("group_shared", -2),
])
def test_sampled_attention_rejects_invalid_arguments(sd, defect, code):
    q, K, V, lens, sp, out, idx = valid_parts(sd)
    s = 16
    idx.shape[2] = 205 + s
    draws = tensor(sd, (2, 32, s), sd.SD_I32)
    w = tensor(sd, (2, 32, 205 + s), sd.SD_F32)
    if defect == "draws_null":
        draws = None
    elif defect == "draws_dtype":
        draws.dtype = sd.SD_F32
    elif defect == "draws_rows":
        draws.shape[1] = 31
    elif defect == "weights_shape":
        w.shape[2] = 205
    elif defect == "weights_dtype":
        w.dtype = sd.SD_BF16
    elif defect == "idx_short_of_draws":
        idx.shape[2] = 205 + s - 1   # the top-k part must still hold 205
    elif defect == "group_shared":
        sp.group_shared = 1
        idx.shape[1] = draws.shape[1] = w.shape[1] = 8
    rc = sd.lib.sparse_decode_sampled_attention(
        C.byref(q), C.byref(K), C.byref(V), lens, C.byref(sp),
        C.byref(draws) if draws is not None else None, C.byref(out), C.byref(idx), C.byref(w),
        None)
    assert rc == code
