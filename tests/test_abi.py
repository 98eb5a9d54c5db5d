"""The C-ABI library: it loads, exports every symbol include/w2v.h declares, the
binding's structs match the header, and argument errors are reported before
anything is launched (no GPU needed for these)."""
import ctypes
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "w2v.h")


@pytest.fixture(scope="module")
def w2v():
    import paper_1606_07822_amd as w2v
    if not os.path.exists(w2v.LIB_PATH):
        pytest.skip("libw2v.so not built")
    return w2v


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(w2v_[a-z_0-9]+)\s*\(", text)))


def test_header_declares_the_four_calls():
    names = declared_functions()
    for n in ("w2v_build_vocab", "w2v_build_huffman", "w2v_train_hs_epoch", "w2v_hs_loglik"):
        assert n in names


def test_library_exports_every_declared_symbol(w2v):
    lib = ctypes.CDLL(w2v.LIB_PATH)
    missing = [n for n in declared_functions() if not hasattr(lib, n)]
    assert not missing, missing


def test_struct_layouts_match_header(w2v):
    # offsets the header implies (natural alignment, LP64)
    assert w2v.CModel.V.offset == 16 and w2v.CModel.vocab_counts.offset == 32
    assert w2v.CModel.points.offset == 72 and ctypes.sizeof(w2v.CModel) == 80
    assert w2v.CParams.sample.offset == 16 and w2v.CParams.corpus_tokens.offset == 40
    assert w2v.CParams.seed.offset == 56 and w2v.CParams.write_policy.offset == 80
    assert w2v.CParams.hot_k.offset == 88 and w2v.CParams.cache_mode.offset == 96
    assert w2v.CParams.span_refresh.offset == 100 and w2v.CParams.span_stash.offset == 104
    assert w2v.CParams.stash_from.offset == 108
    assert ctypes.sizeof(w2v.CParams) == 112


def test_vocab_argument_errors(w2v):
    L = w2v.lib()
    V = ctypes.c_int32(0)
    tw = ctypes.c_int64(0)
    fake = ctypes.c_void_p(0x1000)
    rc = L.w2v_build_vocab(fake, 10, 0, 5, fake, fake, fake, fake, None, ctypes.byref(V), ctypes.byref(tw), fake, 1 << 20,
                           None)
    assert rc == w2v.W2V_E_ARG and "id_space" in w2v.last_error()
    rc = L.w2v_build_vocab(fake, -1, 10, 5, fake, fake, fake, fake, None, ctypes.byref(V), ctypes.byref(tw), fake,
                           1 << 20, None)
    assert rc == w2v.W2V_E_ARG
    rc = L.w2v_build_vocab(fake, 10, 10, 5, fake, fake, fake, fake, None, ctypes.byref(V), ctypes.byref(tw), fake, 8,
                           None)
    assert rc == w2v.W2V_E_WORKSPACE and "workspace" in w2v.last_error()
    rc = L.w2v_build_vocab(fake, 10, 10, 5, fake, fake, fake, fake, fake, ctypes.byref(V), ctypes.byref(tw), fake,
                           1 << 20, None)
    assert rc == w2v.W2V_E_ARG and "alias" in w2v.last_error()


def test_huffman_argument_errors(w2v):
    L = w2v.lib()
    fake = ctypes.c_void_p(0x1000)
    a = ctypes.c_int64(0)
    b = ctypes.c_int32(0)
    assert L.w2v_build_huffman(fake, 1, fake, fake, fake, None, 0, ctypes.byref(a), ctypes.byref(b), fake, 1 << 20,
                               None) == w2v.W2V_E_ARG
    need = L.w2v_build_huffman_workspace_bytes(1000)
    assert need > 1000 * (8 + 8)
    assert L.w2v_build_huffman(fake, 1000, fake, fake, fake, None, 0, ctypes.byref(a), ctypes.byref(b), fake, need - 1,
                               None) == w2v.W2V_E_WORKSPACE


def _model(w2v, **kw):
    m = w2v.CModel(0x1000, 0x2000, 100, 50, 64, 0, 0x3000, 1000, 0x4000, 0x5000, 0x6000, 0x7000)
    for k, v in kw.items():
        setattr(m, k, v)
    return m


def _params(w2v, **kw):
    p = w2v.Params(window=5, corpus_tokens=1000).c()
    for k, v in kw.items():
        setattr(p, k, v)
    return p


@pytest.mark.parametrize("mk,pk,msg", [
    (dict(V=1), {}, "V must"),
    (dict(dim=0), {}, "dim"),
    (dict(dim=2000, row_stride=2000), {}, "dim"),
    (dict(row_stride=49), {}, "row_stride"),
    (dict(row_stride=66), {}, "row_stride"),
    (dict(syn0=0x1004), {}, "aligned"),
    (dict(points=0), {}, "Huffman"),
    ({}, dict(window=0), "window"),
    ({}, dict(window=11), "window"),
    ({}, dict(doc_len=0), "doc_len"),
    ({}, dict(sample=1.5), "sample"),
    ({}, dict(first_raw_index=7), "first_raw_index"),
    ({}, dict(arch=3), "arch"),
    ({}, dict(mode=1, arch=2), "synchronous"),
    ({}, dict(mode=1, arch=1), "synchronous"),
    ({}, dict(epoch=1, n_epochs=1), "epoch"),
    ({}, dict(flush_every=0), "flush_every"),
    ({}, dict(cache_k=-1), "cache_k"),
    ({}, dict(cache_k=100), "cache_k"),
    ({}, dict(alpha0=0.0), "alpha0"),
    ({}, dict(hot_k=-1), "hot_k"),
    ({}, dict(write_policy=8), "needs bit 1"),
    ({}, dict(write_policy=13), "needs bit 1"),
    ({}, dict(write_policy=16), "write_policy"),
    ({}, dict(flush_policy=2), "flush_policy"),
    ({}, dict(cache_mode=2), "cache_mode"),
    ({}, dict(span_refresh=-1), "span_refresh"),
    ({}, dict(span_stash=2), "span_stash"),
    ({}, dict(stash_from=-1), "stash_from"),
])
def test_train_argument_errors(w2v, mk, pk, msg):
    L = w2v.lib()
    m = _model(w2v, **mk)
    p = _params(w2v, **pk)
    rc = L.w2v_train_hs_epoch(ctypes.byref(m), ctypes.c_void_p(0x8000), 1000, ctypes.byref(p), None,
                              ctypes.c_void_p(0x9000), 1 << 40, None)
    assert rc == w2v.W2V_E_ARG
    assert msg in w2v.last_error()


def test_workspace_queries_grow_with_input(w2v):
    m = _model(w2v)
    p = _params(w2v)
    L = w2v.lib()
    a = L.w2v_train_workspace_bytes(ctypes.byref(m), 10_000, ctypes.byref(p))
    b = L.w2v_train_workspace_bytes(ctypes.byref(m), 1_000_000, ctypes.byref(p))
    assert 0 < a < b
    ps = _params(w2v, mode=1)
    assert L.w2v_train_workspace_bytes(ctypes.byref(m), 10_000, ctypes.byref(ps)) > a
    assert L.w2v_hs_loglik_workspace_bytes(ctypes.byref(m), 10_000, ctypes.byref(p)) > 0
    assert L.w2v_sample_pairs_workspace_bytes(100, 10_000, ctypes.byref(p)) > 0


def test_binding_refuses_host_tensors(w2v):
    import torch
    with pytest.raises(ValueError):
        w2v.build_vocab(torch.zeros(10, dtype=torch.int32), 10)


@pytest.mark.parametrize("args,msg", [
    ((0, 10, 4, 4, 0, 1, 1), "NULL"),
    ((0x1000, 0, 4, 4, 0, 1, 1), "rows"),
    ((0x1000, 10, 5, 4, 0, 1, 1), "cols"),
    ((0x1000, 10, 4, 4, 4, 1, 1), "mode"),
    ((0x1000, 10, 4, 4, 0, 0, 1), "workgroups"),
])
def test_probe_argument_errors(args, msg):
    import bench_probe
    ms = ctypes.c_float(0.0)
    m, rows, cols, stride, mode, wg, it = args
    rc = bench_probe.lib().w2v_probe_rows(ctypes.c_void_p(m) if m else None, rows, cols, stride, mode, wg, it,
                                          ctypes.byref(ms), None)
    assert rc == -1
    assert msg in bench_probe.last_error()


def test_probe_is_not_in_the_library(w2v):
    import bench_probe
    assert not hasattr(w2v.lib(), "w2v_probe_rows")
    assert hasattr(bench_probe.lib(), "w2v_probe_rows")


def test_struct_offset_of_negative(w2v):
    assert w2v.CParams.negative.offset == 92


@pytest.mark.parametrize("mk,pk,table,L,msg", [
    ({}, {}, 0, 20, "noise_table"),
    ({}, {}, 0x9000, 0, "log2_size"),
    ({}, {}, 0x9000, 31, "log2_size"),
    ({}, dict(negative=0), 0x9000, 20, "negative"),
    ({}, dict(negative=12), 0x9000, 20, "negative"),
    (dict(dim=400, row_stride=448), dict(negative=8), 0x9000, 20, "negative"),
    (dict(dim=600, row_stride=640), dict(negative=2), 0x9000, 20, "dim"),
    ({}, dict(arch=1), 0x9000, 20, "skip-gram"),
    ({}, dict(mode=1), 0x9000, 20, "skip-gram"),
    ({}, dict(window=11), 0x9000, 20, "window"),
])
def test_train_ns_argument_errors(w2v, mk, pk, table, L, msg):
    lib = w2v.lib()
    m = _model(w2v, **mk)
    p = _params(w2v, **pk)
    rc = lib.w2v_train_ns_epoch(ctypes.byref(m), ctypes.c_void_p(table) if table else None, L,
                                ctypes.c_void_p(0x8000), 1000, ctypes.byref(p), None, ctypes.c_void_p(0xA000), 1 << 30,
                                None)
    assert rc == w2v.W2V_E_ARG, w2v.last_error()
    assert msg in w2v.last_error()


def test_train_ns_needs_no_tree_but_a_workspace(w2v):
    lib = w2v.lib()
    m = _model(w2v, codelen=0, code=0, point_off=0, points=0)
    p = _params(w2v)
    need = lib.w2v_train_ns_workspace_bytes(ctypes.byref(m), 1000, ctypes.byref(p))
    assert need > 0
    rc = lib.w2v_train_ns_epoch(ctypes.byref(m), ctypes.c_void_p(0x9000), 20, ctypes.c_void_p(0x8000), 1000,
                                ctypes.byref(p), None, ctypes.c_void_p(0xA000), need - 1, None)
    assert rc == w2v.W2V_E_WORKSPACE


def test_noise_table_and_objective_argument_errors(w2v):
    lib = w2v.lib()
    fake = ctypes.c_void_p(0x1000)
    tot = ctypes.c_int64(0)
    assert lib.w2v_build_noise_table(fake, 0, 10, fake, ctypes.byref(tot), fake, 1 << 20, None) == w2v.W2V_E_ARG
    assert lib.w2v_build_noise_table(fake, 10, 0, fake, ctypes.byref(tot), fake, 1 << 20, None) == w2v.W2V_E_ARG
    assert lib.w2v_build_noise_table(None, 10, 10, fake, ctypes.byref(tot), fake, 1 << 20, None) == w2v.W2V_E_ARG
    need = lib.w2v_noise_table_workspace_bytes(1000)
    assert need >= 2 * 1001 * 8
    assert lib.w2v_build_noise_table(fake, 1000, 10, fake, ctypes.byref(tot), fake, need - 1,
                                     None) == w2v.W2V_E_WORKSPACE
    m = _model(w2v)
    p = _params(w2v, negative=0)
    s = ctypes.c_double(0)
    n = ctypes.c_int64(0)
    assert lib.w2v_ns_objective(ctypes.byref(m), fake, 10, fake, 100, ctypes.byref(p), ctypes.byref(s),
                                ctypes.byref(n), None, fake, 1 << 30, None) == w2v.W2V_E_ARG
    assert "negative" in w2v.last_error()
    p = _params(w2v)
    assert lib.w2v_sample_negatives(fake, 100, 10, fake, 100, ctypes.byref(p), None, 10, None, 0, ctypes.byref(n),
                                    ctypes.byref(ctypes.c_uint64(0)), fake, 1 << 30, None) == w2v.W2V_E_ARG
    assert "noise_table" in w2v.last_error()


def test_launch_reports_need_pointers(w2v):
    L = w2v.lib()
    a, b, c = ctypes.c_int32(-1), ctypes.c_int32(-1), ctypes.c_int32(-1)
    assert L.w2v_last_train_launch(None, ctypes.byref(b)) == w2v.W2V_E_ARG
    assert L.w2v_last_train_resources(ctypes.byref(a), None, ctypes.byref(c)) == w2v.W2V_E_ARG


# Host-side choice of the skip-gram word-row span (write_policy bit 3): half-width or 0, no launch.
@pytest.mark.parametrize("mk,pk,span", [
    (dict(dim=300, row_stride=320), dict(write_policy=15, cache_k=31), 5),
    (dict(dim=300, row_stride=320), dict(write_policy=15, cache_k=0, window=3), 5),
    (dict(dim=300, row_stride=320), dict(write_policy=11, cache_k=0), 5),
    (dict(dim=150, row_stride=192), dict(write_policy=15, window=1), 5),
    (dict(dim=129, row_stride=132), dict(write_policy=15), 5),
    (dict(dim=128, row_stride=128), dict(write_policy=15), 0),
    (dict(dim=50, row_stride=64), dict(write_policy=15), 0),
    (dict(dim=450, row_stride=512), dict(write_policy=15, window=2), 2),
    (dict(dim=450, row_stride=512), dict(write_policy=15, window=3), 0),
    (dict(dim=600, row_stride=640), dict(write_policy=15, window=1), 0),
    (dict(dim=300, row_stride=320), dict(write_policy=15, window=6), 0),
    (dict(dim=300, row_stride=320), dict(write_policy=7), 0),
    (dict(dim=300, row_stride=320), dict(write_policy=11, cache_k=31), 0),   # cached rows not stored
    (dict(dim=300, row_stride=320), dict(write_policy=15, arch=1), 5),
    (dict(dim=300, row_stride=320), dict(write_policy=15, arch=1, hot_k=1024), 5),
    (dict(dim=450, row_stride=512), dict(write_policy=15, arch=1, window=5), 5),
    (dict(dim=100, row_stride=128), dict(write_policy=15, arch=1), 0),
    (dict(dim=300, row_stride=320), dict(write_policy=7, arch=1), 0),
    (dict(dim=300, row_stride=320), dict(write_policy=15, arch=2), 0),
    (dict(dim=300, row_stride=320), dict(write_policy=15, mode=1), 0),
    (dict(dim=300, row_stride=320), dict(write_policy=15, hot_k=8), 0),
    (dict(dim=300, row_stride=320), dict(write_policy=15, cache_mode=1), 0),
])
def test_train_word_span(w2v, mk, pk, span):
    m = _model(w2v, **mk)
    p = _params(w2v, **pk)
    assert w2v.lib().w2v_train_word_span(ctypes.byref(m), ctypes.byref(p)) == span


def test_train_word_span_argument_errors(w2v):
    L = w2v.lib()
    assert L.w2v_train_word_span(None, ctypes.byref(_params(w2v))) == -1
    assert "NULL" in w2v.last_error()
    assert L.w2v_train_word_span(ctypes.byref(_model(w2v)), ctypes.byref(_params(w2v, write_policy=8))) == -1
    assert "needs bit 1" in w2v.last_error()


def test_noalloc_loglik_rejects_what_the_scratch_cannot_hold(w2v):
    """Checked on the host before any device call: a model of V = 1M and 10M tokens needs more
    workspace than the static scratch."""
    fake = ctypes.c_void_p(0x1000)
    cm = w2v.CModel(syn0=fake, syn1=fake, V=1_000_000, dim=300, row_stride=320, vocab_counts=fake, train_words=10**9,
                    codelen=fake, code=fake, point_off=fake, points=fake)
    p = w2v.Params(window=5).c()
    need = w2v.lib().w2v_hs_loglik_workspace_bytes(ctypes.byref(cm), 10_000_000, ctypes.byref(p))
    assert need > w2v.lib().w2v_noalloc_scratch_bytes() == 64 << 20
    s, n, nn = ctypes.c_double(0), ctypes.c_int64(0), ctypes.c_int64(0)
    rc = w2v.lib().w2v_hs_loglik_noalloc(ctypes.byref(cm), fake, 10_000_000, ctypes.byref(p), ctypes.byref(s),
                                         ctypes.byref(n), ctypes.byref(nn), None)
    assert rc == w2v.W2V_E_RANGE and "scratch" in w2v.last_error()
    rc = w2v.lib().w2v_hs_loglik_noalloc(ctypes.byref(cm), fake, 10, ctypes.byref(p), None, ctypes.byref(n),
                                         ctypes.byref(nn), None)
    assert rc == w2v.W2V_E_ARG
