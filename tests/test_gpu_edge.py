"""Degenerate and boundary inputs of the training and evaluation paths on the
GPU (through the C ABI): empty and fully dropped streams, documents too short
for a window, the smallest tree (V = 2) and vector size (d = 1), a ragged last
document, a corpus fed in whole-document chunks, the widest window, rows
packed with no padding, padding columns that hold NaN, and the deepest tree
the codes allow (64 levels).
"""
import types

import numpy as np
import pytest

import oracle
import synth
from gpu_common import oracle_side, row_rel_err

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def w2v():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_1606_07822_amd as w2v
    w2v.lib()
    return w2v


def to_dev(a):
    import torch
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def tiny_model(w2v, s, dim=16):
    voc = w2v.build_vocab(to_dev(s.tok), s.w.vocab, s.w.min_count)
    tree = w2v.build_huffman(voc.vocab_counts)
    syn0, syn1 = synth.init_weights(s.voc.V, dim, syn1_scale=0.1)
    return voc, tree, syn0, syn1


@pytest.mark.parametrize("mode,arch", [(0, 0), (0, 1), (0, 2), (1, 0)])
@pytest.mark.parametrize("case", ["empty", "all_dropped", "doc_len_1"])
def test_nothing_to_train_leaves_the_model_alone(w2v, mode, arch, case):
    s = oracle_side("tiny_sg_v1k_d50")
    voc, tree, syn0, syn1 = tiny_model(w2v, s)
    model = w2v.make_model(syn0, syn1, voc, tree)
    before = [t.cpu().numpy().copy() for t in model.vectors()]
    doc_len = 1000
    if case == "empty":
        tok = to_dev(np.zeros(1, np.int32))[:0]
    elif case == "all_dropped":
        tok = to_dev(np.full(2500, -1, np.int32))
    else:
        tok = to_dev(s.tv[:3000])
        doc_len = 1                       # one token per document: centres without window words
    p = w2v.Params(window=2, mode=mode, arch=arch, doc_len=doc_len, corpus_tokens=max(1, tok.numel()), cache_k=7)
    st = w2v.train_hs_epoch(model, tok, p).cpu().numpy()
    n = tok.numel()
    assert st[0] == n and st[3] == 0 and st[4] == 0
    assert st[1] == (0 if case != "doc_len_1" else int((s.tv[:3000] >= 0).sum()))
    for a, b in zip(before, (t.cpu().numpy() for t in model.vectors())):
        np.testing.assert_array_equal(a, b)
    sg, npairs, nnodes = w2v.hs_loglik(model, tok, w2v.Params(window=2, doc_len=doc_len))
    assert (sg, npairs, nnodes) == (0.0, 0, 0)


def test_negative_sampling_on_empty_stream(w2v):
    s = oracle_side("tiny_sg_v1k_d50")
    voc = w2v.build_vocab(to_dev(s.tok), s.w.vocab, s.w.min_count)
    noise = w2v.build_noise_table(voc.vocab_counts)
    syn0, _ = synth.init_weights(s.voc.V, 8)
    model = w2v.make_ns_model(syn0, np.ones((s.voc.V, 8), np.float32), voc)
    tok = to_dev(np.zeros(1, np.int32))[:0]
    st = w2v.train_ns_epoch(model, noise, tok, w2v.Params(window=2, corpus_tokens=1)).cpu().numpy()
    assert list(st) == [0, 0, 0, 0, 0]
    np.testing.assert_array_equal(model.vectors()[0].cpu().numpy(), syn0)
    assert w2v.ns_objective(model, noise, tok, w2v.Params(window=2)) == (0.0, 0, 0)


@pytest.mark.parametrize("dim", [1, 3, 64])
def test_two_word_vocabulary(w2v, dim):
    # the smallest tree: one inner node, codes {0} and {1}
    rng = np.random.default_rng(dim)
    tok = rng.choice([3, 7], size=4000, p=[0.6, 0.4]).astype(np.int32)
    voc = w2v.build_vocab(to_dev(tok), 10, 1)
    assert voc.V == 2
    tree = w2v.build_huffman(voc.vocab_counts)
    ov = oracle.build_vocab(tok, 10, 1)
    ot = oracle.build_huffman(ov.vocab_counts)
    tv = oracle.remap(tok, ov.id_to_vocab)
    syn0, syn1 = synth.init_weights(2, dim, syn1_scale=0.2)
    a0, a1 = syn0.copy(), syn1.copy()
    op = oracle.params(2, dim, window=3, train_words=ov.train_words, corpus_tokens=tok.size, order=1, cache_k=1,
                       flush_every=10)
    ost = oracle.train(a0, a1, ot, tv, op)
    model = w2v.make_model(syn0, syn1, voc, tree)
    p = w2v.Params(window=3, corpus_tokens=tok.size, workers=1, cache_k=1, flush_every=10)
    st = w2v.train_hs_epoch(model, to_dev(tv), p).cpu().numpy()
    assert list(st) == list(ost)
    g0, g1 = (t.cpu().numpy() for t in model.vectors())
    assert row_rel_err(g0, a0) <= 1e-4 and row_rel_err(g1[:1], a1) <= 1e-4


@pytest.mark.parametrize("n", [1, 999, 2500, 3001])
def test_ragged_last_document(w2v, n):
    s = oracle_side("sg_v30k_d100")
    voc = w2v.build_vocab(to_dev(s.tok), s.w.vocab, s.w.min_count)
    tree = w2v.build_huffman(voc.vocab_counts)
    tv = s.tv[:n]
    syn0, syn1 = synth.init_weights(s.voc.V, 100, syn1_scale=0.005)
    a0, a1 = syn0.copy(), syn1.copy()
    op = oracle.params(s.voc.V, 100, window=5, sample=1e-3, train_words=s.voc.train_words, corpus_tokens=s.tv.size,
                       order=1, cache_k=31, flush_every=10)
    ost = oracle.train(a0, a1, s.tree, tv, op)
    model = w2v.make_model(syn0, syn1, voc, tree)
    p = w2v.Params(window=5, sample=1e-3, corpus_tokens=s.tv.size, workers=1, cache_k=31, flush_every=10)
    st = w2v.train_hs_epoch(model, to_dev(tv), p).cpu().numpy()
    assert list(st) == list(ost)
    g0, g1 = (t.cpu().numpy() for t in model.vectors())
    assert row_rel_err(g0, a0) <= 1e-4 and row_rel_err(g1[:s.voc.V - 1], a1) <= 1e-4


# The longest documents (65,535 raw tokens: 16-bit offsets, up to 512 segments of kept centres) at raw
# positions past 2^32, with the learning rate of a later epoch: one worker against the oracle.
@pytest.mark.parametrize("dim,wp,arch", [(100, 5, 0), (300, 15, 0), (300, 15, 1)])
def test_longest_documents_far_into_the_run(w2v, dim, wp, arch):
    s = oracle_side("sg_v30k_d100")
    voc = w2v.build_vocab(to_dev(s.tok), s.w.vocab, s.w.min_count)
    tree = w2v.build_huffman(voc.vocab_counts)
    tv = s.tv[:70_000]   # one whole document (about 50,000 kept centres, 390 segments) and a ragged one
    first, doc_len, corpus = 65535 * 70_000, 65535, 5_000_000_000
    syn0, syn1 = synth.init_weights(s.voc.V, dim, syn1_scale=0.5 / dim)
    a0, a1 = syn0.copy(), syn1.copy()
    op = oracle.params(s.voc.V, dim, window=5, sample=1e-3, train_words=s.voc.train_words, corpus_tokens=corpus,
                       doc_len=doc_len, first_raw_index=first, epoch=1, n_epochs=3, order=1, cache_k=31,
                       flush_every=10, arch=arch)
    ost = oracle.train(a0, a1, s.tree, tv, op)
    model = w2v.make_model(syn0, syn1, voc, tree)
    p = w2v.Params(window=5, sample=1e-3, corpus_tokens=corpus, doc_len=doc_len, first_raw_index=first, epoch=1,
                   n_epochs=3, workers=1, cache_k=31, flush_every=10, write_policy=wp, arch=arch)
    st = w2v.train_hs_epoch(model, to_dev(tv), p).cpu().numpy()
    assert list(st) == list(ost)
    g0, g1 = (t.cpu().numpy() for t in model.vectors())
    assert row_rel_err(g0, a0) <= 1e-4 and row_rel_err(g1[:s.voc.V - 1], a1) <= 1e-4


@pytest.mark.parametrize("arch", [0, 2])
def test_chunked_stream_equals_whole_stream(w2v, arch):
    # without a cache one worker's result depends only on the centre sequence and the raw positions,
    # so feeding whole documents in two calls (first_raw_index) gives the same bits
    s = oracle_side("sg_v30k_d100")
    voc = w2v.build_vocab(to_dev(s.tok), s.w.vocab, s.w.min_count)
    tree = w2v.build_huffman(voc.vocab_counts)
    tv = to_dev(s.tv[:6000])
    syn0, syn1 = synth.init_weights(s.voc.V, 64, syn1_scale=0.01)
    m1 = w2v.make_model(syn0, syn1, voc, tree)
    m2 = w2v.make_model(syn0, syn1, voc, tree)
    base = dict(window=5, sample=1e-3, corpus_tokens=s.tv.size, workers=1, cache_k=0, arch=arch)
    st = w2v.train_hs_epoch(m1, tv, w2v.Params(**base)).cpu().numpy()
    sa = w2v.train_hs_epoch(m2, tv[:4000], w2v.Params(**base)).cpu().numpy()
    sb = w2v.train_hs_epoch(m2, tv[4000:], w2v.Params(first_raw_index=4000, **base)).cpu().numpy()
    assert list(st) == list(sa + sb)
    for a, b in zip(m1.vectors(), m2.vectors()):
        np.testing.assert_array_equal(a.cpu().numpy(), b.cpu().numpy())


def test_widest_window_and_widest_rows(w2v):
    # window 10 (up to 20 window words, two register groups) at the widest vector size, d = 1024
    s = oracle_side("sg_v30k_d100")
    voc = w2v.build_vocab(to_dev(s.tok), s.w.vocab, s.w.min_count)
    tree = w2v.build_huffman(voc.vocab_counts)
    tv = s.tv[:2000]
    syn0, syn1 = synth.init_weights(s.voc.V, 1024, syn1_scale=0.5 / 1024)
    a0, a1 = syn0.copy(), syn1.copy()
    op = oracle.params(s.voc.V, 1024, window=10, sample=1e-3, train_words=s.voc.train_words,
                       corpus_tokens=s.tv.size, order=1, cache_k=15, flush_every=10)
    ost = oracle.train(a0, a1, s.tree, tv, op)
    model = w2v.make_model(syn0, syn1, voc, tree)
    p = w2v.Params(window=10, sample=1e-3, corpus_tokens=s.tv.size, workers=1, cache_k=15, flush_every=10)
    st = w2v.train_hs_epoch(model, to_dev(tv), p).cpu().numpy()
    assert list(st) == list(ost)
    g0, g1 = (t.cpu().numpy() for t in model.vectors())
    assert row_rel_err(g0, a0) <= 1e-4 and row_rel_err(g1[:s.voc.V - 1], a1) <= 1e-4


# Row strides of dim rounded up to 4 only (no padding past the lanes' last element group): every row
# access must stop at dim columns, or it reads and writes the next row. write_policy 5 and 1 take the
# store-only walk (buffer loads/stores) and the general one.
@pytest.mark.parametrize("dim,wp", [(300, 5), (300, 1), (100, 5), (452, 5), (60, 5)])
def test_packed_rows_match_oracle(w2v, dim, wp):
    s = oracle_side("sg_v30k_d100")
    voc = w2v.build_vocab(to_dev(s.tok), s.w.vocab, s.w.min_count)
    tree = w2v.build_huffman(voc.vocab_counts)
    tv = s.tv[:3000]
    syn0, syn1 = synth.init_weights(s.voc.V, dim, syn1_scale=0.5 / dim)
    a0, a1 = syn0.copy(), syn1.copy()
    op = oracle.params(s.voc.V, dim, window=5, sample=1e-3, train_words=s.voc.train_words, corpus_tokens=s.tv.size,
                       order=1, cache_k=31, flush_every=10)
    ost = oracle.train(a0, a1, s.tree, tv, op)
    model = w2v.make_model(syn0, syn1, voc, tree, stride=(dim + 3) // 4 * 4)
    p = w2v.Params(window=5, sample=1e-3, corpus_tokens=s.tv.size, workers=1, cache_k=31, flush_every=10,
                   write_policy=wp)
    st = w2v.train_hs_epoch(model, to_dev(tv), p).cpu().numpy()
    assert list(st) == list(ost)
    g0, g1 = (t.cpu().numpy() for t in model.vectors())
    assert row_rel_err(g0, a0) <= 1e-4 and row_rel_err(g1[:s.voc.V - 1], a1) <= 1e-4


# Padding columns are ignored: NaN there leaves the trained columns bit for bit as with zeros.
@pytest.mark.parametrize("wp,arch", [(5, 0), (1, 0), (5, 1), (5, 2)])
def test_padding_contents_are_ignored(w2v, wp, arch):
    s = oracle_side("sg_v30k_d100")
    voc = w2v.build_vocab(to_dev(s.tok), s.w.vocab, s.w.min_count)
    tree = w2v.build_huffman(voc.vocab_counts)
    tv = to_dev(s.tv[:4000])
    syn0, syn1 = synth.init_weights(s.voc.V, 300, syn1_scale=0.5 / 300)
    p = w2v.Params(window=5, sample=1e-3, corpus_tokens=s.tv.size, workers=1, cache_k=31, flush_every=10,
                   write_policy=wp, arch=arch)
    out = []
    for pad in (0.0, float("nan")):
        model = w2v.make_model(syn0, syn1, voc, tree, pad_value=pad)
        w2v.train_hs_epoch(model, tv, p)
        out.append([t.cpu().numpy() for t in model.vectors()])
    for a, b in zip(*out):
        np.testing.assert_array_equal(a, b)


# Cache sizes around the LDS budget at dim 300 (12 wavefronts of centre records, 24 KiB, plus 2 * k rows of
# 320 floats): k = 20 crosses the 64 KiB default launch limit only with the records counted, k = 54 is the
# largest that fits, k = 55 is refused.
@pytest.mark.parametrize("k", [20, 54, 55])
def test_cache_sizes_around_the_lds_budget(w2v, k):
    s = oracle_side("sg_v30k_d100")
    voc = w2v.build_vocab(to_dev(s.tok), s.w.vocab, s.w.min_count)
    tree = w2v.build_huffman(voc.vocab_counts)
    tv = s.tv[:2000]
    syn0, syn1 = synth.init_weights(s.voc.V, 300, syn1_scale=0.5 / 300)
    model = w2v.make_model(syn0, syn1, voc, tree)
    p = w2v.Params(window=5, sample=1e-3, corpus_tokens=s.tv.size, workers=1, cache_k=k, flush_every=10)
    if k == 55:
        with pytest.raises(w2v.W2VError) as e:
            w2v.train_hs_epoch(model, to_dev(tv), p)
        assert e.value.code == w2v.W2V_E_ARG and "LDS" in str(e.value)
        return
    a0, a1 = syn0.copy(), syn1.copy()
    op = oracle.params(s.voc.V, 300, window=5, sample=1e-3, train_words=s.voc.train_words, corpus_tokens=s.tv.size,
                       order=1, cache_k=k, flush_every=10)
    ost = oracle.train(a0, a1, s.tree, tv, op)
    st = w2v.train_hs_epoch(model, to_dev(tv), p).cpu().numpy()
    assert list(st) == list(ost)
    g0, g1 = (t.cpu().numpy() for t in model.vectors())
    assert row_rel_err(g0, a0) <= 1e-4 and row_rel_err(g1[:s.voc.V - 1], a1) <= 1e-4


def test_launch_resources_are_reported(w2v):
    s = oracle_side("sg_v30k_d100")
    voc, tree, syn0, syn1 = tiny_model(w2v, s, dim=300)
    model = w2v.make_model(syn0, syn1, voc, tree)
    w2v.train_hs_epoch(model, to_dev(s.tv[:20000]), w2v.Params(window=5, sample=1e-3, corpus_tokens=s.tv.size))
    r = w2v.last_train_resources()
    # dim 300: 12 wavefronts of 2 KiB records plus 2 * 31 cached rows of 320 floats
    assert r["lds_bytes_per_workgroup"] >= 12 * 2048 + 2 * 31 * 320 * 4
    assert 0 < r["vgprs"] <= 512 and 1 <= r["waves_per_simd"] <= 8


# Delta-only cache (cache_mode 1): LDS holds only the workgroup's change of each cached row, so twice as
# many rows fit; with one worker it is the same computation as the copy-and-original cache of the oracle.
@pytest.mark.parametrize("arch,k,dim,wp", [(0, 31, 100, 1), (0, 31, 300, 5), (0, 31, 300, 0), (1, 31, 300, 5),
                                           (2, 31, 100, 5), (0, 108, 300, 5), (0, 7, 64, 7)])
def test_delta_only_cache_single_worker_matches_oracle(w2v, arch, k, dim, wp):
    s = oracle_side("sg_v30k_d100")
    voc = w2v.build_vocab(to_dev(s.tok), s.w.vocab, s.w.min_count)
    tree = w2v.build_huffman(voc.vocab_counts)
    tv = s.tv[:3000]
    syn0, syn1 = synth.init_weights(s.voc.V, dim, syn1_scale=0.5 / dim)
    a0, a1 = syn0.copy(), syn1.copy()
    alpha0 = 0.05 if arch == 1 else 0.025
    # the reversed orientation is the oracle's pair-major order with its orientation flag
    order = dict(order=0, orient=1) if arch == 2 else dict(order=1, arch=arch)
    op = oracle.params(s.voc.V, dim, window=5, sample=1e-3, train_words=s.voc.train_words, corpus_tokens=s.tv.size,
                       cache_k=k, flush_every=10, alpha0=alpha0, **order)
    ost = oracle.train(a0, a1, s.tree, tv, op)
    model = w2v.make_model(syn0, syn1, voc, tree)
    p = w2v.Params(window=5, sample=1e-3, corpus_tokens=s.tv.size, workers=1, cache_k=k, flush_every=10,
                   write_policy=wp, arch=arch, alpha0=alpha0, cache_mode=1)
    st = w2v.train_hs_epoch(model, to_dev(tv), p).cpu().numpy()
    assert list(st) == list(ost)
    g0, g1 = (t.cpu().numpy() for t in model.vectors())
    assert row_rel_err(g0, a0) <= 1e-4 and row_rel_err(g1[:s.voc.V - 1], a1) <= 1e-4


def test_delta_only_cache_lds_budget(w2v):
    # dim 300: 12 x 2 KiB of centre records plus k rows of 320 floats; k = 109 no longer fits
    s = oracle_side("sg_v30k_d100")
    voc, tree, syn0, syn1 = tiny_model(w2v, s, dim=300)
    model = w2v.make_model(syn0, syn1, voc, tree)
    p = w2v.Params(window=5, sample=1e-3, corpus_tokens=s.tv.size, workers=1, cache_k=109, cache_mode=1)
    with pytest.raises(w2v.W2VError) as e:
        w2v.train_hs_epoch(model, to_dev(s.tv[:2000]), p)
    assert e.value.code == w2v.W2V_E_ARG and "LDS" in str(e.value)


def fib_counts():
    fib = [1, 1]
    while len(fib) < 65:
        fib.append(fib[-1] + fib[-2])
    return np.array(sorted(fib, reverse=True), np.int64)


# The deepest tree the 64-bit codes allow: Fibonacci counts over 65 words give paths of 1 to 64 inner
# nodes (one leaf at each depth up to 63, two at 64), so a path fills all 64 lanes of a wavefront and its
# last code bit is bit 63. Training on a stream that visits every word, and the log-likelihood of the
# trained model, match the oracle; the cache covers the top 31 of the 64 levels or none of them.
@pytest.mark.parametrize("dim,k,wp,arch", [(300, 31, 15, 0), (300, 31, 5, 0), (100, 7, 1, 0), (64, 0, 0, 0),
                                          (300, 31, 15, 1), (100, 31, 5, 2)])
def test_deepest_tree_matches_oracle(w2v, dim, k, wp, arch):
    counts = fib_counts()
    V = counts.size
    ot = oracle.build_huffman(counts)
    assert int(ot.codelen.max()) == 64
    tree = w2v.build_huffman(to_dev(counts))
    assert tree.max_len == 64
    np.testing.assert_array_equal(tree.code.cpu().numpy().view(np.uint64), ot.code)
    np.testing.assert_array_equal(tree.points.cpu().numpy(), ot.points)
    voc = types.SimpleNamespace(vocab_counts=to_dev(counts), train_words=int(counts.sum()))
    tv = np.random.default_rng(11).integers(0, V, 3000).astype(np.int32)
    syn0, syn1 = synth.init_weights(V, dim, syn1_scale=0.5 / dim)
    a0, a1 = syn0.copy(), syn1.copy()
    op = oracle.params(V, dim, window=5, sample=0.0, train_words=voc.train_words, corpus_tokens=tv.size,
                       cache_k=k, flush_every=10, order=0 if arch == 2 else 1, orient=1 if arch == 2 else 0,
                       arch=1 if arch == 1 else 0)
    ost = oracle.train(a0, a1, ot, tv, op)
    model = w2v.make_model(syn0, syn1, voc, tree)
    p = w2v.Params(window=5, sample=0.0, corpus_tokens=tv.size, cache_k=k, flush_every=10, workers=1,
                   write_policy=wp, arch=arch)
    st = w2v.train_hs_epoch(model, to_dev(tv), p).cpu().numpy()
    assert list(st) == list(ost)
    g0, g1 = (t.cpu().numpy() for t in model.vectors())
    assert row_rel_err(g0, a0) <= 1e-4 and row_rel_err(g1[:V - 1], a1) <= 1e-4
    # the held-out objective of the oracle's trained model, walked over the full 64-node paths
    pe = oracle.params(V, dim, window=5, sample=0.0, train_words=voc.train_words, seed=synth.SEED_EVAL,
                       arch=1 if arch == 1 else 0)
    so, npo, nno = oracle.loglik(a0, a1, ot, tv, pe)
    sg, npg, nng = w2v.hs_loglik(w2v.make_model(a0, a1, voc, tree), to_dev(tv),
                                 w2v.Params(window=5, sample=0.0, seed=synth.SEED_EVAL, arch=1 if arch == 1 else 0))
    assert (npg, nng) == (npo, nno)
    assert abs(sg - so) <= 1e-6 * abs(so)


# Synchronous mode on the deepest tree: batches of 32 centres against a snapshot, 64-node paths. (With
# batches of 256 over these 65 words every row takes dozens of summed changes per batch and the model
# diverges on both sides -- the oracle reaches 1e14 -- past the range of the GPU's fixed-point sums.)
@pytest.mark.parametrize("dim", [100, 300])
def test_deepest_tree_sync_mode_matches_oracle(w2v, dim):
    counts = fib_counts()
    V = counts.size
    ot = oracle.build_huffman(counts)
    tree = w2v.build_huffman(to_dev(counts))
    voc = types.SimpleNamespace(vocab_counts=to_dev(counts), train_words=int(counts.sum()))
    tv = np.random.default_rng(12).integers(0, V, 3000).astype(np.int32)
    syn0, syn1 = synth.init_weights(V, dim, syn1_scale=0.5 / dim)
    a0, a1 = syn0.copy(), syn1.copy()
    op = oracle.params(V, dim, window=5, sample=0.0, train_words=voc.train_words, corpus_tokens=tv.size,
                       sync_batch=32)
    ost = oracle.train_sync(a0, a1, ot, tv, op, n_batches=-1)
    assert np.abs(a0).max() < 10 and np.abs(a1).max() < 10   # a regime that does not diverge
    model = w2v.make_model(syn0, syn1, voc, tree)
    p = w2v.Params(window=5, sample=0.0, corpus_tokens=tv.size, mode=1, sync_batch=32)
    st = w2v.train_hs_epoch(model, to_dev(tv), p).cpu().numpy()
    assert list(st) == list(ost)
    g0, g1 = (t.cpu().numpy() for t in model.vectors())
    assert row_rel_err(g0, a0) <= 1e-4 and row_rel_err(g1[:V - 1], a1) <= 1e-4

