"""GPU parity: the HIP path (through the C ABI) against the CPU oracle.

Integer work (counts, vocabulary order, Huffman codes/points, keep thresholds,
sampled pairs) must match bit for bit. Floating-point work: synchronous-mode
embeddings within 1e-4 (row-wise relative, ∞-norm), a single sequential
worker within 1e-4 of the oracle's centre-major order, evaluation
log-likelihood within 1e-6 relative on the same model, and asynchronous
training's held-out log-likelihood within 1 % of the oracle's.
"""
import json
import math
import os

import numpy as np
import pytest

import oracle
import synth
from gpu_common import corpus, gated, ll_gate, log, oracle_side, row_rel_err

pytestmark = pytest.mark.gpu
GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


@pytest.fixture(scope="module")
def w2v():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_1606_07822_amd as w2v
    w2v.lib()
    return w2v


@pytest.fixture(scope="module")
def torch_mod():
    import torch
    return torch


def to_dev(a):
    import torch
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def gpu_side(w2v, side):
    voc = w2v.build_vocab(to_dev(side.tok), side.w.vocab, side.w.min_count)
    tree = w2v.build_huffman(voc.vocab_counts)
    return voc, tree


# ------------------------------------------------------------- vocabulary
@pytest.mark.parametrize("name,n", [("tiny_sg_v1k_d50", None), ("sg_v30k_d100", None), ("sg_v100k_d200", None)])
def test_vocab_bit_exact(w2v, name, n):
    log(f"vocab {name}")
    s = oracle_side(name, n)
    voc = w2v.build_vocab(to_dev(s.tok), s.w.vocab, s.w.min_count)
    assert voc.V == s.voc.V and voc.train_words == s.voc.train_words
    np.testing.assert_array_equal(voc.counts_by_id.cpu().numpy(), s.voc.counts)
    np.testing.assert_array_equal(voc.vocab_ids.cpu().numpy(), s.voc.vocab_ids)
    np.testing.assert_array_equal(voc.vocab_counts.cpu().numpy(), s.voc.vocab_counts)
    np.testing.assert_array_equal(voc.id_to_vocab.cpu().numpy(), s.voc.id_to_vocab)
    np.testing.assert_array_equal(voc.tokens.cpu().numpy(), s.tv)


@pytest.mark.parametrize("case", ["empty", "single_id", "min_count_0", "id_space_1", "ragged_big_space", "all_dropped",
                                  "lds_bin_edge", "unaligned_stream"])
def test_vocab_edge_cases(w2v, case):
    rng = np.random.default_rng(5)
    id_space, mc = 1000, 5
    offset = 0
    if case == "lds_bin_edge":
        # ids on both sides of the count kernel's LDS bins (36,864) and at the end of the id space
        id_space = 36_866
        tok = np.concatenate([rng.integers(36_860, 36_866, 50_000), rng.integers(0, 8, 50_000),
                              rng.integers(0, id_space, 1_001)]).astype(np.int32)
        rng.shuffle(tok)
    elif case == "unaligned_stream":
        # a stream that starts 4 bytes past a 16-byte boundary: the remap takes its one-token path
        tok = rng.integers(0, 300, 100_003).astype(np.int32)
        offset = 1
    elif case == "empty":
        tok = np.zeros(0, np.int32)
    elif case == "single_id":
        tok = np.full(777, 3, np.int32)
    elif case == "min_count_0":
        tok = rng.integers(0, 50, 300).astype(np.int32); mc = 0
    elif case == "id_space_1":
        tok = np.zeros(100, np.int32); id_space = 1
    elif case == "ragged_big_space":
        id_space = 3_000_017
        tok = (rng.zipf(1.1, 2_000_003) % id_space).astype(np.int32)
    else:
        tok = np.arange(1000, dtype=np.int32)
    if offset:
        dev = to_dev(np.concatenate([np.zeros(offset, np.int32), tok]))[offset:]
    else:
        dev = to_dev(tok) if tok.size else to_dev(np.zeros(1, np.int32))[:0]
    voc = w2v.build_vocab(dev, id_space, mc)
    o = oracle.build_vocab(tok, id_space, mc)
    assert voc.V == o.V and voc.train_words == o.train_words
    np.testing.assert_array_equal(voc.counts_by_id.cpu().numpy(), o.counts)
    np.testing.assert_array_equal(voc.vocab_ids.cpu().numpy(), o.vocab_ids)
    np.testing.assert_array_equal(voc.id_to_vocab.cpu().numpy(), o.id_to_vocab)
    np.testing.assert_array_equal(voc.tokens.cpu().numpy(), oracle.remap(tok, o.id_to_vocab))


def test_vocab_out_of_range_token_is_an_error(w2v):
    tok = np.array([0, 1, 2, 5000, 3], np.int32)
    with pytest.raises(w2v.W2VError) as e:
        w2v.build_vocab(to_dev(tok), 1000, 1)
    assert e.value.code == w2v.W2V_E_RANGE


# ------------------------------------------------------------- Huffman
def check_tree(w2v, counts):
    t = w2v.build_huffman(to_dev(counts))
    o = oracle.build_huffman(counts)
    np.testing.assert_array_equal(t.codelen.cpu().numpy(), o.codelen)
    np.testing.assert_array_equal(t.code.cpu().numpy().view(np.uint64), o.code)
    np.testing.assert_array_equal(t.point_off.cpu().numpy(), o.point_off)
    np.testing.assert_array_equal(t.points.cpu().numpy(), o.points)
    assert t.max_len == int(o.codelen.max())


@pytest.mark.parametrize("V,hi,seed", [(2, 10, 0), (3, 3, 1), (17, 5, 2), (1000, 4, 3), (4097, 100, 4),
                                       (50_000, 20, 5), (50_000, 10**6, 6)])
def test_huffman_random_counts_bit_exact(w2v, V, hi, seed):
    rng = np.random.default_rng(seed)
    check_tree(w2v, np.sort(rng.integers(1, hi, V))[::-1].astype(np.int64))


def test_huffman_equal_counts(w2v):
    check_tree(w2v, np.full(1 << 12, 9, np.int64))
    check_tree(w2v, np.full(5000, 5, np.int64))


@pytest.mark.parametrize("V,s,N", [(30_000, 1.0, 10**7), (100_000, 1.0, 10**8), (1_000_000, 1.05, 10**9)])
def test_huffman_zipf_vocab_bit_exact(w2v, V, s, N):
    log(f"huffman zipf V={V}")
    p = synth.zipf_probs(V, s)
    counts = np.maximum(np.floor(p * N), 5).astype(np.int64)
    counts = np.sort(counts)[::-1].copy()
    check_tree(w2v, counts)


def test_huffman_counts_out_of_order_is_an_error(w2v):
    with pytest.raises(w2v.W2VError) as e:
        w2v.build_huffman(to_dev(np.array([9, 7, 7, 8, 2], np.int64)))
    assert e.value.code == w2v.W2V_E_ARG


@pytest.mark.parametrize("V,seed", [(2049, 7), (4096 + 3, 8), (20_000, 9)])
def test_huffman_few_distinct_counts_bit_exact(w2v, V, seed):
    # long generations of equal counts: merges that span several chunks of the parallel merge
    rng = np.random.default_rng(seed)
    check_tree(w2v, np.sort(rng.choice([1, 2, 3, 5, 8, 1000], V))[::-1].astype(np.int64))


# Sizes around the parallel merge's chunk (2,048 picks) and count shapes that give long and short
# generations: uniform, few distinct values, geometric-like, heavy-tailed.
@pytest.mark.parametrize("case", range(24))
def test_huffman_varied_shapes_bit_exact(w2v, case):
    rng = np.random.default_rng(100 + case)
    V = [2, 3, 4, 1023, 1024, 1025, 2047, 2048, 2049, 4095, 4097, 6145][case % 12] if case < 12 else \
        int(rng.integers(2, 60_000))
    kind = case % 4
    if kind == 0:
        counts = rng.integers(1, 1000, V)
    elif kind == 1:
        counts = rng.choice([1, 1, 2, 3, 100], V)
    elif kind == 2:
        counts = np.floor(1.5 ** rng.uniform(0, 40, V)).astype(np.int64) + 1
    else:
        counts = np.floor(1e6 / rng.pareto(1.1, V).clip(1e-3)).astype(np.int64) + 1
    check_tree(w2v, np.sort(counts.astype(np.int64))[::-1].copy())


def test_huffman_too_deep_is_an_error(w2v):
    fib = [1, 1]
    while len(fib) < 70:
        fib.append(fib[-1] + fib[-2])
    with pytest.raises(w2v.W2VError) as e:
        w2v.build_huffman(to_dev(np.array(sorted(fib, reverse=True), np.int64)))
    assert e.value.code == w2v.W2V_E_RANGE


# ------------------------------------------------------------- sampling
@pytest.mark.parametrize("name,t", [("sg_v30k_d100", 1e-3), ("sg_v100k_d200", 1e-4), ("sg_v100k_d200", 1e-5)])
def test_keep_thresholds_bit_exact(w2v, name, t):
    s = oracle_side(name)
    thr = w2v.keep_thresholds(to_dev(s.voc.vocab_counts), t, s.voc.train_words).cpu().numpy().view(np.uint64)
    np.testing.assert_array_equal(thr, oracle.keep_thresholds(s.voc.vocab_counts, t, s.voc.train_words))


def pairs_both(w2v, s, tv, **kw):
    p = w2v.Params(window=kw.get("window", s.w.window), sample=kw.get("sample", s.w.sample),
                   doc_len=kw.get("doc_len", 1000), seed=kw.get("seed", 3), epoch=kw.get("epoch", 0),
                   first_raw_index=kw.get("first", 0))
    op = oracle.params(s.voc.V, 8, window=p.window, sample=p.sample, train_words=s.voc.train_words,
                       doc_len=p.doc_len, seed=p.seed, epoch=p.epoch, first_raw_index=p.first_raw_index)
    cap = kw.get("cap", None)
    o = oracle.sample_pairs(tv, op, s.voc.vocab_counts, cap=cap)
    g = w2v.sample_pairs(to_dev(tv), s.voc.V, to_dev(s.voc.vocab_counts), s.voc.train_words, p,
                         cap=o.total if cap is None else cap, want_mask=True)
    return o, g


@pytest.mark.parametrize("name,n,kw", [
    ("tiny_sg_v1k_d50", None, {}),
    ("tiny_sg_v1k_d50", None, dict(window=1)),
    ("tiny_sg_v1k_d50", None, dict(window=10, doc_len=333)),
    ("sg_v30k_d100", 2_000_500, {}),                     # ragged last document
    ("sg_v30k_d100", 2_000_000, dict(first=7_000_000, epoch=2, seed=11)),
    # raw positions past 2^32 (the counter's high word) and the longest documents the 16-bit offsets hold
    ("sg_v30k_d100", 1_000_000, dict(first=6_000_000_000, epoch=1, seed=5)),
    ("sg_v30k_d100", 400_000, dict(doc_len=65535, first=65535 * 70_000)),
])
def test_pairs_bit_exact(w2v, name, n, kw):
    s = oracle_side(name)
    tv = s.tv[:n] if n else s.tv
    o, g = pairs_both(w2v, s, tv, **kw)
    assert g.total == o.total and g.n_kept == o.n_kept and g.checksum == o.checksum
    np.testing.assert_array_equal(g.keep_mask.cpu().numpy(), o.keep_mask)
    np.testing.assert_array_equal(g.centre.cpu().numpy(), o.centre)
    np.testing.assert_array_equal(g.context.cpu().numpy(), o.context)


@pytest.mark.parametrize("name", ["sg_v30k_d100", "sg_v100k_d200"])
def test_pairs_checksum_full_corpus(w2v, name):
    log(f"pairs checksum {name}")
    s = oracle_side(name)
    o, g = pairs_both(w2v, s, s.tv, cap=0)
    assert (g.total, g.n_kept, g.checksum) == (o.total, o.n_kept, o.checksum)


# ------------------------------------------------------------- evaluation
# d = 100, 300 and 600 take the kernels with 2, 5 and 10 elements per lane; window 5 and 10 put up to 10
# and 20 words in a centre's window, more than one group of words for the d = 300 kernel (8 per walk)
@pytest.mark.parametrize("dim,window,n_held", [(100, 5, None), (300, 5, 200_000), (300, 10, 200_000),
                                                (600, 5, 200_000)])
def test_loglik_matches_oracle_on_the_same_model(w2v, dim, window, n_held):
    log(f"loglik d={dim} window={window}")
    s = oracle_side("sg_v30k_d100")
    voc, tree = gpu_side(w2v, s)
    syn0, syn1 = synth.init_weights(s.voc.V, dim, syn1_scale=30.0 / math.sqrt(dim))
    syn0 = syn0 * np.float32(dim / 5)   # entries up to 0.1: dot products of order 1 at every d
    model = w2v.make_model(syn0, syn1, voc, tree)
    held = corpus("sg_v30k_d100", heldout=True)[:n_held]
    hv = oracle.remap(held, s.voc.id_to_vocab)
    p = w2v.Params(window=window, sample=1e-3, seed=synth.SEED_EVAL)
    sg, npg, nng = w2v.hs_loglik(model, to_dev(hv), p)
    op = oracle.params(s.voc.V, dim, window=window, sample=1e-3, train_words=s.voc.train_words,
                       seed=synth.SEED_EVAL)
    so, npo, nno = oracle.loglik(syn0, syn1, s.tree, hv, op)
    assert (npg, nng) == (npo, nno)
    assert abs(sg - so) <= 1e-6 * abs(so)


# CBOW's objective (§2's softmax with the mean of the window vectors as input): one term per centre
# with a window; h is summed in the same order on both sides, so only the fp64 dot products and the
# logarithms differ in rounding. d = 300 covers five elements per lane with a ragged last one.
@pytest.mark.parametrize("name,n,scale", [("tiny_sg_v1k_d50", None, 0.3), ("sg_v30k_d100", 2_000_000, 0.3),
                                          ("cbow_v100k_d300", 2_000_000, 0.05)])
def test_loglik_cbow_matches_oracle_on_the_same_model(w2v, name, n, scale):
    s = oracle_side(name, n)
    voc, tree = gpu_side(w2v, s)
    syn0, syn1 = synth.init_weights(s.voc.V, s.w.dim, syn1_scale=scale)
    syn0 *= 20.0                                    # words far from zero, so h carries weight
    model = w2v.make_model(syn0, syn1, voc, tree)
    hv = oracle.remap(corpus(name, heldout=True), s.voc.id_to_vocab)[:300_000]
    p = w2v.Params(window=s.w.window, sample=s.w.sample, seed=synth.SEED_EVAL, arch=1)
    sg, ng, nng = w2v.hs_loglik(model, to_dev(hv), p)
    op = oracle.params(s.voc.V, s.w.dim, window=s.w.window, sample=s.w.sample, train_words=s.voc.train_words,
                       seed=synth.SEED_EVAL, arch=1)
    so, no, nno = oracle.loglik(syn0, syn1, s.tree, hv, op)
    log(f"  CBOW LL {name}: gpu {sg / ng:.9f} oracle {so / no:.9f} over {ng} centres")
    assert (ng, nng) == (no, nno) and ng > 0
    assert abs(sg - so) <= 1e-9 * abs(so)
    # the pairs' objective on the same stream counts more terms (every window word of a centre)
    _, npairs, _ = w2v.hs_loglik(model, to_dev(hv), w2v.Params(window=s.w.window, sample=s.w.sample,
                                                               seed=synth.SEED_EVAL))
    assert npairs > ng


def test_loglik_cbow_at_zero_syn1_closed_form(w2v):
    s = oracle_side("tiny_sg_v1k_d50")
    voc, tree = gpu_side(w2v, s)
    syn0, syn1 = synth.init_weights(s.voc.V, s.w.dim)
    model = w2v.make_model(syn0, syn1, voc, tree)
    sg, nc, nnodes = w2v.hs_loglik(model, voc.tokens, w2v.Params(window=2, seed=4, arch=1))
    assert nc > 0
    assert abs(sg + math.log(2.0) * nnodes) <= 1e-9 * nnodes


def test_loglik_at_zero_syn1_closed_form(w2v):
    s = oracle_side("tiny_sg_v1k_d50")
    voc, tree = gpu_side(w2v, s)
    syn0, syn1 = synth.init_weights(s.voc.V, s.w.dim)
    model = w2v.make_model(syn0, syn1, voc, tree)
    sg, npairs, nnodes = w2v.hs_loglik(model, voc.tokens, w2v.Params(window=2, seed=4))
    assert npairs > 0
    assert abs(sg + math.log(2.0) * nnodes) <= 1e-9 * nnodes


# ------------------------------------------------------------- synchronous mode
# Batches of >= 1024 centres at alpha 0.025 diverge within ten batches (the oracle too: the top
# inner nodes take the whole batch's gradient at once), so the ten-batch cases use 256 centres.
@pytest.mark.parametrize("name,n,batches,B", [("tiny_sg_v1k_d50", None, 1, 4096), ("tiny_sg_v1k_d50", None, 10, 256),
                                              ("sg_v30k_d100", 1_000_000, 1, 4096),
                                              ("sg_v30k_d100", 1_000_000, 10, 256),
                                              ("tiny_sg_v1k_d50", 20_000, 3, 1)])
def test_sync_mode_within_1e4(w2v, name, n, batches, B):
    log(f"sync {name} batches={batches}")
    s = oracle_side(name)
    nk_needed = batches * B
    # the token prefix holding exactly `batches` batches of kept centres (whole documents past it are cut)
    tv = s.tv if n is None else s.tv[:n]
    voc, tree = gpu_side(w2v, s)
    syn0, syn1 = synth.init_weights(s.voc.V, s.w.dim, syn1_scale=0.5 / s.w.dim)
    # GPU runs every batch of tv; the oracle stops after `batches`: cut tv so both see the same batches
    op = oracle.params(s.voc.V, s.w.dim, window=s.w.window, sample=s.w.sample, train_words=s.voc.train_words,
                       corpus_tokens=s.tv.size, sync_batch=B)
    pr = oracle.sample_pairs(tv, op, s.voc.vocab_counts, cap=0)
    kept_prefix = np.cumsum(pr.keep_mask)
    cut = int(np.searchsorted(kept_prefix, nk_needed)) + 1 if kept_prefix[-1] > nk_needed else tv.size
    tv = tv[:cut]
    a0, a1 = syn0.copy(), syn1.copy()
    ost = oracle.train_sync(a0, a1, s.tree, tv, op, n_batches=-1)
    model = w2v.make_model(syn0, syn1, voc, tree)
    p = w2v.Params(window=s.w.window, sample=s.w.sample, corpus_tokens=s.tv.size, mode=1, sync_batch=B)
    st = w2v.train_hs_epoch(model, to_dev(tv), p).cpu().numpy()
    assert list(st) == list(ost)
    g0, g1 = (t.cpu().numpy() for t in model.vectors())
    g1 = g1[:s.voc.V - 1]
    assert row_rel_err(g0, a0) <= 1e-4
    assert row_rel_err(g1, a1) <= 1e-4
    # rows no pair touched are bit-identical
    np.testing.assert_array_equal(g0[(a0 == syn0).all(1)], syn0[(a0 == syn0).all(1)])


def test_sync_mode_is_deterministic(w2v):
    s = oracle_side("tiny_sg_v1k_d50")
    voc, tree = gpu_side(w2v, s)
    syn0, syn1 = synth.init_weights(s.voc.V, s.w.dim, syn1_scale=0.01)
    outs = []
    for _ in range(2):
        model = w2v.make_model(syn0, syn1, voc, tree)
        w2v.train_hs_epoch(model, voc.tokens, w2v.Params(window=2, corpus_tokens=s.tv.size, mode=1, sync_batch=512))
        outs.append([t.cpu().numpy() for t in model.vectors()])
    np.testing.assert_array_equal(outs[0][0], outs[1][0])
    np.testing.assert_array_equal(outs[0][1], outs[1][1])


# ------------------------------------------------------------- asynchronous mode
# One wavefront reproduces the oracle's centre-major order up to rounding. dim picks the kernel variant
# (elements per lane 2, 4, 5, 8, 16; up to 256 columns every chunk is prefetched, above only past the
# cached prefix); write_policy 0 (atomic adds of the change), 1 (row stores) and 5 (row stores, cached rows
# included) take different write-back paths, 7 and 2 store word vectors too (a word repeated in a window adds
# atomically); window 10 gives skip-gram windows wider than one register group at dim >= 200 (parked gradients).
@pytest.mark.parametrize("arch,k,F,ndocs,dim,wp,win", [
    (0, 0, 10, 5, 100, 1, 5), (0, 31, 10, 5, 100, 1, 5), (0, 7, 1, 5, 100, 1, 5), (1, 0, 10, 5, 100, 1, 5),
    (1, 31, 10, 5, 100, 1, 5),
    (0, 0, 10, 3, 300, 1, 5), (0, 31, 10, 3, 300, 1, 5), (0, 31, 10, 3, 300, 0, 5), (1, 0, 10, 3, 300, 1, 5),
    (1, 31, 10, 3, 300, 1, 5), (1, 31, 10, 3, 300, 0, 5),
    (0, 31, 10, 2, 300, 1, 10), (0, 31, 10, 2, 300, 0, 10), (1, 31, 10, 2, 300, 1, 10),
    (0, 31, 10, 2, 200, 1, 10), (0, 31, 10, 2, 450, 1, 5), (1, 31, 10, 2, 450, 1, 5), (0, 31, 10, 2, 600, 1, 5),
    (1, 31, 10, 2, 600, 1, 5), (0, 15, 10, 2, 1024, 0, 3),
    (0, 31, 10, 5, 100, 5, 5), (0, 31, 10, 3, 300, 5, 5), (0, 31, 10, 2, 300, 5, 10), (1, 31, 10, 3, 300, 5, 5),
    (0, 31, 10, 2, 450, 5, 5),
    (0, 31, 10, 5, 100, 7, 5), (0, 31, 10, 5, 300, 7, 5), (0, 0, 10, 3, 300, 2, 5), (1, 31, 10, 3, 300, 7, 5),
])
def test_single_worker_matches_oracle_centre_major(w2v, arch, k, F, ndocs, dim, wp, win):
    log(f"single worker arch={arch} k={k} F={F} docs={ndocs} dim={dim} write_policy={wp} window={win}")
    s = oracle_side("sg_v30k_d100")
    voc, tree = gpu_side(w2v, s)
    tv = s.tv[:ndocs * 1000]
    syn0, syn1 = synth.init_weights(s.voc.V, dim, syn1_scale=0.5 / dim)
    a0, a1 = syn0.copy(), syn1.copy()
    alpha0 = 0.05 if arch else 0.025
    op = oracle.params(s.voc.V, dim, window=win, sample=1e-3, train_words=s.voc.train_words,
                       corpus_tokens=s.tv.size, cache_k=k, flush_every=F, order=1, arch=arch, alpha0=alpha0)
    ost = oracle.train(a0, a1, s.tree, tv, op)
    model = w2v.make_model(syn0, syn1, voc, tree)
    p = w2v.Params(window=win, sample=1e-3, corpus_tokens=s.tv.size, cache_k=k, flush_every=F, workers=1, arch=arch,
                   alpha0=alpha0, write_policy=wp)
    st = w2v.train_hs_epoch(model, to_dev(tv), p).cpu().numpy()
    assert list(st) == list(ost)
    g0, g1 = (t.cpu().numpy() for t in model.vectors())
    assert row_rel_err(g0, a0) <= 1e-4
    assert row_rel_err(g1[:s.voc.V - 1], a1) <= 1e-4


# write_policy 15 keeps word rows in registers across consecutive centres (skip-gram and CBOW, rows of 129 to
# 512 floats, window <= 5; skip-gram <= 2 above 320 floats); one wavefront still reproduces the centre-major
# oracle. The
# 1e3-word corpus without subsampling repeats its frequent words within most spans of ten kept positions
# (the slots holding one word are kept equal); window 10 at dim 300 and rows of 128 floats or fewer fall
# back to the per-centre path (the bit is ignored there).
@pytest.mark.parametrize("arch", [0, 1])
@pytest.mark.parametrize("name,sample,k,F,ndocs,dim,win", [
    ("sg_v30k_d100", 1e-3, 31, 10, 3, 300, 5), ("sg_v30k_d100", 1e-3, 0, 10, 3, 300, 5),
    ("sg_v30k_d100", 1e-3, 31, 1, 3, 300, 3), ("sg_v30k_d100", 1e-3, 31, 10, 3, 200, 5),
    ("sg_v30k_d100", 1e-3, 31, 10, 2, 450, 2), ("sg_v30k_d100", 1e-3, 31, 10, 2, 256, 1),
    ("sg_v30k_d100", 1e-3, 31, 10, 2, 300, 10), ("sg_v30k_d100", 1e-3, 31, 10, 3, 100, 5),
    ("tiny_sg_v1k_d50", 0.0, 31, 10, 4, 300, 5), ("tiny_sg_v1k_d50", 0.0, 7, 3, 4, 200, 4),
    ("tiny_sg_v1k_d50", 0.0, 0, 10, 3, 450, 2), ("tiny_sg_v1k_d50", 0.0, 31, 10, 3, 50, 5),
    ("tiny_sg_v1k_d50", 0.0, 31, 10, 3, 150, 3), ("sg_v30k_d100", 1e-3, 31, 10, 3, 64, 5),
])
def test_single_worker_word_rows_kept_across_centres(w2v, arch, name, sample, k, F, ndocs, dim, win):
    log(f"word rows kept across centres arch={arch} {name} t={sample} k={k} F={F} docs={ndocs} dim={dim} "
        f"window={win}")
    s = oracle_side(name)
    voc, tree = gpu_side(w2v, s)
    tv = s.tv[:ndocs * 1000]
    syn0, syn1 = synth.init_weights(s.voc.V, dim, syn1_scale=0.5 / dim)
    a0, a1 = syn0.copy(), syn1.copy()
    alpha0 = 0.05 if arch else 0.025
    op = oracle.params(s.voc.V, dim, window=win, sample=sample, train_words=s.voc.train_words,
                       corpus_tokens=s.tv.size, cache_k=k, flush_every=F, order=1, arch=arch, alpha0=alpha0)
    ost = oracle.train(a0, a1, s.tree, tv, op)
    model = w2v.make_model(syn0, syn1, voc, tree)
    p = w2v.Params(window=win, sample=sample, corpus_tokens=s.tv.size, cache_k=k, flush_every=F, workers=1,
                   write_policy=15, arch=arch, alpha0=alpha0)
    st = w2v.train_hs_epoch(model, to_dev(tv), p).cpu().numpy()
    assert list(st) == list(ost)
    g0, g1 = (t.cpu().numpy() for t in model.vectors())
    assert row_rel_err(g0, a0) <= 1e-4
    assert row_rel_err(g1[:s.voc.V - 1], a1) <= 1e-4
    untouched = np.all(a0 == syn0, axis=1)
    np.testing.assert_array_equal(g0[untouched], syn0[untouched])


# CBOW with the word-row span takes hot_k 0 by default (the store-only walk); with hot rows that take atomic
# adds it walks the general path, which one worker must match too.
@pytest.mark.parametrize("name,sample,k,dim", [
    ("tiny_sg_v1k_d50", 0.0, 31, 300), ("sg_v30k_d100", 1e-3, 31, 300), ("sg_v30k_d100", 1e-3, 0, 256),
])
def test_single_worker_cbow_span_with_hot_rows(w2v, name, sample, k, dim):
    log(f"CBOW span with hot rows {name} t={sample} k={k} dim={dim}")
    s = oracle_side(name)
    voc, tree = gpu_side(w2v, s)
    tv = s.tv[:3000]
    syn0, syn1 = synth.init_weights(s.voc.V, dim, syn1_scale=0.5 / dim)
    a0, a1 = syn0.copy(), syn1.copy()
    op = oracle.params(s.voc.V, dim, window=5, sample=sample, train_words=s.voc.train_words,
                       corpus_tokens=s.tv.size, cache_k=k, flush_every=10, order=1, arch=1, alpha0=0.05)
    ost = oracle.train(a0, a1, s.tree, tv, op)
    model = w2v.make_model(syn0, syn1, voc, tree)
    p = w2v.Params(window=5, sample=sample, corpus_tokens=s.tv.size, cache_k=k, flush_every=10, workers=1,
                   write_policy=15, arch=1, alpha0=0.05, hot_k=1024)
    assert w2v.train_word_span(model, p) == 5
    st = w2v.train_hs_epoch(model, to_dev(tv), p).cpu().numpy()
    assert list(st) == list(ost)
    g0, g1 = (t.cpu().numpy() for t in model.vectors())
    assert row_rel_err(g0, a0) <= 1e-4 and row_rel_err(g1[:s.voc.V - 1], a1) <= 1e-4


# With span_stash the row of the word that becomes the next centre waits in LDS and re-enters the span from
# there; one wavefront holds the only copy that changes, so it still reproduces the centre-major oracle
# (repeated words included: the tiny corpus without subsampling repeats words in most spans).
@pytest.mark.parametrize("arch,name,sample,k,dim,sfrom", [
    (0, "tiny_sg_v1k_d50", 0.0, 31, 300, 0), (0, "sg_v30k_d100", 1e-3, 31, 300, 0), (0, "sg_v30k_d100", 1e-3, 0, 200, 0),
    (1, "tiny_sg_v1k_d50", 0.0, 31, 300, 0), (0, "tiny_sg_v1k_d50", 0.0, 54, 300, 0),
    (0, "tiny_sg_v1k_d50", 0.0, 31, 300, 40), (0, "sg_v30k_d100", 1e-3, 31, 300, 2000),
    # the benchmark's LDS: 48 cached rows and their originals beside the centre records and the stash
    (0, "sg_v30k_d100", 1e-3, 48, 300, 2000), (1, "sg_v30k_d100", 1e-3, 48, 300, 0),
])
def test_single_worker_span_stash_matches_oracle(w2v, arch, name, sample, k, dim, sfrom):
    log(f"span stash arch={arch} {name} t={sample} k={k} dim={dim} from={sfrom}")
    s = oracle_side(name)
    voc, tree = gpu_side(w2v, s)
    tv = s.tv[:3000]
    syn0, syn1 = synth.init_weights(s.voc.V, dim, syn1_scale=0.5 / dim)
    alpha0 = 0.05 if arch else 0.025
    a0, a1 = syn0.copy(), syn1.copy()
    op = oracle.params(s.voc.V, dim, window=5, sample=sample, train_words=s.voc.train_words,
                       corpus_tokens=s.tv.size, cache_k=k, flush_every=10, order=1, arch=arch, alpha0=alpha0)
    ost = oracle.train(a0, a1, s.tree, tv, op)
    model = w2v.make_model(syn0, syn1, voc, tree)
    p = w2v.Params(window=5, sample=sample, corpus_tokens=s.tv.size, cache_k=k, flush_every=10, workers=1,
                   write_policy=15, arch=arch, alpha0=alpha0, span_stash=1, stash_from=sfrom)
    assert w2v.train_word_span(model, p) == 5
    st = w2v.train_hs_epoch(model, to_dev(tv), p).cpu().numpy()
    assert list(st) == list(ost)
    g0, g1 = (t.cpu().numpy() for t in model.vectors())
    assert row_rel_err(g0, a0) <= 1e-4 and row_rel_err(g1[:s.voc.V - 1], a1) <= 1e-4


# span_refresh writes the span's frequent words back and reads them again after every centre. One wavefront
# reads what it wrote, so it still reproduces the centre-major oracle; the result can differ from the run
# without it in rounding only (slots holding the same word take each other's changes in different orders, and
# the refresh decides which slot's rounding is kept).
@pytest.mark.parametrize("arch,name,sample,dim,refresh", [
    (0, "tiny_sg_v1k_d50", 0.0, 300, 10), (0, "tiny_sg_v1k_d50", 0.0, 300, 10**6), (0, "sg_v30k_d100", 1e-3, 200, 500),
    (1, "tiny_sg_v1k_d50", 0.0, 300, 50),
])
def test_span_refresh_single_worker_matches_oracle(w2v, arch, name, sample, dim, refresh):
    log(f"span refresh arch={arch} {name} dim={dim} refresh={refresh}")
    s = oracle_side(name)
    voc, tree = gpu_side(w2v, s)
    tv = s.tv[:3000]
    syn0, syn1 = synth.init_weights(s.voc.V, dim, syn1_scale=0.5 / dim)
    alpha0 = 0.05 if arch else 0.025
    a0, a1 = syn0.copy(), syn1.copy()
    op = oracle.params(s.voc.V, dim, window=5, sample=sample, train_words=s.voc.train_words,
                       corpus_tokens=s.tv.size, cache_k=31, flush_every=10, order=1, arch=arch, alpha0=alpha0)
    ost = oracle.train(a0, a1, s.tree, tv, op)
    out = []
    for r in (0, refresh):
        model = w2v.make_model(syn0, syn1, voc, tree)
        p = w2v.Params(window=5, sample=sample, corpus_tokens=s.tv.size, cache_k=31, flush_every=10, workers=1,
                       write_policy=15, arch=arch, alpha0=alpha0, span_refresh=r)
        assert w2v.train_word_span(model, p) == 5
        st = w2v.train_hs_epoch(model, to_dev(tv), p).cpu().numpy()
        assert list(st) == list(ost)
        g0, g1 = (t.cpu().numpy() for t in model.vectors())
        assert row_rel_err(g0, a0) <= 1e-4 and row_rel_err(g1[:s.voc.V - 1], a1) <= 1e-4
        out.append((g0, g1))
    assert row_rel_err(out[1][0], out[0][0]) <= 1e-5


def same_vocab_and_tree(voc, tree, s):
    # the inputs of an asynchronous run are deterministic: a quality miss is then the training's own
    np.testing.assert_array_equal(voc.id_to_vocab.cpu().numpy(), s.voc.id_to_vocab)
    np.testing.assert_array_equal(voc.vocab_counts.cpu().numpy(), s.voc.vocab_counts)
    np.testing.assert_array_equal(tree.code.cpu().numpy().view(np.uint64), s.tree.code)
    np.testing.assert_array_equal(tree.points.cpu().numpy(), s.tree.points)


def async_ll(w2v, s, held, **kw):
    voc, tree = gpu_side(w2v, s)
    same_vocab_and_tree(voc, tree, s)
    syn0, syn1 = synth.init_weights(s.voc.V, s.w.dim)
    model = w2v.make_model(syn0, syn1, voc, tree)
    p = w2v.Params(window=s.w.window, sample=s.w.sample, corpus_tokens=s.tv.size, arch=s.w.arch, alpha0=s.w.alpha0,
                   **kw)
    w2v.train_hs_epoch(model, voc.tokens, p)
    hv = to_dev(oracle.remap(held, s.voc.id_to_vocab))
    sg, npairs, _ = w2v.hs_loglik(model, hv, w2v.Params(window=s.w.window, sample=s.w.sample, seed=synth.SEED_EVAL,
                                                        arch=s.w.arch))
    return sg / npairs, npairs


@pytest.mark.parametrize("kw", [dict(cache_k=0), dict(cache_k=31, flush_every=10, flush_policy=0, write_policy=0),
                                dict(cache_k=31), dict(cache_k=31, write_policy=0)])
def test_async_loglik_within_1pct_tiny(w2v, kw):
    s = oracle_side("tiny_sg_v1k_d50")
    held = corpus("tiny_sg_v1k_d50", heldout=True)
    syn0, syn1 = synth.init_weights(s.voc.V, s.w.dim)
    op = oracle.params(s.voc.V, s.w.dim, window=2, train_words=s.voc.train_words, corpus_tokens=s.tv.size,
                       cache_k=31, flush_every=10)
    oracle.train(syn0, syn1, s.tree, s.tv, op)
    hv = oracle.remap(held, s.voc.id_to_vocab)
    pe = oracle.params(s.voc.V, s.w.dim, window=2, train_words=s.voc.train_words, seed=4)
    s0, _, _ = oracle.loglik(*synth.init_weights(s.voc.V, s.w.dim), s.tree, hv, pe)
    so, npo, _ = oracle.loglik(syn0, syn1, s.tree, hv, pe)

    def run():
        g, npg = async_ll(w2v, s, held, **kw)
        assert npg == npo
        return g

    gated(run, so / npo, s0 / npo)


def golden(name):
    path = os.path.join(GOLDEN, f"oracle_ll_{name}.json")
    if not os.path.exists(path):
        pytest.skip(f"no stored oracle result {path}")
    return json.load(open(path))


# Every case must also keep at least 0.9 of the oracle's gain over the untrained model (the 1 % bound alone
# would let the 1e7-token workload lose 62 % of it). Default asynchronous mode (top-31 cache in LDS, write-back of the workgroups' averaged change every
# 1000 centres, Hogwild row stores in HBM and in the LDS copy) at full occupancy; the same with atomic adds
# of the change everywhere (write_policy 0) or in LDS only (1); no cache; and the cache with the paper's
# summed write-back, which is stable only at low concurrency (256 wavefronts). CBOW's default also adds
# the change atomically on the 1024 hot rows below the cache. write_policy 7 (word rows stored too) is
# the benchmark's setting; cache_mode 1 the delta-only cache.
@pytest.mark.parametrize("name,kw,min_frac", [
    ("sg_v30k_d100", {}, 0.9),
    ("sg_v30k_d100", dict(write_policy=7), 0.9),
    ("sg_v30k_d100", dict(write_policy=0), 0.9),
    ("sg_v30k_d100", dict(write_policy=1), 0.9),
    ("sg_v30k_d100", dict(cache_k=0), 0.9),
    ("sg_v30k_d100", dict(workers=256, cache_k=31, flush_every=10, flush_policy=0, write_policy=0), 0.9),
    ("sg_v30k_d100", dict(cache_mode=1), 0.9),
    ("sg_v30k_d100", dict(cache_mode=1, cache_k=63, flush_every=100), 0.9),
    ("sg_v100k_d200", {}, 0.9),
    ("sg_v100k_d200", dict(write_policy=0), 0.9),
    ("sg_v100k_d200", dict(write_policy=1), 0.9),
    ("sg_v100k_d200", dict(write_policy=7), 0.9),
    ("sg_v100k_d200", dict(write_policy=15), 0.9),
    ("sg_v100k_d200", dict(write_policy=15, span_stash=1), 0.9),
    ("sg_v100k_d200", dict(cache_mode=1), 0.9),
    ("cbow_v100k_d300", {}, 0.9),
    ("cbow_v100k_d300", dict(write_policy=7), 0.9),
    ("cbow_v100k_d300", dict(write_policy=15), 0.9),
    ("cbow_v100k_d300", dict(write_policy=15, span_stash=1), 0.9),
    ("cbow_v100k_d300", dict(write_policy=15, hot_k=1024), 0.9),
])
def test_async_loglik_within_1pct_of_stored_oracle(w2v, name, kw, min_frac):
    log(f"async LL {name} {kw}")
    gold = golden(name)
    s = oracle_side(name)
    assert s.voc.V == gold["V"] and s.voc.train_words == gold["train_words"]
    held = corpus(name, heldout=True)

    def run():
        g, npg = async_ll(w2v, s, held, **kw)
        assert npg == gold["heldout_pairs"]
        return g

    gated(run, gold["mean_ll"], gold["init_mean_ll"], min_frac)


# ------------------------------------------------------------- memory probe
def test_probe_rows_read_modify_write_counts(w2v, torch_mod):
    from bench_probe import probe_rows
    torch = torch_mod
    # 1 workgroup = 12 wavefronts x 4 rows x iters visits, each adding 1 to the first cols floats of a row;
    # the adds are plain read-modify-writes, so two visits of one row at the same time may count once
    m = torch.zeros(1000, 320, dtype=torch.float32, device="cuda")
    ms = probe_rows(m, 300, mode=1, workgroups=1, iters=3)
    assert ms > 0
    h = m.cpu().numpy()
    assert h[:, 300:].sum() == 0
    assert np.all(h == np.round(h)) and h.min() >= 0
    visits = 12 * 4 * 3
    assert 0.8 * visits * 300 <= h.sum() <= visits * 300
    ms = probe_rows(m, 300, mode=0, workgroups=2, iters=2)
    assert ms > 0 and m.cpu().numpy().sum() == h.sum()   # reads leave the matrix alone
    ms = probe_rows(m, 300, mode=2, workgroups=2, iters=100)
    assert ms > 0 and m.cpu().numpy().sum() == h.sum()
    # streaming write: 2 workgroups x 12 wavefronts x 4 rows x 11 rounds cover rows 0..1055, clipped to 1000;
    # round i writes the value i
    m.zero_()
    probe_rows(m, 320, mode=3, workgroups=2, iters=11)
    h = m.cpu().numpy()
    rows = np.arange(1000)
    assert np.array_equal(h, np.repeat(((rows // 4) % 11).astype(np.float32)[:, None], 320, axis=1))


# ------------------------------------------------------------- reversed orientation, several epochs
# arch 2: each window word's path is walked with the centre's vector as input, which takes each pair's
# gradient before the next pair -- the oracle's pair-major order with the orientation flag, exactly.
@pytest.mark.parametrize("k,dim,wp,win", [(0, 100, 1, 5), (31, 100, 1, 5), (31, 300, 5, 5), (31, 300, 0, 5),
                                          (7, 200, 5, 10), (31, 600, 5, 3)])
def test_single_worker_reversed_orientation(w2v, k, dim, wp, win):
    log(f"single worker reversed k={k} dim={dim} write_policy={wp} window={win}")
    s = oracle_side("sg_v30k_d100")
    voc, tree = gpu_side(w2v, s)
    tv = s.tv[:3000]
    syn0, syn1 = synth.init_weights(s.voc.V, dim, syn1_scale=0.5 / dim)
    a0, a1 = syn0.copy(), syn1.copy()
    op = oracle.params(s.voc.V, dim, window=win, sample=1e-3, train_words=s.voc.train_words,
                       corpus_tokens=s.tv.size, cache_k=k, flush_every=10, order=0, orient=1)
    ost = oracle.train(a0, a1, s.tree, tv, op)
    model = w2v.make_model(syn0, syn1, voc, tree)
    p = w2v.Params(window=win, sample=1e-3, corpus_tokens=s.tv.size, cache_k=k, flush_every=10, workers=1, arch=2,
                   write_policy=wp)
    st = w2v.train_hs_epoch(model, to_dev(tv), p).cpu().numpy()
    assert list(st) == list(ost)
    g0, g1 = (t.cpu().numpy() for t in model.vectors())
    assert row_rel_err(g0, a0) <= 1e-4
    assert row_rel_err(g1[:s.voc.V - 1], a1) <= 1e-4


# Later epochs draw other subsamples and windows (Philox counter) and continue the learning-rate decay.
@pytest.mark.parametrize("arch", [0, 2])
def test_single_worker_second_epoch(w2v, arch):
    s = oracle_side("sg_v30k_d100")
    voc, tree = gpu_side(w2v, s)
    tv = s.tv[:3000]
    syn0, syn1 = synth.init_weights(s.voc.V, 100, syn1_scale=0.005)
    a0, a1 = syn0.copy(), syn1.copy()
    model = w2v.make_model(syn0, syn1, voc, tree)
    for e in range(2):
        op = oracle.params(s.voc.V, 100, window=5, sample=1e-3, train_words=s.voc.train_words, corpus_tokens=tv.size,
                           cache_k=31, flush_every=10, order=1 if arch == 0 else 0, orient=1 if arch == 2 else 0,
                           epoch=e, n_epochs=2)
        ost = oracle.train(a0, a1, s.tree, tv, op)
        p = w2v.Params(window=5, sample=1e-3, corpus_tokens=tv.size, cache_k=31, flush_every=10, workers=1,
                       arch=arch, epoch=e, n_epochs=2)
        st = w2v.train_hs_epoch(model, to_dev(tv), p).cpu().numpy()
        assert list(st) == list(ost)
    g0, g1 = (t.cpu().numpy() for t in model.vectors())
    assert row_rel_err(g0, a0) <= 1e-4
    assert row_rel_err(g1[:s.voc.V - 1], a1) <= 1e-4


@pytest.mark.parametrize("name,gold,arch,epochs", [
    ("sg_v30k_d100", "sg_v30k_d100_orient1", 2, 1),
    ("sg_v30k_d100", "sg_v30k_d100_epochs3", 0, 3),
])
def test_async_loglik_reversed_and_epochs(w2v, name, gold, arch, epochs):
    log(f"async LL {gold}")
    g = golden(gold)
    s = oracle_side(name)
    assert s.voc.V == g["V"] and s.voc.train_words == g["train_words"]
    voc, tree = gpu_side(w2v, s)
    same_vocab_and_tree(voc, tree, s)
    syn0, syn1 = synth.init_weights(s.voc.V, s.w.dim)
    hv = to_dev(oracle.remap(corpus(name, heldout=True), s.voc.id_to_vocab))

    def run():
        model = w2v.make_model(syn0, syn1, voc, tree)
        for e in range(epochs):
            p = w2v.Params(window=s.w.window, sample=s.w.sample, corpus_tokens=s.tv.size, arch=arch,
                           alpha0=s.w.alpha0, epoch=e, n_epochs=epochs)
            st = w2v.train_hs_epoch(model, voc.tokens, p).cpu().numpy()
            assert list(st) == (g["stats"][e] if epochs > 1 else g["stats"])
        sg, npairs, _ = w2v.hs_loglik(model, hv, w2v.Params(window=s.w.window, sample=s.w.sample,
                                                            seed=synth.SEED_EVAL))
        assert npairs == g["heldout_pairs"]
        return sg / npairs

    gated(run, g["mean_ll"], g["init_mean_ll"], 0.9)
