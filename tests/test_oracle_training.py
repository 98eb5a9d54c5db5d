"""Pins of the oracle's objective and updates (Algorithm 1, Cached Skipgram HS).

What fixes these other than the oracle itself:
  * the hierarchical softmax is a distribution: sum_v P(v|x) = 1 (fp64);
  * log-likelihood at syn1 = 0 is -ln 2 per node (closed form), for the
    pairs' objective and for CBOW's;
  * CBOW's objective equals log P(v|h) of the softmax above with h the mean
    of the materialised context rows of each centre (rebuilt in numpy);
  * one update of Algorithm 1 equals alpha times the gradient of log P(v|w),
    by central finite differences (skip-gram, CBOW, synchronous mode);
  * from syn1 = 0 one pair gives syn1[n_j] = alpha (1/2 - t_j) x_w and leaves
    x_w unchanged (closed form);
  * the cache of Algorithm 1 with one worker changes nothing beyond the
    rounding of its flush (invariant of the caching scheme, §3.2);
  * swapping the window and node loops is exact when a window holds no
    repeated word (invariant);
  * with the reversed orientation, a centre's pairs are gradient steps of
    log P(w|v) taken one after the other, each at the model the previous one
    left (finite differences).
"""
import math

import numpy as np
import pytest

import oracle
import synth


def small_model(V, dim, seed, syn1_scale=0.3):
    rng = np.random.default_rng(seed)
    counts = np.sort(rng.integers(5, 500, V))[::-1].astype(np.int64)
    tree = oracle.build_huffman(counts)
    syn0 = ((rng.random((V, dim)) - 0.5) * 0.6).astype(np.float32)
    syn1 = ((rng.random((V - 1, dim)) * 2 - 1) * syn1_scale).astype(np.float32)
    return tree, syn0, syn1


# ----------------------------------------------------------- the objective
@pytest.mark.parametrize("V,dim,seed", [(2, 3, 0), (7, 4, 1), (50, 8, 2), (1000, 16, 3)])
def test_hs_probabilities_sum_to_one(V, dim, seed):
    tree, _, syn1 = small_model(V, dim, seed, syn1_scale=1.0)
    rng = np.random.default_rng(seed + 100)
    s1 = syn1.astype(np.float64)
    for _ in range(3):
        x = rng.normal(size=dim) * 2.0
        total = sum(math.exp(oracle.log_prob(x, s1, tree, v)) for v in range(V))
        assert abs(total - 1.0) < 1e-12


def test_loglik_at_zero_syn1_is_minus_ln2_per_node():
    w = synth.WORKLOADS["tiny_sg_v1k_d50"]
    tok = synth.workload_corpus(w)
    voc = oracle.build_vocab(tok, w.vocab, w.min_count)
    tree = oracle.build_huffman(voc.vocab_counts)
    tv = oracle.remap(tok, voc.id_to_vocab)
    syn0, syn1 = synth.init_weights(voc.V, w.dim)
    p = oracle.params(voc.V, w.dim, window=w.window, train_words=voc.train_words, corpus_tokens=tok.size, seed=4)
    s, npairs, nnodes = oracle.loglik(syn0, syn1, tree, tv, p)
    assert npairs > 0
    assert abs(s - (-math.log(2.0) * nnodes)) < 1e-6 * nnodes


def test_cbow_loglik_at_zero_syn1_is_minus_ln2_per_node():
    w = synth.WORKLOADS["tiny_sg_v1k_d50"]
    tok = synth.workload_corpus(w)
    voc = oracle.build_vocab(tok, w.vocab, w.min_count)
    tree = oracle.build_huffman(voc.vocab_counts)
    tv = oracle.remap(tok, voc.id_to_vocab)
    syn0, syn1 = synth.init_weights(voc.V, w.dim)
    p = oracle.params(voc.V, w.dim, window=w.window, train_words=voc.train_words, seed=4, arch=1)
    s, ncentres, nnodes = oracle.loglik(syn0, syn1, tree, tv, p)
    assert ncentres > 0
    assert nnodes == int(tree.codelen[tv].astype(np.int64).sum())     # every centre has a window here
    assert abs(s - (-math.log(2.0) * nnodes)) < 1e-6 * nnodes


@pytest.mark.parametrize("window,sample", [(2, 0.0), (5, 1e-2)])
def test_cbow_loglik_is_log_prob_of_the_window_mean(window, sample):
    """CBOW's objective, rebuilt from the materialised pairs: per centre, h = the mean of its context
    rows (numpy, fp64), scored with the softmax whose normalisation is pinned above."""
    w = synth.WORKLOADS["tiny_sg_v1k_d50"]
    tok = synth.workload_corpus(w)[:8000]
    voc = oracle.build_vocab(tok, w.vocab, 1)
    tree = oracle.build_huffman(voc.vocab_counts)
    tv = oracle.remap(tok, voc.id_to_vocab)
    rng = np.random.default_rng(7)
    syn0 = ((rng.random((voc.V, w.dim)) - 0.5) * 0.6).astype(np.float32)
    syn1 = ((rng.random((voc.V - 1, w.dim)) * 2 - 1) * 0.3).astype(np.float32)
    p = oracle.params(voc.V, w.dim, window=window, sample=sample, train_words=voc.train_words, seed=4, arch=1)
    s, ncentres, nnodes = oracle.loglik(syn0, syn1, tree, tv, p)
    pr = oracle.sample_pairs(tv, p, voc.vocab_counts)
    s1 = syn1.astype(np.float64)
    ref, centres = 0.0, 0
    for c in np.unique(pr.centre):
        ctx = pr.context[pr.centre == c]
        h = syn0[tv[ctx]].astype(np.float64).mean(axis=0)
        ref += oracle.log_prob(h, s1, tree, int(tv[c]))
        centres += 1
    assert ncentres == centres > 100
    assert abs(s - ref) <= 1e-12 * abs(ref)
    # the skip-gram objective on the same stream is a different number (one term per pair)
    p0 = oracle.params(voc.V, w.dim, window=window, sample=sample, train_words=voc.train_words, seed=4)
    s0, npairs, _ = oracle.loglik(syn0, syn1, tree, tv, p0)
    assert npairs == pr.total > ncentres and abs(s0 - s) > 1.0


# ------------------------------------------------------- one-pair updates
def one_pair_corpus(v, w):
    """Two kept tokens, window 1, no subsampling: the first centre's only pair is (v, w)."""
    return np.array([v, w], np.int32)


def fd_grad_x(x, syn1, tree, v, h=1e-6):
    g = np.zeros_like(x)
    for k in range(x.size):
        e = np.zeros_like(x); e[k] = h
        g[k] = (oracle.log_prob(x + e, syn1, tree, v) - oracle.log_prob(x - e, syn1, tree, v)) / (2 * h)
    return g


def fd_grad_y(x, syn1, tree, v, n, h=1e-6):
    g = np.zeros(syn1.shape[1])
    for k in range(syn1.shape[1]):
        a = syn1.copy(); a[n, k] += h
        b = syn1.copy(); b[n, k] -= h
        g[k] = (oracle.log_prob(x, a, tree, v) - oracle.log_prob(x, b, tree, v)) / (2 * h)
    return g


@pytest.mark.parametrize("V,dim,seed", [(6, 4, 0), (13, 5, 1), (20, 8, 2)])
@pytest.mark.parametrize("order", [0, 1])
def test_skipgram_pair_update_is_alpha_times_gradient(V, dim, seed, order):
    tree, syn0, syn1 = small_model(V, dim, seed)
    v, w = V - 1, 1                      # a deep word and another one
    tok = one_pair_corpus(v, w)
    alpha = 0.025
    p = oracle.params(V, dim, window=1, alpha0=alpha, corpus_tokens=2, max_centres=1, order=order)
    a0, a1 = syn0.copy(), syn1.copy()
    st = oracle.train(a0, a1, tree, tok, p)
    assert st[3] == 1 and st[4] == tree.codelen[v]
    x = syn0[w].astype(np.float64)
    s1 = syn1.astype(np.float64)
    gx = fd_grad_x(x, s1, tree, v)
    np.testing.assert_allclose(a0[w] - syn0[w], alpha * gx, rtol=2e-4, atol=2e-8)
    others = [r for r in range(V) if r != w]
    np.testing.assert_array_equal(a0[others], syn0[others])
    pts, _ = tree.path(v)
    for n in range(V - 1):
        if n in pts:
            gy = fd_grad_y(x, s1, tree, v, n)
            np.testing.assert_allclose(a1[n] - syn1[n], alpha * gy, rtol=2e-4, atol=2e-8)
        else:
            np.testing.assert_array_equal(a1[n], syn1[n])


@pytest.mark.parametrize("V,dim,seed", [(6, 4, 0), (13, 5, 1), (20, 8, 2)])
def test_reversed_orientation_pairs_are_sequential_gradient_steps(V, dim, seed):
    tree, syn0, syn1 = small_model(V, dim, seed)
    v, w1, w2 = 2, V - 1, 1
    tok = np.array([v, w1, w2], np.int32)
    alpha = 0.025
    # a sampler seed whose first centre (v) takes both neighbours: half-width 2
    for s in range(200):
        p = oracle.params(V, dim, window=2, alpha0=alpha, corpus_tokens=3, max_centres=1, orient=1, seed=s)
        pr = oracle.sample_pairs(tok, p, tree.vocab_counts)
        if list(pr.centre[:2]) == [0, 0] and list(pr.context[:2]) == [1, 2]:
            break
    else:
        pytest.fail("no seed gives the first centre a half-width of 2")
    a0, a1 = syn0.copy(), syn1.copy()
    st = oracle.train(a0, a1, tree, tok, p)
    assert st[3] == 2 and st[4] == int(tree.codelen[w1]) + int(tree.codelen[w2])
    x = syn0[v].astype(np.float64)
    y = syn1.astype(np.float64)
    for w in (w1, w2):                   # each pair at the state the previous one left
        gx = fd_grad_x(x, y, tree, w)
        pts, _ = tree.path(w)
        gy = {n: fd_grad_y(x, y, tree, w, n) for n in pts}
        x = x + alpha * gx
        for n in pts:
            y[n] = y[n] + alpha * gy[n]
    np.testing.assert_allclose(a0[v], x, rtol=2e-4, atol=2e-8)
    np.testing.assert_allclose(a1, y, rtol=2e-4, atol=2e-8)
    others = [r for r in range(V) if r != v]
    np.testing.assert_array_equal(a0[others], syn0[others])


def test_one_step_from_zero_syn1_closed_form():
    V, dim = 9, 6
    tree, syn0, _ = small_model(V, dim, 5)
    syn1 = np.zeros((V - 1, dim), np.float32)
    v, w = 3, 7
    alpha = 0.05
    p = oracle.params(V, dim, window=1, alpha0=alpha, corpus_tokens=2, max_centres=1)
    a0, a1 = syn0.copy(), syn1.copy()
    oracle.train(a0, a1, tree, one_pair_corpus(v, w), p)
    np.testing.assert_array_equal(a0, syn0)            # e = sum g * 0 = 0
    pts, bits = tree.path(v)
    for n, t in zip(pts, bits):
        np.testing.assert_allclose(a1[n], alpha * (0.5 - t) * syn0[w], rtol=1e-6)


@pytest.mark.parametrize("V,dim,seed", [(8, 4, 0), (15, 6, 1)])
def test_cbow_update_is_alpha_times_gradient_wrt_mean(V, dim, seed):
    tree, syn0, syn1 = small_model(V, dim, seed)
    # centre v at position 1 with window words at positions 0 and 2 (window 1 -> eff 1)
    v, w1, w2 = V - 2, 0, 2
    tok = np.array([w1, v, w2], np.int32)
    alpha = 0.05
    # skip the first centre (position 0) by running two centres and undoing nothing: instead run
    # with max_centres=2 on a corpus whose first centre has no effect is impossible, so check the
    # second centre directly against a model advanced by the first.
    p1 = oracle.params(V, dim, window=1, alpha0=alpha, corpus_tokens=3, max_centres=1, arch=1)
    b0, b1 = syn0.copy(), syn1.copy()
    oracle.train(b0, b1, tree, tok, p1)
    p2 = oracle.params(V, dim, window=1, alpha0=alpha, corpus_tokens=3, max_centres=2, arch=1)
    a0, a1 = syn0.copy(), syn1.copy()
    oracle.train(a0, a1, tree, tok, p2)
    h = (b0[w1].astype(np.float64) + b0[w2].astype(np.float64)) / 2
    s1 = b1.astype(np.float64)
    gh = fd_grad_x(h, s1, tree, v)
    # C-tool convention: the full hidden-layer gradient is added to each window vector
    np.testing.assert_allclose(a0[w1] - b0[w1], alpha * gh, rtol=2e-4, atol=2e-8)
    np.testing.assert_allclose(a0[w2] - b0[w2], alpha * gh, rtol=2e-4, atol=2e-8)
    for n in tree.path(v)[0]:
        gy = fd_grad_y(h, s1, tree, v, n)
        np.testing.assert_allclose(a1[n] - b1[n], alpha * gy, rtol=2e-4, atol=2e-8)


def test_sync_batch_is_sum_of_gradients_at_the_snapshot():
    V, dim = 10, 5
    tree, syn0, syn1 = small_model(V, dim, 9)
    tok = np.array([1, 8, 4, 8, 6], np.int32)     # a repeated word: order must not matter
    alpha = 0.025
    p = oracle.params(V, dim, window=1, alpha0=alpha, corpus_tokens=tok.size, sync_batch=5)
    a0, a1 = syn0.copy(), syn1.copy()
    st = oracle.train_sync(a0, a1, tree, tok, p, n_batches=1)
    assert st[2] == 5
    # expected: every pair (centre c, context x) of window 1
    s0 = syn0.astype(np.float64)
    s1 = syn1.astype(np.float64)
    d0 = np.zeros_like(s0)
    d1 = np.zeros_like(s1)
    for j in range(tok.size):
        for c in (j - 1, j + 1):
            if 0 <= c < tok.size:
                v, w = tok[j], tok[c]
                d0[w] += alpha * fd_grad_x(s0[w], s1, tree, v)
                for n in tree.path(v)[0]:
                    d1[n] += alpha * fd_grad_y(s0[w], s1, tree, v, n)
    np.testing.assert_allclose(a0 - syn0, d0, rtol=5e-4, atol=2e-7)
    np.testing.assert_allclose(a1 - syn1, d1, rtol=5e-4, atol=2e-7)


# --------------------------------------------------------------- invariants
def tiny_setup(sample=0.0, window=3, n=20_000, V=300, dim=12, seed=0, distinct=False):
    rng = np.random.default_rng(seed)
    if distinct:
        # no id repeats within any run of 2*window+1 consecutive tokens
        tok = np.arange(n, dtype=np.int32) % V
    else:
        tok = (rng.zipf(1.2, n) - 1).astype(np.int32) % V
    voc = oracle.build_vocab(tok, V, 1)
    tree = oracle.build_huffman(voc.vocab_counts)
    tv = oracle.remap(tok, voc.id_to_vocab)
    syn0 = ((rng.random((voc.V, dim)) - 0.5) / dim).astype(np.float32)
    syn1 = ((rng.random((voc.V - 1, dim)) - 0.5) * 0.2).astype(np.float32)
    return voc, tree, tv, syn0, syn1


def test_loop_interchange_is_bit_exact_without_repeated_words():
    voc, tree, tv, syn0, syn1 = tiny_setup(distinct=True, V=97)
    base = dict(window=3, train_words=voc.train_words, corpus_tokens=tv.size, sample=0.0)
    outs = []
    for order in (0, 1):
        a0, a1 = syn0.copy(), syn1.copy()
        oracle.train(a0, a1, tree, tv, oracle.params(voc.V, syn0.shape[1], order=order, **base))
        outs.append((a0, a1))
    np.testing.assert_array_equal(outs[0][0], outs[1][0])
    np.testing.assert_array_equal(outs[0][1], outs[1][1])


@pytest.mark.parametrize("k,u", [(1, 1), (7, 10), (31, 10), (31, 100)])
def test_cache_with_one_worker_matches_no_cache(k, u):
    voc, tree, tv, syn0, syn1 = tiny_setup(seed=4)
    base = dict(window=3, train_words=voc.train_words, corpus_tokens=tv.size, sample=1e-3)
    ref0, ref1 = syn0.copy(), syn1.copy()
    oracle.train(ref0, ref1, tree, tv, oracle.params(voc.V, syn0.shape[1], **base))
    a0, a1 = syn0.copy(), syn1.copy()
    oracle.train(a0, a1, tree, tv, oracle.params(voc.V, syn0.shape[1], cache_k=k, flush_every=u, **base))
    # differs only by the rounding of weight + (cached - original)
    assert np.abs(a1 - ref1).max() <= 1e-5 * max(1.0, np.abs(ref1).max())
    assert np.abs(a0 - ref0).max() <= 1e-5 * max(1.0, np.abs(ref0).max())
    assert not np.array_equal(ref1, syn1)


def test_training_raises_likelihood_of_the_training_stream():
    # Algorithm 1 is SGD on sum log P(v|w): the likelihood of the pairs it trains on must rise
    w = synth.Workload("t", 300_000, 2_000, 1.0, 10, 32, 5, 0.0, heldout_tokens=50_000)
    tok = synth.workload_corpus(w)
    voc = oracle.build_vocab(tok, w.vocab, w.min_count)
    tree = oracle.build_huffman(voc.vocab_counts)
    tv = oracle.remap(tok, voc.id_to_vocab)
    syn0, syn1 = synth.init_weights(voc.V, w.dim)
    pe = oracle.params(voc.V, w.dim, window=w.window, train_words=voc.train_words, corpus_tokens=tok.size, seed=4)
    ll0 = oracle.loglik(syn0, syn1, tree, tv[:50_000], pe)
    for e in range(3):
        p = oracle.params(voc.V, w.dim, window=w.window, train_words=voc.train_words, corpus_tokens=tok.size,
                          epoch=e, n_epochs=3, alpha0=0.025)
        oracle.train(syn0, syn1, tree, tv, p)
    ll1 = oracle.loglik(syn0, syn1, tree, tv[:50_000], pe)
    assert ll1[1] == ll0[1]
    assert ll1[0] / ll1[1] > ll0[0] / ll0[1] + 0.1
