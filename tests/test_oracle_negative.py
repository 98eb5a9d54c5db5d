"""Pins of the oracle's negative-sampling path (the objective named in §2,
trained with Ji et al.'s shared-negative mini-batch as §3.2 describes it).

What fixes these other than the oracle itself:
  * the noise weight of a count c lies within c^(1/4)/2 + 1 below c^(3/4)
    and never above it (closed-form bound of the integer square roots);
  * every word fills within one entry of T * weight / total of the noise
    table (a consequence of the table's definition, brute force);
  * negatives are drawn in proportion to the weights (chi-squared), never
    equal the centre word, and change with the seed and the epoch;
  * one centre's update equals alpha times the gradient of its window's
    objective at the values before the update (central finite differences);
  * the objective at zero output vectors is -ln 2 per term (closed form);
  * training raises the objective of the pairs it trains on.
"""
import math

import numpy as np
import pytest

import oracle
import synth


@pytest.mark.parametrize("seed", [0, 1])
def test_noise_weight_is_three_quarter_power_within_its_bound(seed):
    rng = np.random.default_rng(seed)
    c = np.concatenate([np.arange(1, 5000), rng.integers(1, 2**31 - 1, 20000),
                        np.array([2**31 - 1, 10**9, 65535, 65536, 65537, 4, 9, 15, 16, 17])]).astype(np.int64)
    w, tot = oracle.noise_weights(c)
    assert tot == int(w.sum())
    cf = c.astype(np.float64)
    exact = cf ** 0.75
    assert np.all(w <= exact + 1e-6 * exact)
    assert np.all(w >= exact - cf ** 0.25 / 2 - 1)
    assert np.all(w >= 1)


@pytest.mark.parametrize("V,L,seed", [(2, 4, 0), (7, 10, 1), (300, 16, 2), (5000, 20, 3)])
def test_noise_table_counts_within_one_of_the_weights(V, L, seed):
    rng = np.random.default_rng(seed)
    counts = np.sort(rng.zipf(1.3, V) + 4)[::-1].astype(np.int64)
    t = oracle.noise_table(counts, L)
    w, tot = oracle.noise_weights(counts)
    got = np.bincount(t, minlength=V)
    assert got.sum() == 1 << L
    assert np.all(np.abs(got - w * (1 << L) / tot) < 1.0)
    assert np.all(np.diff(t) >= 0)            # words in vocabulary order along the table
    if L <= 10:                               # brute force: entry i lies in its word's weight interval
        pref = np.concatenate([[0], np.cumsum(w)])
        for i in range(1 << L):
            u = (i * tot) >> L
            assert pref[t[i]] <= u < pref[t[i] + 1]


def small_stream(V=200, n=60_000, seed=7):
    w = synth.Workload("ns", n, V, 1.0, 0, 16, 3, 0.0, heldout_tokens=10_000)
    tok = synth.corpus(n, V, 1.0, 0, seed)
    voc = oracle.build_vocab(tok, V, 1)
    return w, voc, oracle.remap(tok, voc.id_to_vocab)


def test_negatives_follow_the_noise_distribution():
    w, voc, tv = small_stream()
    L = 16
    table = oracle.noise_table(voc.vocab_counts, L)
    p = oracle.params(voc.V, 8, window=3, train_words=voc.train_words, negative=7)
    r = oracle.sample_negatives(tv, p, voc.vocab_counts, table, L, cap=10**6)
    neg = r.negatives
    assert r.n_kept == tv.size == neg.shape[0]
    centres = tv[tv >= 0]
    assert not np.any(neg == centres[:, None])                       # never the centre word
    wt, tot = oracle.noise_weights(voc.vocab_counts)
    exp_p = np.bincount(table, minlength=voc.V) / table.size
    # dropped draws are exactly the draws that hit the centre word
    drop = (neg < 0).mean()
    assert abs(drop - float((exp_p[centres]).mean())) < 5 * math.sqrt(drop / neg.size) + 1e-4
    got = np.bincount(neg[neg >= 0], minlength=voc.V).astype(np.float64)
    # chi-squared against the table's distribution, conditioned on not being the centre (approximately)
    cond = exp_p * (1 - np.bincount(centres, minlength=voc.V) / centres.size)
    cond /= cond.sum()
    e = cond * got.sum()
    m = e > 20
    chi2 = float((((got - e) ** 2) / e)[m].sum())
    dof = int(m.sum()) - 1
    assert chi2 < dof + 6 * math.sqrt(2 * dof)


def test_negatives_depend_on_seed_and_epoch():
    w, voc, tv = small_stream(n=5000)
    table = oracle.noise_table(voc.vocab_counts, 12)
    base = dict(window=3, train_words=voc.train_words, negative=5)
    a = oracle.sample_negatives(tv, oracle.params(voc.V, 8, **base), voc.vocab_counts, table, 12, cap=5000)
    b = oracle.sample_negatives(tv, oracle.params(voc.V, 8, **base), voc.vocab_counts, table, 12, cap=5000)
    c = oracle.sample_negatives(tv, oracle.params(voc.V, 8, seed=9, **base), voc.vocab_counts, table, 12, cap=5000)
    d = oracle.sample_negatives(tv, oracle.params(voc.V, 8, epoch=1, n_epochs=2, **base), voc.vocab_counts, table,
                                12, cap=5000)
    assert np.array_equal(a.negatives, b.negatives) and a.checksum == b.checksum
    assert (a.negatives != c.negatives).mean() > 0.5 and (a.negatives != d.negatives).mean() > 0.5


def ns_objective_np(X, Y, targets):
    """sum over window rows q of log sig(x_q . y_t0) + sum_{k>=1, t_k>=0} log sig(-x_q . y_tk), fp64."""
    s = 0.0
    for x in X:
        for k, t in enumerate(targets):
            if t < 0:
                continue
            z = float(x @ Y[t])
            u = z if k == 0 else -z
            s += -math.log1p(math.exp(-u)) if u >= 0 else u - math.log1p(math.exp(u))
    return s


@pytest.mark.parametrize("V,dim,K,seed", [(12, 4, 3, 0), (30, 6, 5, 1), (9, 5, 8, 2)])
def test_centre_update_is_alpha_times_gradient(V, dim, K, seed):
    rng = np.random.default_rng(seed)
    counts = np.sort(rng.integers(5, 500, V))[::-1].astype(np.int64)
    L = 10
    table = oracle.noise_table(counts, L)
    syn0 = ((rng.random((V, dim)) - 0.5) * 0.8).astype(np.float32)
    syn1 = ((rng.random((V, dim)) - 0.5) * 0.8).astype(np.float32)
    v, w1, w2 = 1, 4, V - 2
    tok = np.array([w1, v, w2], np.int32)
    alpha = 0.025
    # a sampler seed whose second centre (v) takes both neighbours; only the first two centres train
    for s in range(300):
        p = oracle.params(V, dim, window=2, alpha0=alpha, corpus_tokens=3, max_centres=2, negative=K, seed=s,
                          train_words=int(counts.sum()))
        pr = oracle.sample_pairs(tok, p, counts)
        first = pr.centre == 0
        if list(pr.context[~first][:2]) == [0, 2] and list(pr.centre[~first][:2]) == [1, 1]:
            break
    else:
        pytest.fail("no seed gives the second centre both neighbours")
    negs = oracle.sample_negatives(tok, p, counts, table, L, cap=3).negatives
    a0, a1 = syn0.copy(), syn1.copy()
    # state after the first centre (w1 with its window), then the second centre's update
    p1 = oracle.params(V, dim, window=2, alpha0=alpha, corpus_tokens=3, max_centres=1, negative=K, seed=s,
                       train_words=int(counts.sum()))
    oracle.train_ns(a0, a1, counts, table, L, tok, p1)
    b0, b1 = syn0.copy(), syn1.copy()
    st = oracle.train_ns(b0, b1, counts, table, L, tok, p)
    targets = [v] + list(negs[1])
    assert st[3] == int(first.sum()) + 2
    X = np.stack([a0[w1], a0[w2]]).astype(np.float64)
    Y = a1.astype(np.float64)
    h = 1e-6
    gX = np.zeros_like(X)
    for q in range(2):
        for i in range(dim):
            e = np.zeros_like(X); e[q, i] = h
            gX[q, i] = (ns_objective_np(X + e, Y, targets) - ns_objective_np(X - e, Y, targets)) / (2 * h)
    gY = np.zeros_like(Y)
    for t in set(tt for tt in targets if tt >= 0):
        for i in range(dim):
            e = np.zeros_like(Y); e[t, i] = h
            gY[t, i] = (ns_objective_np(X, Y + e, targets) - ns_objective_np(X, Y - e, targets)) / (2 * h)
    np.testing.assert_allclose(b0[[w1, w2]] - a0[[w1, w2]], alpha * gX, rtol=2e-4, atol=2e-8)
    np.testing.assert_allclose(b1 - a1, alpha * gY, rtol=2e-4, atol=2e-8)
    others = [r for r in range(V) if r not in (w1, w2)]
    np.testing.assert_array_equal(b0[others], a0[others])


def test_objective_at_zero_output_vectors_is_minus_ln2_per_term():
    w, voc, tv = small_stream(n=20_000)
    table = oracle.noise_table(voc.vocab_counts, 14)
    syn0 = synth.init_weights(voc.V, 16)[0]
    syn1 = np.zeros((voc.V, 16), np.float32)
    p = oracle.params(voc.V, 16, window=3, train_words=voc.train_words, negative=5, seed=4)
    s, npairs, nterms = oracle.ns_objective(syn0, syn1, voc.vocab_counts, table, 14, tv, p)
    assert npairs > 0 and npairs <= nterms <= 6 * npairs
    assert abs(s + math.log(2.0) * nterms) <= 1e-9 * nterms


def test_training_raises_the_objective():
    w, voc, tv = small_stream(n=100_000)
    table = oracle.noise_table(voc.vocab_counts, 16)
    syn0, _ = synth.init_weights(voc.V, 16)
    syn1 = np.zeros((voc.V, 16), np.float32)
    pe = oracle.params(voc.V, 16, window=3, train_words=voc.train_words, negative=5, seed=4)
    s0, n0, t0 = oracle.ns_objective(syn0, syn1, voc.vocab_counts, table, 16, tv[:20_000], pe)
    for e in range(3):
        p = oracle.params(voc.V, 16, window=3, train_words=voc.train_words, corpus_tokens=tv.size, negative=5,
                          epoch=e, n_epochs=3)
        st = oracle.train_ns(syn0, syn1, voc.vocab_counts, table, 16, tv, p)
        assert st[2] == tv.size and st[3] > 0 and st[4] > st[3]
    s1, n1, t1 = oracle.ns_objective(syn0, syn1, voc.vocab_counts, table, 16, tv[:20_000], pe)
    assert (n1, t1) == (n0, t0)
    assert s1 / n1 > s0 / n0 + 0.1
