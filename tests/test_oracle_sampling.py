"""Pins of the oracle's sampling, learning-rate schedule and counter-based RNG.

  * Philox4x32-10 against the published known-answer vectors (golden file);
  * subsampling ("downsample", §4.1): t = 0 keeps every in-vocabulary token;
    per-word keep rates agree with the keep probability within 5 sigma;
  * window ("windowsize", §4.1): every centre's contexts are the kept tokens
    of its own document within its effective half-width, which is uniform on
    {1..W} (chi-square);
  * learning rate ("update alpha", Algorithm 1): starts at alpha0, is
    piecewise constant over 10,000-token blocks, decreases, floors at
    1e-4 alpha0.
"""
import os

import numpy as np
import pytest
from scipy import stats

import oracle
import synth

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def test_philox_known_answers():
    n = 0
    for line in open(os.path.join(GOLDEN, "philox4x32_10_kat.txt")):
        if line.startswith("#") or not line.strip():
            continue
        v = [int(x, 16) for x in line.split()]
        assert oracle.philox4x32_10(v[0:4], v[4:6]) == v[6:10]
        n += 1
    assert n == 3


def corpus_v(n=200_000, V=2000, topics=10, seed=1):
    tok = synth.corpus(n, V, 1.0, topics, seed)
    voc = oracle.build_vocab(tok, V, 5)
    return voc, oracle.remap(tok, voc.id_to_vocab)


def test_no_subsampling_keeps_every_in_vocab_token():
    voc, tv = corpus_v()
    p = oracle.params(voc.V, 8, window=5, sample=0.0, train_words=voc.train_words, corpus_tokens=tv.size)
    pr = oracle.sample_pairs(tv, p, voc.vocab_counts)
    assert pr.n_kept == int((tv >= 0).sum())
    np.testing.assert_array_equal(pr.keep_mask.astype(bool), tv >= 0)


def test_keep_rate_matches_keep_probability():
    voc, tv = corpus_v(n=1_000_000)
    t = 1e-3
    p = oracle.params(voc.V, 8, window=5, sample=t, train_words=voc.train_words, corpus_tokens=tv.size)
    pr = oracle.sample_pairs(tv, p, voc.vocab_counts, cap=0)
    mask = pr.keep_mask.astype(bool)
    for v in range(0, 40):
        occ = tv == v
        nv = int(occ.sum())
        q = t * voc.train_words / voc.vocab_counts[v]
        pk = min(1.0, np.sqrt(q) + q)
        kept = int(mask[occ].sum())
        sd = np.sqrt(nv * pk * (1 - pk)) + 1e-9
        assert abs(kept - nv * pk) <= 5 * sd + 1, (v, kept, nv * pk)
    # thresholds in units of 2^-32
    thr = oracle.keep_thresholds(voc.vocab_counts, t, voc.train_words)
    assert thr.dtype == np.uint64 and (thr <= (1 << 32)).all()
    assert (np.diff(thr.astype(np.float64)) >= 0).all()   # rarer words are kept more often


def test_keep_thresholds_exact_where_the_probability_is_a_dyadic_fraction():
    """The keep probability min(1, sqrt(q) + q), q = t N / count, in units of 2^-32, at counts where q is
    a power of two so that sqrt(q) + q is exact: t = 0.25, N = 100 (q = 1/4, 1/16, 1/64, 1, 1/2, 4)."""
    counts = np.array([100, 400, 1600, 25, 50, 6, 6400], dtype=np.int64)
    thr = oracle.keep_thresholds(counts, 0.25, 100)
    assert list(thr) == [3 << 30,                  # 1/2 + 1/4 = 3/4
                         5 << 28,                  # 1/4 + 1/16 = 5/16
                         9 << 26,                  # 1/8 + 1/64 = 9/64
                         1 << 32, 1 << 32,         # q = 1: 2; q = 1/2: 1.207..., kept always
                         1 << 32,                  # q = 25/6 > 1
                         (1 << 32) // 16 + (1 << 32) // 256]   # q = 1/256: 1/16 + 1/256
    assert list(oracle.keep_thresholds(counts, 0.0, 100)) == [1 << 32] * counts.size   # t = 0: keep all


def kept_runs(tv, mask, doc_len):
    """Per document, the global raw indices of kept tokens."""
    out = []
    for lo in range(0, tv.size, doc_len):
        idx = np.nonzero(mask[lo:lo + doc_len])[0] + lo
        out.append(idx)
    return out


@pytest.mark.parametrize("W,sample", [(1, 0.0), (2, 0.0), (5, 1e-3)])
def test_windows_are_contiguous_within_documents_and_uniform(W, sample):
    voc, tv = corpus_v(n=300_000)
    p = oracle.params(voc.V, 8, window=W, sample=sample, train_words=voc.train_words, corpus_tokens=tv.size)
    pr = oracle.sample_pairs(tv, p, voc.vocab_counts)
    mask = pr.keep_mask.astype(bool)
    runs = kept_runs(tv, mask, 1000)
    pos = {}
    for d, r in enumerate(runs):
        for j, g in enumerate(r):
            pos[int(g)] = (d, j, len(r))
    assert pr.n_kept == len(pos)
    # group contexts per centre (pairs are in stream order)
    by_centre = {}
    for c, x in zip(pr.centre.tolist(), pr.context.tolist()):
        by_centre.setdefault(c, []).append(x)
    widths = []
    for c, xs in by_centre.items():
        d, j, n = pos[c]
        js = [pos[x][1] for x in xs]
        assert all(pos[x][0] == d for x in xs)              # same document
        assert js == sorted(js) and j not in js              # ascending, centre excluded
        e = max(abs(a - j) for a in js)
        assert e <= W
        expect = [a for a in range(j - e, j + e + 1) if a != j and 0 <= a < n]
        assert js == expect                                  # every kept token within reach
        if j - W >= 0 and j + W < n:                          # not cut by a document edge
            widths.append(e)
    h = np.bincount(widths, minlength=W + 1)[1:]
    assert (h > 0).all()
    if W > 1:
        assert stats.chisquare(h).pvalue > 1e-4
    # a centre with no context contributes no pair
    assert sum(len(v) for v in by_centre.values()) == pr.total


def test_sampling_depends_on_seed_and_epoch_only():
    voc, tv = corpus_v(n=50_000)
    kw = dict(window=5, sample=1e-3, train_words=voc.train_words, corpus_tokens=tv.size)
    a = oracle.sample_pairs(tv, oracle.params(voc.V, 8, seed=3, **kw), voc.vocab_counts)
    b = oracle.sample_pairs(tv, oracle.params(voc.V, 8, seed=3, **kw), voc.vocab_counts)
    c = oracle.sample_pairs(tv, oracle.params(voc.V, 8, seed=4, **kw), voc.vocab_counts)
    d = oracle.sample_pairs(tv, oracle.params(voc.V, 8, seed=3, epoch=1, **kw), voc.vocab_counts)
    assert a.checksum == b.checksum and a.total == b.total
    assert a.checksum != c.checksum and a.checksum != d.checksum


def test_chunked_stream_equals_whole_stream():
    # documents are keyed by global raw index: two halves (whole documents) give the same pairs
    voc, tv = corpus_v(n=60_000)
    kw = dict(window=5, sample=1e-3, train_words=voc.train_words, corpus_tokens=tv.size)
    whole = oracle.sample_pairs(tv, oracle.params(voc.V, 8, **kw), voc.vocab_counts)
    h1 = oracle.sample_pairs(tv[:30_000], oracle.params(voc.V, 8, **kw), voc.vocab_counts)
    h2 = oracle.sample_pairs(tv[30_000:], oracle.params(voc.V, 8, first_raw_index=30_000, **kw), voc.vocab_counts)
    np.testing.assert_array_equal(whole.centre, np.concatenate([h1.centre, h2.centre]))
    np.testing.assert_array_equal(whole.context, np.concatenate([h1.context, h2.context]))


def test_learning_rate_schedule():
    a0, N, E = 0.025, 1_234_567, 3
    al = [oracle.alpha(a0, i, e, E, N) for e in range(E) for i in (0, 9_999, 10_000, 600_000, N - 1)]
    assert al[0] == np.float32(a0)
    assert al[1] == al[0] and al[2] < al[1]                  # one step per 10,000 tokens
    assert all(x >= y for x, y in zip(al, al[1:]))
    assert oracle.alpha(a0, N - 1, E - 1, E, N) > a0 * 1e-4 * 0.999
    assert oracle.alpha(a0, 10 * N, E - 1, E, N) == np.float32(a0 * 1e-4)   # floor
    # linear decay: half-way through the run alpha is about alpha0 / 2
    mid = oracle.alpha(a0, N // 2, 1, E, N)
    assert abs(mid - a0 / 2) < a0 * 0.01
