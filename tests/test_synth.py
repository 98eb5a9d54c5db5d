"""The seeded corpus generator (input recipe of every workload)."""
import numpy as np
import pytest
from scipy import stats

import synth


def test_deterministic_and_thread_independent():
    a = synth.corpus(50_000, 5000, 1.05, 20, 7, threads=1)
    b = synth.corpus(50_000, 5000, 1.05, 20, 7, threads=4)
    c = synth.corpus(50_000, 5000, 1.05, 20, 8, threads=4)
    np.testing.assert_array_equal(a, b)
    assert not np.array_equal(a, c)
    assert a.min() >= 0 and a.max() < 5000


def test_plain_zipf_rank_frequencies():
    V, s, n = 200, 1.0, 400_000
    tok = synth.corpus(n, V, s, 0, 3)
    obs = np.bincount(tok, minlength=V)
    p = synth.zipf_probs(V, s)
    np.testing.assert_allclose(p, np.arange(1, V + 1) ** -s / (np.arange(1, V + 1) ** -s).sum(), rtol=1e-12)
    assert stats.chisquare(obs, p * n).pvalue > 1e-4


def test_topic_documents_reweight_their_subset():
    V, T, n, doc = 1000, 4, 400_000, 1000
    tok = synth.corpus(n, V, 1.0, T, 5, doc_len=doc)
    sub = synth.topic_subset(5, 2, V)
    assert sub.size == round(0.05 * V) and np.unique(sub).size == sub.size
    docs = [k for k in range(n // doc) if synth.doc_topic(5, k, T) == 2]
    assert len(docs) > 20
    toks = np.concatenate([tok[k * doc:(k + 1) * doc] for k in docs])
    p = synth.zipf_probs(V, 1.0)
    w = p.copy()
    w[sub] *= 20.0
    w /= w.sum()
    obs = np.bincount(toks, minlength=V)
    # compare the subset's share and the head of the distribution
    share = np.isin(toks, sub).mean()
    sd = np.sqrt(w[sub].sum() * (1 - w[sub].sum()) / toks.size)
    assert abs(share - w[sub].sum()) < 6 * sd
    top = np.argsort(-w)[:50]
    exp = w[top] * toks.size
    assert stats.chisquare(np.append(obs[top], toks.size - obs[top].sum()),
                           np.append(exp, toks.size - exp.sum())).pvalue > 1e-4


def test_workload_table():
    w = synth.WORKLOADS["sg_v1m_d300"]
    assert (w.n_tokens, w.vocab, w.dim, w.window, w.sample, w.topics) == (10**9, 10**6, 300, 5, 1e-5, 200)
    assert synth.WORKLOADS["cbow_v100k_d300"].arch == 1
    s0, s1 = synth.init_weights(100, 30)
    assert s0.shape == (100, 30) and s1.shape == (99, 30) and (s1 == 0).all()
    assert np.abs(s0).max() <= 0.5 / 30
