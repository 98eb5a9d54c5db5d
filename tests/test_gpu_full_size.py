"""GPU parity at the full size of the 1e9-token workload (V = 1M, d = 300).

The HIP path runs on the whole corpus in the launch configuration that the
benchmark times; the oracle checks what it can afford at that size:
- vocabulary and Huffman tree of the whole corpus, live, bit for bit;
- the training sampler's pair count, kept count, pair checksum and pair-node
  update count over the whole corpus, from the stored oracle result
  (tests/golden/oracle_sampler_sg_v1m_d300.json, written by make_golden.py);
- the first synchronous batches (4096 centres, and ten of 256) within 1e-4;
- one sequential worker on the first documents within 1e-4 of the oracle's
  centre-major order (the deepest paths of any workload here);
- asynchronous training on the first 1e8 tokens: held-out log-likelihood
  within 1 % of the stored oracle result for the same prefix.
"""
import functools
import json
import math
import os

import numpy as np
import pytest

import oracle
import synth
from gpu_common import corpus, gated, log, row_rel_err

pytestmark = pytest.mark.gpu
GOLDEN = os.path.join(os.path.dirname(__file__), "golden")
NAME = "sg_v1m_d300"
PREFIX = 100_000_000


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


def golden(fname):
    path = os.path.join(GOLDEN, fname)
    if not os.path.exists(path):
        pytest.skip(f"no stored oracle result {path}")
    return json.load(open(path))


@functools.lru_cache(maxsize=1)
def oracle_full():
    """The oracle's vocabulary and tree of the whole corpus (the token stream itself stays raw)."""
    w = synth.WORKLOADS[NAME]
    tok = corpus(NAME)
    voc = oracle.build_vocab(tok, w.vocab, w.min_count)
    tree = oracle.build_huffman(voc.vocab_counts)
    return w, tok, voc, tree


@functools.lru_cache(maxsize=2)
def oracle_prefix(n):
    w, tok, voc, _ = oracle_full()
    return oracle.remap(tok[:n], voc.id_to_vocab)


@functools.lru_cache(maxsize=1)
def gpu_full(w2v):
    w, tok, _, _ = oracle_full()
    voc = w2v.build_vocab(to_dev(tok), w.vocab, w.min_count)
    tree = w2v.build_huffman(voc.vocab_counts)
    return voc, tree


def test_full_vocab_and_tree_bit_exact(w2v):
    log("full-size vocabulary and tree")
    w, tok, ov, ot = oracle_full()
    voc, tree = gpu_full(w2v)
    assert voc.V == ov.V and voc.train_words == ov.train_words
    np.testing.assert_array_equal(voc.counts_by_id.cpu().numpy(), ov.counts)
    np.testing.assert_array_equal(voc.vocab_ids.cpu().numpy(), ov.vocab_ids)
    np.testing.assert_array_equal(voc.id_to_vocab.cpu().numpy(), ov.id_to_vocab)
    np.testing.assert_array_equal(tree.codelen.cpu().numpy(), ot.codelen)
    np.testing.assert_array_equal(tree.code.cpu().numpy().view(np.uint64), ot.code)
    np.testing.assert_array_equal(tree.point_off.cpu().numpy(), ot.point_off)
    np.testing.assert_array_equal(tree.points.cpu().numpy(), ot.points)
    # the remapped stream on sampled positions (the whole stream is compared at smaller sizes)
    idx = np.random.default_rng(0).integers(0, tok.size, 1_000_000)
    np.testing.assert_array_equal(voc.tokens[to_dev(idx)].cpu().numpy(), ov.id_to_vocab[tok[idx]])


def test_full_sampler_matches_stored_oracle(w2v):
    g = golden(f"oracle_sampler_{NAME}.json")
    w, _, ov, _ = oracle_full()
    assert (g["V"], g["train_words"]) == (ov.V, ov.train_words)
    voc, _ = gpu_full(w2v)
    p = w2v.Params(window=w.window, sample=w.sample, seed=synth.SEED_TRAIN)
    pr = w2v.sample_pairs(voc.tokens, voc.V, voc.vocab_counts, voc.train_words, p, cap=0)
    assert (pr.total, pr.n_kept, pr.checksum) == (g["pairs"], g["kept"], g["pairs_checksum"])


@pytest.mark.parametrize("batches,B", [(1, 4096), (10, 256)])
def test_full_sync_first_batches_within_1e4(w2v, batches, B):
    log(f"full-size sync batches={batches} B={B}")
    w, _, ov, ot = oracle_full()
    voc, tree = gpu_full(w2v)
    tv = oracle_prefix(200_000)
    op = oracle.params(ov.V, w.dim, window=w.window, sample=w.sample, train_words=ov.train_words,
                       corpus_tokens=w.n_tokens, sync_batch=B)
    pr = oracle.sample_pairs(tv, op, ov.vocab_counts, cap=0)
    kept = np.cumsum(pr.keep_mask)
    assert kept[-1] > batches * B
    tv = tv[:int(np.searchsorted(kept, batches * B)) + 1]
    syn0, syn1 = synth.init_weights(ov.V, w.dim, syn1_scale=0.5 / w.dim)
    a0, a1 = syn0.copy(), syn1.copy()
    ost = oracle.train_sync(a0, a1, ot, tv, op, n_batches=-1)
    model = w2v.make_model(syn0, syn1, voc, tree)
    p = w2v.Params(window=w.window, sample=w.sample, corpus_tokens=w.n_tokens, mode=1, sync_batch=B)
    st = w2v.train_hs_epoch(model, to_dev(tv), p).cpu().numpy()
    assert list(st) == list(ost)
    g0, g1 = (t.cpu().numpy() for t in model.vectors())
    touched0 = ~(a0 == syn0).all(1)
    touched1 = ~(a1 == syn1).all(1)
    assert row_rel_err(g0[touched0], a0[touched0]) <= 1e-4
    assert row_rel_err(g1[:ov.V - 1][touched1], a1[touched1]) <= 1e-4
    np.testing.assert_array_equal(g0[~touched0], syn0[~touched0])
    np.testing.assert_array_equal(g1[:ov.V - 1][~touched1], syn1[~touched1])


@pytest.mark.parametrize("k,wp", [(31, 5), (31, 0), (0, 1), (31, 15), (0, 11)])
def test_full_single_worker_matches_oracle_centre_major(w2v, k, wp):
    log(f"full-size single worker k={k} write_policy={wp}")
    w, _, ov, ot = oracle_full()
    voc, tree = gpu_full(w2v)
    tv = oracle_prefix(200_000)[:3000]
    syn0, syn1 = synth.init_weights(ov.V, w.dim, syn1_scale=0.5 / w.dim)
    a0, a1 = syn0.copy(), syn1.copy()
    op = oracle.params(ov.V, w.dim, window=w.window, sample=w.sample, train_words=ov.train_words,
                       corpus_tokens=w.n_tokens, cache_k=k, flush_every=10, order=1)
    ost = oracle.train(a0, a1, ot, tv, op)
    model = w2v.make_model(syn0, syn1, voc, tree)
    p = w2v.Params(window=w.window, sample=w.sample, corpus_tokens=w.n_tokens, cache_k=k, flush_every=10,
                   workers=1, write_policy=wp)
    st = w2v.train_hs_epoch(model, to_dev(tv), p).cpu().numpy()
    assert list(st) == list(ost)
    g0, g1 = (t.cpu().numpy() for t in model.vectors())
    touched0 = ~(a0 == syn0).all(1)
    touched1 = ~(a1 == syn1).all(1)
    assert touched1.sum() > 1000
    assert row_rel_err(g0[touched0], a0[touched0]) <= 1e-4
    assert row_rel_err(g1[:ov.V - 1][touched1], a1[touched1]) <= 1e-4
    np.testing.assert_array_equal(g1[:ov.V - 1][~touched1], syn1[~touched1])


@pytest.mark.parametrize("wp", [5, 7, 15])
def test_full_prefix_async_loglik_within_1pct(w2v, wp):
    g = golden(f"oracle_ll_{NAME}_first{PREFIX}.json")
    w, _, ov, _ = oracle_full()
    assert (g["V"], g["train_words"], g["train_tokens"]) == (ov.V, ov.train_words, PREFIX)
    voc, tree = gpu_full(w2v)
    syn0, syn1 = synth.init_weights(voc.V, w.dim)
    held = to_dev(oracle.remap(corpus(NAME, heldout=True), ov.id_to_vocab))

    def run():
        model = w2v.make_model(syn0, syn1, voc, tree)
        p = w2v.Params(window=w.window, sample=w.sample, alpha0=w.alpha0, corpus_tokens=PREFIX,
                       seed=synth.SEED_TRAIN, write_policy=wp)
        st = w2v.train_hs_epoch(model, voc.tokens[:PREFIX], p).cpu().numpy()
        assert list(st) == g["stats"]
        s, npairs, _ = w2v.hs_loglik(model, held, w2v.Params(window=w.window, sample=w.sample,
                                                             seed=synth.SEED_EVAL))
        assert npairs == g["heldout_pairs"]
        return s / npairs

    gated(run, g["mean_ll"], g["init_mean_ll"], 0.9)
