"""Write the oracle's full-epoch results that the GPU tests compare against.

Calls only the CPU oracle (and the input generator). For a workload it runs
one epoch of Algorithm 1 as printed (one sequential worker, top-31 inner-node
cache flushed every 10 centre words, §4.1 / Figure 1's c31 setting) from the
seeded initial model and stores the held-out mean log-likelihood per pair.

    python tests/golden/make_golden.py sg_v30k_d100 [more names...]
    python tests/golden/make_golden.py sg_v1m_d300 --train-tokens 100000000
    python tests/golden/make_golden.py sg_v1m_d300 --sampler

With --orient 1 the pairs walk the window word's path with the centre's
vector as input; with --epochs E the corpus is trained E times with the
learning rate decaying over all of them; both add to the file name.

With --train-tokens N the vocabulary and tree still come from the whole
corpus, but training covers only its first N tokens (whole documents; the
learning rate decays over those N), and the result is stored as
oracle_ll_<name>_first<N>.json: a bounded sample of a workload whose full
epoch is too long for one core.

With --ns K it trains skip-gram with K shared negatives instead (noise table
of 2^ceil(log2(64 V)) entries, at least 2^10 and at most 2^27, output vectors
starting at zero) and stores the held-out negative-sampling objective as
oracle_ns<K>_<name>.json.

With --sampler it stores, as oracle_sampler_<name>.json, digests of the
oracle's vocabulary and Huffman tree for the whole corpus and the count and
checksum of the training seed's (centre, context) pairs: the integer parts of
the path at a size where the tests cannot afford to run the oracle live.
"""
from __future__ import annotations

import hashlib
import json
import os
import sys
import time

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(os.path.dirname(HERE))
sys.path.insert(0, ROOT)

import numpy as np  # noqa: E402

import oracle  # noqa: E402
import synth  # noqa: E402


def run(name: str, cache_k: int = 31, flush_every: int = 10, train_tokens: int = 0, orient: int = 0,
        epochs: int = 1) -> dict:
    w = synth.WORKLOADS[name]
    assert train_tokens % w.doc_len == 0, "a training prefix must be whole documents"
    t0 = time.time()
    tok = synth.workload_corpus(w)
    held = synth.workload_corpus(w, heldout=True)
    voc = oracle.build_vocab(tok, w.vocab, w.min_count)
    tree = oracle.build_huffman(voc.vocab_counts)
    tv = oracle.remap(tok[:train_tokens] if train_tokens else tok, voc.id_to_vocab)
    del tok
    hv = oracle.remap(held, voc.id_to_vocab)
    syn0, syn1 = synth.init_weights(voc.V, w.dim)
    pe = oracle.params(voc.V, w.dim, window=w.window, sample=w.sample, train_words=voc.train_words,
                       seed=synth.SEED_EVAL, arch=w.arch)
    s0, npairs, _ = oracle.loglik(syn0, syn1, tree, hv, pe)
    t1 = time.time()
    stats = []
    for e in range(epochs):
        p = oracle.params(voc.V, w.dim, window=w.window, sample=w.sample, alpha0=w.alpha0,
                          train_words=voc.train_words, corpus_tokens=tv.size, seed=synth.SEED_TRAIN,
                          cache_k=cache_k, flush_every=flush_every, order=0, orient=orient, arch=w.arch,
                          epoch=e, n_epochs=epochs)
        stats.append([int(x) for x in oracle.train(syn0, syn1, tree, tv, p)])
    t2 = time.time()
    s1, npairs1, _ = oracle.loglik(syn0, syn1, tree, hv, pe)
    assert npairs1 == npairs
    h = hashlib.sha256()
    h.update(syn0.tobytes())
    h.update(syn1.tobytes())
    src = open(oracle.SRC_PATH, "rb").read()
    return {
        "workload": name,
        "train_tokens": int(tv.size),
        "V": voc.V,
        "train_words": voc.train_words,
        "dim": w.dim,
        "cache_k": cache_k,
        "flush_every": flush_every,
        "order": "as printed (pair-major)",
        "orient": orient,
        "epochs": epochs,
        "stats": stats[0] if epochs == 1 else stats,
        "heldout_pairs": int(npairs),
        "init_mean_ll": s0 / npairs,
        "mean_ll": s1 / npairs,
        "model_sha256": h.hexdigest(),
        "oracle_source_sha256": hashlib.sha256(src).hexdigest(),
        "train_seconds_single_core": round(t2 - t1, 1),
        "total_seconds": round(time.time() - t0, 1),
    }


def noise_log2(V: int) -> int:
    return max(10, min(27, (64 * V - 1).bit_length()))


def run_ns(name: str, K: int) -> dict:
    w = synth.WORKLOADS[name]
    t0 = time.time()
    tok = synth.workload_corpus(w)
    held = synth.workload_corpus(w, heldout=True)
    voc = oracle.build_vocab(tok, w.vocab, w.min_count)
    tv = oracle.remap(tok, voc.id_to_vocab)
    del tok
    hv = oracle.remap(held, voc.id_to_vocab)
    L = noise_log2(voc.V)
    table = oracle.noise_table(voc.vocab_counts, L)
    syn0, _ = synth.init_weights(voc.V, w.dim)
    syn1 = np.zeros((voc.V, w.dim), np.float32)
    pe = oracle.params(voc.V, w.dim, window=w.window, sample=w.sample, train_words=voc.train_words,
                       seed=synth.SEED_EVAL, negative=K)
    s0, npairs, nterms = oracle.ns_objective(syn0, syn1, voc.vocab_counts, table, L, hv, pe)
    p = oracle.params(voc.V, w.dim, window=w.window, sample=w.sample, alpha0=w.alpha0, train_words=voc.train_words,
                      corpus_tokens=tv.size, seed=synth.SEED_TRAIN, negative=K)
    t1 = time.time()
    st = oracle.train_ns(syn0, syn1, voc.vocab_counts, table, L, tv, p)
    t2 = time.time()
    s1, np1, nt1 = oracle.ns_objective(syn0, syn1, voc.vocab_counts, table, L, hv, pe)
    assert (np1, nt1) == (npairs, nterms)
    return {
        "workload": name,
        "negative": K,
        "log2_table": L,
        "V": voc.V,
        "train_words": voc.train_words,
        "dim": w.dim,
        "stats": [int(x) for x in st],
        "heldout_pairs": int(npairs),
        "heldout_terms": int(nterms),
        "init_mean_objective": s0 / npairs,
        "mean_objective": s1 / npairs,
        "oracle_source_sha256": hashlib.sha256(open(oracle.SRC_PATH, "rb").read()).hexdigest(),
        "train_seconds_single_core": round(t2 - t1, 1),
        "total_seconds": round(time.time() - t0, 1),
    }


def sampler(name: str) -> dict:
    w = synth.WORKLOADS[name]
    t0 = time.time()
    tok = synth.workload_corpus(w)
    voc = oracle.build_vocab(tok, w.vocab, w.min_count)
    tree = oracle.build_huffman(voc.vocab_counts)
    tv = oracle.remap(tok, voc.id_to_vocab)
    del tok
    # whole-document chunks placed in the global stream by first_raw_index; the checksum is a
    # sum over pairs mod 2^64, so chunk checksums add up
    chunk = 10_000 * w.doc_len
    total = kept = nodes = checksum = 0
    for off in range(0, tv.size, chunk):
        part = tv[off:off + chunk]
        p = oracle.params(voc.V, 8, window=w.window, sample=w.sample, train_words=voc.train_words,
                          seed=synth.SEED_TRAIN, first_raw_index=off)
        pr = oracle.sample_pairs(part, p, voc.vocab_counts, want_mask=False)
        total += pr.total
        kept += pr.n_kept
        checksum = (checksum + pr.checksum) % (1 << 64)
        nodes += int(tree.codelen[part[pr.centre - off]].astype(np.int64).sum())
    def sha(*arrays):
        h = hashlib.sha256()
        for a in arrays:
            h.update(np.ascontiguousarray(a).tobytes())
        return h.hexdigest()

    return {
        "workload": name,
        "n_tokens": int(tv.size),
        "V": voc.V,
        "train_words": voc.train_words,
        "counts_by_id_sha256": sha(voc.counts),
        "vocab_ids_sha256": sha(voc.vocab_ids),
        "id_to_vocab_sha256": sha(voc.id_to_vocab),
        "codelen_code_sha256": sha(tree.codelen, tree.code),
        "point_off_points_sha256": sha(tree.point_off, tree.points),
        "max_codelen": int(tree.codelen.max()),
        "seed": synth.SEED_TRAIN,
        "pairs": total,
        "kept": kept,
        "pair_node_updates": nodes,
        "pairs_checksum": checksum,
        "oracle_source_sha256": hashlib.sha256(open(oracle.SRC_PATH, "rb").read()).hexdigest(),
        "total_seconds": round(time.time() - t0, 1),
    }


if __name__ == "__main__":
    import argparse
    ap = argparse.ArgumentParser()
    ap.add_argument("names", nargs="+")
    ap.add_argument("--train-tokens", type=int, default=0)
    ap.add_argument("--sampler", action="store_true")
    ap.add_argument("--orient", type=int, default=0, help="1: the window word's path, the centre's vector as input")
    ap.add_argument("--epochs", type=int, default=1)
    ap.add_argument("--ns", type=int, default=0, help="negatives per centre: train with negative sampling")
    a = ap.parse_args()
    for name in a.names:
        if a.ns:
            r = run_ns(name, a.ns)
            with open(os.path.join(HERE, f"oracle_ns{a.ns}_{name}.json"), "w") as f:
                json.dump(r, f, indent=1)
            print(json.dumps(r), flush=True)
            continue
        if a.sampler:
            r = sampler(name)
            with open(os.path.join(HERE, f"oracle_sampler_{name}.json"), "w") as f:
                json.dump(r, f, indent=1)
            print(json.dumps(r), flush=True)
            continue
        r = run(name, train_tokens=a.train_tokens, orient=a.orient, epochs=a.epochs)
        suffix = ((f"_orient{a.orient}" if a.orient else "") + (f"_epochs{a.epochs}" if a.epochs > 1 else "")
                  + (f"_first{a.train_tokens}" if a.train_tokens else ""))
        path = os.path.join(HERE, f"oracle_ll_{name}{suffix}.json")
        with open(path, "w") as f:
            json.dump(r, f, indent=1)
        print(json.dumps(r), flush=True)
