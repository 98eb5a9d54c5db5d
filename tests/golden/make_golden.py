"""Write the oracle's full-epoch results that the GPU tests compare against.

Calls only the CPU oracle (and the input generator). For a workload it runs
one epoch of Algorithm 1 as printed (one sequential worker, top-31 inner-node
cache flushed every 10 centre words, §4.1 / Figure 1's c31 setting) from the
seeded initial model and stores the held-out mean log-likelihood per pair.

    python tests/golden/make_golden.py sg_v30k_d100 [more names...]
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


def run(name: str, cache_k: int = 31, flush_every: int = 10) -> dict:
    w = synth.WORKLOADS[name]
    t0 = time.time()
    tok = synth.workload_corpus(w)
    held = synth.workload_corpus(w, heldout=True)
    voc = oracle.build_vocab(tok, w.vocab, w.min_count)
    tree = oracle.build_huffman(voc.vocab_counts)
    tv = oracle.remap(tok, voc.id_to_vocab)
    del tok
    hv = oracle.remap(held, voc.id_to_vocab)
    syn0, syn1 = synth.init_weights(voc.V, w.dim)
    pe = oracle.params(voc.V, w.dim, window=w.window, sample=w.sample, train_words=voc.train_words,
                       seed=synth.SEED_EVAL)
    s0, npairs, _ = oracle.loglik(syn0, syn1, tree, hv, pe)
    p = oracle.params(voc.V, w.dim, window=w.window, sample=w.sample, alpha0=w.alpha0, train_words=voc.train_words,
                      corpus_tokens=tv.size, seed=synth.SEED_TRAIN, cache_k=cache_k, flush_every=flush_every,
                      order=0, arch=w.arch)
    t1 = time.time()
    st = oracle.train(syn0, syn1, tree, tv, p)
    t2 = time.time()
    s1, npairs1, _ = oracle.loglik(syn0, syn1, tree, hv, pe)
    assert npairs1 == npairs
    h = hashlib.sha256()
    h.update(syn0.tobytes())
    h.update(syn1.tobytes())
    src = open(oracle.SRC_PATH, "rb").read()
    return {
        "workload": name,
        "V": voc.V,
        "train_words": voc.train_words,
        "dim": w.dim,
        "cache_k": cache_k,
        "flush_every": flush_every,
        "order": "as printed (pair-major)",
        "stats": [int(x) for x in st],
        "heldout_pairs": int(npairs),
        "init_mean_ll": s0 / npairs,
        "mean_ll": s1 / npairs,
        "model_sha256": h.hexdigest(),
        "oracle_source_sha256": hashlib.sha256(src).hexdigest(),
        "train_seconds_single_core": round(t2 - t1, 1),
        "total_seconds": round(time.time() - t0, 1),
    }


if __name__ == "__main__":
    for name in sys.argv[1:]:
        r = run(name)
        path = os.path.join(HERE, f"oracle_ll_{name}.json")
        with open(path, "w") as f:
            json.dump(r, f, indent=1)
        print(json.dumps(r), flush=True)
