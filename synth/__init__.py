"""Seeded synthetic inputs shared by the GPU path's tests, the bench and the CPU oracle.

This package produces data only (word-id streams, initial weights, the
workload table). It holds none of the word2vec arithmetic; the GPU library and
the oracle each implement that on their own.
"""
from __future__ import annotations

import ctypes
import os
from dataclasses import dataclass, field, replace

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libsynth.so")

# Seeds of the input recipe (one per role).
SEED_CORPUS = 1
SEED_HELDOUT = 2
SEED_TRAIN = 3
SEED_EVAL = 4
SEED_INIT = 5


@dataclass(frozen=True)
class Workload:
    """One synthetic workload: corpus shape plus the training settings run on it."""

    name: str
    n_tokens: int
    vocab: int            # id space of the generator (word ids 0..vocab-1)
    zipf_s: float
    topics: int           # 0 = plain i.i.d. Zipf
    dim: int
    window: int
    sample: float         # subsampling threshold t (0 = off)
    arch: int = 0         # 0 skip-gram, 1 CBOW
    min_count: int = 5
    alpha0: float = 0.025
    doc_len: int = 1000
    heldout_tokens: int = 1_000_000
    topic_frac: float = 0.05
    topic_boost: float = 20.0
    extra: dict = field(default_factory=dict)

    def scaled(self, n_tokens: int, heldout_tokens: int | None = None) -> "Workload":
        return replace(self, n_tokens=n_tokens,
                       heldout_tokens=self.heldout_tokens if heldout_tokens is None else heldout_tokens)


# The five workloads: a tiny one the oracle finishes in well under a second,
# three mid-size ones, and the large skip-gram one (V = 1M, d = 300).
WORKLOADS = {
    "tiny_sg_v1k_d50": Workload("tiny_sg_v1k_d50", 100_000, 1_000, 1.0, 0, 50, 2, 0.0,
                                heldout_tokens=100_000),
    "sg_v30k_d100": Workload("sg_v30k_d100", 10_000_000, 30_000, 1.0, 50, 100, 5, 1e-3),
    "sg_v100k_d200": Workload("sg_v100k_d200", 100_000_000, 100_000, 1.0, 50, 200, 5, 1e-4),
    "cbow_v100k_d300": Workload("cbow_v100k_d300", 100_000_000, 100_000, 1.0, 50, 300, 5, 1e-4,
                                arch=1, alpha0=0.05),
    "sg_v1m_d300": Workload("sg_v1m_d300", 1_000_000_000, 1_000_000, 1.05, 200, 300, 5, 1e-5),
}


def _lib():
    if not os.path.exists(LIB_PATH):
        raise RuntimeError(f"{LIB_PATH} is not built; run __graft_entry__.build()")
    lib = ctypes.CDLL(LIB_PATH)
    lib.synth_corpus.restype = ctypes.c_int
    lib.synth_corpus.argtypes = [ctypes.c_int64, ctypes.c_int32, ctypes.c_double, ctypes.c_int32,
                                 ctypes.c_double, ctypes.c_double, ctypes.c_int32, ctypes.c_uint64,
                                 ctypes.c_int32, ctypes.c_void_p]
    lib.synth_zipf_probs.restype = ctypes.c_int
    lib.synth_zipf_probs.argtypes = [ctypes.c_int32, ctypes.c_double, ctypes.c_void_p]
    lib.synth_topic_subset.restype = ctypes.c_int
    lib.synth_topic_subset.argtypes = [ctypes.c_uint64, ctypes.c_int32, ctypes.c_int32, ctypes.c_int32,
                                       ctypes.c_void_p]
    lib.synth_topic_size.restype = ctypes.c_int32
    lib.synth_topic_size.argtypes = [ctypes.c_int32, ctypes.c_double]
    lib.synth_doc_topic.restype = ctypes.c_int32
    lib.synth_doc_topic.argtypes = [ctypes.c_uint64, ctypes.c_int64, ctypes.c_int32]
    return lib


_LIB = None


def lib():
    global _LIB
    if _LIB is None:
        _LIB = _lib()
    return _LIB


def corpus(n_tokens: int, vocab: int, zipf_s: float, topics: int, seed: int, *, doc_len: int = 1000,
           topic_frac: float = 0.05, topic_boost: float = 20.0, threads: int = 0,
           out: np.ndarray | None = None) -> np.ndarray:
    """int32[n_tokens] word ids drawn from the Zipf + topic generator."""
    if out is None:
        out = np.empty(n_tokens, dtype=np.int32)
    assert out.dtype == np.int32 and out.flags.c_contiguous and out.size == n_tokens
    rc = lib().synth_corpus(n_tokens, vocab, zipf_s, topics, topic_frac, topic_boost, doc_len, seed,
                            threads, out.ctypes.data)
    if rc != 0:
        raise RuntimeError("synth_corpus failed")
    return out


def workload_corpus(w: Workload, heldout: bool = False, threads: int = 0) -> np.ndarray:
    n = w.heldout_tokens if heldout else w.n_tokens
    seed = SEED_HELDOUT if heldout else SEED_CORPUS
    return corpus(n, w.vocab, w.zipf_s, w.topics, seed, doc_len=w.doc_len, topic_frac=w.topic_frac,
                  topic_boost=w.topic_boost, threads=threads)


def zipf_probs(vocab: int, zipf_s: float) -> np.ndarray:
    p = np.empty(vocab, dtype=np.float64)
    lib().synth_zipf_probs(vocab, zipf_s, p.ctypes.data)
    return p


def topic_subset(seed: int, tau: int, vocab: int, frac: float = 0.05) -> np.ndarray:
    m = lib().synth_topic_size(vocab, frac)
    out = np.empty(m, dtype=np.int32)
    lib().synth_topic_subset(seed, tau, vocab, m, out.ctypes.data)
    return out


def doc_topic(seed: int, doc: int, topics: int) -> int:
    return int(lib().synth_doc_topic(seed, doc, topics))


def init_weights(V: int, dim: int, seed: int = SEED_INIT, syn1_scale: float = 0.0):
    """Initial model: syn0 ~ U(-0.5/d, 0.5/d); syn1 = 0, or U(-s, s) when syn1_scale > 0.

    Returns fp32 arrays of shape [V, dim] and [V-1, dim].
    """
    rng = np.random.default_rng(seed)
    syn0 = ((rng.random((V, dim), dtype=np.float64) - 0.5) / dim).astype(np.float32)
    if syn1_scale > 0:
        syn1 = ((rng.random((max(V - 1, 0), dim), dtype=np.float64) * 2 - 1) * syn1_scale).astype(np.float32)
    else:
        syn1 = np.zeros((max(V - 1, 0), dim), dtype=np.float32)
    return syn0, syn1
