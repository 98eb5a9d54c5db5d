"""CPU oracle for hierarchical-softmax word2vec (ctypes wrapper over liboracle.so).

TEST INFRASTRUCTURE ONLY. Only the tests, ``__graft_entry__.smoke()`` and the
benchmark's CPU-baseline leg may import this package. The GPU library and its
Python binding never do.

Every function follows Vuurens, Eickhoff and de Vries, "Efficient Parallel
Learning of Word2Vec": Algorithm 1 (Cached Skipgram HS) for training, §2 for
the hierarchical softmax over a binary Huffman tree, §4.1 for the settings
(mintf, windowsize, vectorsize, downsample). Negative sampling, named in §2
as the alternative objective, follows Ji et al.'s shared-negative mini-batch
as the opening of §3.2 describes it. The readings used where the paper
is silent are listed at the top of ``w2v_oracle.c``.

Parity pins (what fixes the oracle other than itself) live in
``tests/test_oracle_*.py``. The Philox generator is pinned by the published
known-answer vectors; the tree by Kraft equality, exhaustive search and an
independent quadratic construction; the objective by normalisation; the
updates by finite differences and closed forms.
"""
from __future__ import annotations

import ctypes
import os
from dataclasses import dataclass

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
# W2V_ORACLE_LIB names another build of the same source (e.g. one made with -march=native).
LIB_PATH = os.environ.get("W2V_ORACLE_LIB") or os.path.join(_HERE, "liboracle.so")
SRC_PATH = os.path.join(_HERE, "w2v_oracle.c")

P = ctypes.c_void_p
I32, I64, U64, F32, F64 = ctypes.c_int32, ctypes.c_int64, ctypes.c_uint64, ctypes.c_float, ctypes.c_double


class Params(ctypes.Structure):
    _fields_ = [("V", I32), ("dim", I32), ("window", I32), ("doc_len", I32), ("sample", F64),
                ("alpha0", F32), ("epoch", I32), ("n_epochs", I32), ("train_words", I64),
                ("corpus_tokens", I64), ("first_raw_index", I64), ("seed", U64), ("cache_k", I32),
                ("flush_every", I32), ("order", I32), ("orient", I32), ("arch", I32), ("sync_batch", I32),
                ("max_centres", I64), ("negative", I32), ("reserved", I32)]


class _Tree(ctypes.Structure):
    _fields_ = [("vocab_counts", P), ("codelen", P), ("code", P), ("point_off", P), ("points", P)]


def build(force: bool = False) -> str:
    """Compile liboracle.so with gcc (plain C, no FMA contraction)."""
    import subprocess
    if force or not os.path.exists(LIB_PATH) or os.path.getmtime(LIB_PATH) < os.path.getmtime(SRC_PATH):
        subprocess.check_call(["gcc", "-O3", "-march=x86-64-v3", "-std=c11", "-Wall", "-Wextra", "-ffp-contract=off", "-fPIC",
                               "-shared", SRC_PATH, "-o", LIB_PATH, "-lm"])
    return LIB_PATH


_LIB = None


def lib():
    global _LIB
    if _LIB is None:
        if not os.path.exists(LIB_PATH):
            build()
        L = ctypes.CDLL(LIB_PATH)
        L.or_count.restype = I64
        L.or_count.argtypes = [P, I64, I32, P]
        L.or_vocab.restype = I32
        L.or_vocab.argtypes = [P, I32, I64, P, P, P, P]
        L.or_remap.restype = None
        L.or_remap.argtypes = [P, I64, P, P]
        L.or_huffman.restype = ctypes.c_int
        L.or_huffman.argtypes = [P, I32, P, P, P]
        L.or_huffman_codes.restype = ctypes.c_int
        L.or_huffman_codes.argtypes = [P, P, I32, P, P, P, P, I64]
        L.or_philox4x32_10.restype = None
        L.or_philox4x32_10.argtypes = [P, P, P]
        L.or_keep_thresholds.restype = None
        L.or_keep_thresholds.argtypes = [P, I32, F64, I64, P]
        L.or_alpha.restype = F32
        L.or_alpha.argtypes = [F32, I64, I32, I32, I64]
        L.or_sample_pairs.restype = I64
        L.or_sample_pairs.argtypes = [P, I64, ctypes.POINTER(Params), P, P, P, I64, P, P, P]
        L.or_train.restype = ctypes.c_int
        L.or_train.argtypes = [P, P, ctypes.POINTER(_Tree), P, I64, ctypes.POINTER(Params), P]
        L.or_train_sync.restype = ctypes.c_int
        L.or_train_sync.argtypes = [P, P, ctypes.POINTER(_Tree), P, I64, ctypes.POINTER(Params), I64, P]
        L.or_log_prob.restype = F64
        L.or_log_prob.argtypes = [P, P, I32, ctypes.POINTER(_Tree), I32]
        L.or_log_prob_f64.restype = F64
        L.or_log_prob_f64.argtypes = [P, P, I32, ctypes.POINTER(_Tree), I32]
        L.or_loglik.restype = ctypes.c_int
        L.or_loglik.argtypes = [P, P, ctypes.POINTER(_Tree), P, I64, ctypes.POINTER(Params), P, P, P]
        L.or_noise_weights.restype = I64
        L.or_noise_weights.argtypes = [P, I32, P]
        L.or_noise_table.restype = ctypes.c_int
        L.or_noise_table.argtypes = [P, I32, I32, P]
        L.or_sample_negatives.restype = I64
        L.or_sample_negatives.argtypes = [P, I64, ctypes.POINTER(Params), P, P, I32, P, I64, P, P]
        L.or_train_ns.restype = ctypes.c_int
        L.or_train_ns.argtypes = [P, P, P, P, I32, P, I64, ctypes.POINTER(Params), P]
        L.or_ns_objective.restype = ctypes.c_int
        L.or_ns_objective.argtypes = [P, P, P, P, I32, P, I64, ctypes.POINTER(Params), P, P, P]
        _LIB = L
    return _LIB


def _ptr(a: np.ndarray):
    assert a.flags.c_contiguous
    return a.ctypes.data


# ---------------------------------------------------------------- vocabulary
@dataclass
class Vocab:
    counts: np.ndarray        # int64[id_space]
    vocab_ids: np.ndarray     # int32[V]
    vocab_counts: np.ndarray  # int64[V]
    id_to_vocab: np.ndarray   # int32[id_space]
    train_words: int
    bad: int

    @property
    def V(self) -> int:
        return int(self.vocab_ids.size)


def build_vocab(tokens: np.ndarray, id_space: int, min_count: int) -> Vocab:
    tokens = np.ascontiguousarray(tokens, dtype=np.int32)
    counts = np.empty(id_space, np.int64)
    bad = lib().or_count(_ptr(tokens), tokens.size, id_space, _ptr(counts))
    ids = np.empty(id_space, np.int32)
    vc = np.empty(id_space, np.int64)
    i2v = np.empty(id_space, np.int32)
    tw = ctypes.c_int64(0)
    V = lib().or_vocab(_ptr(counts), id_space, min_count, _ptr(ids), _ptr(vc), _ptr(i2v), ctypes.byref(tw))
    return Vocab(counts, ids[:V].copy(), vc[:V].copy(), i2v, int(tw.value), int(bad))


def remap(tokens: np.ndarray, id_to_vocab: np.ndarray) -> np.ndarray:
    tokens = np.ascontiguousarray(tokens, dtype=np.int32)
    out = np.empty_like(tokens)
    lib().or_remap(_ptr(tokens), tokens.size, _ptr(id_to_vocab), _ptr(out))
    return out


# --------------------------------------------------------------- Huffman tree
@dataclass
class Tree:
    vocab_counts: np.ndarray  # int64[V]
    parent: np.ndarray        # int32[2V-1]  (inner index a, -1 at the root)
    bit: np.ndarray           # uint8[2V-1]
    node_count: np.ndarray    # int64[2V-1]
    codelen: np.ndarray       # uint8[V]
    code: np.ndarray          # uint64[V]
    point_off: np.ndarray     # int32[V+1]
    points: np.ndarray        # int32[sum len]

    @property
    def V(self) -> int:
        return int(self.codelen.size)

    def path(self, v: int):
        pts = self.points[self.point_off[v]:self.point_off[v + 1]]
        bits = [(int(self.code[v]) >> j) & 1 for j in range(int(self.codelen[v]))]
        return list(map(int, pts)), bits

    def c(self) -> _Tree:
        return _Tree(_ptr(self.vocab_counts), _ptr(self.codelen), _ptr(self.code), _ptr(self.point_off),
                     _ptr(self.points))


def build_huffman(vocab_counts: np.ndarray) -> Tree:
    vc = np.ascontiguousarray(vocab_counts, dtype=np.int64)
    V = int(vc.size)
    parent = np.empty(2 * V - 1, np.int32)
    bit = np.empty(2 * V - 1, np.uint8)
    ncount = np.empty(2 * V - 1, np.int64)
    if lib().or_huffman(_ptr(vc), V, _ptr(parent), _ptr(bit), _ptr(ncount)) != 0:
        raise ValueError("Huffman construction needs V >= 2")
    codelen = np.empty(V, np.uint8)
    code = np.empty(V, np.uint64)
    off = np.empty(V + 1, np.int32)
    if lib().or_huffman_codes(_ptr(parent), _ptr(bit), V, _ptr(codelen), _ptr(code), _ptr(off), None, 0) != 0:
        raise ValueError("code longer than 64 bits")
    points = np.empty(int(off[V]), np.int32)
    lib().or_huffman_codes(_ptr(parent), _ptr(bit), V, _ptr(codelen), _ptr(code), _ptr(off), _ptr(points),
                           points.size)
    return Tree(vc, parent, bit, ncount, codelen, code, off, points)


# --------------------------------------------------------------------- Philox
def philox4x32_10(ctr, key):
    c = np.asarray(ctr, dtype=np.uint32)
    k = np.asarray(key, dtype=np.uint32)
    out = np.empty(4, np.uint32)
    lib().or_philox4x32_10(_ptr(c), _ptr(k), _ptr(out))
    return [int(x) for x in out]


def keep_thresholds(vocab_counts: np.ndarray, sample: float, train_words: int) -> np.ndarray:
    vc = np.ascontiguousarray(vocab_counts, dtype=np.int64)
    thr = np.empty(vc.size, np.uint64)
    lib().or_keep_thresholds(_ptr(vc), vc.size, sample, train_words, _ptr(thr))
    return thr


def alpha(alpha0: float, raw_pos: int, epoch: int, n_epochs: int, corpus_tokens: int) -> float:
    return float(lib().or_alpha(alpha0, raw_pos, epoch, n_epochs, corpus_tokens))


# ------------------------------------------------------------------- sampling
def params(V: int, dim: int, *, window: int, sample: float = 0.0, alpha0: float = 0.025, train_words: int = 0,
           corpus_tokens: int = 0, seed: int = 3, epoch: int = 0, n_epochs: int = 1, doc_len: int = 1000,
           first_raw_index: int = 0, cache_k: int = 0, flush_every: int = 10, order: int = 0, orient: int = 0,
           arch: int = 0, sync_batch: int = 4096, max_centres: int = -1, negative: int = 5) -> Params:
    return Params(V, dim, window, doc_len, sample, alpha0, epoch, n_epochs, train_words, corpus_tokens,
                  first_raw_index, seed, cache_k, flush_every, order, orient, arch, sync_batch, max_centres, negative,
                  0)


@dataclass
class Pairs:
    centre: np.ndarray   # int64 global raw index
    context: np.ndarray  # int64 global raw index
    total: int
    n_kept: int
    checksum: int
    keep_mask: np.ndarray | None


def sample_pairs(tokens_v: np.ndarray, p: Params, vocab_counts: np.ndarray, cap: int | None = None,
                 want_mask: bool = True) -> Pairs:
    tok = np.ascontiguousarray(tokens_v, dtype=np.int32)
    vc = np.ascontiguousarray(vocab_counts, dtype=np.int64)
    if cap is None:
        # first pass: count only
        nk = ctypes.c_int64(0)
        cs = ctypes.c_uint64(0)
        total = lib().or_sample_pairs(_ptr(tok), tok.size, ctypes.byref(p), _ptr(vc), None, None, 0, None,
                                      ctypes.byref(nk), ctypes.byref(cs))
        cap = int(total)
    c = np.empty(cap, np.int64)
    x = np.empty(cap, np.int64)
    mask = np.empty(tok.size, np.uint8) if want_mask else None
    nk = ctypes.c_int64(0)
    cs = ctypes.c_uint64(0)
    total = lib().or_sample_pairs(_ptr(tok), tok.size, ctypes.byref(p), _ptr(vc), _ptr(c), _ptr(x), cap,
                                  _ptr(mask) if mask is not None else None, ctypes.byref(nk), ctypes.byref(cs))
    if total < 0:
        raise RuntimeError("or_sample_pairs failed")
    m = min(cap, int(total))
    return Pairs(c[:m], x[:m], int(total), int(nk.value), int(cs.value), mask)


# ------------------------------------------------------------------- training
def train(syn0: np.ndarray, syn1: np.ndarray, tree: Tree, tokens_v: np.ndarray, p: Params) -> np.ndarray:
    """In place on syn0 [V,d] / syn1 [V-1,d] (fp32). Returns stats int64[5]."""
    assert syn0.dtype == np.float32 and syn1.dtype == np.float32
    tok = np.ascontiguousarray(tokens_v, dtype=np.int32)
    st = np.zeros(5, np.int64)
    t = tree.c()
    if lib().or_train(_ptr(syn0), _ptr(syn1), ctypes.byref(t), _ptr(tok), tok.size, ctypes.byref(p), _ptr(st)):
        raise RuntimeError("or_train failed")
    return st


def train_sync(syn0: np.ndarray, syn1: np.ndarray, tree: Tree, tokens_v: np.ndarray, p: Params,
               n_batches: int = -1) -> np.ndarray:
    assert syn0.dtype == np.float32 and syn1.dtype == np.float32
    tok = np.ascontiguousarray(tokens_v, dtype=np.int32)
    st = np.zeros(5, np.int64)
    t = tree.c()
    if lib().or_train_sync(_ptr(syn0), _ptr(syn1), ctypes.byref(t), _ptr(tok), tok.size, ctypes.byref(p),
                           n_batches, _ptr(st)):
        raise RuntimeError("or_train_sync failed")
    return st


def log_prob(x: np.ndarray, syn1: np.ndarray, tree: Tree, v: int) -> float:
    t = tree.c()
    if x.dtype == np.float64:
        return float(lib().or_log_prob_f64(_ptr(x), _ptr(syn1), x.size, ctypes.byref(t), v))
    return float(lib().or_log_prob(_ptr(x), _ptr(syn1), x.size, ctypes.byref(t), v))


def loglik(syn0: np.ndarray, syn1: np.ndarray, tree: Tree, tokens_v: np.ndarray, p: Params):
    """(sum of the held-out objective, n_terms, n_nodes).

    p.arch 0: log P(v|w) summed over the sampler's pairs (v, w).
    p.arch 1 (CBOW): log P(v|h) summed over the sampler's centres that have a
    window, h = the mean of the window words' vectors.
    """
    tok = np.ascontiguousarray(tokens_v, dtype=np.int32)
    s = ctypes.c_double(0)
    npairs = ctypes.c_int64(0)
    nn = ctypes.c_int64(0)
    t = tree.c()
    if lib().or_loglik(_ptr(syn0), _ptr(syn1), ctypes.byref(t), _ptr(tok), tok.size, ctypes.byref(p),
                       ctypes.byref(s), ctypes.byref(npairs), ctypes.byref(nn)):
        raise RuntimeError("or_loglik failed")
    return float(s.value), int(npairs.value), int(nn.value)


# ---------------------------------------------------------- negative sampling
def noise_weights(vocab_counts: np.ndarray):
    """(weights int64[V], total): isqrt(c * isqrt(c)) per word (unigram^(3/4) in integers)."""
    vc = np.ascontiguousarray(vocab_counts, dtype=np.int64)
    w = np.empty(vc.size, np.int64)
    tot = lib().or_noise_weights(_ptr(vc), vc.size, _ptr(w))
    return w, int(tot)


def noise_table(vocab_counts: np.ndarray, log2_size: int) -> np.ndarray:
    vc = np.ascontiguousarray(vocab_counts, dtype=np.int64)
    t = np.empty(1 << log2_size, np.int32)
    if lib().or_noise_table(_ptr(vc), vc.size, log2_size, _ptr(t)) != 0:
        raise ValueError("bad noise-table input")
    return t


@dataclass
class Negatives:
    negatives: np.ndarray   # int32[min(cap, kept)][K], -1 = dropped (equal to the centre)
    n_kept: int
    checksum: int


def sample_negatives(tokens_v: np.ndarray, p: Params, vocab_counts: np.ndarray, table: np.ndarray, log2_size: int,
                     cap: int = 0) -> Negatives:
    tok = np.ascontiguousarray(tokens_v, dtype=np.int32)
    vc = np.ascontiguousarray(vocab_counts, dtype=np.int64)
    out = np.empty((max(cap, 0), p.negative), np.int32)
    nk = ctypes.c_int64(0)
    cs = ctypes.c_uint64(0)
    r = lib().or_sample_negatives(_ptr(tok), tok.size, ctypes.byref(p), _ptr(vc), _ptr(table), log2_size,
                                  _ptr(out) if cap > 0 else None, cap, ctypes.byref(nk), ctypes.byref(cs))
    if r < 0:
        raise RuntimeError("or_sample_negatives failed")
    return Negatives(out[:min(cap, int(nk.value))], int(nk.value), int(cs.value))


def train_ns(syn0: np.ndarray, syn1: np.ndarray, vocab_counts: np.ndarray, table: np.ndarray, log2_size: int,
             tokens_v: np.ndarray, p: Params) -> np.ndarray:
    """Skip-gram with shared negatives, in place on syn0 [V,d] / syn1 [V,d]. Returns stats int64[5]."""
    assert syn0.dtype == np.float32 and syn1.dtype == np.float32 and syn1.shape[0] == syn0.shape[0]
    tok = np.ascontiguousarray(tokens_v, dtype=np.int32)
    vc = np.ascontiguousarray(vocab_counts, dtype=np.int64)
    st = np.zeros(5, np.int64)
    if lib().or_train_ns(_ptr(syn0), _ptr(syn1), _ptr(vc), _ptr(table), log2_size, _ptr(tok), tok.size,
                         ctypes.byref(p), _ptr(st)):
        raise RuntimeError("or_train_ns failed")
    return st


def ns_objective(syn0: np.ndarray, syn1: np.ndarray, vocab_counts: np.ndarray, table: np.ndarray, log2_size: int,
                 tokens_v: np.ndarray, p: Params):
    """(sum over the sampler's pairs of the negative-sampling objective, n_pairs, n_terms)."""
    tok = np.ascontiguousarray(tokens_v, dtype=np.int32)
    vc = np.ascontiguousarray(vocab_counts, dtype=np.int64)
    s = ctypes.c_double(0)
    npairs = ctypes.c_int64(0)
    nt = ctypes.c_int64(0)
    if lib().or_ns_objective(_ptr(syn0), _ptr(syn1), _ptr(vc), _ptr(table), log2_size, _ptr(tok), tok.size,
                             ctypes.byref(p), ctypes.byref(s), ctypes.byref(npairs), ctypes.byref(nt)):
        raise RuntimeError("or_ns_objective failed")
    return float(s.value), int(npairs.value), int(nt.value)
