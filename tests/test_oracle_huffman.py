"""Pins of the oracle's vocabulary and Huffman tree (§2: the output layer is a
binary Huffman tree, a word is predicted by the turns on its root path).

What fixes these other than the oracle itself:
  * counts and vocabulary order against numpy's bincount / Python's sort;
  * Kraft equality (a full binary prefix code), checked in integers;
  * optimality: the weighted code length equals the minimum over every merge
    sequence, found by exhaustive search (V <= 8);
  * the construction rule (two-queue merge, leaf wins ties, first child gets
    bit 0) by an independent quadratic "scan for the minimum" construction;
  * textbook special cases (V = 2; 2^m equal counts give length m);
  * the generation-wise construction that the GPU's parallel merge follows
    (each generation's picks are a stable merge of the leaf queue with the
    inner nodes it started with) gives the same tree, bit for bit.
"""
import functools
import math

import numpy as np
import pytest

import oracle


# ---------------------------------------------------------------- vocabulary
def test_counts_and_vocab_order_match_independent_recount():
    rng = np.random.default_rng(11)
    id_space = 500
    tok = (rng.zipf(1.3, 50_000) - 1) % id_space
    tok = tok.astype(np.int32)
    voc = oracle.build_vocab(tok, id_space, 5)
    np.testing.assert_array_equal(voc.counts, np.bincount(tok, minlength=id_space))
    expect = sorted([i for i in range(id_space) if voc.counts[i] >= 5], key=lambda i: (-voc.counts[i], i))
    np.testing.assert_array_equal(voc.vocab_ids, np.array(expect, np.int32))
    assert voc.train_words == int(voc.counts[voc.counts >= 5].sum())
    assert voc.counts.sum() == tok.size
    for r, i in enumerate(expect):
        assert voc.id_to_vocab[i] == r
    dropped = voc.counts < 5
    assert (voc.id_to_vocab[dropped] == -1).all()
    tv = oracle.remap(tok, voc.id_to_vocab)
    np.testing.assert_array_equal(tv, voc.id_to_vocab[tok])


def test_out_of_range_tokens_are_counted_as_bad():
    tok = np.array([0, 1, 2, 7, -1, 3], np.int32)
    voc = oracle.build_vocab(tok, 4, 1)
    assert voc.bad == 2
    np.testing.assert_array_equal(voc.counts, [1, 1, 1, 1])


# -------------------------------------------------------------- Huffman: pins
def kraft_ok(codelen):
    L = int(max(codelen))
    return sum(1 << (L - int(l)) for l in codelen) == (1 << L)


@functools.lru_cache(maxsize=None)
def best_merge_cost(ws):
    """Minimum total merge cost (= weighted code length) over all merge sequences."""
    if len(ws) <= 1:
        return 0
    best = None
    n = len(ws)
    for i in range(n):
        for j in range(i + 1, n):
            s = ws[i] + ws[j]
            rest = tuple(sorted(ws[:i] + ws[i + 1:j] + ws[j + 1:] + (s,)))
            c = s + best_merge_cost(rest)
            if best is None or c < best:
                best = c
    return best


def naive_tree(counts):
    """Rule R7 written as 'repeatedly take the smallest active node' (O(V^2)).

    Ordering key of an active node: (count, 0 for a leaf / 1 for an inner node,
    position), where a leaf's position is its place in ascending-count order
    (vocabulary index V-1 first) and an inner node's is its creation index.
    """
    V = len(counts)
    active = [(int(counts[v]), 0, V - 1 - v, ("leaf", v)) for v in range(V)]
    parent = {}
    bit = {}
    for a in range(V - 1):
        picked = []
        for b in range(2):
            m = min(range(len(active)), key=lambda i: active[i][:3])
            picked.append(active.pop(m))
            parent[picked[-1][3]] = a
            bit[picked[-1][3]] = b
        active.append((picked[0][0] + picked[1][0], 1, a, ("inner", a)))
    codes, paths = [], []
    for v in range(V):
        node = ("leaf", v)
        up = []
        while node in parent:
            up.append((parent[node], bit[node]))
            node = ("inner", parent[node])
        up.reverse()
        paths.append([p for p, _ in up])
        codes.append(sum(b << j for j, (_, b) in enumerate(up)))
    return codes, paths


def desc_counts(rng, V, hi):
    return np.sort(rng.integers(1, hi, V))[::-1].astype(np.int64)


@pytest.mark.parametrize("V", [2, 3, 4, 5, 6, 7, 8])
@pytest.mark.parametrize("seed", range(6))
def test_weighted_length_is_optimal_by_exhaustive_search(V, seed):
    rng = np.random.default_rng(1000 * V + seed)
    counts = desc_counts(rng, V, 12 if seed % 2 else 1000)   # small range -> many ties
    t = oracle.build_huffman(counts)
    assert kraft_ok(t.codelen)
    cost = int((counts * t.codelen.astype(np.int64)).sum())
    assert cost == best_merge_cost(tuple(sorted(int(c) for c in counts)))


@pytest.mark.parametrize("V,seed", [(v, s) for v in (2, 3, 9, 17, 64, 200) for s in range(4)])
def test_codes_and_points_match_quadratic_construction(V, seed):
    rng = np.random.default_rng(7 * V + seed)
    counts = desc_counts(rng, V, 4 if seed == 0 else (30 if seed == 1 else 10_000))
    t = oracle.build_huffman(counts)
    codes, paths = naive_tree(counts)
    for v in range(V):
        pts, bits = t.path(v)
        assert pts == paths[v]
        assert int(t.code[v]) == codes[v]
        assert int(t.codelen[v]) == len(paths[v])
        assert pts[0] == V - 2  # root first


def test_two_words():
    t = oracle.build_huffman(np.array([10, 3], np.int64))
    assert list(t.codelen) == [1, 1]
    assert sorted(int(c) for c in t.code) == [0, 1]
    assert int(t.code[1]) == 0   # the smaller count leaves its queue first: bit 0
    assert list(t.points) == [0, 0]


@pytest.mark.parametrize("m", [1, 2, 3, 4, 6, 10])
def test_equal_counts_power_of_two_give_balanced_tree(m):
    t = oracle.build_huffman(np.full(1 << m, 7, np.int64))
    assert (t.codelen == m).all()
    # balanced: every leaf has a distinct code
    assert len(set(int(c) for c in t.code)) == 1 << m


def test_inner_node_counts_are_nondecreasing_and_cover_the_corpus():
    rng = np.random.default_rng(3)
    counts = desc_counts(rng, 3000, 100_000)
    t = oracle.build_huffman(counts)
    V = counts.size
    inner = t.node_count[V:]
    assert (np.diff(inner) >= 0).all()
    assert inner[-1] == counts.sum()   # the root covers everything
    # top-k inner nodes by count are exactly the last k created (reading of isFrequent)
    for k in (1, 7, 31):
        top = set(np.argsort(-inner, kind="stable")[:k].tolist())
        if len(set(inner[sorted(top)])) == k and inner[V - 2 - k] < inner[V - 1 - k]:
            assert top == set(range(V - 1 - k, V - 1))


def test_zipf_vocab_kraft_and_depth():
    # a realistic skewed vocabulary: Kraft equality and code lengths fit 64 bits
    V = 30000
    counts = np.floor(1e7 / np.arange(1, V + 1)).astype(np.int64) + 5
    t = oracle.build_huffman(counts)
    assert kraft_ok(t.codelen)
    assert t.codelen.max() <= 64
    assert t.point_off[-1] == int(t.codelen.astype(np.int64).sum())
    # entropy bound: H <= mean length < H + 1
    p = counts / counts.sum()
    H = float(-(p * np.log2(p)).sum())
    L = float((p * t.codelen).sum())
    assert H <= L < H + 1


def test_code_longer_than_64_bits_is_rejected():
    # Fibonacci counts give a maximally skewed tree: depth V-1
    fib = [1, 1]
    while len(fib) < 70:
        fib.append(fib[-1] + fib[-2])
    counts = np.array(sorted(fib, reverse=True), np.int64)
    with pytest.raises(ValueError):
        oracle.build_huffman(counts)


def test_v_below_two_is_rejected():
    with pytest.raises(ValueError):
        oracle.build_huffman(np.array([5], np.int64))


# ---------------------------------------------------------------- generations
def generation_tree(counts):
    """The tree built generation by generation: while an inner node that existed when a generation began is
    still queued, the inner front is such an "old" node, so the generation's picks are the stable merge of
    the leaf queue with the old nodes (a leaf first on a tie), cut after the last old node; merge a0 + j
    takes picks 2j (bit 0) and 2j + 1 (bit 1). An odd last pick (the last old node) opens one more merge
    with the smaller of the leaf front and the generation's first node. (The GPU builds the tree so.)"""
    V = counts.size
    leaf = counts[::-1].astype(np.int64)                      # ascending; position p is word V-1-p
    icount = np.zeros(max(V - 1, 1), np.int64)
    parent = np.full(2 * V - 1, -1, np.int32)
    bit = np.zeros(2 * V - 1, np.uint8)
    pl = ih = a = 0

    def put(child, node, b):
        parent[child] = node
        bit[child] = b

    while a < V - 1:
        a0 = a
        if a0 == ih:                                          # no inner node yet: two leaves
            put(V - 1 - pl, a, 0)
            put(V - 2 - pl, a, 1)
            icount[a] = leaf[pl] + leaf[pl + 1]
            pl, a = pl + 2, a + 1
            continue
        old = icount[ih:a0]
        nl = int(np.searchsorted(leaf[pl:], old[-1], side="right"))   # leaves at most the last old count
        vals = np.concatenate([leaf[pl:pl + nl], old])
        ids = np.concatenate([V - 1 - (pl + np.arange(nl)), V + ih + np.arange(old.size)])
        # stable merge, leaves before old nodes on a tie (leaves come first in the concatenation)
        order = np.argsort(vals, kind="stable")
        vals, ids = vals[order], ids[order]
        m = vals.size // 2
        for j in range(m):
            put(ids[2 * j], a0 + j, 0)
            put(ids[2 * j + 1], a0 + j, 1)
        icount[a0:a0 + m] = vals[0:2 * m:2] + vals[1:2 * m:2]
        a = a0 + m
        pl, ih = pl + nl, a0
        if vals.size % 2:                                     # the last old node opens one more merge
            put(ids[-1], a, 0)
            if pl < V and (a == a0 or leaf[pl] <= icount[a0]):
                put(V - 1 - pl, a, 1)
                icount[a] = vals[-1] + leaf[pl]
                pl += 1
            else:
                put(V + a0, a, 1)
                icount[a] = vals[-1] + icount[a0]
                ih += 1
            a += 1
    return parent, bit


@pytest.mark.parametrize("V,hi,seed", [(2, 9, 1), (3, 2, 2), (5, 3, 3), (64, 2, 4), (1000, 5, 5), (1000, 10**6, 6),
                                       (30_000, 50, 7)])
def test_generation_wise_construction_equals_the_two_queue_merge(V, hi, seed):
    rng = np.random.default_rng(seed)
    counts = np.sort(rng.integers(1, hi, V))[::-1].astype(np.int64)
    t = oracle.build_huffman(counts)
    parent, bit = generation_tree(counts)
    np.testing.assert_array_equal(parent, t.parent)
    np.testing.assert_array_equal(bit, t.bit)


def test_generation_wise_construction_on_zipf_and_equal_counts():
    p = 1.0 / np.arange(1, 20_001) ** 1.05
    for counts in (np.maximum(np.floor(p / p.sum() * 1e8), 5).astype(np.int64), np.full(4096, 7, np.int64)):
        counts = np.sort(counts)[::-1].copy()
        t = oracle.build_huffman(counts)
        parent, bit = generation_tree(counts)
        np.testing.assert_array_equal(parent, t.parent)
        np.testing.assert_array_equal(bit, t.bit)
