"""MI355X hierarchical-softmax word2vec: Python binding of libw2v.so.

Argument marshalling only: every step runs in the library's HIP kernels.
PyTorch provides device memory and the current stream. The library never
allocates device memory; workspaces are torch uint8 tensors made here.

Entry points mirror the C ABI in include/w2v.h:
    build_vocab, build_huffman, train_hs_epoch, hs_loglik
    build_noise_table, train_ns_epoch, ns_objective (negative sampling)
plus the test hooks sample_pairs, keep_thresholds and sample_negatives.
"""
from __future__ import annotations

import ctypes
import os
from dataclasses import dataclass, field

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libw2v.so")

W2V_OK, W2V_E_ARG, W2V_E_RANGE, W2V_E_WORKSPACE, W2V_E_DEVICE = 0, -1, -2, -3, -4
N_STATS = 5
STAT_NAMES = ("raw_tokens", "in_vocab_tokens", "kept_centres", "pairs", "node_updates")

P = ctypes.c_void_p
I32, I64, U64 = ctypes.c_int32, ctypes.c_int64, ctypes.c_uint64


class W2VError(RuntimeError):
    def __init__(self, code: int, msg: str):
        super().__init__(f"w2v error {code}: {msg}")
        self.code = code


class CModel(ctypes.Structure):
    _fields_ = [("syn0", P), ("syn1", P), ("V", I32), ("dim", I32), ("row_stride", I32), ("reserved0", I32),
                ("vocab_counts", P), ("train_words", I64), ("codelen", P), ("code", P), ("point_off", P),
                ("points", P)]


class CParams(ctypes.Structure):
    _fields_ = [("arch", I32), ("mode", I32), ("window", I32), ("doc_len", I32), ("sample", ctypes.c_double),
                ("alpha0", ctypes.c_float), ("epoch", I32), ("n_epochs", I32), ("reserved1", I32),
                ("corpus_tokens", I64), ("first_raw_index", I64), ("seed", U64), ("cache_k", I32),
                ("flush_every", I32), ("sync_batch", I32), ("workers", I32), ("write_policy", I32),
                ("flush_policy", I32), ("hot_k", I32), ("negative", I32), ("cache_mode", I32),
                ("span_refresh", I32), ("span_stash", I32), ("stash_from", I32)]


assert ctypes.sizeof(CModel) == 80 and ctypes.sizeof(CParams) == 112

_LIB = None


def lib() -> ctypes.CDLL:
    """The loaded libw2v.so; raises if it has not been built."""
    global _LIB
    if _LIB is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing: build it with __graft_entry__.build() "
                               "(there is no fallback implementation)")
        L = ctypes.CDLL(LIB_PATH)
        L.w2v_last_error.restype = ctypes.c_char_p
        L.w2v_last_error.argtypes = []
        L.w2v_build_vocab_workspace_bytes.restype = ctypes.c_size_t
        L.w2v_build_vocab_workspace_bytes.argtypes = [I32]
        L.w2v_build_vocab.restype = ctypes.c_int
        L.w2v_build_vocab.argtypes = [P, I64, I32, I64, P, P, P, P, P, P, P, P, ctypes.c_size_t, P]
        L.w2v_build_huffman_workspace_bytes.restype = ctypes.c_size_t
        L.w2v_build_huffman_workspace_bytes.argtypes = [I32]
        L.w2v_build_huffman.restype = ctypes.c_int
        L.w2v_build_huffman.argtypes = [P, I32, P, P, P, P, I64, P, P, P, ctypes.c_size_t, P]
        L.w2v_train_workspace_bytes.restype = ctypes.c_size_t
        L.w2v_train_workspace_bytes.argtypes = [ctypes.POINTER(CModel), I64, ctypes.POINTER(CParams)]
        L.w2v_train_hs_epoch.restype = ctypes.c_int
        L.w2v_train_hs_epoch.argtypes = [ctypes.POINTER(CModel), P, I64, ctypes.POINTER(CParams), P, P,
                                         ctypes.c_size_t, P]
        L.w2v_last_train_kernel_ms.restype = ctypes.c_int
        L.w2v_last_train_kernel_ms.argtypes = [ctypes.POINTER(ctypes.c_float)]
        L.w2v_train_word_span.restype = I32
        L.w2v_train_word_span.argtypes = [ctypes.POINTER(CModel), ctypes.POINTER(CParams)]
        L.w2v_last_train_launch.restype = ctypes.c_int
        L.w2v_last_train_launch.argtypes = [ctypes.POINTER(I32), ctypes.POINTER(I32)]
        L.w2v_hs_loglik_workspace_bytes.restype = ctypes.c_size_t
        L.w2v_hs_loglik_workspace_bytes.argtypes = [ctypes.POINTER(CModel), I64, ctypes.POINTER(CParams)]
        L.w2v_hs_loglik.restype = ctypes.c_int
        L.w2v_hs_loglik.argtypes = [ctypes.POINTER(CModel), P, I64, ctypes.POINTER(CParams), P, P, P, P,
                                    ctypes.c_size_t, P]
        L.w2v_sample_pairs_workspace_bytes.restype = ctypes.c_size_t
        L.w2v_sample_pairs_workspace_bytes.argtypes = [I32, I64, ctypes.POINTER(CParams)]
        L.w2v_sample_pairs.restype = ctypes.c_int
        L.w2v_sample_pairs.argtypes = [P, I64, I32, P, I64, ctypes.POINTER(CParams), P, P, I64, P, P, P, P, P,
                                       ctypes.c_size_t, P]
        L.w2v_keep_thresholds.restype = ctypes.c_int
        L.w2v_keep_thresholds.argtypes = [P, I32, ctypes.c_double, I64, P, P]
        L.w2v_noise_table_workspace_bytes.restype = ctypes.c_size_t
        L.w2v_noise_table_workspace_bytes.argtypes = [I32]
        L.w2v_build_noise_table.restype = ctypes.c_int
        L.w2v_build_noise_table.argtypes = [P, I32, I32, P, P, P, ctypes.c_size_t, P]
        L.w2v_train_ns_workspace_bytes.restype = ctypes.c_size_t
        L.w2v_train_ns_workspace_bytes.argtypes = [ctypes.POINTER(CModel), I64, ctypes.POINTER(CParams)]
        L.w2v_train_ns_epoch.restype = ctypes.c_int
        L.w2v_train_ns_epoch.argtypes = [ctypes.POINTER(CModel), P, I32, P, I64, ctypes.POINTER(CParams), P, P,
                                         ctypes.c_size_t, P]
        L.w2v_ns_objective_workspace_bytes.restype = ctypes.c_size_t
        L.w2v_ns_objective_workspace_bytes.argtypes = [ctypes.POINTER(CModel), I64, ctypes.POINTER(CParams)]
        L.w2v_ns_objective.restype = ctypes.c_int
        L.w2v_ns_objective.argtypes = [ctypes.POINTER(CModel), P, I32, P, I64, ctypes.POINTER(CParams), P, P, P, P,
                                       ctypes.c_size_t, P]
        L.w2v_noalloc_scratch_bytes.restype = ctypes.c_size_t
        L.w2v_noalloc_scratch_bytes.argtypes = []
        L.w2v_hs_loglik_noalloc.restype = ctypes.c_int
        L.w2v_hs_loglik_noalloc.argtypes = [ctypes.POINTER(CModel), P, I64, ctypes.POINTER(CParams), P, P, P, P]
        L.w2v_sample_negatives_workspace_bytes.restype = ctypes.c_size_t
        L.w2v_sample_negatives_workspace_bytes.argtypes = [I32, I64, ctypes.POINTER(CParams)]
        L.w2v_sample_negatives.restype = ctypes.c_int
        L.w2v_sample_negatives.argtypes = [P, I64, I32, P, I64, ctypes.POINTER(CParams), P, I32, P, I64, P, P, P,
                                           ctypes.c_size_t, P]
        _LIB = L
    return _LIB


def last_error() -> str:
    return lib().w2v_last_error().decode()


def _check(rc: int):
    if rc != W2V_OK:
        raise W2VError(rc, last_error())


def _dev_ptr(t: torch.Tensor | None, dtype: torch.dtype, name: str):
    if t is None:
        return None
    if not t.is_cuda:
        raise ValueError(f"{name} must be a GPU tensor")
    if t.dtype != dtype:
        raise ValueError(f"{name} must be {dtype}, got {t.dtype}")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    return t.data_ptr()


def _stream(device: torch.device | None = None) -> int:
    return torch.cuda.current_stream(device).cuda_stream


def _workspace(nbytes: int, device) -> torch.Tensor:
    return torch.empty(max(int(nbytes), 1), dtype=torch.uint8, device=device)


# ---------------------------------------------------------------- vocabulary
@dataclass
class Vocab:
    counts_by_id: torch.Tensor   # int64[id_space]
    vocab_ids: torch.Tensor      # int32[V]
    vocab_counts: torch.Tensor   # int64[V]
    id_to_vocab: torch.Tensor    # int32[id_space]
    V: int
    train_words: int
    tokens: torch.Tensor | None  # int32[n] vocabulary indices (-1 = dropped)


def build_vocab(tokens: torch.Tensor, id_space: int, min_count: int = 5, remap: bool = True) -> Vocab:
    """Count ids, keep count >= min_count, order by (count desc, id asc); optionally remap tokens."""
    dev = tokens.device
    n = tokens.numel()
    counts = torch.empty(id_space, dtype=torch.int64, device=dev)
    ids = torch.empty(id_space, dtype=torch.int32, device=dev)
    vc = torch.empty(id_space, dtype=torch.int64, device=dev)
    i2v = torch.empty(id_space, dtype=torch.int32, device=dev)
    out = torch.empty(n, dtype=torch.int32, device=dev) if remap else None
    ws = _workspace(lib().w2v_build_vocab_workspace_bytes(id_space), dev)
    V = ctypes.c_int32(0)
    tw = ctypes.c_int64(0)
    _check(lib().w2v_build_vocab(_dev_ptr(tokens, torch.int32, "tokens"), n, id_space, min_count,
                                 counts.data_ptr(), ids.data_ptr(), vc.data_ptr(), i2v.data_ptr(),
                                 out.data_ptr() if out is not None else None, ctypes.byref(V), ctypes.byref(tw),
                                 ws.data_ptr(), ws.numel(), _stream(dev)))
    v = V.value
    return Vocab(counts, ids[:v], vc[:v], i2v, v, tw.value, out)


# ---------------------------------------------------------------- Huffman
@dataclass
class Tree:
    codelen: torch.Tensor    # uint8[V]
    code: torch.Tensor       # int64[V] (bit patterns of uint64)
    point_off: torch.Tensor  # int32[V+1]
    points: torch.Tensor     # int32[sum len]
    max_len: int


def build_huffman(vocab_counts: torch.Tensor) -> Tree:
    dev = vocab_counts.device
    V = vocab_counts.numel()
    vc = vocab_counts.contiguous()
    codelen = torch.empty(V, dtype=torch.uint8, device=dev)
    code = torch.empty(V, dtype=torch.int64, device=dev)
    off = torch.empty(V + 1, dtype=torch.int32, device=dev)
    ws = _workspace(lib().w2v_build_huffman_workspace_bytes(V), dev)
    plen = ctypes.c_int64(0)
    mlen = ctypes.c_int32(0)
    # codes are at most 64 long: one call with a buffer of that bound builds the tree once
    points = torch.empty(max(V * min(64, V - 1), 1), dtype=torch.int32, device=dev)
    _check(lib().w2v_build_huffman(_dev_ptr(vc, torch.int64, "vocab_counts"), V, codelen.data_ptr(),
                                   code.data_ptr(), off.data_ptr(), points.data_ptr(), points.numel(),
                                   ctypes.byref(plen), ctypes.byref(mlen), ws.data_ptr(), ws.numel(), _stream(dev)))
    return Tree(codelen, code, off, points[:plen.value], mlen.value)


# ---------------------------------------------------------------- model
def padded_stride(dim: int) -> int:
    """Row stride in floats: dim rounded up to 32 (128-byte rows)."""
    return (dim + 31) // 32 * 32


@dataclass
class Model:
    syn0: torch.Tensor          # float32[V, stride]
    syn1: torch.Tensor          # float32[V-1, stride]
    dim: int
    vocab_counts: torch.Tensor  # int64[V]
    train_words: int
    tree: Tree

    @property
    def V(self) -> int:
        return self.syn0.shape[0]

    @property
    def stride(self) -> int:
        return self.syn0.shape[1]

    def c(self) -> CModel:
        for name, t in (("syn0", self.syn0), ("syn1", self.syn1)):
            _dev_ptr(t, torch.float32, name)
        tr = self.tree
        return CModel(self.syn0.data_ptr(), self.syn1.data_ptr(), self.V, self.dim, self.stride, 0,
                      _dev_ptr(self.vocab_counts, torch.int64, "vocab_counts"), self.train_words,
                      tr.codelen.data_ptr() if tr else None, tr.code.data_ptr() if tr else None,
                      tr.point_off.data_ptr() if tr else None, tr.points.data_ptr() if tr else None)

    def vectors(self) -> tuple[torch.Tensor, torch.Tensor]:
        """(syn0[:, :dim], syn1[:, :dim]) views."""
        return self.syn0[:, :self.dim], self.syn1[:, :self.dim]


def make_model(syn0_init, syn1_init, vocab: Vocab, tree: Tree, device="cuda", stride: int | None = None,
               pad_value: float = 0.0) -> Model:
    """Copy [V, dim] initial weights (numpy or torch) into device rows of `stride` floats (default
    padded_stride(dim)); the padding columns hold pad_value."""
    s0 = torch.as_tensor(syn0_init, dtype=torch.float32)
    s1 = torch.as_tensor(syn1_init, dtype=torch.float32)
    V, dim = s0.shape
    stride = padded_stride(dim) if stride is None else stride
    syn0 = torch.full((V, stride), pad_value, dtype=torch.float32, device=device)
    syn1 = torch.full((max(V - 1, 1), stride), pad_value, dtype=torch.float32, device=device)
    syn0[:, :dim].copy_(s0)
    syn1[:V - 1, :dim].copy_(s1)
    return Model(syn0, syn1, dim, vocab.vocab_counts.contiguous(), vocab.train_words, tree)


# CBOW applies one update per node and centre, so its row stores lose more of
# the contended upper nodes' changes than skip-gram's; by default those rows
# take atomic adds there -- except with the word-row span (write_policy bit 3),
# where the stored rows measured both faster and no worse (1e8 tokens, d = 300:
# 254 instead of 488 ms, held-out CBOW objective -10.066 instead of -10.096).
HOT_K_CBOW = 1024


@dataclass
class Params:
    """Fields of w2v_params (include/w2v.h). hot_k=None picks 0 for skip-gram
    and HOT_K_CBOW for CBOW (0 for CBOW with the word-row span, write_policy bit 3)."""
    window: int
    sample: float = 0.0
    alpha0: float = 0.025
    arch: int = 0
    mode: int = 0
    doc_len: int = 1000
    epoch: int = 0
    n_epochs: int = 1
    corpus_tokens: int = 0
    first_raw_index: int = 0
    seed: int = 3
    cache_k: int = 31
    flush_every: int = 1000
    sync_batch: int = 4096
    workers: int = 0
    write_policy: int = 5
    flush_policy: int = 1
    hot_k: int | None = None
    negative: int = 5
    cache_mode: int = 0
    span_refresh: int = 0
    span_stash: int = 0
    stash_from: int = 0
    extra: dict = field(default_factory=dict)

    def c(self) -> CParams:
        return CParams(self.arch, self.mode, self.window, self.doc_len, float(self.sample), float(self.alpha0),
                       self.epoch, self.n_epochs, 0, self.corpus_tokens, self.first_raw_index, self.seed,
                       self.cache_k, self.flush_every, self.sync_batch, self.workers, self.write_policy,
                       self.flush_policy, self.resolved_hot_k(), self.negative, self.cache_mode, self.span_refresh,
                       self.span_stash, self.stash_from)

    def resolved_hot_k(self) -> int:
        if self.hot_k is not None:
            return self.hot_k
        return HOT_K_CBOW if self.arch == 1 and not (self.write_policy & 8) else 0


# ---------------------------------------------------------------- training
def train_hs_epoch(model: Model, tokens: torch.Tensor, p: Params, stats: torch.Tensor | None = None,
                   workspace: torch.Tensor | None = None) -> torch.Tensor:
    """One pass over tokens (vocabulary indices). Returns the device stats tensor int64[5]; does not sync."""
    dev = tokens.device
    cm, cp = model.c(), p.c()
    if cp.corpus_tokens <= 0:
        cp.corpus_tokens = tokens.numel()
    need = lib().w2v_train_workspace_bytes(ctypes.byref(cm), tokens.numel(), ctypes.byref(cp))
    if workspace is None or workspace.numel() < need:
        workspace = _workspace(need, dev)
    if stats is None:
        stats = torch.zeros(N_STATS, dtype=torch.int64, device=dev)
    _check(lib().w2v_train_hs_epoch(ctypes.byref(cm), _dev_ptr(tokens, torch.int32, "tokens"), tokens.numel(),
                                    ctypes.byref(cp), _dev_ptr(stats, torch.int64, "stats"), workspace.data_ptr(),
                                    workspace.numel(), _stream(dev)))
    return stats


def train_workspace_bytes(model: Model, n_tokens: int, p: Params) -> int:
    cm, cp = model.c(), p.c()
    if cp.corpus_tokens <= 0:
        cp.corpus_tokens = n_tokens
    return int(lib().w2v_train_workspace_bytes(ctypes.byref(cm), n_tokens, ctypes.byref(cp)))


def train_word_span(model: Model, p: Params) -> int:
    """Half-width of the word-row span kept in registers across centres for these settings (0: none)."""
    cm, cp = model.c(), p.c()
    if cp.corpus_tokens <= 0:
        cp.corpus_tokens = 1
    h = int(lib().w2v_train_word_span(ctypes.byref(cm), ctypes.byref(cp)))
    if h < 0:
        raise W2VError(W2V_E_ARG, last_error())
    return h


def last_train_kernel_ms() -> float:
    ms = ctypes.c_float(0)
    _check(lib().w2v_last_train_kernel_ms(ctypes.byref(ms)))
    return float(ms.value)


def last_train_launch() -> tuple[int, int]:
    """(workgroups, wavefronts) of the last asynchronous training launch."""
    g = ctypes.c_int32(0)
    wv = ctypes.c_int32(0)
    _check(lib().w2v_last_train_launch(ctypes.byref(g), ctypes.byref(wv)))
    return g.value, wv.value


def last_train_resources() -> dict:
    """LDS bytes per workgroup, VGPRs per lane and wavefronts per SIMD of the last asynchronous training
    launch."""
    lds, vg, occ = ctypes.c_int32(0), ctypes.c_int32(0), ctypes.c_int32(0)
    _check(lib().w2v_last_train_resources(ctypes.byref(lds), ctypes.byref(vg), ctypes.byref(occ)))
    return {"lds_bytes_per_workgroup": lds.value, "vgprs": vg.value, "waves_per_simd": occ.value}


def hs_loglik(model: Model, tokens: torch.Tensor, p: Params):
    """(sum of the held-out objective, n_terms, n_nodes). Synchronises.

    p.arch 0/2: log P(v|w) summed over the sampler's pairs; p.arch 1 (CBOW):
    log P(v|h) summed over the sampled centres with a window, h = the mean of
    the window words' vectors.
    """
    dev = tokens.device
    cm, cp = model.c(), p.c()
    ws = _workspace(lib().w2v_hs_loglik_workspace_bytes(ctypes.byref(cm), tokens.numel(), ctypes.byref(cp)), dev)
    s = ctypes.c_double(0)
    npairs = ctypes.c_int64(0)
    nn = ctypes.c_int64(0)
    _check(lib().w2v_hs_loglik(ctypes.byref(cm), _dev_ptr(tokens, torch.int32, "tokens"), tokens.numel(),
                               ctypes.byref(cp), ctypes.byref(s), ctypes.byref(npairs), ctypes.byref(nn),
                               ws.data_ptr(), ws.numel(), _stream(dev)))
    return s.value, npairs.value, nn.value


def hs_loglik_noalloc(model: Model, tokens: torch.Tensor, p: Params):
    """hs_loglik on the library's static scratch (no workspace is allocated). Synchronises."""
    dev = tokens.device
    cm, cp = model.c(), p.c()
    s = ctypes.c_double(0)
    npairs = ctypes.c_int64(0)
    nn = ctypes.c_int64(0)
    _check(lib().w2v_hs_loglik_noalloc(ctypes.byref(cm), _dev_ptr(tokens, torch.int32, "tokens"), tokens.numel(),
                                       ctypes.byref(cp), ctypes.byref(s), ctypes.byref(npairs), ctypes.byref(nn),
                                       _stream(dev)))
    return s.value, npairs.value, nn.value


# ---------------------------------------------------------------- test hooks
@dataclass
class Pairs:
    centre: torch.Tensor | None
    context: torch.Tensor | None
    total: int
    n_kept: int
    checksum: int
    keep_mask: torch.Tensor | None


def sample_pairs(tokens: torch.Tensor, V: int, vocab_counts: torch.Tensor, train_words: int, p: Params,
                 cap: int = 0, want_mask: bool = False) -> Pairs:
    dev = tokens.device
    cp = p.c()
    n = tokens.numel()
    ws = _workspace(lib().w2v_sample_pairs_workspace_bytes(V, n, ctypes.byref(cp)), dev)
    c = torch.empty(max(cap, 1), dtype=torch.int64, device=dev)
    x = torch.empty(max(cap, 1), dtype=torch.int64, device=dev)
    mask = torch.empty(max(n, 1), dtype=torch.uint8, device=dev) if want_mask else None
    npairs = ctypes.c_int64(0)
    nk = ctypes.c_int64(0)
    cs = ctypes.c_uint64(0)
    _check(lib().w2v_sample_pairs(_dev_ptr(tokens, torch.int32, "tokens"), n, V,
                                  _dev_ptr(vocab_counts, torch.int64, "vocab_counts"), train_words, ctypes.byref(cp),
                                  c.data_ptr() if cap else None, x.data_ptr() if cap else None, cap,
                                  mask.data_ptr() if mask is not None else None, ctypes.byref(npairs),
                                  ctypes.byref(nk), ctypes.byref(cs), ws.data_ptr(), ws.numel(), _stream(dev)))
    m = min(cap, npairs.value)
    return Pairs(c[:m] if cap else None, x[:m] if cap else None, npairs.value, nk.value, cs.value,
                 mask[:n] if mask is not None else None)


def keep_thresholds(vocab_counts: torch.Tensor, sample: float, train_words: int) -> torch.Tensor:
    V = vocab_counts.numel()
    thr = torch.empty(V, dtype=torch.int64, device=vocab_counts.device)
    _check(lib().w2v_keep_thresholds(_dev_ptr(vocab_counts, torch.int64, "vocab_counts"), V, float(sample),
                                     train_words, thr.data_ptr(), _stream(vocab_counts.device)))
    return thr


def kernel_source_hash() -> str:
    """First 16 hex digits of sha256 over the training kernel's sources (ties stored counter data to a build)."""
    import hashlib
    h = hashlib.sha256()
    for f in ("train.hip", "w2v_internal.h"):
        with open(os.path.join(os.path.dirname(os.path.abspath(__file__)), "csrc", f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()[:16]


# ---------------------------------------------------------- negative sampling
@dataclass
class Noise:
    table: torch.Tensor   # int32[2^log2_size] vocabulary indices
    log2_size: int
    total_weight: int


def noise_log2_size(V: int) -> int:
    """A table of about 64 entries per word: 2^ceil(log2(64 V)), between 2^10 and 2^27."""
    return max(10, min(27, (64 * max(V, 1) - 1).bit_length()))


def build_noise_table(vocab_counts: torch.Tensor, log2_size: int | None = None) -> Noise:
    V = vocab_counts.numel()
    L = noise_log2_size(V) if log2_size is None else log2_size
    dev = vocab_counts.device
    table = torch.empty(1 << L, dtype=torch.int32, device=dev)
    ws = _workspace(lib().w2v_noise_table_workspace_bytes(V), dev)
    tot = ctypes.c_int64(0)
    _check(lib().w2v_build_noise_table(_dev_ptr(vocab_counts, torch.int64, "vocab_counts"), V, L, table.data_ptr(),
                                       ctypes.byref(tot), ws.data_ptr(), ws.numel(), _stream(dev)))
    return Noise(table, L, tot.value)


def make_ns_model(syn0_init, syn1_init, vocab: Vocab, device="cuda", stride: int | None = None,
                  pad_value: float = 0.0) -> Model:
    """[V, dim] input and output vectors in device rows of `stride` floats (default padded_stride(dim);
    padding columns hold pad_value), no tree."""
    s0 = torch.as_tensor(syn0_init, dtype=torch.float32)
    s1 = torch.as_tensor(syn1_init, dtype=torch.float32)
    V, dim = s0.shape
    if tuple(s1.shape) != (V, dim):
        raise ValueError("output vectors must be [V, dim]")
    stride = padded_stride(dim) if stride is None else stride
    syn0 = torch.full((V, stride), pad_value, dtype=torch.float32, device=device)
    syn1 = torch.full((V, stride), pad_value, dtype=torch.float32, device=device)
    syn0[:, :dim].copy_(s0)
    syn1[:, :dim].copy_(s1)
    return Model(syn0, syn1, dim, vocab.vocab_counts.contiguous(), vocab.train_words, None)


def train_ns_epoch(model: Model, noise: Noise, tokens: torch.Tensor, p: Params,
                   stats: torch.Tensor | None = None) -> torch.Tensor:
    """One pass of skip-gram with shared negatives. Returns the device stats int64[5]; does not sync."""
    dev = tokens.device
    cm, cp = model.c(), p.c()
    if cp.corpus_tokens <= 0:
        cp.corpus_tokens = tokens.numel()
    ws = _workspace(lib().w2v_train_ns_workspace_bytes(ctypes.byref(cm), tokens.numel(), ctypes.byref(cp)), dev)
    if stats is None:
        stats = torch.zeros(N_STATS, dtype=torch.int64, device=dev)
    _check(lib().w2v_train_ns_epoch(ctypes.byref(cm), _dev_ptr(noise.table, torch.int32, "noise table"),
                                    noise.log2_size, _dev_ptr(tokens, torch.int32, "tokens"), tokens.numel(),
                                    ctypes.byref(cp), _dev_ptr(stats, torch.int64, "stats"), ws.data_ptr(),
                                    ws.numel(), _stream(dev)))
    return stats


def ns_objective(model: Model, noise: Noise, tokens: torch.Tensor, p: Params):
    """(sum of the negative-sampling objective over the sampler's pairs, n_pairs, n_terms). Synchronises."""
    dev = tokens.device
    cm, cp = model.c(), p.c()
    ws = _workspace(lib().w2v_ns_objective_workspace_bytes(ctypes.byref(cm), tokens.numel(), ctypes.byref(cp)), dev)
    s = ctypes.c_double(0)
    npairs = ctypes.c_int64(0)
    nt = ctypes.c_int64(0)
    _check(lib().w2v_ns_objective(ctypes.byref(cm), _dev_ptr(noise.table, torch.int32, "noise table"),
                                  noise.log2_size, _dev_ptr(tokens, torch.int32, "tokens"), tokens.numel(),
                                  ctypes.byref(cp), ctypes.byref(s), ctypes.byref(npairs), ctypes.byref(nt),
                                  ws.data_ptr(), ws.numel(), _stream(dev)))
    return s.value, npairs.value, nt.value


@dataclass
class Negatives:
    negatives: torch.Tensor | None   # int32[min(cap, kept), K], -1 = dropped
    n_kept: int
    checksum: int


def sample_negatives(tokens: torch.Tensor, V: int, vocab_counts: torch.Tensor, train_words: int, p: Params,
                     noise: Noise, cap: int = 0) -> Negatives:
    dev = tokens.device
    cp = p.c()
    n = tokens.numel()
    ws = _workspace(lib().w2v_sample_negatives_workspace_bytes(V, n, ctypes.byref(cp)), dev)
    out = torch.empty(max(cap, 1) * p.negative, dtype=torch.int32, device=dev)
    nk = ctypes.c_int64(0)
    cs = ctypes.c_uint64(0)
    _check(lib().w2v_sample_negatives(_dev_ptr(tokens, torch.int32, "tokens"), n, V,
                                      _dev_ptr(vocab_counts, torch.int64, "vocab_counts"), train_words,
                                      ctypes.byref(cp), _dev_ptr(noise.table, torch.int32, "noise table"),
                                      noise.log2_size, out.data_ptr() if cap else None, cap, ctypes.byref(nk),
                                      ctypes.byref(cs), ws.data_ptr(), ws.numel(), _stream(dev)))
    m = min(cap, nk.value)
    return Negatives(out[:m * p.negative].view(m, p.negative) if cap else None, nk.value, cs.value)
