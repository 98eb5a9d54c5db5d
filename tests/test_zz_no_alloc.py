"""The allocation-free log-likelihood entry point (w2v_hs_loglik_noalloc), called through the C ABI,
against w2v_hs_loglik on the same model and tokens: two calls in a row on the static scratch, the
second with a smaller input, and a CBOW evaluation after them. Both entry points run the same
kernels in a fixed summation order, so the results must be identical."""
import ctypes
import os

import numpy as np
import pytest

import oracle
import synth
from gpu_common import corpus, log, oracle_side

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def w2v():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_1606_07822_amd as w2v
    w2v.lib()
    return w2v


def noalloc_call(w2v, model, tokens, p):
    import torch
    cm, cp = model.c(), p.c()
    s = ctypes.c_double(0.0)
    npairs = ctypes.c_int64(0)
    nn = ctypes.c_int64(0)
    rc = w2v.lib().w2v_hs_loglik_noalloc(ctypes.byref(cm), ctypes.c_void_p(tokens.data_ptr()), tokens.numel(),
                                         ctypes.byref(cp), ctypes.byref(s), ctypes.byref(npairs), ctypes.byref(nn),
                                         ctypes.c_void_p(torch.cuda.current_stream().cuda_stream))
    assert rc == w2v.W2V_OK, w2v.last_error()
    return s.value, npairs.value, nn.value


def test_noalloc_loglik_matches_workspace_loglik(w2v):
    import torch
    name = "sg_v30k_d100"
    s = oracle_side(name)
    voc = w2v.build_vocab(torch.from_numpy(s.tok).cuda(), s.w.vocab, s.w.min_count)
    tree = w2v.build_huffman(voc.vocab_counts)
    syn0, syn1 = synth.init_weights(s.voc.V, s.w.dim, syn1_scale=0.3)
    model = w2v.make_model(syn0, syn1, voc, tree)
    held = torch.from_numpy(oracle.remap(corpus(name, heldout=True), s.voc.id_to_vocab)).cuda()
    assert w2v.lib().w2v_hs_loglik_workspace_bytes(ctypes.byref(model.c()), held.numel(),
                                                   ctypes.byref(w2v.Params(window=5).c())) \
        <= w2v.lib().w2v_noalloc_scratch_bytes()
    for n, arch in ((held.numel(), 0), (300_000, 0), (200_000, 1)):
        log(f"noalloc loglik: {n} tokens, arch {arch}")
        tok = held[:n]
        p = w2v.Params(window=s.w.window, sample=s.w.sample, seed=synth.SEED_EVAL, arch=arch)
        got = noalloc_call(w2v, model, tok, p)
        ref = w2v.hs_loglik(model, tok, p)
        assert got == ref and got[1] > 0, (got, ref)
