"""Benchmark: trained words/sec of hierarchical-softmax skip-gram on one MI355X.

One step = the whole path over the synthetic corpus, resident in HBM: reset
of the model to the initial vectors (device copy), vocabulary (count, order,
remap), Huffman tree (codes, points), one training epoch (subsampling,
window draws, path walks, top-31 LDS cache), held-out log-likelihood. value = in-vocabulary raw tokens of the epoch / step time
(the classic tool's "words" count, taken before subsampling).

The JSON line also carries the roofline of the training kernel (algorithmic
bytes per launch from the byte model below, over the kernel's duration timed
with HIP events on its stream) and the CPU oracle's rate on a bounded sample.

Per-centre byte model (survey_model; roofline.achieved for a kernel without
the word-row span), per kept centre v with P > 0 window words (fp32 rows of
d floats):
    8 d (len(v) - cached(v))   inner-node rows read and written once
  + 8 d P                      window rows read once and updated once
  + 4 len(v) + 9               path indices, code, length
plus the cache traffic of each workgroup: fill 4 d k, write-back 8 d k per
flush and at the end.

Span model (span_model; roofline.achieved for a kernel that keeps word rows
across centres, write_policy bit 3): the word rows of a span of H kept
positions on each side of the centre stay in registers, so the 8 d P term
becomes 8 d per row entering a span: per work unit (a segment of consecutive
kept centres j0 .. j1-1 of a document with nk kept words) the rows of its
first centre's span, then per later centre the previous centre's row and the
row H positions ahead when it exists; each is read once and written back
once. This is what that kernel's algorithm moves: the per-centre model counts
window rows it never moves, so its quotient by the epoch time is no
bandwidth and can exceed the HBM peak on a fast device (it is reported
beside the roofline as survey_model).

With --cpu-child DIR the script is instead the CPU baseline's pinned child
process (see cpu_baseline).
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_HBM_GBS = 8000.0


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=3)
    ap.add_argument("--warmup", type=int, default=1)
    ap.add_argument("--workload", default="sg_v1m_d300")
    ap.add_argument("--cpu-seconds", type=float, default=15.0, help="target length of the CPU oracle sample")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    # the paper's experiments cache the top 31 nodes (48 also fit one workgroup's LDS beside the centre
    # records and the stash: 0.8 % shorter epoch, same held-out LL, but fewer algorithmic bytes per launch)
    ap.add_argument("--cache-k", type=int, default=31)
    ap.add_argument("--flush-every", type=int, default=1000)
    ap.add_argument("--flush-policy", type=int, default=1)
    ap.add_argument("--cache-mode", type=int, default=0, help="0 = cached copy and original, 1 = delta-only")
    ap.add_argument("--write-policy", type=int, default=None,
                    help="default 15 (every row stored, word rows kept across centres); with --ns, 1 (target "
                         "rows stored, word rows added)")
    ap.add_argument("--workers", type=int, default=0)
    ap.add_argument("--span-refresh", type=int, default=0,
                    help="words below this index leave the word-row span and are read again after every centre")
    ap.add_argument("--span-stash", type=int, default=1, choices=(0, 1),
                    help="1: the re-entering centre row of the word-row span waits in LDS instead of being read "
                         "again from memory")
    ap.add_argument("--stash-from", type=int, default=10000,
                    help="with --span-stash 1: only words of vocabulary index >= this re-enter from the stash")
    ap.add_argument("--no-loglik", action="store_true", help="leave the held-out log-likelihood out of the step")
    ap.add_argument("--no-probe", action="store_true", help="skip the random-row memory probe")
    ap.add_argument("--sweep-cache", action="store_true",
                    help="instead of the benchmark line: one JSON line per (cache_k, flush_every) of the "
                         "cache-size x write-back-interval grid (epoch kernel time and held-out log-likelihood)")
    ap.add_argument("--ns", type=int, default=0,
                    help="measure skip-gram with this many shared negatives (negative sampling) instead of the "
                         "hierarchical softmax; same workload and JSON layout, its own byte model")
    ap.add_argument("--sweep-k", default="0,1,3,7,15,31,63")
    ap.add_argument("--sweep-f", default="1,10,100,1000")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="first write, then read, 1.28 GB of rows once each (reference dispatches for HBM byte counters)")
    args = ap.parse_args()
    if args.write_policy is None:
        args.write_policy = 1 if args.ns else 15
    return args


def log(msg):
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


def algorithmic_bytes(torch, voc, tree, mask, doc_len, dim, k, flush_every, n_groups):
    """Sum of the byte model over the epoch (see the module docstring)."""
    V = voc.V
    dev = mask.device
    lens = tree.codelen.to(torch.int64)
    first = V - 1 - k
    seg = torch.repeat_interleave(torch.arange(V, device=dev), lens)
    unc = torch.zeros(V, dtype=torch.int64, device=dev).index_add_(0, seg, (tree.points < first).to(torch.int64))
    n = mask.numel()
    n_docs = (n + doc_len - 1) // doc_len
    m = torch.zeros(n_docs * doc_len, dtype=torch.bool, device=dev)
    m[:n] = mask.bool()
    per_doc = m.view(n_docs, doc_len).sum(1)
    m.view(n_docs, doc_len)[per_doc < 2] = False          # centres without a window word do nothing
    v = voc.tokens[m[:n]].to(torch.int64)
    centres = int(v.numel())
    node_rows = int(unc[v].sum().item())
    path_len = int(lens[v].sum().item())
    return centres, node_rows, path_len, per_doc.where(per_doc >= 2, 0)


def span_rows(torch, per_doc, span, seg_len=128):
    """Word rows entering a span of `span` kept positions each side of the centre, over every work unit."""
    nk = per_doc.to(torch.int64)
    n_seg = (nk + seg_len - 1) // seg_len
    doc = torch.repeat_interleave(torch.arange(nk.numel(), device=nk.device), n_seg)
    first = torch.repeat_interleave(n_seg.cumsum(0) - n_seg, n_seg)
    j0 = (torch.arange(doc.numel(), device=nk.device) - first) * seg_len
    nkd = nk[doc]
    j1 = torch.minimum(nkd, j0 + seg_len)
    zero = torch.zeros_like(j0)
    start = torch.clamp(j0, max=span) + torch.clamp(nkd - 1 - j0, max=span)
    behind = j1 - 1 - j0                                                   # previous centre's row
    ahead = torch.maximum(zero, torch.minimum(j1 - 2, nkd - 2 - span) - j0 + 1)   # row span positions ahead
    return int((start + behind + ahead).sum().item())


def main():
    args = parse()
    if args.gpus != 1:
        print(json.dumps({"error": "this benchmark runs on one GPU only: the training path is single-GPU "
                                   "(its sharding is a design, not code)", "n_gpus": args.gpus}))
        sys.exit(2)
    import numpy as np
    import torch

    import bench_probe
    import paper_1606_07822_amd as w2v
    import synth

    w = synth.WORKLOADS[args.workload]
    dev = torch.device("cuda:0")
    t0 = time.time()
    tok_np = synth.workload_corpus(w, threads=16)
    held_np = synth.workload_corpus(w, heldout=True, threads=16)
    log(f"generated {w.n_tokens:,} + {w.heldout_tokens:,} tokens in {time.time() - t0:.1f}s")
    tok = torch.from_numpy(tok_np).to(dev)

    if args.ns:
        return ns_main(args, torch, w2v, synth, w, tok, tok_np, held_np, dev)

    # first pass builds the model's shapes (same vocabulary every step: deterministic)
    voc = w2v.build_vocab(tok, w.vocab, w.min_count)
    tree = w2v.build_huffman(voc.vocab_counts)
    syn0, syn1 = synth.init_weights(voc.V, w.dim)
    model = w2v.make_model(syn0, syn1, voc, tree, dev)
    del syn0, syn1
    # every step trains one epoch from the same initial model (a device copy, 2.6 GB at V = 1M, d = 300)
    init0, init1 = model.syn0.clone(), model.syn1.clone()
    p = w2v.Params(window=w.window, sample=w.sample, alpha0=w.alpha0, arch=w.arch, corpus_tokens=w.n_tokens,
                   seed=synth.SEED_TRAIN, cache_k=args.cache_k, flush_every=args.flush_every,
                   flush_policy=args.flush_policy, write_policy=args.write_policy, workers=args.workers,
                   cache_mode=args.cache_mode, span_refresh=args.span_refresh, span_stash=args.span_stash,
                   stash_from=args.stash_from)
    pe = w2v.Params(window=w.window, sample=w.sample, seed=synth.SEED_EVAL, arch=w.arch)
    # held-out tokens as vocabulary indices (input preparation; the vocabulary is the same every step)
    held = torch.from_numpy(voc.id_to_vocab.cpu().numpy()[held_np]).to(dev)
    ll_init = None if args.no_loglik else w2v.hs_loglik(model, held, pe)
    ws = torch.empty(w2v.train_workspace_bytes(model, w.n_tokens, p), dtype=torch.uint8, device=dev)
    stats = torch.zeros(w2v.N_STATS, dtype=torch.int64, device=dev)

    if args.sweep_cache:
        sweep_cache(args, torch, w2v, synth, w, voc, tree, model, held, pe, ws, stats)
        return

    calib = None
    if args.copy_calibration:
        # dispatches of known size for scaling the HBM byte counters: every row of a
        # 1e6 x 320 float matrix written once, then read once (the training kernel's accesses)
        rows, cols = 1_000_000, 320
        m = torch.empty(rows, cols, dtype=torch.float32, device=dev)
        iters = -(-rows // (256 * 12 * 4))
        bench_probe.probe_rows(m, cols, 3, 256, iters)
        bench_probe.probe_rows(m, cols, 2, 256, iters)
        torch.cuda.synchronize()
        del m
        calib = {"rows": rows, "row_bytes": 4 * cols, "write_dispatch": "k_probe<3, 5>", "read_dispatch": "k_probe<2, 5>"}

    # byte model of one launch (the sampler's keep mask with the training seed)
    pr = w2v.sample_pairs(voc.tokens, voc.V, voc.vocab_counts, voc.train_words, p, cap=0, want_mask=True)
    centres, node_rows, path_len, per_doc = algorithmic_bytes(torch, voc, tree, pr.keep_mask, p.doc_len, w.dim,
                                                              args.cache_k, args.flush_every, 0)
    pairs = pr.total
    span = w2v.train_word_span(model, p)
    word_rows = span_rows(torch, per_doc, span) if span else pairs
    del per_doc
    del pr
    torch.cuda.empty_cache()

    def step():
        model.syn0.copy_(init0)
        model.syn1.copy_(init1)
        v = w2v.build_vocab(tok, w.vocab, w.min_count)
        t = w2v.build_huffman(v.vocab_counts)
        model.tree = t
        model.vocab_counts = v.vocab_counts
        w2v.train_hs_epoch(model, v.tokens, p, stats=stats, workspace=ws)
        kms = w2v.last_train_kernel_ms()
        ll = None
        if not args.no_loglik:
            ll = w2v.hs_loglik(model, held, pe)
        return kms, ll

    for i in range(args.warmup):
        step()
        log(f"warmup {i} done")
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    kms_all, lls = [], []
    for i in range(args.steps):
        kms, ll = step()
        kms_all.append(kms)
        lls.append(ll)
        log(f"step {i} train kernel {kms:.1f} ms")
    torch.cuda.synchronize()
    dt = time.perf_counter() - t0
    st = stats.cpu().numpy()
    ms_per_step = dt * 1e3 / args.steps
    words = int(st[1])
    value = words / (ms_per_step / 1e3)
    kernel_ms = sum(kms_all) / len(kms_all)
    # the step's stages timed one by one in one more step, after the timed ones (synchronising between them)
    stage_ms = {}

    def lap(name, t):
        torch.cuda.synchronize()
        now = time.perf_counter()
        stage_ms[name] = (now - t) * 1e3
        return now

    t = time.perf_counter()
    model.syn0.copy_(init0)
    model.syn1.copy_(init1)
    t = lap("model_reset", t)
    v = w2v.build_vocab(tok, w.vocab, w.min_count)
    t = lap("vocab", t)
    tr = w2v.build_huffman(v.vocab_counts)
    model.tree = tr
    model.vocab_counts = v.vocab_counts
    t = lap("huffman", t)
    w2v.train_hs_epoch(model, v.tokens, p, workspace=ws)
    t = lap("epoch", t)
    if not args.no_loglik:
        w2v.hs_loglik(model, held, pe)
        t = lap("heldout_loglik", t)
    del v, tr

    # roofline of the training kernel
    d = w.dim
    n_groups, n_waves = w2v.last_train_launch()
    flushes = centres // max(1, args.flush_every) + n_groups
    cache_bytes = n_groups * 4 * d * args.cache_k + flushes * 8 * d * args.cache_k
    # the per-centre byte model B(v): every window word's row read and updated once per pair (8 d P)
    byte_model = 8 * d * node_rows + 8 * d * pairs + 4 * path_len + 9 * centres + cache_bytes
    # the tighter count for a kernel that keeps word rows across centres: 8 d per row entering a span
    byte_span = 8 * d * node_rows + 8 * d * word_rows + 4 * path_len + 9 * centres + cache_bytes
    achieved_model = byte_model / (kernel_ms / 1e3) / 1e9
    achieved_span = byte_span / (kernel_ms / 1e3) / 1e9
    # the roofline counts what the kernel that runs moves: the span model when it keeps word rows across centres
    span_run = w2v.train_word_span(model, p) > 0
    byte_alg = byte_span if span_run else byte_model
    achieved = byte_alg / (kernel_ms / 1e3) / 1e9
    # the inner-node rows alone (uncached path rows, cache fill and write-backs): the node-vector traffic
    node_bytes = 8 * d * node_rows + n_groups * 4 * d * args.cache_k + flushes * 8 * d * args.cache_k
    node_gbps = node_bytes / (kernel_ms / 1e3) / 1e9
    res = w2v.last_train_resources()
    cfg_keys = {"cache_k": args.cache_k, "flush_every": args.flush_every, "flush_policy": args.flush_policy,
                "write_policy": args.write_policy, "cache_mode": args.cache_mode, "span_refresh": args.span_refresh,
                "span_stash": args.span_stash, "stash_from": args.stash_from}
    traffic = None
    tfile = os.path.join(ROOT, "profiles", f"traffic_{args.workload}.json")
    if os.path.exists(tfile):
        # counters taken on this kernel source and these settings only
        t = json.load(open(tfile))
        if t.get("kernel_source") == w2v.kernel_source_hash() and t.get("settings") == cfg_keys:
            traffic = t.get("hbm_bytes_per_launch")

    # learning achieved against the sequential oracle's full epoch on the same workload, when stored:
    # (init - gpu) / (init - oracle) of the held-out mean log-likelihood
    ll_final = (lls[-1][0] / lls[-1][1]) if lls and lls[-1] else None
    oracle_ll = gain_frac = None
    gfile = os.path.join(ROOT, "tests", "golden", f"oracle_ll_{args.workload}.json")
    if ll_final is not None and ll_init and os.path.exists(gfile):
        g = json.load(open(gfile))
        oracle_ll = g["mean_ll"]
        gain_frac = (ll_final - ll_init[0] / ll_init[1]) / (oracle_ll - g["init_mean_ll"])

    # the training kernel moves whole padded rows (row_stride >= 64 * ceil(d / 64) floats) when it can
    share = 64 * (-(-d // 64))
    probe = None if args.no_probe else memory_probe(torch, w2v, voc.V, min(share, model.stride), model.stride, dev)

    cpu = None
    if not args.no_cpu_baseline:
        cpu = cpu_baseline(w, tok_np, args)

    line = {
        "metric": "trained words/sec, HS skip-gram V=1M d=300 fp32; % of HBM roofline",
        "value": value,
        "unit": "words/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_per_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic (seeded Zipf + topic-mixture corpus standing in for the paper's text corpus)",
        "config": {"workload": args.workload, "tokens": w.n_tokens, "vocab_ids": w.vocab, "V": voc.V, "dim": d,
                   "window": w.window, "sample": w.sample, "min_count": w.min_count, "epochs_per_step": 1,
                   "cache_k": args.cache_k, "flush_every": args.flush_every, "flush_policy": args.flush_policy,
                   "write_policy": args.write_policy, "cache_mode": args.cache_mode, "span_refresh": args.span_refresh,
                   "span_stash": args.span_stash, "stash_from": args.stash_from,
                   "step": "model reset + vocab + huffman + epoch" +
                   ("" if args.no_loglik else " + held-out loglik")},
        "roofline": {"bound": "hbm", "achieved": achieved, "peak": PEAK_HBM_GBS, "unit": "GB/s",
                     "frac": achieved / PEAK_HBM_GBS, "traffic": traffic},
        "train_kernel_ms": kernel_ms,
        "train_kernel_words_per_s": words / (kernel_ms / 1e3),
        "stats": dict(zip(w2v.STAT_NAMES, map(int, st))),
        "pair_node_updates_per_s": int(st[4]) / (kernel_ms / 1e3),
        "stage_ms": stage_ms,
        "kept_centres_per_s": int(st[2]) / (kernel_ms / 1e3),
        "pairs_per_s": int(st[3]) / (kernel_ms / 1e3),
        "algorithmic_bytes_per_launch": byte_alg,
        "byte_model": "span" if span_run else "per-centre",
        "byte_model_terms": {"node_rows": node_rows, "pairs": pairs, "path_nodes": path_len, "centres": centres,
                             "span_word_rows": word_rows, "cache_fill_and_writeback_bytes": cache_bytes,
                             "dim": d, "workgroups": n_groups, "flushes": flushes},
        "span_model": {"bytes_per_launch": byte_span, "GBps": achieved_span, "frac": achieved_span / PEAK_HBM_GBS},
        "survey_model": {"bytes_per_launch": byte_model, "GBps": achieved_model, "frac": achieved_model / PEAK_HBM_GBS},
        "node_vector_traffic": {"bytes_per_launch": node_bytes, "GBps": node_gbps, "frac": node_gbps / PEAK_HBM_GBS},
        "word_span": span,
        "heldout_mean_ll": ll_final,
        "heldout_init_mean_ll": (ll_init[0] / ll_init[1]) if ll_init else None,
        "oracle_mean_ll": oracle_ll,
        "gain_fraction_vs_oracle": gain_frac,
        "cpu_baseline": cpu,
        "memory_probe": probe,
        "counter_calibration": calib,
        "kernel_source": w2v.kernel_source_hash(),
        "launch": {"workgroups": n_groups, "wavefronts": n_waves, **res},
    }
    print(json.dumps(line), flush=True)


def ns_main(args, torch, w2v, synth, w, tok, tok_np, held_np, dev):
    """Negative sampling on the same workload: one step = vocabulary + noise table + one epoch of
    shared-negative training + held-out objective. Byte model per kept centre with P > 0 window words
    and T targets (the centre word and its kept negatives): 8 d (P + T) (each row read once, then
    changed once by an atomic add) + 4 K (table entries) + 9 (centre metadata)."""
    import numpy as np
    K = args.ns
    voc = w2v.build_vocab(tok, w.vocab, w.min_count)
    noise = w2v.build_noise_table(voc.vocab_counts)
    syn0, _ = synth.init_weights(voc.V, w.dim)
    model = w2v.make_ns_model(syn0, np.zeros((voc.V, w.dim), np.float32), voc, dev)
    del syn0
    init0, init1 = model.syn0.clone(), model.syn1.clone()
    p = w2v.Params(window=w.window, sample=w.sample, alpha0=w.alpha0, corpus_tokens=w.n_tokens,
                   seed=synth.SEED_TRAIN, negative=K, workers=args.workers, write_policy=args.write_policy)
    pe = w2v.Params(window=w.window, sample=w.sample, seed=synth.SEED_EVAL, negative=K)
    held = torch.from_numpy(voc.id_to_vocab.cpu().numpy()[held_np]).to(dev)
    stats = torch.zeros(w2v.N_STATS, dtype=torch.int64, device=dev)

    # byte model: every kept centre's targets (negatives hook) and which centres have window words
    pr = w2v.sample_pairs(voc.tokens, voc.V, voc.vocab_counts, voc.train_words, p, cap=0, want_mask=True)
    neg = w2v.sample_negatives(voc.tokens, voc.V, voc.vocab_counts, voc.train_words, p, noise, cap=pr.n_kept)
    n = pr.keep_mask.numel()
    n_docs = (n + p.doc_len - 1) // p.doc_len
    m = torch.zeros(n_docs * p.doc_len, dtype=torch.bool, device=dev)
    m[:n] = pr.keep_mask.bool()
    per_doc = m.view(n_docs, p.doc_len).sum(1)
    active = torch.repeat_interleave(per_doc >= 2, per_doc)          # kept centres, stream order
    targets = int((1 + (neg.negatives[active] >= 0).sum(1)).sum().item())
    centres = int(active.sum().item())
    byte_total = 8 * w.dim * (pr.total + targets) + 4 * K * centres + 9 * centres
    del pr, neg, m, active
    torch.cuda.empty_cache()

    def step():
        model.syn0.copy_(init0)
        model.syn1.copy_(init1)
        v = w2v.build_vocab(tok, w.vocab, w.min_count)
        nz = w2v.build_noise_table(v.vocab_counts)
        model.vocab_counts = v.vocab_counts
        w2v.train_ns_epoch(model, nz, v.tokens, p, stats=stats)
        kms = w2v.last_train_kernel_ms()
        obj = None if args.no_loglik else w2v.ns_objective(model, nz, held, pe)
        return kms, obj

    for i in range(args.warmup):
        step()
        log(f"warmup {i} done")
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    kms_all, objs = [], []
    for i in range(args.steps):
        kms, obj = step()
        kms_all.append(kms)
        objs.append(obj)
        log(f"step {i} train kernel {kms:.1f} ms")
    torch.cuda.synchronize()
    dt = time.perf_counter() - t0
    st = stats.cpu().numpy()
    ms_per_step = dt * 1e3 / args.steps
    words = int(st[1])
    kernel_ms = sum(kms_all) / len(kms_all)
    achieved = byte_total / (kernel_ms / 1e3) / 1e9
    n_groups, n_waves = w2v.last_train_launch()
    res = w2v.last_train_resources()
    cpu = None if args.no_cpu_baseline else cpu_baseline(w, tok_np, args, negative=K)
    line = {
        "metric": f"trained words/sec, skip-gram with {K} shared negatives V=1M d=300 fp32; % of HBM roofline",
        "value": words / (ms_per_step / 1e3),
        "unit": "words/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_per_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic (seeded Zipf + topic-mixture corpus standing in for the paper's text corpus)",
        "config": {"workload": args.workload, "tokens": w.n_tokens, "V": voc.V, "dim": w.dim, "window": w.window,
                   "sample": w.sample, "negative": K, "noise_table_entries": int(noise.table.numel()),
                   "write_policy": args.write_policy,
                   "step": "model reset + vocab + noise table + epoch" + ("" if args.no_loglik else " + held-out objective")},
        "roofline": {"bound": "hbm", "achieved": achieved, "peak": PEAK_HBM_GBS, "unit": "GB/s",
                     "frac": achieved / PEAK_HBM_GBS, "traffic": None},
        "train_kernel_ms": kernel_ms,
        "train_kernel_words_per_s": words / (kernel_ms / 1e3),
        "stats": dict(zip(("raw_tokens", "in_vocab_tokens", "kept_centres", "pairs", "pair_target_updates"),
                          map(int, st))),
        "algorithmic_bytes_per_launch": byte_total,
        "heldout_mean_objective": (objs[-1][0] / objs[-1][1]) if objs and objs[-1] else None,
        "cpu_baseline": cpu,
        "launch": {"workgroups": n_groups, "wavefronts": n_waves, **res},
    }
    print(json.dumps(line), flush=True)


def sweep_cache(args, torch, w2v, synth, w, voc, tree, model, held, pe, ws, stats):
    """Cache size k x write-back interval F (centres per workgroup): the GPU form of the paper's
    study of the number of cached nodes and of the update interval. Every point starts from the same
    initial model and trains one epoch with the default write policies; k = 0 has no cache, so one F."""
    syn0, syn1 = synth.init_weights(voc.V, w.dim)
    s0 = torch.from_numpy(syn0).to(model.syn0.device)
    s1 = torch.from_numpy(syn1).to(model.syn0.device)
    del syn0, syn1
    for k in (int(x) for x in args.sweep_k.split(",")):
        for f in ((1,) if k == 0 else tuple(int(x) for x in args.sweep_f.split(","))):
            model.syn0.zero_()
            model.syn1.zero_()
            model.syn0[:, :w.dim].copy_(s0)
            model.syn1[:voc.V - 1, :w.dim].copy_(s1)
            p = w2v.Params(window=w.window, sample=w.sample, alpha0=w.alpha0, arch=w.arch, corpus_tokens=w.n_tokens,
                           seed=synth.SEED_TRAIN, cache_k=k, flush_every=f, flush_policy=args.flush_policy,
                           write_policy=args.write_policy, workers=args.workers, cache_mode=args.cache_mode)
            head = {"sweep": "cache_k x flush_every", "workload": args.workload, "cache_k": k, "flush_every": f,
                    "flush_policy": args.flush_policy, "write_policy": args.write_policy,
                    "cache_mode": args.cache_mode}
            try:
                w2v.train_hs_epoch(model, voc.tokens, p, stats=stats, workspace=ws)
            except w2v.W2VError as e:   # e.g. a cache that does not fit LDS
                log(f"k={k} F={f}: {e}")
                print(json.dumps({**head, "error": str(e)}), flush=True)
                continue
            kms = w2v.last_train_kernel_ms()
            s, npairs, _ = w2v.hs_loglik(model, held, pe)
            st = stats.cpu().numpy()
            line = {**head, "train_kernel_ms": kms, "words_per_s": int(st[1]) / (kms / 1e3),
                    "pair_node_updates_per_s": int(st[4]) / (kms / 1e3), "heldout_mean_ll": s / npairs}
            log(f"k={k} F={f}: {kms:.0f} ms, LL {s / npairs:.5f}")
            print(json.dumps(line), flush=True)


def memory_probe(torch, w2v, rows, cols, stride, dev):
    import bench_probe
    """Practical memory ceiling of the training kernel's access pattern: rows of
    cols floats (the padded row the kernel moves; rows = V) at hashed positions,
    four in flight per wavefront on the same launch shape, read and
    read-modify-written."""
    m = torch.zeros(rows, stride, dtype=torch.float32, device=dev)
    wg, iters = 256, 1000
    visits = wg * 12 * 4 * iters
    out = {"rows": rows, "row_bytes": 4 * cols, "row_visits": visits}
    for mode, name in ((0, "read"), (1, "rmw")):
        bench_probe.probe_rows(m, cols, mode, wg, iters)                 # warm-up
        ms = bench_probe.probe_rows(m, cols, mode, wg, iters)
        moved = visits * 4 * cols * (2 if mode else 1)
        out[f"{name}_GBps"] = moved / (ms / 1e3) / 1e9
        out[f"{name}_rows_per_s"] = visits / (ms / 1e3)
    del m
    torch.cuda.empty_cache()
    return out


def _cpu_model() -> str:
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    import platform
    return platform.processor() or "unknown"


def cpu_baseline(w, tok_np, args, negative=0):
    """The oracle (single-threaded C) on a prefix of the same corpus, timed on this host.

    The oracle is compiled for this host (gcc -O3 -march=native -ffp-contract=off) into a temporary
    directory, and the timed run is a child process pinned to one core with taskset, which reads the
    vocabulary counts and the token prefix from that directory: nothing else runs on that core, and
    the GPU process is not involved.
    """
    import shutil
    import subprocess
    import tempfile

    import numpy as np

    import oracle

    t0 = time.time()
    voc = oracle.build_vocab(tok_np, w.vocab, w.min_count)
    log(f"oracle vocabulary in {time.time() - t0:.1f}s")
    tmp = tempfile.mkdtemp(prefix="w2v_cpu_")
    try:
        n_pre = min(w.n_tokens, 16_000 * w.doc_len)
        np.save(os.path.join(tmp, "vocab_counts.npy"), voc.vocab_counts)
        np.save(os.path.join(tmp, "tokens.npy"), oracle.remap(tok_np[:n_pre], voc.id_to_vocab))
        with open(os.path.join(tmp, "job.json"), "w") as f:
            json.dump({"workload": w.name, "train_words": voc.train_words, "negative": negative,
                       "cpu_seconds": args.cpu_seconds}, f)
        lib = os.path.join(tmp, "liboracle_native.so")
        build = ["gcc", "-O3", "-march=native", "-std=c11", "-ffp-contract=off", "-fPIC", "-shared",
                 oracle.SRC_PATH, "-o", lib, "-lm"]
        env = dict(os.environ)
        try:
            subprocess.run(build, check=True, capture_output=True)
            env["W2V_ORACLE_LIB"] = lib
            build_s = "gcc -O3 -march=native -ffp-contract=off (single-threaded C)"
        except (OSError, subprocess.CalledProcessError):
            build_s = "the committed liboracle.so (gcc -O3 -march=x86-64-v3 -ffp-contract=off); native build failed"
        cores = sorted(os.sched_getaffinity(0))
        core = cores[-1]
        cmd = [sys.executable, os.path.abspath(__file__), "--cpu-child", tmp]
        pin = None
        if shutil.which("taskset"):
            cmd = ["taskset", "-c", str(core)] + cmd
            pin = f"taskset -c {core}"
        r = subprocess.run(cmd, env=env, capture_output=True, text=True, timeout=600)
        if r.returncode != 0:
            log(f"CPU baseline child failed: {r.stderr[-2000:]}")
            return None
        out = json.loads(r.stdout.strip().splitlines()[-1])
    finally:
        shutil.rmtree(tmp, ignore_errors=True)
    out.update({"unit": "words/s", "cores": 1, "kind": "oracle", "cpu_model": _cpu_model(),
                "nproc": os.cpu_count(), "cores_allowed": len(cores), "pinned": pin, "build": build_s})
    return out


def cpu_child(tmp):
    """Child process of cpu_baseline: calibrate on 20 documents, then time about cpu_seconds of training."""
    import numpy as np

    import oracle
    import synth

    job = json.load(open(os.path.join(tmp, "job.json")))
    w = synth.WORKLOADS[job["workload"]]
    vc = np.load(os.path.join(tmp, "vocab_counts.npy"))
    tv_all = np.load(os.path.join(tmp, "tokens.npy"))
    V, K = int(vc.size), int(job["negative"])
    p = oracle.params(V, w.dim, window=w.window, sample=w.sample, alpha0=w.alpha0, train_words=job["train_words"],
                      corpus_tokens=w.n_tokens, seed=synth.SEED_TRAIN, cache_k=31, flush_every=10, arch=w.arch,
                      negative=K if K else 5)
    if K:
        L = max(10, min(27, (64 * V - 1).bit_length()))
        table = oracle.noise_table(vc, L)

        def fresh():
            s0, _ = synth.init_weights(V, w.dim)
            return s0, np.zeros((V, w.dim), np.float32)

        def run(s0, s1, tv):
            return oracle.train_ns(s0, s1, vc, table, L, tv, p)
        what = f"one epoch of shared-negative training (K={K})"
    else:
        tree = oracle.build_huffman(vc)

        def fresh():
            return synth.init_weights(V, w.dim)

        def run(s0, s1, tv):
            return oracle.train(s0, s1, tree, tv, p)
        what = "one epoch of Algorithm 1 with the top-31 cache flushed every 10 centres (u=10)"
    syn0, syn1 = fresh()
    run(syn0, syn1, tv_all[:2 * w.doc_len])                     # warms the pages up
    n_cal = min(tv_all.size, 20 * w.doc_len)
    t0 = time.perf_counter()
    run(syn0, syn1, tv_all[:n_cal])
    per_tok = (time.perf_counter() - t0) / n_cal
    n = int(min(tv_all.size, max(n_cal, job["cpu_seconds"] / max(per_tok, 1e-9))))
    n = (n // w.doc_len) * w.doc_len or n_cal
    syn0, syn1 = fresh()
    t0 = time.perf_counter()
    st = run(syn0, syn1, tv_all[:n])
    dt = time.perf_counter() - t0
    print(json.dumps({"value": float(st[1]) / dt, "seconds": dt, "tokens": n,
                      "sample": f"first {n:,} tokens ({n // w.doc_len} documents) of the same corpus, {what}, "
                                f"{dt:.1f}s on one pinned host core"}), flush=True)


if __name__ == "__main__":
    if len(sys.argv) == 3 and sys.argv[1] == "--cpu-child":
        cpu_child(sys.argv[2])
    else:
        main()
