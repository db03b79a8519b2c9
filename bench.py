"""Benchmark of the trie-automaton mask path on one MI355X.

One step = one pass of the whole device hot path over one batch:
  1. the device compile: the zero fill of the dense [N, W] bitmask table (the
     dominant kernel) with the suffix probes running beside it on a second
     stream, then every valid (node, token) bit set by 64-bit atomics,
  3. the mask apply on [B, V] logits,
  4. the state advance of the B rows.
Inputs (trie and vocabulary tables, node ids, tokens, logits) are resident in
HBM before the timed region; the host trie build and the uploads are reported
separately as the end-to-end compile time.

value = (node, token) pairs resolved per second = N * V per step / step time.

Usage: python bench.py [--gpus 1] [--steps K] [--warmup W] [--config 4]
"""
from __future__ import annotations

import argparse
import hashlib
import json
import math
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "compile ms + (node,token) pairs/s; mask-apply GB/s at B=256 (bit-exact)"
HBM_PEAK_GBPS = 8000.0  # MI355X HBM3E, AMD published peak


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--config", type=int, default=4)
    ap.add_argument("--repr", choices=["auto", "full", "tail", "lists"], default="auto",
                    help="mask representation: full dense table, tail compression (dense rows for "
                         "branching nodes, lists for tails), or lists only; auto = full for one set, "
                         "lists for a forest")
    ap.add_argument("--apply-iters", type=int, default=1000)
    ap.add_argument("--apply-warmup", type=int, default=200)
    ap.add_argument("--cpu-seconds", type=float, default=12.0,
                    help="wall-clock budget of the oracle's CPU-baseline sample")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--calib-copy-mib", type=int, default=0,
                    help="also run one device copy of this size (counter calibration)")
    return ap.parse_args()


def kernels_sha() -> str:
    p = os.path.join(ROOT, "paper_2608_12574_amd", "csrc", "kernels.hip")
    return hashlib.sha256(open(p, "rb").read()).hexdigest()[:16]


def load_traffic(name: str, sha: str):
    """HBM bytes per launch from the committed counter summary, if it was taken
    on the current kernels (else None)."""
    p = os.path.join(ROOT, "profiles", name)
    if not os.path.exists(p):
        return None
    d = json.load(open(p))
    if d.get("kernels_sha") != sha:
        return None
    return d


def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only: this path has no multi-GPU mode (asked for --gpus {args.gpus}).",
              file=sys.stderr)
        sys.exit(2)

    import torch

    import paper_2608_12574_amd as P
    import workloads as W

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    dev = torch.device("cuda", 0)
    torch.cuda.set_device(dev)
    P.lib()
    sha = kernels_sha()

    t = time.time()
    w = W.config(args.config)
    gen_s = time.time() - t
    K, V, B = w.K, w.V, w.batch
    logit_dtype = torch.bfloat16 if w.dtype == "bf16" else torch.float32
    esize = 2 if w.dtype == "bf16" else 4
    rep = args.repr if args.repr != "auto" else ("lists" if w.set_offsets is not None else "full")
    flags = P.FLAG_TIMING | {"full": 0, "tail": P.FLAG_TAIL_LISTS, "lists": P.FLAG_NO_TABLE}[rep]
    print(f"[bench] workload {w.name}: K={K} V={V} B={B} ({gen_s:.1f}s to generate)", flush=True)

    # ---- end-to-end compile (host trie + vocabulary + upload + device) ----
    # cold: the vocabulary tables are built from the token list on every call;
    # warm: they come from a Vocab built once per tokenizer.
    def timed_compile(vocab):
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        hh = P.compile(w.strings, vocab, sets=w.set_offsets, flags=flags)
        torch.cuda.synchronize()
        return hh, (time.perf_counter() - t0) * 1e3

    cold, warm = [], []
    phases_cold = None
    for i in range(3):
        hh, ms = timed_compile(w.vocab)
        cold.append(ms)
        phases_cold = hh.timing()
        hh.close()
    t0 = time.perf_counter()
    voc = P.Vocab(w.vocab)
    torch.cuda.synchronize()
    vocab_ms = (time.perf_counter() - t0) * 1e3
    h = None
    for i in range(3):
        if h is not None:
            h.close()
        h, ms = timed_compile(voc)
        warm.append(ms)
    phases_warm = h.timing()
    N = h.num_nodes
    Wd = h.words_per_row
    M = h.valid_pairs()
    print(f"[bench] compiled: N={N} W={Wd} valid pairs={M} end-to-end cold {min(cold):.1f} ms, "
          f"warm {min(warm):.1f} ms (vocabulary build {vocab_ms:.1f} ms once)", flush=True)

    # ---- serving inputs, resident on the device ----
    if w.node_mode == "uniform":
        nodes_np = W.uniform_nodes(w.config_id, N, B)
    elif w.node_mode == "set_roots":
        nodes_np = h.roots[:B].astype(np.int32)
    else:
        nodes_np = np.zeros(B, dtype=np.int32)
    ids = torch.as_tensor(nodes_np, device=dev)
    nbuf = max(2, math.ceil((1 << 30) / (B * V * esize)))  # >= 1 GiB of distinct logits
    gen = torch.Generator(device=dev)
    gen.manual_seed(w.config_id)
    bufs = [torch.randn((B, V), generator=gen, device=dev, dtype=torch.float32).to(logit_dtype)
            for _ in range(nbuf)]
    probe = bufs[0].clone()
    h.apply_mask(ids, probe)
    toks = probe.float().argmax(dim=1).to(torch.int32)  # a valid token per live row
    out = torch.empty_like(ids)
    del probe

    has_table = h.row_stride_words > 0

    def step(i, ev=None):
        """device compile (table: probes beside the zero fill, then the marks;
        sparse handles: the lists), apply, advance."""
        if ev is not None:
            ev[0].record()
        h.rebuild()
        if ev is not None:
            ev[1].record()
        h.apply_mask(ids, bufs[i % nbuf])
        if ev is not None:
            ev[2].record()
        h.advance(ids, toks, out=out)
        if ev is not None:
            ev[3].record()

    for i in range(args.warmup):
        step(i)
    evs = [[torch.cuda.Event(enable_timing=True) for _ in range(4)] for _ in range(args.steps)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(args.steps):
        step(i, evs[i])
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    ms_step = wall * 1e3 / args.steps
    dev_ms = np.mean([e[0].elapsed_time(e[1]) for e in evs])     # device compile of one step
    apply_ms = np.mean([e[1].elapsed_time(e[2]) for e in evs])
    adv_ms = np.mean([e[2].elapsed_time(e[3]) for e in evs])
    pairs_per_s = N * V / (ms_step / 1e3)

    # ---- the dominant kernel alone: the table's zero fill (one launch per rebuild) ----
    zero_ms = mark_ms = float("nan")
    if has_table:
        zev = [[torch.cuda.Event(enable_timing=True) for _ in range(3)] for _ in range(args.steps)]
        for e in zev:
            e[0].record()
            h.rebuild(phases=P.PHASE_ZERO)
            e[1].record()
            h.rebuild(phases=P.PHASE_MARK)
            e[2].record()
        torch.cuda.synchronize()
        zero_ms = float(np.mean([e[0].elapsed_time(e[1]) for e in zev]))
        mark_ms = float(np.mean([e[1].elapsed_time(e[2]) for e in zev]))
    print(f"[bench] step {ms_step:.3f} ms (device compile {dev_ms:.3f}, apply {apply_ms:.4f}, advance {adv_ms:.4f}); "
          f"alone: zero {zero_ms:.3f}, probes+marks {mark_ms:.3f}", flush=True)

    # ---- mask apply alone: the paper's protocol (200 warm-up + 1,000 timed) ----
    for i in range(args.apply_warmup):
        h.apply_mask(ids, bufs[i % nbuf])
    a0, a1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    a0.record()
    for i in range(args.apply_iters):
        h.apply_mask(ids, bufs[i % nbuf])
    a1.record()
    torch.cuda.synchronize()
    apply_us = a0.elapsed_time(a1) * 1e3 / args.apply_iters
    apply_bytes = B * (Wd * 8 + V * esize)
    apply_gbps = apply_bytes / (apply_us * 1e-6) / 1e9

    # ---- workloads that decode from their roots: apply over the whole trajectory ----
    # Rows start at their root, take the argmax of their masked logits (a uniformly
    # random valid token, the logits being i.i.d.), advance, and restart at their
    # root once final; the apply figure is then the average over the decode steps.
    traj_us = None
    if w.node_mode in ("root", "set_roots") and w.decode_steps > 1:
        fin_dev = torch.as_tensor(h.is_final.astype(np.bool_), device=dev)
        cur = ids.clone()
        traj = []
        for s in range(w.decode_steps):
            traj.append(cur.clone())
            lg = bufs[s % nbuf].clone()
            h.apply_mask(cur, lg)
            tk = lg.float().argmax(dim=1).to(torch.int32)
            nxt = h.advance(cur, tk)
            cur = torch.where((nxt < 0) | fin_dev[nxt.clamp(min=0).long()], ids, nxt)
            del lg
        torch.cuda.synchronize()
        for i in range(args.apply_warmup):
            h.apply_mask(traj[i % len(traj)], bufs[i % nbuf])
        torch.cuda.synchronize()
        a0.record()
        for i in range(args.apply_iters):
            h.apply_mask(traj[i % len(traj)], bufs[i % nbuf])
        a1.record()
        torch.cuda.synchronize()
        traj_us = a0.elapsed_time(a1) * 1e3 / args.apply_iters
        root_us, root_gbps = apply_us, apply_gbps
        apply_us = traj_us
        apply_gbps = apply_bytes / (apply_us * 1e-6) / 1e9

    # ---- advance latency ----
    torch.cuda.synchronize()
    a0.record()
    for i in range(1000):
        h.advance(ids, toks, out=out)
    a1.record()
    torch.cuda.synchronize()
    advance_us = a0.elapsed_time(a1) * 1e3 / 1000

    # ---- achievable write bandwidth on this device: a 4 GiB fill ----
    fill = torch.empty(1 << 32, dtype=torch.uint8, device=dev)
    fill.zero_()
    torch.cuda.synchronize()
    a0.record()
    for _ in range(5):
        fill.zero_()
    a1.record()
    torch.cuda.synchronize()
    fill_gbps = 5 * (1 << 32) / (a0.elapsed_time(a1) * 1e-3) / 1e9
    del fill

    if args.calib_copy_mib:
        src = torch.ones(args.calib_copy_mib << 20, dtype=torch.uint8, device=dev)
        dst = torch.empty_like(src)
        dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst

    # ---- roofline of the dominant kernel ----
    # dense handles: the table's zero fill, N*W*8 bytes written once;
    # sparse handles (forests): the lists phase, whose algorithmic output is the
    # M valid token ids plus N+1 row offsets (4 bytes each).
    table_bytes = h.dense_rows * Wd * 8 if has_table else (M + N + 1) * 4
    tr = load_traffic(f"k_zero_{w.name}_traffic.json", sha) if has_table else None
    kern_ms = zero_ms if has_table else dev_ms
    roofline = {
        "kernel": "k_zero" if has_table else "k_probe+k_scan+k_fill",
        "bound": "hbm",
        "achieved": round(table_bytes / (kern_ms * 1e-3) / 1e9, 1),
        "peak": HBM_PEAK_GBPS,
        "unit": "GB/s",
        "frac": round(table_bytes / (kern_ms * 1e-3) / 1e9 / HBM_PEAK_GBPS, 4),
        "traffic": tr["bytes_per_launch"] if tr else None,
        "algorithmic_bytes": table_bytes,
        "avg_launch_ms": round(float(kern_ms), 4),
    }
    tra = load_traffic(f"k_apply_{w.name}_traffic.json", sha)
    roofline_apply = {
        "kernel": "k_apply",
        "bound": "hbm",
        "achieved": round(apply_gbps, 1),
        "peak": HBM_PEAK_GBPS,
        "unit": "GB/s",
        "frac": round(apply_gbps / HBM_PEAK_GBPS, 4),
        "traffic": tra["bytes_per_launch"] if tra else None,
        "algorithmic_bytes": apply_bytes,
        "avg_launch_us": round(apply_us, 3),
    }

    # ---- CPU baseline: the oracle on a bounded sample, one thread ----
    cpu = None
    exact = None
    if not args.no_cpu_baseline:
        import oracle
        t = time.perf_counter()
        o = oracle.Oracle(w.strings, w.vocab, set_offsets=w.set_offsets)
        build_s = time.perf_counter() - t
        rng = np.random.default_rng(99)
        done, rows_done = 0.0, 0
        sample_nodes = []
        t = time.perf_counter()
        while time.perf_counter() - t < args.cpu_seconds:
            nodes = rng.integers(0, o.N, size=64).astype(np.int32)
            rows = o.mask_rows(nodes)
            sample_nodes.append((nodes, rows))
            rows_done += 64
        done = time.perf_counter() - t
        opps = rows_done * V / done
        cpu = {"value": round(opps, 1), "unit": "pairs/s", "cores": 1, "kind": "oracle",
               "sample": f"{rows_done} random rows x V={V} tokens of {w.name} ({done:.1f} s, one thread), "
                         f"trie build {build_s * 1e3:.0f} ms; full table extrapolates to "
                         f"{N * V / opps:.0f} s",
               "host_cpus": os.cpu_count()}
        # the same rows on the GPU must be bit-identical
        exact = True
        for nodes, rows in sample_nodes[:8]:
            got = h.export_rows(torch.as_tensor(nodes, device=dev)).cpu().numpy().view(np.uint64)
            exact = exact and bool(np.array_equal(got, rows))

    result = {
        "metric": METRIC,
        "value": round(pairs_per_s, 1),
        "unit": "(node,token) pairs/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "u64",
        "data": "synthetic",
        "config": {"workload": f"{w.name}: {w.description}", "repr": rep, "K": K, "V": V, "N": N, "B": B,
                   "logits_dtype": w.dtype, "num_sets": w.num_sets, "valid_pairs": M},
        "roofline": roofline,
        "roofline_apply": roofline_apply,
        "cpu_baseline": cpu,
        "compile_ms": {"end_to_end_cold_min": round(min(cold), 3), "end_to_end_cold_all": [round(x, 3) for x in cold],
                       "end_to_end_warm_min": round(min(warm), 3), "end_to_end_warm_all": [round(x, 3) for x in warm],
                       "vocabulary_build_once": round(vocab_ms, 3),
                       "device": round(float(dev_ms), 4),
                       "device_zero_alone_ms": round(zero_ms, 4),
                       "device_probe_mark_alone_ms": round(mark_ms, 4),
                       "device_frac_of_hbm_roofline": round(table_bytes / (dev_ms * 1e-3) / 1e9 / HBM_PEAK_GBPS, 4),
                       "phases_cold": phases_cold, "phases_warm": phases_warm},
        "apply": {"us": round(apply_us, 3), "GBps": round(apply_gbps, 1), "bytes": apply_bytes,
                  "frac_of_hbm_roofline": round(apply_gbps / HBM_PEAK_GBPS, 4), "iters": args.apply_iters,
                  "rows": (f"{w.decode_steps}-step decode trajectory from the roots" if traj_us is not None
                           else w.node_mode),
                  "first_step_at_roots": ({"us": round(root_us, 3), "GBps": round(root_gbps, 1),
                                           "frac_of_hbm_roofline": round(root_gbps / HBM_PEAK_GBPS, 4)}
                                          if traj_us is not None else None)},
        "advance_us": round(advance_us, 3),
        "fill_GBps_4GiB": round(fill_gbps, 1),
        "bit_exact_sampled_rows": exact,
        "kernels_sha": sha,
    }
    h.close()
    voc.close()
    print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()
