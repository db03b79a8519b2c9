"""Benchmark of the trie-automaton mask path on one MI355X.

One step = one pass of the whole device hot path over one batch:
  1. the device compile of the handle's masks from its resident trie and
     vocabulary tables: for the full dense [N, W] bitmask table, the zero fill
     of the table (the dominant kernel) and the probe pass that sets every valid
     (node, token) bit with 64-bit atomics; for a forest, the sparse valid lists;
  2. the mask apply on [B, V] logits;
  3. the state advance of the B rows.
Inputs (trie and vocabulary tables, node ids, tokens, logits) are resident in
HBM before the timed region; the host trie build and the uploads are reported
separately as the end-to-end compile time, which starts from the strings in
the C ABI's CSR form (packing a Python list into it is timed on its own).

The same line also reports the workload under tail compression
(TAM_FLAG_TAIL_LISTS: dense rows only for branching nodes, tails read back from
the probe's hits), which gives bit-identical masks from a much smaller table,
and with rows built on demand (TAM_FLAG_LAZY_ROWS: no mask at compile, a row
cache filled by the decode steps).

value = (node, token) pairs resolved per second = N * V per step / step time.

Usage: python bench.py [--gpus 1] [--steps K] [--warmup W] [--config 4] [--repr auto|full|tail|lists]
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
# A serving process that compiles on the host: OpenMP worker threads of torch's
# CPU ops otherwise spin for milliseconds after each parallel region, on every
# core, and the compile's host threads then run several times slower.  Set
# before torch is imported; an explicit setting in the environment wins.
os.environ.setdefault("OMP_WAIT_POLICY", "PASSIVE")

METRIC = "compile ms + (node,token) pairs/s; mask-apply GB/s at B=256 (bit-exact)"
HBM_PEAK_GBPS = 8000.0  # MI355X HBM3E, AMD published peak
# TAM_FLAG_TAIL_LISTS (8), TAM_FLAG_NO_TABLE (2); tail_lists = tail compression
# without a table (the branching nodes keep sparse lists)
FLAGS = {"full": 0, "tail": 8, "lists": 2, "tail_lists": 10}


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--config", type=int, default=4)
    ap.add_argument("--repr", choices=["auto", "full", "tail", "lists", "tail_lists"], default="auto",
                    help="mask representation of the headline figures: full dense table, tail "
                         "compression (dense rows for branching nodes), lists only, or tail "
                         "compression with lists for the branching nodes; auto = full for one set, "
                         "tail_lists for a forest")
    ap.add_argument("--no-secondary", action="store_true",
                    help="skip the other representations (tail compression; for a forest lists and "
                         "tail compression) and the rows built on demand")
    ap.add_argument("--apply-iters", type=int, default=1000)
    ap.add_argument("--apply-warmup", type=int, default=200)
    ap.add_argument("--cpu-seconds", type=float, default=12.0,
                    help="wall-clock budget of the oracle's CPU-baseline sample")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--calib-copy-mib", type=int, default=0,
                    help="also run one device copy of this size (counter calibration)")
    ap.add_argument("--profile-apply", choices=["roots", "trajectory", "uniform"], default=None,
                    help="profiling run: compile once, then only mask apply (--apply-warmup + --apply-iters "
                         "calls) on the workload's root rows, its decode trajectory, or uniform rows, so that "
                         "every apply dispatch a profiler records is of that kind; prints one JSON line")
    return ap.parse_args()


def kernels_sha() -> str:
    """Hash of the device code (kernels.hip and device_tables.hpp, the
    definitions the kernels share with the host), with comments and whitespace
    removed: the counter summaries under profiles/ are valid while it matches
    (comment edits do not change what was measured)."""
    import re
    h = hashlib.sha256()
    for name in ("kernels.hip", "device_tables.hpp"):
        src = open(os.path.join(ROOT, "paper_2608_12574_amd", "csrc", name), encoding="utf-8").read()
        src = re.sub(r"/\*.*?\*/", " ", src, flags=re.S)
        src = re.sub(r"//[^\n]*", " ", src)
        h.update(" ".join(src.split()).encode())
    return h.hexdigest()[:16]


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


def hbm_roofline(kernel, nbytes, ms, traffic=None):
    gbps = nbytes / (ms * 1e-3) / 1e9
    return {"kernel": kernel, "bound": "hbm", "achieved": round(gbps, 1), "peak": HBM_PEAK_GBPS,
            "unit": "GB/s", "frac": round(gbps / HBM_PEAK_GBPS, 4),
            "traffic": traffic["bytes_per_launch"] if traffic else None,
            "algorithmic_bytes": int(nbytes), "avg_launch_ms": round(float(ms), 4)}


class Bench:
    def __init__(self, args, torch, P, W, w, dev):
        self.args, self.torch, self.P, self.W, self.w, self.dev = args, torch, P, W, w, dev
        self.V, self.B = w.V, w.batch
        self.logit_dtype = torch.bfloat16 if w.dtype == "bf16" else torch.float32
        self.esize = 2 if w.dtype == "bf16" else 4
        # >= 1 GiB of distinct logits, so the 256 MB Infinity Cache is defeated
        self.nbuf = max(2, math.ceil((1 << 30) / (self.B * self.V * self.esize)))
        gen = torch.Generator(device=dev)
        gen.manual_seed(w.config_id)
        self.bufs = [torch.randn((self.B, self.V), generator=gen, device=dev, dtype=torch.float32)
                     .to(self.logit_dtype) for _ in range(self.nbuf)]
        self.voc = None
        self.vocab_ms = None
        self.oracle, self.sample = None, None  # set by the CPU-baseline leg
        # the strings in the C ABI's input form (CSR bytes + offsets); packing a
        # Python list is timed on its own
        from paper_2608_12574_amd.tam import csr
        t0 = time.perf_counter()
        self.packed = csr(w.strings)
        self.pack_ms = (time.perf_counter() - t0) * 1e3
        t0 = time.perf_counter()
        self.packed_vocab = csr(w.vocab)
        self.vocab_pack_ms = (time.perf_counter() - t0) * 1e3

    def event(self):
        return self.torch.cuda.Event(enable_timing=True)

    def structure(self, h):
        """The paper's structural diagnostics of the workload.  Prefix sharing
        (appendix "Prefix Sharing Analysis"): r = |T| / N_chars per set, |T| the
        trie's nodes without the terminator nodes (the root counted, as in the
        worked example's 29 nodes for 44 characters) and N_chars the bytes of
        the set's distinct strings.  Valid-set sizes by depth (the appendix's
        "Valid set size distribution"): |valid[n]| of every node, counted on the
        device from the handle's rows (tam_valid_counts)."""
        torch, w = self.torch, self.w
        offs = list(w.set_offsets) if w.set_offsets is not None else [0, len(w.strings)]
        roots = list(h.roots) + [h.num_nodes]
        rs, nodes_t, chars_t, k_t = [], 0, 0, 0
        for j in range(len(offs) - 1):
            d = set(w.strings[int(offs[j]):int(offs[j + 1])])
            chars = sum(len(x) for x in d)
            nodes = int(roots[j + 1] - roots[j]) - len(d)  # without the terminator nodes
            rs.append(nodes / max(chars, 1))
            nodes_t, chars_t, k_t = nodes_t + nodes, chars_t + chars, k_t + len(d)
        N = h.num_nodes
        cnt = np.empty(N, dtype=np.int64)
        step = 1 << 22
        for a in range(0, N, step):
            ids = torch.arange(a, min(N, a + step), dtype=torch.int32, device=self.dev)
            cnt[a:a + ids.numel()] = h.valid_counts(ids).cpu().numpy()
        depth = h.depth
        D = int(depth.max()) + 1
        nodes_d = np.bincount(depth, minlength=D)
        sum_d = np.bincount(depth, weights=cnt, minlength=D)
        max_d = np.zeros(D, dtype=np.int64)
        np.maximum.at(max_d, depth, cnt)
        keep = nodes_d > 0
        res = {"prefix_sharing": {"strings": k_t, "N_chars": chars_t, "trie_nodes": nodes_t,
                                  "r": round(nodes_t / chars_t, 4), "sets": len(rs)},
               "valid_by_depth": {"depth": np.flatnonzero(keep).tolist(), "nodes": nodes_d[keep].tolist(),
                                  "mean": np.round(sum_d[keep] / nodes_d[keep], 2).tolist(),
                                  "max": max_d[keep].tolist()},
               "valid_pairs_from_counts": int(cnt.sum())}
        if len(rs) > 1:
            res["prefix_sharing"]["r_per_set"] = {"min": round(min(rs), 4), "median": round(float(np.median(rs)), 4),
                                                  "max": round(max(rs), 4)}
        top = min(D, 9)
        print(f"[bench] structure: r = {nodes_t}/{chars_t} = {nodes_t / chars_t:.3f}; |valid| by depth "
              + ", ".join(f"{d}: mean {sum_d[d] / max(nodes_d[d], 1):.1f} max {max_d[d]} ({nodes_d[d]} nodes)"
                          for d in range(top)), flush=True)
        return res

    def parity(self, h, ids):
        """Bit-exactness of a timed handle against the oracle (None without it):
        the oracle's sampled rows against the handle's exported rows; apply on
        the timed batch and on a batch of sampled rows, raw bits against the
        oracle's apply; advance of those rows on a valid token each and on
        random ids (out of range included) against the oracle's advance."""
        if self.oracle is None:
            return None
        torch, W, o, dev = self.torch, self.W, self.oracle, self.dev
        nodes, rows = self.sample
        k = min(len(nodes), 2048)
        got = h.export_rows(torch.as_tensor(nodes[:k], device=dev)).cpu().numpy().view(np.uint64)
        rows_ok = bool(np.array_equal(got, rows[:k]))
        bits_t = torch.int16 if self.esize == 2 else torch.int32
        bits_np = np.uint16 if self.esize == 2 else np.uint32
        odt = 1 if self.esize == 2 else 0
        g = torch.Generator()
        g.manual_seed(77)
        apply_ok, advance_ok = True, True
        rng = np.random.default_rng(78)
        batches = [ids.cpu().numpy().astype(np.int32), nodes[: self.B].astype(np.int32)]
        for bi, id_np in enumerate(batches):
            x = torch.randn((len(id_np), self.V), generator=g).to(self.logit_dtype)
            exp = o.apply(id_np, x.view(bits_t).numpy().view(bits_np), odt)
            xd = x.to(dev)
            idt = torch.as_tensor(id_np, device=dev)
            h.apply_mask(idt, xd)
            apply_ok = apply_ok and bool(np.array_equal(xd.view(bits_t).cpu().numpy().view(bits_np), exp))
            vrows = rows[: self.B] if bi == 1 else o.mask_rows(id_np)
            for toks in (W.choose_valid_tokens(rng, vrows, self.V),
                         rng.integers(-1, self.V + 1, size=len(id_np)).astype(np.int32)):
                out = h.advance(idt, torch.as_tensor(toks, device=dev)).cpu().numpy()
                advance_ok = advance_ok and bool(np.array_equal(out, o.advance(id_np, toks)))
        return {"rows_checked": int(k), "rows": rows_ok, "apply_rows_checked": int(sum(len(b) for b in batches)),
                "apply": apply_ok, "advance_checked": int(2 * sum(len(b) for b in batches)),
                "advance": advance_ok}

    def fresh_logits(self, seed):
        """Unmasked logits (the rotating buffers are masked in place by the timed
        applies, so token choices are made on fresh ones)."""
        torch = self.torch
        g = torch.Generator(device=self.dev)
        g.manual_seed(1000 + seed)
        return torch.randn((self.B, self.V), generator=g, device=self.dev).to(self.logit_dtype)

    def graph_us(self, call, n, replays=10):
        """Microseconds per call of `call` (a library call that only launches
        kernels), captured n times in a HIP graph and replayed."""
        torch = self.torch
        s = torch.cuda.Stream()
        s.wait_stream(torch.cuda.current_stream())
        with torch.cuda.stream(s):
            call()
        torch.cuda.current_stream().wait_stream(s)
        torch.cuda.synchronize()
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g):
            for _ in range(n):
                call()
        g.replay()
        torch.cuda.synchronize()
        e0, e1 = self.event(), self.event()
        e0.record()
        for _ in range(replays):
            g.replay()
        e1.record()
        torch.cuda.synchronize()
        del g
        return e0.elapsed_time(e1) * 1e3 / (n * replays)

    def compile_times(self, flags, cold_runs):
        """End-to-end compile (host trie + vocabulary + upload + device), cold
        (vocabulary tables built by the call) and warm (from a Vocab built once)."""
        torch, P, w = self.torch, self.P, self.w

        def timed(vocab):
            torch.cuda.synchronize()
            t0 = time.perf_counter()
            hh = P.compile(self.packed, vocab, sets=w.set_offsets, flags=flags)
            torch.cuda.synchronize()
            return hh, (time.perf_counter() - t0) * 1e3

        cold, phases_cold = [], None
        for _ in range(cold_runs):
            hh, ms = timed(self.packed_vocab)
            cold.append(ms)
            phases_cold = hh.timing()
            hh.close()
        if self.voc is None:
            t0 = time.perf_counter()
            self.voc = P.Vocab(self.packed_vocab)
            torch.cuda.synchronize()
            self.vocab_ms = (time.perf_counter() - t0) * 1e3
        warm, h = [], None
        for _ in range(10):
            if h is not None:
                h.close()
            h, ms = timed(self.voc)
            warm.append(ms)
        return h, cold, warm, phases_cold, h.timing()

    def one_set_compile_ms(self, flags, runs=20):
        """A forest's first set compiled on its own, warm (the latency of one new
        query's set), minimum over runs; None for a single-set workload.  The
        first few compiles of a process enqueue their small uploads several
        times slower than later ones, hence the runs."""
        torch, P, w = self.torch, self.P, self.w
        if w.set_offsets is None:
            return None
        from paper_2608_12574_amd.tam import csr
        one = csr(w.strings[int(w.set_offsets[0]):int(w.set_offsets[1])])
        ts = []
        for _ in range(runs):
            torch.cuda.synchronize()
            t0 = time.perf_counter()
            hh = P.compile(one, self.voc, flags=flags)
            torch.cuda.synchronize()
            ts.append((time.perf_counter() - t0) * 1e3)
            hh.close()
        return round(min(ts), 3)

    def measure(self, rep, steps, warmup, cold_runs):
        torch, P, W, w, dev = self.torch, self.P, self.W, self.w, self.dev
        B, V, bufs, nbuf = self.B, self.V, self.bufs, self.nbuf
        flags = P.FLAG_TIMING | FLAGS[rep]
        h, cold, warm, phases_cold, phases_warm = self.compile_times(flags, cold_runs)
        N, Wd, M = h.num_nodes, h.words_per_row, h.valid_pairs()
        print(f"[bench] {rep}: N={N} W={Wd} dense rows={h.dense_rows} valid pairs={M} end-to-end"
              f"{f' cold {min(cold):.1f} ms,' if cold else ''} warm {min(warm):.1f} ms", flush=True)

        # serving inputs, resident on the device
        if w.node_mode == "uniform":
            nodes_np = W.uniform_nodes(w.config_id, N, B)
        elif w.node_mode == "set_roots":
            nodes_np = h.roots[:B].astype(np.int32)
        else:
            nodes_np = np.zeros(B, dtype=np.int32)
        ids = torch.as_tensor(nodes_np, device=dev)
        probe = self.fresh_logits(0)
        h.apply_mask(ids, probe)
        toks = probe.float().argmax(dim=1).to(torch.int32)  # a valid token per live row
        out = torch.empty_like(ids)
        del probe

        def step(i, ev=None):
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

        # the timed steps run on a handle without timing events and with no
        # events of their own (event records between the kernels slow them)
        timed_h = P.compile(self.packed, self.voc, sets=w.set_offsets, flags=FLAGS[rep])
        hh = h
        h = timed_h
        for i in range(warmup):
            step(i)
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for i in range(steps):
            step(i)
        torch.cuda.synchronize()
        ms_step = (time.perf_counter() - t0) * 1e3 / steps
        h = hh
        timed_h.close()
        # the same steps with events between the parts, for the breakdown
        evs = [[self.event() for _ in range(4)] for _ in range(steps)]
        for i in range(steps):
            step(i, evs[i])
        torch.cuda.synchronize()
        dev_ms = float(np.mean([e[0].elapsed_time(e[1]) for e in evs]))
        apply_step_ms = float(np.mean([e[1].elapsed_time(e[2]) for e in evs]))
        adv_step_ms = float(np.mean([e[2].elapsed_time(e[3]) for e in evs]))

        # the device phases alone: zero fill, probe pass (marks, or list
        # counts), the whole lists phase (probe pass, prefix sum, fill)
        alone = {}
        for name, ph in (("zero", P.PHASE_ZERO), ("probe_marks", P.PHASE_MARK), ("probe_counts", P.PHASE_COUNT),
                         ("lists", P.PHASE_LISTS)):
            try:
                h.rebuild(phases=ph)
            except P.TamError:
                continue
            ev = [[self.event() for _ in range(2)] for _ in range(steps)]
            for e in ev:
                e[0].record()
                h.rebuild(phases=ph)
                e[1].record()
            torch.cuda.synchronize()
            alone[name] = float(np.mean([e[0].elapsed_time(e[1]) for e in ev]))
        h.rebuild()  # leave a complete table and lists
        print(f"[bench] {rep}: step {ms_step:.3f} ms (device compile {dev_ms:.3f}, apply {apply_step_ms:.4f}, "
              f"advance {adv_step_ms:.4f}); alone: " + ", ".join(f"{k} {v:.3f}" for k, v in alone.items()),
              flush=True)

        # mask apply alone: the paper's protocol (200 warm-up + 1,000 timed)
        def time_apply(id_list, iters=None):
            iters = iters or self.args.apply_iters
            for i in range(self.args.apply_warmup):
                h.apply_mask(id_list[i % len(id_list)], bufs[i % nbuf])
            a0, a1 = self.event(), self.event()
            torch.cuda.synchronize()
            a0.record()
            for i in range(iters):
                h.apply_mask(id_list[i % len(id_list)], bufs[i % nbuf])
            a1.record()
            torch.cuda.synchronize()
            return a0.elapsed_time(a1) * 1e3 / iters

        apply_bytes = B * (Wd * 8 + V * self.esize)
        # uniform rows: a decode moves every row each step, so the timed calls
        # take 64 id lists in turn and each call reads its mask rows from HBM;
        # the same ids every call (their rows then stay in the caches) are
        # reported beside
        same_rows = None
        if w.node_mode == "uniform":
            id_lists = [ids] + [torch.as_tensor(W.uniform_nodes(w.config_id, N, B, seed_extra=1 + k), device=dev)
                                for k in range(63)]
            s_us = time_apply([ids], max(20, self.args.apply_iters // 5))
            same_rows = {"us": round(s_us, 3), "GBps": round(apply_bytes / (s_us * 1e-6) / 1e9, 1),
                         "frac_of_hbm_roofline": round(apply_bytes / (s_us * 1e-6) / 1e9 / HBM_PEAK_GBPS, 4)}
        else:
            id_lists = [ids]
        apply_us = time_apply(id_lists)
        root_us = None
        # workloads that decode from their roots: apply over the whole trajectory.
        # Rows take the argmax of their masked logits (a uniformly random valid
        # token, the logits being i.i.d.), advance, and restart at their root
        # once final.
        if w.node_mode in ("root", "set_roots") and w.decode_steps > 1:
            fin_dev = torch.as_tensor(h.is_final.astype(np.bool_), device=dev)
            cur, traj = ids.clone(), []
            for s in range(w.decode_steps):
                traj.append(cur.clone())
                lg = self.fresh_logits(1 + s)
                h.apply_mask(cur, lg)
                nxt = h.advance(cur, lg.float().argmax(dim=1).to(torch.int32))
                cur = torch.where((nxt < 0) | fin_dev[nxt.clamp(min=0).long()], ids, nxt)
                del lg
            root_us, apply_us = apply_us, time_apply(traj)
            id_lists = traj
        apply_gbps = apply_bytes / (apply_us * 1e-6) / 1e9

        # logit reads no masking in place can avoid: a 16-byte chunk holding
        # both valid and invalid tokens must be read; the algorithmic bytes
        # above leave them out.  Counted from the exported rows of the timed ids.
        def mixed_chunks(id_tensor):
            rows = h.export_rows(id_tensor)                       # [B, W] int64 words
            E = 16 // self.esize                                  # tokens per chunk
            bytes_ = rows.view(torch.uint8)[:, : (V // 8)]        # whole bytes of full chunks
            if E == 8:
                chunk_bits = bytes_.to(torch.int32)
                full = 0xFF
            else:
                b = bytes_.to(torch.int32)
                chunk_bits = torch.stack([b & 0xF, b >> 4], dim=2).reshape(b.shape[0], -1)
                full = 0xF
            return int(((chunk_bits != 0) & (chunk_bits != full)).sum().item())

        # 128-byte lines of the logits (whole lines only) holding both valid and
        # invalid tokens: lines the call writes in part
        def partial_lines(id_tensor):
            rows = h.export_rows(id_tensor)
            T = 128 // self.esize                                 # tokens per line: 64 or 32
            if T == 64:
                words = rows[:, : V // 64]
                ones = -1
            else:
                w32 = rows.view(torch.int32)[:, : V // 32]
                words, ones = w32, -1
            return int(((words != 0) & (words != ones)).sum().item())

        mixed = float(np.mean([mixed_chunks(x) for x in id_lists]))
        partial = float(np.mean([partial_lines(x) for x in id_lists]))
        required_bytes = apply_bytes + 16 * mixed
        # the same at the memory's granularity: a 128-byte line of logits that
        # holds both valid and invalid tokens is read whole
        required_lines = apply_bytes + 128 * partial
        root_required = None
        if root_us is not None:
            r_lines = apply_bytes + 128 * partial_lines(ids)
            root_required = {"partial_lines": partial_lines(ids), "mixed_chunks": mixed_chunks(ids),
                             "required_bytes_lines": int(r_lines),
                             "frac_of_required_lines": round(r_lines / (root_us * 1e-6) / 1e9 / HBM_PEAK_GBPS, 4)}

        a0, a1 = self.event(), self.event()
        torch.cuda.synchronize()
        a0.record()
        for i in range(1000):
            h.advance(ids, toks, out=out)
        a1.record()
        torch.cuda.synchronize()
        advance_eager_us = a0.elapsed_time(a1) * 1e3 / 1000
        # the same calls replayed from a HIP graph: the device time without the
        # Python call overhead that bounds the eager loop
        advance_us = self.graph_us(lambda: h.advance(ids, toks, out=out), 100)
        calls = [0]

        def apply_next():  # the timed rows and buffers in turn
            k = calls[0]
            calls[0] += 1
            h.apply_mask(id_lists[k % len(id_lists)], bufs[k % nbuf])

        apply_graph_us = self.graph_us(apply_next, 100)

        # the compile kernels, each with its algorithmic bytes: the zero fill
        # writes the dense rows; the probe pass writes the hits, 4 bytes per node
        # and suffix length <= 16 (they hold the tails' masks and feed the
        # lists); the lists' prefix sum and fill write row offsets and entries
        lw = np.minimum(np.minimum(h.depth, h.max_token_len), 16)
        hit_bytes = 4 * int(lw.sum())
        sha = kernels_sha()
        kernels = {}
        if "zero" in alone and h.dense_rows:
            kernels["k_zero"] = hbm_roofline("k_zero", h.dense_rows * Wd * 8, alone["zero"],
                                             load_traffic(f"k_zero_{w.name}_{rep}_traffic.json", sha))
        probe_ms = alone.get("probe_marks", alone.get("probe_counts"))
        if probe_ms is not None:
            kernels["k_probe"] = hbm_roofline("k_probe", hit_bytes, probe_ms,
                                              load_traffic(f"k_probe_{w.name}_{rep}_traffic.json", sha))
        if "lists" in alone and "probe_counts" in alone:
            listed = M if rep == "lists" else None  # plain lists hold every valid pair
            ms = max(alone["lists"] - alone["probe_counts"], 1e-6)
            fill = "k_scan_*+k_fill_records" if rep == "tail_lists" else "k_scan_*+k_fill"
            kernels[fill] = {"kernel": fill, "avg_launch_ms": round(ms, 4),
                                        "algorithmic_bytes": None if listed is None else int((listed + N + 1) * 4),
                                        "achieved": None if listed is None else
                                        round((listed + N + 1) * 4 / (ms * 1e-3) / 1e9, 1), "unit": "GB/s"}
        # the dominant one (longest launch) is the line's roofline
        dom = max((k for k in kernels if k in ("k_zero", "k_probe")), key=lambda k: kernels[k]["avg_launch_ms"])
        roofline = kernels[dom]
        # work of the validity computation: the suffix probes made here, and the
        # (node, token) pairs a walk over first-byte token buckets would test
        tb, to = self.packed_vocab
        lens = np.diff(to)
        first = np.bincount(tb[to[:-1][lens > 0]], minlength=256)
        depth = h.depth
        work = {"suffix_probes": int(np.minimum(np.minimum(depth, h.max_token_len), 16).sum()),
                "tested_pairs_first_byte_buckets": int(first[h.edge_byte[depth > 0]].sum())}
        res = {
            "value": round(N * V / (ms_step / 1e3), 1),
            "ms_per_step": round(ms_step, 4),
            "N": N, "dense_rows": h.dense_rows, "valid_pairs": M,
            "device_bytes": h.device_bytes,
            "roofline": roofline,
            "rooflines_per_kernel": kernels,
            "compile_work": work,
            "compile_ms": {"device": round(dev_ms, 4),
                           "device_alone": {k: round(v, 4) for k, v in alone.items()},
                           "end_to_end_cold_min": round(min(cold), 3) if cold else None,
                           "end_to_end_cold_all": [round(x, 3) for x in cold],
                           "end_to_end_warm_min": round(min(warm), 3),
                           "end_to_end_warm_median": round(float(np.median(warm)), 3),
                           "end_to_end_warm_mean_std": [round(float(np.mean(warm)), 3), round(float(np.std(warm)), 3)],
                           "end_to_end_warm_all": [round(x, 3) for x in warm],
                           "end_to_end_cold_median": round(float(np.median(cold)), 3) if cold else None,
                           "one_set_warm": self.one_set_compile_ms(FLAGS[rep]),
                           "phases_cold": phases_cold, "phases_warm": phases_warm},
            "apply": {"us": round(apply_us, 3), "GBps": round(apply_gbps, 1), "bytes": apply_bytes,
                      "frac_of_hbm_roofline": round(apply_gbps / HBM_PEAK_GBPS, 4),
                      "same_rows_every_call": same_rows,
                      "mixed_chunks_per_call": round(mixed, 1),
                      "partial_lines_per_call": round(partial, 1),
                      "required_bytes": int(required_bytes),
                      "frac_of_required": round(required_bytes / (apply_us * 1e-6) / 1e9 / HBM_PEAK_GBPS, 4),
                      "required_bytes_lines": int(required_lines),
                      "frac_of_required_lines": round(required_lines / (apply_us * 1e-6) / 1e9 / HBM_PEAK_GBPS, 4),
                      "iters": self.args.apply_iters,
                      "rows": (f"{w.decode_steps}-step decode trajectory from the roots" if root_us is not None
                               else "uniform, 64 id lists in turn (new rows every call)" if same_rows
                               else w.node_mode),
                      "first_step_at_roots": (
                          {"us": round(root_us, 3),
                           "GBps": round(apply_bytes / (root_us * 1e-6) / 1e9, 1),
                           "frac_of_hbm_roofline": round(apply_bytes / (root_us * 1e-6) / 1e9 / HBM_PEAK_GBPS, 4),
                           **root_required}
                          if root_us is not None else None)},
            "advance_us": round(advance_us, 3),
            "advance_us_eager": round(advance_eager_us, 3),
            "apply_us_graph": round(apply_graph_us, 3),
            "bit_exact": self.parity(h, ids),
        }
        if res["compile_ms"]["one_set_warm"] is not None:
            print(f"[bench] {rep}: one set alone compiles in {res['compile_ms']['one_set_warm']:.3f} ms (warm)", flush=True)
        print(f"[bench] {rep}: apply {apply_us:.2f} us ({apply_gbps:.0f} GB/s; graph-replayed {apply_graph_us:.2f} us"
              + (f"; same rows every call {same_rows['us']:.2f} us" if same_rows else "") + "), "
              f"advance {advance_us:.2f} us (graph-replayed; eager loop {advance_eager_us:.2f} us)", flush=True)
        return h, res


    def measure_lazy(self, h_ref, reps=5):
        """Rows built on demand (TAM_FLAG_LAZY_ROWS): compile end to end with the
        vocabulary cached (no mask is computed), then a decode of up to 32 steps
        from the workload's start rows, mask apply + advance per step, timed with
        the row cache emptied first (every row built at its first use) and again
        with the cache kept; the main representation's handle runs the same
        trajectory."""
        torch, P, W, w, dev = self.torch, self.P, self.W, self.w, self.dev
        S = max(1, min(w.decode_steps, 32))
        e2e, hz = [], None
        for _ in range(10):  # as many warm runs as the main representation's
            if hz is not None:
                hz.close()
            torch.cuda.synchronize()
            t0 = time.perf_counter()
            hz = P.compile(self.packed, self.voc, sets=w.set_offsets, flags=P.FLAG_LAZY_ROWS | P.FLAG_TIMING)
            torch.cuda.synchronize()
            e2e.append((time.perf_counter() - t0) * 1e3)
        N, B = hz.num_nodes, self.B
        if w.node_mode == "uniform":
            start = W.uniform_nodes(w.config_id, N, B)
        elif w.node_mode == "set_roots":
            start = hz.roots[:B].astype(np.int32)
        else:
            start = np.zeros(B, dtype=np.int32)
        ids0 = torch.as_tensor(start, device=dev)
        fin = torch.as_tensor(hz.is_final.astype(np.bool_), device=dev)
        traj, toks, cur = [], [], ids0.clone()
        for s in range(S):
            lg = self.fresh_logits(1 + s)
            hz.apply_mask(cur, lg)
            tok = lg.float().argmax(dim=1).to(torch.int32)
            nxt = hz.advance(cur, tok)
            traj.append(cur.clone())
            toks.append(tok)
            cur = torch.where((nxt < 0) | fin[nxt.clamp(min=0).long()], ids0, nxt)
            del lg
        distinct = int(np.unique(torch.cat(traj).cpu().numpy()).size)
        out = torch.empty_like(ids0)

        def run(hh, reset):
            ts = []
            for r in range(reps):
                if reset:
                    hh.rebuild()
                e0, e1 = self.event(), self.event()
                e0.record()
                for s in range(S):
                    hh.apply_mask(traj[s], self.bufs[(r * S + s) % self.nbuf])
                    hh.advance(traj[s], toks[s], out=out)
                e1.record()
                torch.cuda.synchronize()
                ts.append(e0.elapsed_time(e1) * 1e3 / S)
            return float(np.median(ts))

        def run_graph(hh, reset):
            """The S steps captured once in a HIP graph and replayed."""
            s = torch.cuda.Stream()
            s.wait_stream(torch.cuda.current_stream())
            with torch.cuda.stream(s):
                for st in range(S):
                    hh.apply_mask(traj[st], self.bufs[st % self.nbuf])
                    hh.advance(traj[st], toks[st], out=out)
            torch.cuda.current_stream().wait_stream(s)
            torch.cuda.synchronize()
            g = torch.cuda.CUDAGraph()
            with torch.cuda.graph(g):
                for st in range(S):
                    hh.apply_mask(traj[st], self.bufs[st % self.nbuf])
                    hh.advance(traj[st], toks[st], out=out)
            ts = []
            for r in range(reps):
                if reset:
                    hh.rebuild()
                e0, e1 = self.event(), self.event()
                e0.record()
                g.replay()
                e1.record()
                torch.cuda.synchronize()
                ts.append(e0.elapsed_time(e1) * 1e3 / S)
            del g
            return float(np.median(ts))

        exact = self.parity(hz, ids0)
        cold, warm, ref = run(hz, True), run(hz, False), run(h_ref, False)
        gcold, gwarm, gref = run_graph(hz, True), run_graph(hz, False), run_graph(h_ref, False)
        res = {"cache_rows": hz.cache_rows, "device_bytes": hz.device_bytes,
               "compile_warm_ms": round(min(e2e), 3), "compile_warm_median": round(float(np.median(e2e)), 3),
               "compile_warm_all": [round(x, 3) for x in e2e],
               "one_set_compile_warm_ms": self.one_set_compile_ms(P.FLAG_LAZY_ROWS),
               "compile_phases": hz.timing(),
               "decode_steps": S, "batch": B, "distinct_rows": distinct,
               "step_us_cache_emptied": round(cold, 2), "step_us_cache_kept": round(warm, 2),
               "step_us_main_repr": round(ref, 2), "bit_exact": exact,
               "graph_replayed": {"step_us_cache_emptied": round(gcold, 2), "step_us_cache_kept": round(gwarm, 2),
                                  "step_us_main_repr": round(gref, 2)}}
        hz.close()
        if res["one_set_compile_warm_ms"] is not None:
            print(f"[bench] lazy rows: one set alone compiles in {res['one_set_compile_warm_ms']:.3f} ms (warm)",
                  flush=True)
        print(f"[bench] lazy rows: compile {min(e2e):.2f} ms, {S} steps x {B} rows ({distinct} distinct): "
              f"{cold:.1f} us/step from an empty cache, {warm:.1f} us/step cache kept, "
              f"{ref:.1f} us/step precomputed; graph-replayed {gcold:.1f} / {gwarm:.1f} / {gref:.1f} us/step",
              flush=True)
        return res


def cpu_model() -> str:
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def cpu_baseline(w, V, seconds, esize):
    """The oracle on a bounded sample of rows, one thread pinned to one core.
    Also the oracle's apply on a few rows, as GB/s of the same algorithmic
    bytes as the GPU apply.  Returns the baseline, the oracle and its sampled
    (nodes, rows), which the parity checks of every timed representation use."""
    import oracle
    prev = None
    try:
        prev = os.sched_getaffinity(0)
        os.sched_setaffinity(0, {min(prev)})
    except (AttributeError, OSError):
        prev = None
    try:
        t = time.perf_counter()
        o = oracle.Oracle(w.strings, w.vocab, set_offsets=w.set_offsets)
        build_s = time.perf_counter() - t
        rng = np.random.default_rng(99)
        rows_done, sample = 0, []
        t = time.perf_counter()
        while time.perf_counter() - t < seconds:
            nodes = rng.integers(0, o.N, size=64).astype(np.int32)
            sample.append((nodes, o.mask_rows(nodes)))
            rows_done += 64
        done = time.perf_counter() - t
        # apply: 8 rows of logits bits at a time, for about a second
        bits = rng.integers(0, 1 << (8 * esize), size=(8, V), dtype=np.uint64).astype(
            np.uint16 if esize == 2 else np.uint32)
        dt = oracle.DTYPE_BF16 if esize == 2 else oracle.DTYPE_FP32
        applied, t = 0, time.perf_counter()
        while time.perf_counter() - t < 1.0:
            o.apply(rng.integers(0, o.N, size=8).astype(np.int32), bits, dt)
            applied += 8
        apply_s = time.perf_counter() - t
    finally:
        if prev is not None:
            os.sched_setaffinity(0, prev)
    opps = rows_done * V / done
    Wd = (V + 63) // 64
    cpu = {"value": round(opps, 1), "unit": "pairs/s", "cores": 1, "kind": "oracle",
           "sample": f"{rows_done} random rows x V={V} tokens of {w.name} ({done:.1f} s, one thread"
                     f"{' pinned to one core' if prev is not None else ''}), trie build {build_s * 1e3:.0f} ms; "
                     f"full table extrapolates to {o.N * V / opps:.0f} s",
           "apply_GBps": round(applied * (Wd * 8 + V * esize) / apply_s / 1e9, 3),
           "host_cpus": os.cpu_count(), "cpu_model": cpu_model()}
    nodes = np.concatenate([n for n, _ in sample])
    rows = np.concatenate([r for _, r in sample])
    return cpu, o, (nodes, rows)


def profile_apply(bench, rep, rows):
    """Mask apply alone on one kind of rows (see --profile-apply)."""
    torch, P, W, w, dev = bench.torch, bench.P, bench.W, bench.w, bench.dev
    B, V, args = bench.B, bench.V, bench.args
    voc = P.Vocab(bench.packed_vocab)
    h = P.compile(bench.packed, voc, sets=w.set_offsets, flags=FLAGS[rep])
    N = h.num_nodes
    if rows == "uniform":
        lists = [torch.as_tensor(W.uniform_nodes(w.config_id, N, B, seed_extra=k), device=dev) for k in range(64)]
    else:
        roots = (h.roots[:B] if w.node_mode == "set_roots" else np.zeros(B)).astype(np.int32)
        lists = [torch.as_tensor(roots, device=dev)]
        if rows == "trajectory":
            fin = torch.as_tensor(h.is_final.astype(np.bool_), device=dev)
            ids, cur, lists = lists[0], lists[0].clone(), []
            for s in range(max(1, w.decode_steps)):
                lists.append(cur.clone())
                lg = bench.fresh_logits(1 + s)
                h.apply_mask(cur, lg)
                nxt = h.advance(cur, lg.float().argmax(dim=1).to(torch.int32))
                cur = torch.where((nxt < 0) | fin[nxt.clamp(min=0).long()], ids, nxt)
                del lg
    torch.cuda.synchronize()
    n = args.apply_warmup + args.apply_iters
    for i in range(args.apply_warmup):
        h.apply_mask(lists[i % len(lists)], bench.bufs[i % bench.nbuf])
    e0, e1 = bench.event(), bench.event()
    e0.record()
    for i in range(args.apply_warmup, n):
        h.apply_mask(lists[i % len(lists)], bench.bufs[i % bench.nbuf])
    e1.record()
    torch.cuda.synchronize()
    us = e0.elapsed_time(e1) * 1e3 / max(1, args.apply_iters)
    Wd = (V + 63) // 64
    apply_bytes = B * (Wd * 8 + V * bench.esize)
    print(json.dumps({"profile": "apply", "workload": w.name, "repr": rep, "rows": rows,
                      "dispatch_lists": len(lists), "calls": n, "us": round(us, 3), "bytes": apply_bytes,
                      "frac_of_hbm_roofline": round(apply_bytes / (us * 1e-6) / 1e9 / HBM_PEAK_GBPS, 4),
                      "kernels_sha": kernels_sha()}), flush=True)
    h.close()
    if args.calib_copy_mib:  # a copy of known size, for the counters' calibration
        src = torch.ones(args.calib_copy_mib << 20, dtype=torch.uint8, device=dev)
        dst = torch.empty_like(src)
        dst.copy_(src)
        torch.cuda.synchronize()


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
    forest = w.set_offsets is not None
    rep = args.repr if args.repr != "auto" else ("tail_lists" if forest else "full")
    print(f"[bench] workload {w.name}: K={K} V={V} B={B} ({gen_s:.1f}s to generate)", flush=True)

    bench = Bench(args, torch, P, W, w, dev)
    if args.profile_apply:
        profile_apply(bench, rep, args.profile_apply)
        return
    cpu = None
    if not args.no_cpu_baseline:
        cpu, bench.oracle, bench.sample = cpu_baseline(w, V, args.cpu_seconds, bench.esize)
    h, main_res = bench.measure(rep, args.steps, args.warmup, cold_runs=5)
    structure = bench.structure(h)

    # achievable write bandwidth on this device: a 4 GiB fill
    fill = torch.empty(1 << 32, dtype=torch.uint8, device=dev)
    fill.zero_()
    a0, a1 = bench.event(), bench.event()
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

    lazy = None if args.no_secondary else bench.measure_lazy(h)
    h.close()

    # character-position masks of fixed formats over the same vocabulary
    # (Appendix, Constraint-Aware Dispatch Beyond Finite Sets): end-to-end
    # compile with the vocabulary cached, and the device pass alone
    formats = {}
    for name, classes in W.formats().items():
        e2e = []
        for _ in range(5):
            torch.cuda.synchronize()
            t0 = time.perf_counter()
            hf = P.compile_format(classes, bench.voc)
            torch.cuda.synchronize()
            e2e.append((time.perf_counter() - t0) * 1e3)
            if _ < 4:
                hf.close()
        ev = [[bench.event() for _ in range(2)] for _ in range(20)]
        for e in ev:
            e[0].record()
            hf.rebuild()
            e[1].record()
        torch.cuda.synchronize()
        formats[name] = {"L": len(classes), "compile_warm_ms": round(min(e2e), 3),
                         "device_ms": round(float(np.mean([e[0].elapsed_time(e[1]) for e in ev])), 4),
                         "valid_pairs": hf.valid_pairs()}
        hf.close()
    print("[bench] character-position masks: " + ", ".join(
        f"{k} {v['device_ms'] * 1e3:.0f} us device / {v['compile_warm_ms']:.2f} ms" for k, v in formats.items()),
        flush=True)

    # the other representations of the same workload
    others = {}
    if not args.no_secondary:
        for r2 in (["lists", "tail"] if forest else ["tail"]):
            if r2 == rep:
                continue
            h2, others[r2] = bench.measure(r2, args.steps, args.warmup, cold_runs=0)
            h2.close()
    secondary = others.get("tail")

    N, M = main_res["N"], main_res["valid_pairs"]
    result = {
        "metric": METRIC,
        "value": main_res["value"],
        "unit": "(node,token) pairs/s",
        "value_note": ("(node, token) pairs resolved per second of the device step; the full table stores one "
                       "bit per pair (roofline 8 pairs per byte x 8 TB/s = 6.4e13 pairs/s), while tail "
                       "compression and lists store no bit for most pairs, so their pairs/s is not comparable "
                       "to that roofline"),
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": main_res["ms_per_step"],
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "u64",
        "data": "synthetic",
        "config": {"workload": f"{w.name}: {w.description}", "repr": rep, "K": K, "V": V, "N": N, "B": B,
                   "logits_dtype": w.dtype, "num_sets": w.num_sets, "valid_pairs": M},
        "roofline": main_res["roofline"],
        "roofline_apply": {"kernel": "k_apply_dense" if rep == "full" else "k_apply", "bound": "hbm",
                           "achieved": main_res["apply"]["GBps"],
                           "peak": HBM_PEAK_GBPS, "unit": "GB/s",
                           "frac": main_res["apply"]["frac_of_hbm_roofline"],
                           "traffic": (load_traffic(f"k_apply_{w.name}_{rep}_traffic.json", sha) or {})
                           .get("bytes_per_launch"),
                           "algorithmic_bytes": main_res["apply"]["bytes"],
                           "avg_launch_us": main_res["apply"]["us"]},
        "cpu_baseline": cpu,
        "compile_ms": dict(main_res["compile_ms"], vocabulary_build_once=round(bench.vocab_ms, 3),
                           python_list_packing=round(bench.pack_ms, 3),
                           python_vocabulary_packing=round(bench.vocab_pack_ms, 3)),
        "apply": main_res["apply"],
        "compile_work": main_res["compile_work"],
        "structure": structure,
        "advance_us": main_res["advance_us"],
        "advance_us_eager": main_res["advance_us_eager"],
        "apply_us_graph": main_res["apply_us_graph"],
        "device_bytes": main_res["device_bytes"],
        "tail_compression": secondary,
        "sparse_lists": others.get("lists"),
        "lazy_rows": lazy,
        "char_position_masks": formats,
        "fill_GBps_4GiB": round(fill_gbps, 1),
        "bit_exact": {"oracle_sample": None if bench.sample is None else
                      f"{len(bench.sample[0])} oracle rows drawn uniformly over the trie; apply and advance on the "
                      f"timed batch and on {B} sampled rows",
                      rep: main_res["bit_exact"],
                      **{r2: others[r2]["bit_exact"] for r2 in others},
                      "lazy": None if lazy is None else lazy["bit_exact"]},
        "kernels_sha": sha,
    }
    for key in ("roofline", "roofline_apply"):  # against the measured fill as well
        r = result[key]
        r["achievable_GBps"] = round(fill_gbps, 1)
        r["frac_of_achievable"] = round(r["achieved"] / fill_gbps, 4)
    bench.voc.close()
    print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()
