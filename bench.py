#!/usr/bin/env python3
"""Benchmark of the SemShareKV hot path on one MI355X.

One step = one pass of the whole path for one 5120-token target prompt against
a cached 5120-token reference prompt, Llama-3-8B attention shape (32 layers,
hidden 4096, 32 query / 8 kv heads, head_dim 128), bf16:
  RoPE-embed of the target embeddings -> 128-bit sign LSH -> top-1 Hamming
  match against the reference codes -> gather of the matched reference K/V
  rows for all 32 layers -> layer 0: full recompute with KV deviation ->
  high-deviation token selection (recompute fraction f) -> layers 1..31:
  partial prefill of the selected tokens over the assembled cache.
The reference side (its RoPE/LSH codes and its own K/V cache) is prepared
once before timing, as at cache-insert time.  Inputs are seeded synthetic
data resident in HBM before the timed region starts.

    python bench.py [--gpus 1] [--steps 20] [--warmup 20] [--frac 0.25]

Prints one JSON line (see the keys below).
"""
from __future__ import annotations

import argparse
import json
import math
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

HBM_PEAK_GBPS = 8000.0          # MI355X HBM3E
BF16_PEAK_TFLOPS = 2500.0       # MI355X dense bf16 MFMA
FP32_PEAK_TFLOPS = 157.3        # MI355X fp32 vector (and fp32 matrix)


def parse():
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=20)
    ap.add_argument("--config", type=int, choices=(2, 4), default=2,
                    help="2: 5120-token prompts (the headline); 4: 32768-token prompts (long context)")
    ap.add_argument("--frac", type=float, default=None,
                    help="recompute fraction of the headline line (default 0.25 at config 2, 0.10 at config 4)")
    ap.add_argument("--sweep", default=None,
                    help="recompute fractions also timed ('' to skip; default 0.10,0.25,0.50,1.00 at config 2, "
                         "none at config 4); 1.00 is the full-prefill analogue")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-budget-s", type=float, default=15.0, help="approximate oracle time of the CPU sample")
    ap.add_argument("--encode", choices=("fused", "two-pass"), default="fused",
                    help="RoPE + LSH of the target in one kernel, or rope_embed then lsh_encode")
    ap.add_argument("--gather", choices=("except", "all"), default="except",
                    help="except: the first layer's deviation reads the matched reference rows directly and the "
                         "layers after it are gathered after the selection, without the recomputed rows; all: "
                         "every layer and row gathered before the first layer")
    ap.add_argument("--gather-stream", choices=("serial", "overlap"), default="serial",
                    help="with --gather except: serial: one gather call for layers 1..L-1 before layer 1; overlap: "
                         "each later layer's gather runs on a second stream (default priority) and that layer's "
                         "attention waits for it (the same results; measured slower: the copies slow the compute "
                         "kernels they share the CUs and HBM with by more than they hide)")
    ap.add_argument("--matcher", choices=("mfma", "xor"), default="mfma",
                    help="top-1 Hamming matcher of the hot path: int8 MFMA or XOR/popcount (bit-identical outputs)")
    ap.add_argument("--vendor-compare", action="store_true",
                    help="instead of the hot path: time the two dominant operations against the platform's own "
                         "library path (torch SDPA for the first layer's causal attention, torch.matmul on hipBLASLt "
                         "for the projection) and print its JSON line")
    ap.add_argument("--fp32", action="store_true",
                    help="instead of the hot path: time the fp32 partial prefill (projection, attention) on the "
                         "tiny fp32 configuration and on a larger fp32 shape and print its JSON line")
    ap.add_argument("--dynamic-recompute", action="store_true",
                    help="time the average attention score per token and the dynamic recompute set instead")
    ap.add_argument("--schedule", choices=("fixed", "dynamic"), default="fixed",
                    help="dynamic: the step with the dynamic recompute set, nested per-layer recompute sets and "
                         "per-layer retention over compacted caches (its own JSON line)")
    ap.add_argument("--alpha-recomp", type=float, default=0.95,
                    help="dynamic schedule: recompute ratio of every layer after the second (nested sets)")
    ap.add_argument("--alpha-retain", type=float, default=0.98,
                    help="dynamic schedule: retention ratio of every layer after the first")
    ap.add_argument("--match-compare", action="store_true",
                    help="time the XOR/popcount and int8-MFMA matchers side by side instead of the hot path")
    ap.add_argument("--bank-similarity", action="store_true",
                    help="instead of the hot path: time the reference retrieval over a bank (a 4096-token target "
                         "against 16 prompts of 4096 tokens, 128- and 256-bit codes) and print its JSON line")
    ap.add_argument("--copy-calibration-mib", type=int, default=0,
                    help="before timing, run one plain device copy of this many MiB (a known-size reference "
                         "for FETCH_SIZE / WRITE_SIZE counter runs)")
    return ap.parse_args()


# HBM bytes per prefill_attention call at f = 0.25 (all 32 attention calls of a
# step averaged), from rocprofv3 FETCH_SIZE and WRITE_SIZE runs of this bench
# scaled by the same counters on a plain copy of known size; valid only for the
# attention source they were taken on (its SHA-256 below), otherwise null.
ATTN_TRAFFIC = {"source_sha256": "655f0832f7023c3c55e80f8258eaed498f72414721d2e5fbce93bf4983d10604",
                "bytes_per_call": 94579646}


def source_sha256(rel):
    import hashlib
    with open(os.path.join(ROOT, rel), "rb") as f:
        return hashlib.sha256(f.read()).hexdigest()


class Path:
    """Device buffers and the step of the hot path (config: 32 Llama-3-8B-shaped layers, 5k tokens)."""

    def __init__(self, torch, ss, cfg):
        import numpy as np

        import workloads
        self.torch, self.ss, self.cfg = torch, ss, cfg
        self.matcher = ss.match_mfma
        self.fused_encode = True
        self.gather_except = True
        self.gather_overlap = False
        self.side = torch.cuda.Stream()  # default priority
        self.gather_done = [torch.cuda.Event() for _ in range(cfg.n_layers)]
        dev = "cuda"
        bf = torch.bfloat16
        T, d, L = cfg.n_tok, cfg.dim, cfg.n_layers
        hq, hkv, D = cfg.n_q_heads, cfg.n_kv_heads, cfg.head_dim
        self.T, self.d, self.L, self.hq, self.hkv, self.D = T, d, L, hq, hkv, D

        def up(a):
            return torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).to(dev).to(bf).contiguous()

        pair = workloads.make_prompt_pair(cfg)
        self.e_ref = up(pair.e_ref)
        self.e_tgt = up(pair.e_tgt)
        self.planes = up(workloads.make_planes(cfg))
        # per-layer Wq/Wk/Wv ~ N(0, 0.02), drawn on the device from a seeded generator
        g = torch.Generator(device=dev)
        self.w = []
        for l in range(L):
            g.manual_seed(1000 * (cfg.cid + 1) + l)
            wq = (torch.randn((hq * D, d), generator=g, device=dev) * 0.02).to(bf)
            wk = (torch.randn((hkv * D, d), generator=g, device=dev) * 0.02).to(bf)
            wv = (torch.randn((hkv * D, d), generator=g, device=dev) * 0.02).to(bf)
            self.w.append((wq, wk, wv))
        # reference side, prepared once (insert time): codes and its own K/V cache
        self.allpos = torch.arange(T, dtype=torch.int32, device=dev)
        e_ref_rot = ss.rope_embed(self.e_ref)
        self.codes_ref = ss.lsh_encode(e_ref_rot, self.planes)
        self.ref_k = torch.zeros((L, T, hkv, D), dtype=bf, device=dev)
        self.ref_v = torch.zeros_like(self.ref_k)
        for l in range(L):
            ss.qkv_rope(self.e_ref, self.allpos, None, self.w[l][1], self.w[l][2], self.ref_k[l], self.ref_v[l], hq,
                        hkv, want_q=False)
        # target-side buffers
        self.e_rot = torch.empty_like(self.e_tgt)
        self.codes_t = torch.empty_like(self.codes_ref)
        self.idx = torch.empty(T, dtype=torch.int32, device=dev)
        self.dist = torch.empty(T, dtype=torch.int32, device=dev)
        self.asm_k = torch.empty_like(self.ref_k)
        self.asm_v = torch.empty_like(self.ref_v)
        self.q_full = torch.empty((T, hq, D), dtype=bf, device=dev)
        self.out_full = torch.empty_like(self.q_full)
        self.sigma = torch.empty(T, dtype=torch.float32, device=dev)
        ws = max(ss.qkv_rope_workspace_bytes(T, hq, hkv, D, bf),
                 ss.prefill_attention_workspace_bytes(T, T, hq, hkv, D, bf))
        self.set_frac(0.25, ws_hint=ws)

    def set_frac(self, frac, ws_hint=0):
        torch, ss = self.torch, self.ss
        bf = torch.bfloat16
        self.frac = frac
        self.n_sel = self.cfg.n_sel(frac)
        n = self.n_sel
        self.sel = torch.empty(n, dtype=torch.int32, device="cuda")
        self.q_sel = torch.empty((n, self.hq, self.D), dtype=bf, device="cuda")
        self.out_sel = torch.empty_like(self.q_sel)
        # the attention work plan of the selection, made once per step and shared by layers 1..L-1
        self.rope_sel = torch.empty(max(16, ss.rope_table_bytes(n, self.D)), dtype=torch.uint8, device="cuda")
        self.plan = torch.empty(max(1, ss.attention_plan_bytes(n, self.T, self.hq, self.hkv, self.D, bf)),
                                dtype=torch.uint8, device="cuda")
        need = max(ws_hint,
                   ss.qkv_rope_workspace_bytes(self.T, self.hq, self.hkv, self.D, bf),
                   ss.prefill_attention_workspace_bytes(self.T, self.T, self.hq, self.hkv, self.D, bf),
                   ss.prefill_attention_workspace_bytes(n, self.T, self.hq, self.hkv, self.D, bf))
        self.ws = torch.empty(need, dtype=torch.uint8, device="cuda")

    # ---- the stages of one step, in order; the per-layer ones take the layer
    def s_encode(self):
        ss = self.ss
        if self.fused_encode:
            ss.rope_lsh_encode(self.e_tgt, self.planes, out=self.codes_t)
        else:
            ss.rope_embed(self.e_tgt, out=self.e_rot)
            ss.lsh_encode(self.e_rot, self.planes, out=self.codes_t)

    def s_match(self):
        self.matcher(self.codes_t, self.codes_ref, idx=self.idx, dist=self.dist)

    def s_gather(self):
        if not self.gather_except:
            self.ss.gather_kv(self.ref_k, self.ref_v, self.idx, out_k=self.asm_k, out_v=self.asm_v)

    def s_qkv0(self):
        ss, hq, hkv = self.ss, self.hq, self.hkv
        wq, wk, wv = self.w[0]
        if self.gather_except:
            # layer 0 recomputes every row, so its gathered rows would feed the deviation only: it reads the
            # matched reference rows directly; layers 1.. are gathered after the selection, without the
            # recomputed rows
            ss.qkv_rope_dev_ref(self.e_tgt, self.allpos, wq, wk, wv, self.asm_k[0], self.asm_v[0], hq, hkv,
                                self.ref_k[0], self.ref_v[0], self.idx, q_out=self.q_full, deviation=self.sigma,
                                workspace=self.ws)
        else:
            ss.qkv_rope(self.e_tgt, self.allpos, wq, wk, wv, self.asm_k[0], self.asm_v[0], hq, hkv,
                        q_out=self.q_full, deviation=self.sigma, want_deviation=True, workspace=self.ws)

    def s_attn0(self):
        self.ss.prefill_attention(self.q_full, self.allpos, self.asm_k[0], self.asm_v[0], self.hkv, out=self.out_full,
                                  workspace=self.ws)

    def s_select(self):
        ss = self.ss
        ss.select_recompute(self.sigma, self.n_sel, out=self.sel)
        ss.attention_plan(self.sel, self.T, self.hq, self.hkv, self.D, out=self.plan)
        ss.rope_table(self.sel, self.T, self.D, out=self.rope_sel)

    def s_gather_rest(self):
        if self.gather_except:
            self.ss.gather_kv(self.ref_k[1:], self.ref_v[1:], self.idx, out_k=self.asm_k[1:], out_v=self.asm_v[1:],
                              except_pos=self.sel)

    def s_gather_layers_async(self):
        """The except-gather of layers 1..L-1 as one call per layer on the side
        stream, after the selection; layer l's attention waits for its event.
        A projection only writes its layer's selected rows, which the gather
        leaves alone, so it need not wait."""
        torch = self.torch
        self.side.wait_stream(torch.cuda.current_stream())
        with torch.cuda.stream(self.side):
            for l in range(1, self.L):
                self.ss.gather_kv(self.ref_k[l:l + 1], self.ref_v[l:l + 1], self.idx, out_k=self.asm_k[l:l + 1],
                                  out_v=self.asm_v[l:l + 1], except_pos=self.sel)
                self.gather_done[l].record(self.side)

    def s_qkv(self, l):
        # the recomputed tokens' rows are read from the target's embeddings in place
        wq, wk, wv = self.w[l]
        self.ss.qkv_rope(self.e_tgt, self.sel, wq, wk, wv, self.asm_k[l], self.asm_v[l], self.hq, self.hkv,
                         q_out=self.q_sel, workspace=self.ws, rope_table=self.rope_sel, x_rows=self.sel)

    def s_attn(self, l):
        self.ss.prefill_attention(self.q_sel, self.sel, self.asm_k[l], self.asm_v[l], self.hkv, out=self.out_sel,
                                  workspace=self.ws, plan=self.plan)

    def step(self):
        """One pass of the hot path."""
        self.s_encode()
        self.s_match()
        self.s_gather()
        self.s_qkv0()
        self.s_attn0()
        self.s_select()
        overlap = self.gather_except and self.gather_overlap
        if overlap:
            self.s_gather_layers_async()
        else:
            self.s_gather_rest()
        main = self.torch.cuda.current_stream()
        for l in range(1, self.L):
            self.s_qkv(l)
            if overlap:
                main.wait_event(self.gather_done[l])  # the last one also covers every earlier gather
            self.s_attn(l)


def time_steps(torch, path, steps, warmup):
    """Times `steps` steps after `warmup` untimed ones: one HIP event pair on
    the launch stream around the whole run."""
    for _ in range(warmup):
        path.step()
    stream = torch.cuda.current_stream()
    t0 = torch.cuda.Event(enable_timing=True)
    t1 = torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    wall0 = time.perf_counter()
    t0.record(stream)
    for _ in range(steps):
        path.step()
    t1.record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - wall0
    return t0.elapsed_time(t1) / steps, wall / steps * 1e3


def stage_times(torch, path, reps):
    """Per-call duration of every stage of a step.  A stage is timed as a run
    of its own calls with the inputs of a real step (one full step first),
    between one HIP event pair on the launch stream: 5 * reps (at least 10)
    calls of a once-per-step stage (some take a few microseconds, so a short
    run would mostly time the host), `reps` passes over layers 1..L-1 of a
    per-layer one.
    No event sits between the calls of a run, so the figure is the kernels'
    time plus the launch gaps of back-to-back calls."""
    path.step()
    stream = torch.cuda.current_stream()
    once = [("rope_lsh", path.s_encode), ("match", path.s_match)]
    once += [("gather_rest", path.s_gather_rest)] if path.gather_except else [("gather", path.s_gather)]
    once += [("qkv0", path.s_qkv0), ("attn0", path.s_attn0), ("select", path.s_select)]
    out = {}
    n_once = max(10, 5 * reps)
    for name, fn in once:
        fn()
        t0, t1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        t0.record(stream)
        for _ in range(n_once):
            fn()
        t1.record(stream)
        torch.cuda.synchronize()
        out[name] = t0.elapsed_time(t1) / n_once
    for name, fn in (("qkv", path.s_qkv), ("attn", path.s_attn)):
        t0, t1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        t0.record(stream)
        for _ in range(reps):
            for l in range(1, path.L):
                fn(l)
        t1.record(stream)
        torch.cuda.synchronize()
        out[name] = t0.elapsed_time(t1) / (reps * (path.L - 1))
    path.step()  # leave every buffer as a plain step leaves it
    torch.cuda.synchronize()
    return out


def flushed_medians(torch, path, reps):
    """Median durations over `reps` single runs, each after a 512 MiB write
    that pushes the previous run's data out of L2 and the 256 MB Infinity
    Cache: one whole step, and one partial-layer prefill_attention call (a
    layer in the middle of the stack).  A HIP event pair on the launch stream
    brackets each run; the flush is outside it."""
    flush = torch.empty(512 << 20, dtype=torch.uint8, device="cuda")
    stream = torch.cuda.current_stream()
    mid = max(1, path.L // 2)

    def runs(fn):
        t = []
        for _ in range(reps):
            flush.fill_(1)
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record(stream)
            fn()
            e1.record(stream)
            torch.cuda.synchronize()
            t.append(e0.elapsed_time(e1))
        t.sort()
        return {"median_ms": t[len(t) // 2] if len(t) % 2 else 0.5 * (t[len(t) // 2 - 1] + t[len(t) // 2]),
                "min_ms": t[0], "max_ms": t[-1]}

    path.step()
    out = {"reps": reps, "flush_bytes": flush.numel(), "step": runs(path.step),
           "attn_partial_layer": runs(lambda: path.s_attn(mid))}
    path.step()
    torch.cuda.synchronize()
    del flush
    return out


def attention_flops(sel_pos, hq, D):
    """4 * D * Hq * sum_s (p_s + 1): QK^T and PV multiply-adds of causal attention."""
    return 4.0 * D * hq * float((sel_pos.astype("float64") + 1.0).sum())


def cpu_baseline(cfg, frac, budget_s):
    """The oracle, as it stands, on a bounded sample of one step: each stage is
    run on a slice of its rows and scaled by work to the full step."""
    import numpy as np

    import oracle as orc
    import workloads
    T, d, L, hq, hkv, D = cfg.n_tok, cfg.dim, cfg.n_layers, cfg.n_q_heads, cfg.n_kv_heads, cfg.head_dim
    n_sel = cfg.n_sel(frac)
    rng = np.random.default_rng(0)
    pair = workloads.make_prompt_pair(cfg)
    planes = workloads.make_planes(cfg)
    w = workloads.make_weights(cfg, 0)
    k, v = workloads.make_cache(cfg, 1, T)
    k, v = k[0].reshape(T, -1), v[0].reshape(T, -1)
    sel = workloads.make_sel_pos(cfg, T, n_sel)
    est = {}
    # sample sizes chosen so the whole sample costs about budget_s on 16 threads
    scale = max(budget_s / 15.0, 0.05)
    nr = max(16, int(256 * scale))
    t = time.perf_counter(); e = orc.rope_embed(pair.e_tgt[:nr], dtype="bf16"); est["rope"] = (time.perf_counter() - t) * T / nr
    t = time.perf_counter(); c = orc.lsh_encode(e, planes); est["lsh"] = (time.perf_counter() - t) * T / nr
    cr = orc.lsh_encode(orc.rope_embed(pair.e_ref[:nr], dtype="bf16"), planes)
    codes_ref = np.tile(cr, (T // nr + 1, 1))[:T]
    t = time.perf_counter(); orc.match(c, codes_ref); est["match"] = (time.perf_counter() - t) * T / nr
    idx = rng.integers(0, T, T).astype(np.int32)
    rows16 = rng.integers(0, 2**16, size=(1, T, hkv * D), dtype=np.uint16)  # one layer's K, bf16 bit patterns
    t = time.perf_counter(); orc.gather_rows(rows16, idx); est["gather"] = (time.perf_counter() - t) * 2 * L
    nq = max(4, int(16 * scale))
    rows = np.sort(rng.choice(n_sel, nq, replace=False))
    t = time.perf_counter()
    orc.qkv_rows(pair.e_tgt[sel[rows]], sel[rows], w.wq, w.wk, w.wv, hq, hkv, D, dtype="bf16")
    per_row_qkv = (time.perf_counter() - t) / nq
    q, _, _ = orc.qkv_rows(pair.e_tgt[sel[rows]], sel[rows], w.wq, w.wk, w.wv, hq, hkv, D, dtype="bf16", want_kv=False)
    t = time.perf_counter()
    orc.attention_rows(q, sel[rows], k, v, hq, hkv, D, dtype="bf16")
    per_key_attn = (time.perf_counter() - t) / float((sel[rows] + 1).sum())
    est["qkv0"] = per_row_qkv * T
    est["attn0"] = per_key_attn * T * (T + 1) / 2
    sigma = rng.exponential(size=T)
    t = time.perf_counter(); orc.select_recompute(sigma, n_sel); est["select"] = time.perf_counter() - t
    est["qkv"] = per_row_qkv * n_sel * (L - 1)
    est["attn"] = per_key_attn * float((sel + 1).sum()) * (L - 1)
    total = sum(est.values())
    sample = (f"oracle on {nr} of {T} rows for RoPE/LSH/match, 1 of {2 * L} gathered layer tensors, {nq} selected "
              f"rows for QKV and attention; each stage scaled by its work to one full step (f={frac}), extrapolated")
    return {"value": T / total, "unit": "tokens/s", "cores": orc.num_threads(), "kind": "oracle", "sample": sample,
            "est_step_s": total, "est_stage_s": {k2: round(v2, 6) for k2, v2 in est.items()}}


def bank_similarity_line(torch, np, ss, cfg, args):
    """Reference retrieval (Appendix A.3 score over a bank): one 4096-token
    target against 16 reference prompts of 4096 tokens (the bank shape),
    seeded synthetic codes, 128 and 256 bits.  Integer VALU bound: 4W + 1
    operations per (target, reference) pair (2W XOR, 2W popcount-accumulate,
    one min), peak 256 CU x 4 SIMD x 16 lanes x 2.4 GHz = 39.3 T ops/s."""
    out = {"metric": "bank_similarity_pairs_per_s", "unit": "pairs/s", "n_gpus": 1, "steps": args.steps,
           "warmup": args.warmup, "higher_is_better": True, "data": "synthetic", "dtype": "u64",
           "config": {"workload": "retrieval over a bank: 4096-token target x 16 prompts x 4096 tokens"}, "by_bits": {}}
    n_tgt, n_prompts, per = 4096, 16, 4096
    for w in (2, 4):
        tgt = torch.from_numpy(cfg_codes(np, cfg, n_tgt, w, 1)).cuda()
        ref = torch.from_numpy(cfg_codes(np, cfg, n_prompts * per, w, 2)).cuda()
        off = torch.arange(n_prompts + 1, dtype=torch.int64, device="cuda") * per
        ws = torch.empty(max(1, ss.semshare.load().semshare_bank_similarity_workspace(n_tgt, n_prompts)),
                         dtype=torch.uint8, device="cuda")
        for _ in range(args.warmup):
            ss.bank_similarity(tgt, ref, off, workspace=ws)
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(args.steps):
            ss.bank_similarity(tgt, ref, off, workspace=ws)
        e1.record()
        torch.cuda.synchronize()
        us = e0.elapsed_time(e1) / args.steps * 1e3
        pairs = n_tgt * n_prompts * per
        ops = pairs * (4 * w + 1)
        out["by_bits"][str(64 * w)] = {"us_per_call": round(us, 2), "pairs_per_s": pairs / (us * 1e-6),
                                        "roofline": {"bound": "alu", "achieved": round(ops / us / 1e6, 2),
                                                     "peak": 39.3, "unit": "T int ops/s",
                                                     "frac": round(ops / us / 1e6 / 39.3, 3)}}
    out["value"] = out["by_bits"]["128"]["pairs_per_s"]
    print(json.dumps(out), flush=True)


def match_compare_line(torch, np, ss, configs, args):
    """The two top-1 Hamming matchers side by side (Sections 4.2, 4.3), on the
    headline shape (5120 x 5120 tokens, 128 bits), the bank shape (4096 x
    16 x 4096, 256 bits) and the long shape (32768 x 32768, 128 bits), seeded
    synthetic codes.  XOR/popcount: integer VALU bound, 4W + 1 operations per
    pair, peak 39.3 T ops/s.  int8 matrix cores: 2 n_b operations per pair
    (one multiply-add per bit), dense int8 peak 5.0 P ops/s.  Both return
    bit-identical outputs (checked here on every shape)."""
    out = {"metric": "match_token_pairs_per_s", "unit": "pairs/s", "n_gpus": 1, "steps": args.steps,
           "warmup": args.warmup, "higher_is_better": True, "data": "synthetic", "dtype": "u64",
           "config": {"workload": "top-1 Hamming match, XOR/popcount vs int8 MFMA"}, "shapes": {}}
    shapes = [("5120x5120_128b", configs[2], 5120, 5120, 2), ("4096x65536_256b", configs[3], 4096, 65536, 4),
              ("32768x32768_128b", configs[4], 32768, 32768, 2)]
    for name, cfg, n_tgt, n_ref, w in shapes:
        tgt = torch.from_numpy(cfg_codes(np, cfg, n_tgt, w, 1)).cuda()
        ref = torch.from_numpy(cfg_codes(np, cfg, n_ref, w, 2)).cuda()
        pairs = n_tgt * n_ref
        row = {}
        res = {}
        for kind, fn in (("xor", ss.match), ("mfma", ss.match_mfma)):
            idx = torch.empty(n_tgt, dtype=torch.int32, device="cuda")
            dist = torch.empty(n_tgt, dtype=torch.int32, device="cuda")
            for _ in range(args.warmup):
                fn(tgt, ref, idx=idx, dist=dist)
            torch.cuda.synchronize()
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record()
            for _ in range(args.steps):
                fn(tgt, ref, idx=idx, dist=dist)
            e1.record()
            torch.cuda.synchronize()
            us = e0.elapsed_time(e1) / args.steps * 1e3
            res[kind] = (idx.cpu(), dist.cpu())
            if kind == "xor":
                ops, peak, unit, bound = pairs * (4 * w + 1), 39.3, "T int ops/s", "alu"
                achieved = ops / us / 1e6
            else:
                ops, peak, unit, bound = pairs * 2 * 64 * w, 5000.0, "T int8 ops/s", "mfma"
                achieved = ops / us / 1e6
            row[kind] = {"us_per_call": round(us, 2), "pairs_per_s": pairs / (us * 1e-6),
                         "roofline": {"bound": bound, "achieved": round(achieved, 1), "peak": peak, "unit": unit,
                                      "frac": round(achieved / peak, 3)}}
        row["identical"] = bool(torch.equal(res["xor"][0], res["mfma"][0]) and torch.equal(res["xor"][1], res["mfma"][1]))
        row["speedup_mfma"] = round(row["xor"]["us_per_call"] / row["mfma"]["us_per_call"], 2)
        out["shapes"][name] = row
        del tgt, ref
    out["value"] = out["shapes"]["5120x5120_128b"]["mfma"]["pairs_per_s"]
    print(json.dumps(out), flush=True)


def dynamic_recompute_line(torch, np, ss, cfg, args):
    """The dynamic recompute step on the headline shape (Section 3 Insight 2,
    Section 4.3.3): average attention score per token of the fully computed
    first layer (5120 tokens, 32 q / 8 kv heads, head_dim 128, bf16, seeded
    synthetic q and K), then AR at 55%, hot / cold and the recompute set.
    Bound: MFMA; the two passes over the causal score matrix do 2 x 2 D flops
    per (head, query, key <= query) pair = 4 D H_q T (T + 1) / 2."""
    import workloads
    T, hq, hkv, D = 5120, 32, 8, 128
    q = torch.from_numpy(workloads.make_rows(cfg, T, hq * D, tag=70)).to("cuda").to(torch.bfloat16).view(T, hq, D)
    k = torch.from_numpy(workloads.make_rows(cfg, T, hkv * D, tag=71)).to("cuda").to(torch.bfloat16).view(T, hkv, D)
    sigma = torch.from_numpy(np.random.default_rng(72).exponential(size=T).astype(np.float32)).cuda()
    mass = torch.empty(T, dtype=torch.float32, device="cuda")
    ws = torch.empty(int(ss.semshare.load().semshare_attention_mass_workspace(T, hq)), dtype=torch.uint8, device="cuda")
    sel = torch.empty(T, dtype=torch.int32, device="cuda")
    counts = torch.empty(3, dtype=torch.int32, device="cuda")

    def run():
        ss.attention_mass(q, k, hq, hkv, mass=mass, workspace=ws)
        ss.dynamic_recompute(mass, sigma, sel_pos=sel, counts=counts)
    for _ in range(args.warmup):
        run()
    torch.cuda.synchronize()
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(3)]
    t_mass = t_sel = 0.0
    for _ in range(args.steps):
        ev[0].record()
        ss.attention_mass(q, k, hq, hkv, mass=mass, workspace=ws)
        ev[1].record()
        ss.dynamic_recompute(mass, sigma, sel_pos=sel, counts=counts)
        ev[2].record()
        torch.cuda.synchronize()
        t_mass += ev[0].elapsed_time(ev[1])
        t_sel += ev[1].elapsed_time(ev[2])
    us_mass, us_sel = t_mass / args.steps * 1e3, t_sel / args.steps * 1e3
    flops = 4 * D * hq * T * (T + 1) / 2
    c = counts.cpu().numpy().tolist()
    # retention (first layer): window of the last (1 - AR/T) rows, ranking,
    # and the compaction of a 32-layer K/V cache to the kept rows
    ar = c[0]
    row_begin = min(T - 1, T - int(np.floor((1.0 - ar / T) * T + 0.5)))
    L = 32
    kc = torch.randn(L, T, hkv, D, device="cuda").to(torch.bfloat16)
    vc = torch.randn(L, T, hkv, D, device="cuda").to(torch.bfloat16)
    score = torch.empty(T, dtype=torch.float32, device="cuda")
    t_win = t_ret = t_cmp = 0.0
    for it in range(args.warmup + args.steps):
        ev[0].record()
        # the window pass takes the row normalisers the full pass left in ws
        ss.attention_mass(q, k, hq, hkv, mass=score, workspace=ws, row_begin=row_begin, reuse_normalisers=True)
        ev[1].record()
        rank, kept, n_kept = ss.retention(mass, score, sel, counts, 0.8)
        ev[2].record()
        torch.cuda.synchronize()
        nk = int(n_kept.cpu().numpy()[0])
        e3, e4 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e3.record()
        ok, ov = ss.gather_kv(kc, vc, kept[:nk])
        e4.record()
        torch.cuda.synchronize()
        if it >= args.warmup:
            t_win += ev[0].elapsed_time(ev[1])
            t_ret += ev[1].elapsed_time(ev[2])
            t_cmp += e3.elapsed_time(e4)
    n = args.steps
    out = {"metric": "dynamic_recompute_us", "value": us_mass + us_sel, "unit": "us", "n_gpus": 1,
           "steps": args.steps, "warmup": args.warmup, "higher_is_better": False, "data": "synthetic", "dtype": "bf16",
           "config": {"workload": "average attention score per token + AR 55% + hot/cold recompute set, 5120 tokens, "
                                  "32q/8kv heads, head_dim 128; then first-layer retention and a 32-layer cache "
                                  "compaction"},
           "attention_mass_us": round(us_mass, 2), "dynamic_select_us": round(us_sel, 2),
           "AR": c[0], "n_recompute": c[1], "n_hot_recompute": c[2],
           "retention": {"window_rows": T - row_begin, "window_mass_us": round(t_win / n * 1e3, 2),
                         "window_reuses_row_normalisers": True,
                         "rank_us": round(t_ret / n * 1e3, 2), "n_kept": nk,
                         "compaction_us": round(t_cmp / n * 1e3, 2),
                         "compaction_GB_per_s": 2 * 2 * L * nk * hkv * D * 2 / (t_cmp / n * 1e-3) / 1e9},
           "roofline": {"kernel": "mass_lse_kernel + mass_col_kernel + mass_final_kernel", "bound": "mfma",
                        "achieved": flops / (us_mass * 1e-6) / 1e12, "peak": BF16_PEAK_TFLOPS, "unit": "TFLOP/s",
                        "frac": flops / (us_mass * 1e-6) / 1e12 / BF16_PEAK_TFLOPS}}
    print(json.dumps(out), flush=True)


def vendor_compare_line(torch, np, ss, cfg, args):
    """The two dominant operations of the step against the platform's own
    library path on the same box, same inputs (5120 tokens, 32 q / 8 kv heads,
    head_dim 128, hidden 4096, bf16): the first layer's causal attention over
    all rows (prefill_attention vs torch's scaled_dot_product_attention, flash
    backend, grouped-query heads), and a partial layer's projection of the
    1280 selected rows (qkv_rope, which also applies RoPE and scatters K/V into
    the cache, vs a plain torch.matmul on hipBLASLt that does neither).  Event
    timing over runs of back-to-back calls; the largest difference between the
    two results is reported as a check."""
    import torch.nn.functional as F
    T, hq, hkv, D, d = cfg.n_tok, cfg.n_q_heads, cfg.n_kv_heads, cfg.head_dim, cfg.dim
    n_sel = cfg.n_sel(0.25)
    bf = torch.bfloat16
    g = torch.Generator(device="cuda").manual_seed(0)
    q = torch.randn(T, hq, D, device="cuda", generator=g).to(bf)
    k = torch.randn(T, hkv, D, device="cuda", generator=g).to(bf)
    v = torch.randn(T, hkv, D, device="cuda", generator=g).to(bf)
    pos = torch.arange(T, dtype=torch.int32, device="cuda")
    reps = max(10, args.steps)

    def timed(fn):
        for _ in range(max(3, args.warmup)):
            fn()
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(reps):
            fn()
        e1.record()
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) / reps * 1e3

    out = torch.empty_like(q)
    ws = torch.empty(ss.prefill_attention_workspace_bytes(T, T, hq, hkv, D, bf), dtype=torch.uint8, device="cuda")
    attn_ours = timed(lambda: ss.prefill_attention(q, pos, k, v, hkv, out=out, workspace=ws))
    qt, kt, vt = (t.transpose(0, 1).unsqueeze(0).contiguous() for t in (q, k, v))
    from torch.nn.attention import SDPBackend, sdpa_kernel
    with sdpa_kernel([SDPBackend.FLASH_ATTENTION]):
        o = F.scaled_dot_product_attention(qt, kt, vt, is_causal=True, enable_gqa=True)
        attn_torch = timed(lambda: F.scaled_dot_product_attention(qt, kt, vt, is_causal=True, enable_gqa=True))
    attn_diff = (o[0].transpose(0, 1).float() - out.float()).abs().max().item()
    fl = 4.0 * D * hq * T * (T + 1) / 2.0
    # projection of the selected rows
    x = (torch.randn(n_sel, d, device="cuda", generator=g) * 0.5).to(bf)
    w = [(torch.randn(r * D, d, device="cuda", generator=g) * 0.02).to(bf) for r in (hq, hkv, hkv)]
    sel = torch.sort(torch.randperm(T, device="cuda", generator=g)[:n_sel])[0].to(torch.int32)
    kc, vc = torch.zeros(T, hkv, D, dtype=bf, device="cuda"), torch.zeros(T, hkv, D, dtype=bf, device="cuda")
    q_out = torch.empty(n_sel, hq, D, dtype=bf, device="cuda")
    ws2 = torch.empty(ss.qkv_rope_workspace_bytes(n_sel, hq, hkv, D, bf), dtype=torch.uint8, device="cuda")
    table = torch.empty(ss.rope_table_bytes(n_sel, D), dtype=torch.uint8, device="cuda")
    ss.rope_table(sel, T, D, out=table)
    qkv_ours = timed(lambda: ss.qkv_rope(x, sel, w[0], w[1], w[2], kc, vc, hq, hkv, q_out=q_out, workspace=ws2,
                                         rope_table=table))
    wcat = torch.cat(w, 0).contiguous()
    y = torch.empty(n_sel, wcat.shape[0], dtype=bf, device="cuda")
    qkv_torch = timed(lambda: torch.matmul(x, wcat.t(), out=y))
    v_diff = (y[:, (hq + hkv) * D:].float().view(n_sel, hkv, D) - vc[sel.long()].float()).abs().max().item()
    qfl = 2.0 * n_sel * (hq + 2 * hkv) * D * d
    out_line = {"metric": "vendor_compare_us", "value": attn_ours, "unit": "us", "n_gpus": 1, "steps": reps,
                "warmup": args.warmup,
                "higher_is_better": False, "data": "synthetic", "dtype": "bf16",
                "config": {"workload": f"first-layer causal attention over {T} tokens (32 q / 8 kv heads, head_dim "
                                       f"128) and the projection of {n_sel} selected rows (hidden 4096 -> 6144)"},
                "attention_layer0": {"ours_us": attn_ours, "torch_sdpa_flash_us": attn_torch,
                                     "ours_TFLOPs": fl / attn_ours / 1e6, "torch_TFLOPs": fl / attn_torch / 1e6,
                                     "speedup": attn_torch / attn_ours, "max_abs_diff": attn_diff},
                "qkv_partial": {"ours_us": qkv_ours, "torch_matmul_us": qkv_torch,
                                "ours_TFLOPs": qfl / qkv_ours / 1e6, "torch_TFLOPs": qfl / qkv_torch / 1e6,
                                "speedup": qkv_torch / qkv_ours, "v_rows_max_abs_diff": v_diff,
                                "note": "ours also applies RoPE to q and k and scatters k and v into the cache"}}
    print(json.dumps(out_line), flush=True)


def fp32_line(torch, np, ss, cfg, args):
    """The fp32 path (VALU kernels, no matrix cores): one partial-prefill
    layer, projection and attention timed separately, on the tiny fp32
    configuration (512 tokens, hidden 256, 4/4 heads, head_dim 64, f = 0.2)
    and on a larger fp32 shape (4096 tokens, hidden 1024, 8/8 heads, f = 0.25).
    Bound: fp32 vector ALU, peak 157.3 TFLOP/s."""
    import workloads
    out = {"metric": "fp32_partial_prefill_TFLOPs", "unit": "TFLOP/s", "n_gpus": 1, "steps": args.steps,
           "warmup": args.warmup, "higher_is_better": True, "data": "synthetic", "dtype": "f32",
           "config": {"workload": "one fp32 partial-prefill layer: 512 tok / hidden 256 / 4-4 heads / D 64 / f 0.2, "
                                  "and 4096 tok / hidden 1024 / 8-8 heads / D 64 / f 0.25"}, "shapes": {}}
    for T, d, hq, hkv, D, f in ((cfg.n_tok, cfg.dim, cfg.n_q_heads, cfg.n_kv_heads, cfg.head_dim, 0.2),
                                (4096, 1024, 8, 8, 64, 0.25)):
        n = int(np.floor(f * T + 0.5))
        g = torch.Generator(device="cuda").manual_seed(T)
        x = torch.randn(n, d, device="cuda", generator=g)
        wq = torch.randn(hq * D, d, device="cuda", generator=g) * 0.02
        wk = torch.randn(hkv * D, d, device="cuda", generator=g) * 0.02
        wv = torch.randn(hkv * D, d, device="cuda", generator=g) * 0.02
        kc = torch.randn(T, hkv, D, device="cuda", generator=g)
        vc = torch.randn(T, hkv, D, device="cuda", generator=g)
        sel = workloads.make_sel_pos(cfg, T, n, tag=500 + T)
        pos = torch.from_numpy(sel).cuda()
        q, _ = ss.qkv_rope(x, pos, wq, wk, wv, kc, vc, hq, hkv)
        o = ss.prefill_attention(q, pos, kc, vc, hkv)
        res = {}
        for name, fn, flops in (("qkv", lambda: ss.qkv_rope(x, pos, wq, wk, wv, kc, vc, hq, hkv, q_out=q),
                                 2.0 * n * (hq + 2 * hkv) * D * d),
                                ("attention", lambda: ss.prefill_attention(q, pos, kc, vc, hkv, out=o),
                                 4.0 * D * hq * float((sel.astype(np.float64) + 1).sum()))):
            for _ in range(args.warmup):
                fn()
            torch.cuda.synchronize()
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record()
            for _ in range(args.steps):
                fn()
            e1.record()
            torch.cuda.synchronize()
            us = e0.elapsed_time(e1) / args.steps * 1e3
            tf = flops / (us * 1e-6) / 1e12
            res[name] = {"us_per_call": round(us, 2), "flops": flops,
                         "roofline": {"bound": "alu", "achieved": tf, "peak": FP32_PEAK_TFLOPS, "unit": "TFLOP/s",
                                      "frac": tf / FP32_PEAK_TFLOPS}}
        out["shapes"][f"{T}tok_h{d}_{hq}x{D}_n{n}"] = res
    out["value"] = list(out["shapes"].values())[-1]["attention"]["roofline"]["achieved"]
    print(json.dumps(out), flush=True)


def dynamic_schedule_line(torch, np, ss, cfg, args):
    """The step with the dynamic schedule on the headline shape (32 Llama-3-8B
    shaped layers, 5120 tokens): first layer in full with the deviation against
    the matched reference rows, the average attention score per token -> AR at
    55% -> hot / cold recompute set (0.5 / 0.1), the retention ranking (window
    of the last 1 - AR/T rows, max(0.8, AR/T) kept on the first layer), then
    per layer a recompute set drawn from the previous one (ratio
    --alpha-recomp) and a kept set falling by --alpha-retain per layer,
    gathered into a compacted cache and attended over.  The ratios are this
    run's choice: the paper states only their trends over depth."""
    from paper_2509_24832_amd.schedule import DynamicSchedule
    path = Path(torch, ss, cfg)
    T, L = path.T, path.L
    ar = [1.0, 1.0] + [args.alpha_recomp] * (L - 2)
    at = [1.0] + [args.alpha_retain] * (L - 1)
    sched = DynamicSchedule(T, path.d, L, path.hq, path.hkv, path.D, path.codes_ref.shape[1], ar, at)
    run = lambda mark=None: sched.run(path.e_tgt, path.planes, path.codes_ref, path.ref_k, path.ref_v, path.w,
                                      mark=mark)
    for _ in range(args.warmup):
        run()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(args.steps):
        run()
    torch.cuda.synchronize()
    ms = (time.perf_counter() - t0) / args.steps * 1e3
    rec = sched.run(path.e_tgt, path.planes, path.codes_ref, path.ref_k, path.ref_v, path.w, record=True)
    kept = rec.kv_rows_kept(T, L)
    n_rec = [rec.counts[1]] + [int(lr.sel.numel()) for lr in rec.layers[1:]]
    out = {"metric": "dynamic_schedule_tokens_per_s", "value": T / (ms * 1e-3), "unit": "tokens/s", "n_gpus": 1,
           "steps": args.steps, "warmup": args.warmup, "ms_per_step": ms, "higher_is_better": True,
           "data": "synthetic", "dtype": "bf16",
           "config": {"workload": "5120-token target vs 5120-token cached reference, 32 Llama-3-8B-shaped "
                                  "attention layers, dynamic recompute set and per-layer retention",
                      "alpha_recomp_after_layer_1": args.alpha_recomp, "alpha_retain_after_layer_0": args.alpha_retain},
           "AR": rec.counts[0], "recomputed_first_to_last": [n_rec[0], n_rec[-1]],
           "recomputed_tokens_total": T + sum(n_rec), "kept_rows_first_layer": rec.n_kept0,
           "kept_rows_last_layer": rec.layers[-1].n_kept if rec.layers else rec.n_kept0,
           "kv_cache_rows_kept_frac": kept, "kv_cache_bytes_saved_frac": 1.0 - kept,
           "timing": "wall clock over the steps (the schedule reads two counts back after the first layer, so the "
                     "host waits for the device there once per step)"}
    print(json.dumps(out), flush=True)


def cfg_codes(np, cfg, n, w, tag):
    """Seeded synthetic code words (uniform bits), the generator of the configs."""
    import workloads
    return workloads.make_codes(cfg, n, w, tag=tag).view(np.int64)


def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py measures one GPU; --gpus {args.gpus} is not supported: every box here has one GPU and "
              "this build has no multi-GPU path (see the sharding notes in DESIGN.md).", file=sys.stderr)
        sys.exit(2)
    import numpy as np
    import torch

    import paper_2509_24832_amd as ss
    from workloads import CONFIGS

    torch.cuda.set_device(0)
    if args.bank_similarity:
        bank_similarity_line(torch, np, ss, CONFIGS[3], args)
        return
    if args.match_compare:
        match_compare_line(torch, np, ss, CONFIGS, args)
        return
    if args.dynamic_recompute:
        dynamic_recompute_line(torch, np, ss, CONFIGS[2], args)
        return
    if args.vendor_compare:
        vendor_compare_line(torch, np, ss, CONFIGS[2], args)
        return
    if args.fp32:
        fp32_line(torch, np, ss, CONFIGS[0], args)
        return
    if args.schedule == "dynamic":
        dynamic_schedule_line(torch, np, ss, CONFIGS[2], args)
        return
    cfg = CONFIGS[args.config]
    if args.frac is None:
        args.frac = 0.25 if cfg.cid == 2 else cfg.recompute_fracs[0]
    if args.sweep is None:
        args.sweep = "0.10,0.25,0.50,1.00" if cfg.cid == 2 else ""
    path = Path(torch, ss, cfg)
    path.matcher = ss.match_mfma if args.matcher == "mfma" else ss.match
    path.fused_encode = args.encode == "fused"
    path.gather_except = args.gather == "except"
    path.gather_overlap = args.gather_stream == "overlap"

    if args.copy_calibration_mib:
        # fill the source, then a 1 GiB buffer that pushes it out of L2 and the
        # 256 MB Infinity Cache, then the copy itself (reads and writes n bytes)
        n = args.copy_calibration_mib << 20
        src = torch.ones(n, dtype=torch.uint8, device="cuda")
        flush = torch.ones(1 << 30, dtype=torch.uint8, device="cuda")
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst, flush
    # headline: plain timed region
    path.set_frac(args.frac)
    ms, wall_ms = time_steps(torch, path, args.steps, args.warmup)
    # per-call durations: each stage timed as a run of its own calls after the timed region
    stages = stage_times(torch, path, max(2, args.steps // 4))
    # medians of single runs with the caches flushed before each (after the timed region, which warmed up)
    flushed = flushed_medians(torch, path, max(20, args.steps))
    sel_h = path.sel.cpu().numpy()
    T, L, hq, hkv, D, d = path.T, path.L, path.hq, path.hkv, path.D, path.d
    n_sel = path.n_sel

    def avg(name):
        return stages.get(name, float("nan"))

    attn_flops = attention_flops(sel_h, hq, D)
    attn0_flops = 4.0 * D * hq * T * (T + 1) / 2.0
    qkv_flops = 2.0 * n_sel * (hq + 2 * hkv) * D * d
    attn_ms, qkv_ms, attn0_ms = avg("attn"), avg("qkv"), avg("attn0")
    gather_rows = (L - 1) * (T - n_sel) if args.gather == "except" else L * T
    gather_bytes = 2.0 * 2 * gather_rows * hkv * D * 2  # read + write, K and V
    gather_ms = avg("gather_rest") if args.gather == "except" else avg("gather")
    match_ms = avg("match")
    pp_ms = (avg("qkv0") + attn0_ms + (L - 1) * (attn_ms + qkv_ms))
    # the dominant call: prefill_attention (attention kernel + combine of cut row tiles),
    # averaged over the 32 calls of a step (layer 0 over all 5120 rows, then
    # 31 partial layers); achieved = algorithmic flops per call / event-timed
    # duration per call
    attn_call_flops = (attn0_flops + (L - 1) * attn_flops) / L
    attn_call_ms = (attn0_ms + (L - 1) * attn_ms) / L
    traffic = None
    if ATTN_TRAFFIC["source_sha256"] and \
            source_sha256("paper_2509_24832_amd/csrc/attention.hip") == ATTN_TRAFFIC["source_sha256"] and \
            abs(args.frac - 0.25) < 1e-9 and cfg.cid == 2:
        traffic = ATTN_TRAFFIC["bytes_per_call"]
    achieved = attn_call_flops / (attn_call_ms * 1e-3) / 1e12
    res = {
        "metric": "partial-prefill tokens/s + LSH match token-pairs/s at "
                  f"{'5k' if cfg.cid == 2 else '32k'} tokens, Llama-3-8B shape",
        "value": T / (ms * 1e-3),
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": f"{T}-token target vs {T}-token cached reference, 32 Llama-3-8B-shaped attention "
                               f"layers (hidden 4096, 32q/8kv heads, head_dim 128), 128-bit LSH, recompute "
                               f"fraction {args.frac}", "n_tok": T, "layers": L, "recompute_frac": args.frac,
                   "n_recompute": n_sel, "matcher": args.matcher, "encode": args.encode, "gather": args.gather,
                   "gather_stream": args.gather_stream if args.gather == "except" else None},
        "partial_prefill_tokens_per_s": T / (pp_ms * 1e-3),
        "match_token_pairs_per_s": T * T / (match_ms * 1e-3),
        "stage_ms": {k: round(v, 4) for k, v in stages.items()},
        "stage_sum_ms_per_step": sum(v for k, v in stages.items() if k not in ("qkv", "attn")) +
                                 (L - 1) * (stages["qkv"] + stages["attn"]),
        "wall_ms_per_step": wall_ms,
        "flushed_median": flushed,
        "gather": {"GB/s": gather_bytes / (gather_ms * 1e-3) / 1e9, "frac_of_hbm": gather_bytes / (gather_ms * 1e-3) / 1e9 / HBM_PEAK_GBPS},
        "attention_TFLOPs": {"partial_layer": attn_flops / (attn_ms * 1e-3) / 1e12,
                             "layer0_full": attn0_flops / (attn0_ms * 1e-3) / 1e12},
        "qkv_gemm_TFLOPs": qkv_flops / (qkv_ms * 1e-3) / 1e12,
        "roofline": {"kernel": "prefill_attention (attention_kernel + combine_kernel; layer 0 also its plan_kernel, layers 1-31 share the plan made after selection)", "bound": "mfma",
                     "achieved": achieved, "peak": BF16_PEAK_TFLOPS, "unit": "TFLOP/s",
                     "frac": achieved / BF16_PEAK_TFLOPS, "traffic": traffic,
                     "flops_per_call": attn_call_flops, "us_per_call": attn_call_ms * 1e3, "calls_per_step": L},
    }
    if args.sweep:
        sweep = {}
        for f in [float(x) for x in args.sweep.split(",") if x]:
            path.set_frac(f)
            m_f, _ = time_steps(torch, path, max(3, args.steps // 2), 2)
            sweep[f"{f:.2f}"] = {"ms_per_step": m_f, "tokens_per_s": T / (m_f * 1e-3), "n_recompute": path.n_sel,
                                 "recomputed_tokens_per_s": (T + (L - 1) * path.n_sel) / (m_f * 1e-3)}
        res["recompute_sweep"] = sweep
    if not args.no_cpu_baseline:
        res["cpu_baseline"] = cpu_baseline(cfg, args.frac, args.cpu_budget_s)
    print(json.dumps(res), flush=True)


if __name__ == "__main__":
    main()
