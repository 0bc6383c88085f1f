"""The layer schedule of one target prompt with the dynamic recompute set and
retention (Sections 4.2, 4.3.3 and 4.3.4; Appendix A.5 and A.6), as a
sequence of libsemshare calls.  Host-side sequencing only: every step runs in
the library's kernels.  The host reads back two counts once per prompt, after
the first layer (AR with the number recomputed, and the number kept on
layer 0); later layers' sizes follow from them on the host (the recompute
counts exactly, the kept counts as a bound, see below), so the layers are
launched without waiting for the device.

Layer indices here start at 0 (the paper's first layer is layer 0):

* layer 0 is recomputed in full; its KV deviation compares every row with the
  matched reference row; its attention covers every row;
* the average attention score per token of layer 0 gives Attention Recovery
  (AR at `thres`), the hot / cold split and the recompute set S_1 of the next
  layer (`w_hot` of the hot tokens and `w_cold` of the cold ones, by
  deviation);
* the window score (the attention of the last 1 - AR/T of the rows) ranks the
  tokens for retention: hot and recomputed tokens first, R_0 =
  max(min_keep, AR/T) T kept on layer 0 (its cache is compacted);
* layer l >= 1 recomputes n_l tokens drawn from layer l-1's by their deviation
  there (n_1 = |S_1|, n_l = round(n_(l-1) alpha_recomp[l]) for l >= 2), keeps
  Retain_l = round(R_0 prod_(j=1..l) alpha_retain[j]) tokens of the ranking
  plus its recomputed ones, gathers only those rows of its reference cache,
  and attends over that compacted cache.

The paper gives the two alpha schedules only qualitatively (recompute ratios
growing with depth, retention ratios falling); they are the caller's input.
"""
from __future__ import annotations

import math
from dataclasses import dataclass, field
from typing import Callable, List, Optional, Sequence

import torch

from . import semshare as ss


@dataclass
class LayerRecord:
    sel: torch.Tensor          # recomputed positions (ascending)
    kept: torch.Tensor         # kept positions (ascending)
    rows: torch.Tensor         # rows of `sel` in the compacted cache
    n_kept: int
    sigma: torch.Tensor        # deviation of the recomputed rows (against the matched reference rows)
    out: torch.Tensor          # attention output of the recomputed rows [n, Hq, D]


@dataclass
class ScheduleRecord:
    idx: torch.Tensor
    sigma0: torch.Tensor
    q0: torch.Tensor
    out0: torch.Tensor
    mass: torch.Tensor
    score: torch.Tensor
    counts: List[int]
    row_begin: int
    rank: torch.Tensor
    kept0: torch.Tensor
    n_kept0: int
    layers: List[LayerRecord] = field(default_factory=list)

    def kv_rows_kept(self, n_tok: int, n_layers: int) -> float:
        """Fraction of the L x T cache rows that stay resident."""
        return (self.n_kept0 + sum(l.n_kept for l in self.layers)) / float(n_tok * n_layers)


class DynamicSchedule:
    """Buffers and calls of the dynamic schedule for prompts of n_tok tokens."""

    def __init__(self, n_tok: int, dim: int, n_layers: int, n_q_heads: int, n_kv_heads: int, head_dim: int,
                 n_words: int, alpha_recomp: Sequence[float], alpha_retain: Sequence[float], thres: float = 0.55,
                 w_hot: float = 0.5, w_cold: float = 0.1, min_keep: float = 0.8, device: str = "cuda"):
        if len(alpha_recomp) < n_layers or len(alpha_retain) < n_layers:
            raise ValueError("one alpha per layer (entries 0 and 1 of alpha_recomp are not used)")
        self.T, self.d, self.L = n_tok, dim, n_layers
        self.hq, self.hkv, self.D = n_q_heads, n_kv_heads, head_dim
        self.alpha_recomp, self.alpha_retain = list(alpha_recomp), list(alpha_retain)
        self.thres, self.w_hot, self.w_cold, self.min_keep = thres, w_hot, w_cold, min_keep
        T, bf, dev = n_tok, torch.bfloat16, device
        i32 = dict(dtype=torch.int32, device=dev)
        f32 = dict(dtype=torch.float32, device=dev)
        self.allpos = torch.arange(T, **i32)
        self.codes = torch.empty((T, n_words), dtype=torch.int64, device=dev)
        self.idx = torch.empty(T, **i32)
        self.dist = torch.empty(T, **i32)
        self.asm_k = torch.empty((n_layers, T, n_kv_heads, head_dim), dtype=bf, device=dev)
        self.asm_v = torch.empty_like(self.asm_k)
        self.kc0 = torch.empty((T, n_kv_heads, head_dim), dtype=bf, device=dev)  # layer 0 after retention
        self.vc0 = torch.empty_like(self.kc0)
        self.q0 = torch.empty((T, n_q_heads, head_dim), dtype=bf, device=dev)
        self.out0 = torch.empty_like(self.q0)
        self.sigma0 = torch.empty(T, **f32)
        self.mass = torch.empty(T, **f32)
        self.score = torch.empty(T, **f32)
        self.mass_ws = torch.empty(max(1, int(ss.load().semshare_attention_mass_workspace(T, n_q_heads))),
                                   dtype=torch.uint8, device=dev)
        self.sel1 = torch.empty(T, **i32)
        self.counts = torch.empty(3, **i32)
        self.sel = [torch.empty(T, **i32) for _ in range(2)]     # S_l, alternating
        self.sig = [torch.empty(T, **f32) for _ in range(2)]     # sigma_l, alternating
        self.q_sel = torch.empty((T, n_q_heads, head_dim), dtype=bf, device=dev)
        ws = max(ss.qkv_rope_workspace_bytes(T, n_q_heads, n_kv_heads, head_dim, bf),
                 ss.prefill_attention_workspace_bytes(T, T, n_q_heads, n_kv_heads, head_dim, bf))
        self.ws = torch.empty(ws, dtype=torch.uint8, device=dev)
        self.plan_buf = torch.empty(max(1, ss.attention_plan_bytes(T, T, n_q_heads, n_kv_heads, head_dim, bf)),
                                    dtype=torch.uint8, device=dev)
        self.table_buf = torch.empty(max(16, ss.rope_table_bytes(T, head_dim)), dtype=torch.uint8, device=dev)

    def _n(self, t: torch.Tensor) -> int:
        return int(t.cpu().numpy()[0])

    def run(self, e_tgt: torch.Tensor, planes: torch.Tensor, codes_ref: torch.Tensor, ref_k: torch.Tensor,
            ref_v: torch.Tensor, weights, record: bool = False,
            mark: Optional[Callable[[str], None]] = None) -> Optional[ScheduleRecord]:
        """One prompt: e_tgt [T, d] raw target embeddings, the reference's codes and per-layer caches
        [L, T_ref, Hkv, D], weights[l] = (wq, wk, wv).  With record, the intermediate results are kept."""
        m = mark or (lambda name: None)
        T, hq, hkv, D = self.T, self.hq, self.hkv, self.D
        clone = (lambda t: t.clone()) if record else (lambda t: t)
        m("start")
        ss.rope_lsh_encode(e_tgt, planes, out=self.codes)
        ss.match_mfma(self.codes, codes_ref, idx=self.idx, dist=self.dist)
        m("match")
        wq, wk, wv = weights[0]
        ss.qkv_rope_dev_ref(e_tgt, self.allpos, wq, wk, wv, self.asm_k[0], self.asm_v[0], hq, hkv, ref_k[0],
                            ref_v[0], self.idx, q_out=self.q0, deviation=self.sigma0, workspace=self.ws)
        ss.prefill_attention(self.q0, self.allpos, self.asm_k[0], self.asm_v[0], hkv, out=self.out0,
                             workspace=self.ws)
        m("layer0")
        ss.attention_mass(self.q0, self.asm_k[0], hq, hkv, mass=self.mass, workspace=self.mass_ws)
        ss.dynamic_recompute(self.mass, self.sigma0, self.thres, self.w_hot, self.w_cold, sel_pos=self.sel1,
                             counts=self.counts)
        counts = [int(c) for c in self.counts.cpu().numpy()]
        ar, n1 = counts[0], counts[1]
        row_begin = min(T - 1, T - int(math.floor((1.0 - ar / T) * T + 0.5)))
        ss.attention_mass(self.q0, self.asm_k[0], hq, hkv, mass=self.score, workspace=self.mass_ws,
                          row_begin=row_begin, reuse_normalisers=True)
        rank, kept0, n_kept0_t = ss.retention(self.mass, self.score, self.sel1, self.counts, self.min_keep)
        n_kept0 = self._n(n_kept0_t)
        ss.gather_kv(self.asm_k[0][None], self.asm_v[0][None], kept0[:n_kept0], out_k=self.kc0[None, :n_kept0],
                     out_v=self.vc0[None, :n_kept0])
        m("select")
        rec = None
        if record:
            rec = ScheduleRecord(clone(self.idx), clone(self.sigma0), clone(self.q0), clone(self.out0),
                                 clone(self.mass), clone(self.score), counts, row_begin, clone(rank), clone(kept0),
                                 n_kept0)
        n_prev, retain = n1, float(n_kept0)
        for l in range(1, self.L):
            cur, prev = self.sel[l % 2], self.sel[(l - 1) % 2]
            if l == 1:
                n_l = n1
                cur[:n_l].copy_(self.sel1[:n_l])
            else:
                n_l = max(1, min(n_prev, int(math.floor(n_prev * self.alpha_recomp[l] + 0.5))))
                ss.select_recompute_nested(self.sig[(l - 1) % 2][:n_prev], prev[:n_prev], n_l, out=cur[:n_l])
            retain *= self.alpha_retain[l]
            n_ret = int(math.floor(retain + 0.5))
            s_l = cur[:n_l]
            kept, src, rows, nk_t = ss.retention_layer(rank, n_ret, s_l, self.idx)
            # The layer keeps at most n_ret + n_l rows (the retained ones and its
            # recomputed ones): its cache, gather, projection and attention are
            # sized by that bound instead of the count on the device.  Rows past
            # the kept ones are gathered too (copies of reference rows, or zeros
            # for indices out of range: finite either way) and never attended,
            # since every recomputed row's causal range ends at its own row,
            # which is a kept one.
            nk = min(T, n_ret + n_l)
            kc, vc = self.asm_k[l][:nk], self.asm_v[l][:nk]
            ss.gather_kv(ref_k[l][None], ref_v[l][None], src[:nk], out_k=kc[None], out_v=vc[None])
            table = ss.rope_table(s_l, T, D, out=self.table_buf)
            wq, wk, wv = weights[l]
            # the recomputed tokens' embeddings are read in place (rows s_l of e_tgt)
            q, sig = ss.qkv_rope(e_tgt, rows, wq, wk, wv, kc, vc, hq, hkv, q_out=self.q_sel[:n_l],
                                 deviation=self.sig[l % 2][:n_l], want_deviation=True, workspace=self.ws,
                                 rope_table=table, x_rows=s_l)
            plan = ss.attention_plan(rows, nk, hq, hkv, D, out=self.plan_buf)
            out = ss.prefill_attention(q, rows, kc, vc, hkv, workspace=self.ws, plan=plan)
            m("layer")
            if record:
                n_kept = self._n(nk_t)
                assert n_kept <= nk, "kept rows beyond their bound"
                rec.layers.append(LayerRecord(clone(s_l), clone(kept[:n_kept]), clone(rows), n_kept, clone(sig), out))
            n_prev = n_l
        return rec
