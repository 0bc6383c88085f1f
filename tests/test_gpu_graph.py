"""The hot path's sequence of calls captured in one HIP graph
(torch.cuda.CUDAGraph) and replayed: every call of the path only launches
kernels on the caller's stream (no allocation, memset or synchronisation
inside the library), so a serving loop can capture it.  Each replay must equal
the eager run of the same calls bit for bit; the eager chain itself is checked
against the oracle in test_gpu_chain.py.  Between replays every output buffer
is cleared and other eager work runs on the same buffers, so a replay that
skipped a call would be caught."""
import pytest
import torch

import paper_2509_24832_amd as ss
import workloads
from workloads import CONFIGS

from helpers import announce, dev, dev_i32

pytestmark = pytest.mark.gpu


def test_chain_graph_replays_equal_eager():
    """Config 1's shape (1024 tokens, hidden 4096, 32 q / 8 kv heads, 128-bit
    LSH, f = 0.25) over two layers: fused RoPE + LSH, MFMA match, first layer
    with the deviation against the matched reference rows and its attention,
    selection with the shared attention plan and RoPE table, gather of the
    second layer without the recomputed rows, partial prefill of the second
    layer."""
    cfg = CONFIGS[1]
    T, hq, hkv, D, L = cfg.n_tok, cfg.n_q_heads, cfg.n_kv_heads, cfg.head_dim, 2
    n_sel = cfg.n_sel(cfg.recompute_fracs[0])
    bf = torch.bfloat16
    announce("graph capture of the config 1 chain, 2 layers")
    pair = workloads.make_prompt_pair(cfg)
    er, et, pl = dev(pair.e_ref, "bf16"), dev(pair.e_tgt, "bf16"), dev(workloads.make_planes(cfg), "bf16")
    W = []
    for l in range(L):
        w = workloads.make_weights(cfg, l)
        W.append(tuple(dev(a, "bf16") for a in (w.wq, w.wk, w.wv)))
    ap = dev_i32(list(range(T)))
    # reference side, prepared before (insert time)
    codes_ref = ss.lsh_encode(ss.rope_embed(er), pl)
    ref_k = torch.empty((L, T, hkv, D), dtype=bf, device="cuda")
    ref_v = torch.empty_like(ref_k)
    for l in range(L):
        ss.qkv_rope(er, ap, None, W[l][1], W[l][2], ref_k[l], ref_v[l], hq, hkv, want_q=False)
    # every buffer the path writes
    out = {
        "codes": torch.empty_like(codes_ref), "idx": torch.empty(T, dtype=torch.int32, device="cuda"),
        "dist": torch.empty(T, dtype=torch.int32, device="cuda"),
        "asm_k": torch.empty_like(ref_k), "asm_v": torch.empty_like(ref_v),
        "q0": torch.empty((T, hq, D), dtype=bf, device="cuda"), "out0": torch.empty((T, hq, D), dtype=bf, device="cuda"),
        "sigma": torch.empty(T, dtype=torch.float32, device="cuda"),
        "sel": torch.empty(n_sel, dtype=torch.int32, device="cuda"),
        "plan": torch.empty(ss.attention_plan_bytes(n_sel, T, hq, hkv, D, bf), dtype=torch.uint8, device="cuda"),
        "rope": torch.empty(ss.rope_table_bytes(n_sel, D), dtype=torch.uint8, device="cuda"),
        "x_sel": torch.empty((n_sel, et.shape[1]), dtype=bf, device="cuda"),
        "q1": torch.empty((n_sel, hq, D), dtype=bf, device="cuda"),
        "out1": torch.empty((n_sel, hq, D), dtype=bf, device="cuda"),
    }
    ws = torch.empty(max(ss.qkv_rope_workspace_bytes(T, hq, hkv, D, bf),
                         ss.prefill_attention_workspace_bytes(T, T, hq, hkv, D, bf),
                         ss.prefill_attention_workspace_bytes(n_sel, T, hq, hkv, D, bf)),
                     dtype=torch.uint8, device="cuda")
    o = out

    def step():
        ss.rope_lsh_encode(et, pl, out=o["codes"])
        ss.match_mfma(o["codes"], codes_ref, idx=o["idx"], dist=o["dist"])
        ss.qkv_rope_dev_ref(et, ap, *W[0], o["asm_k"][0], o["asm_v"][0], hq, hkv, ref_k[0], ref_v[0], o["idx"],
                            q_out=o["q0"], deviation=o["sigma"], workspace=ws)
        ss.prefill_attention(o["q0"], ap, o["asm_k"][0], o["asm_v"][0], hkv, out=o["out0"], workspace=ws)
        ss.select_recompute(o["sigma"], n_sel, out=o["sel"])
        ss.attention_plan(o["sel"], T, hq, hkv, D, out=o["plan"])
        ss.rope_table(o["sel"], T, D, out=o["rope"])
        ss.gather_kv(ref_k[1:], ref_v[1:], o["idx"], out_k=o["asm_k"][1:], out_v=o["asm_v"][1:], except_pos=o["sel"])
        ss.gather_rows(et, o["sel"], out=o["x_sel"])
        ss.qkv_rope(o["x_sel"], o["sel"], *W[1], o["asm_k"][1], o["asm_v"][1], hq, hkv, q_out=o["q1"], workspace=ws,
                    rope_table=o["rope"])
        ss.prefill_attention(o["q1"], o["sel"], o["asm_k"][1], o["asm_v"][1], hkv, out=o["out1"], workspace=ws,
                             plan=o["plan"])

    def snapshot():
        torch.cuda.synchronize()
        return {k: v.clone() for k, v in out.items()}

    def clear():
        for v in out.values():
            v.zero_()

    clear()  # the plan's unused entries (it is sized for the worst case) stay as they were: zero on both sides
    step()
    eager = snapshot()
    assert int((eager["out1"] != 0).sum()) > 0 and int((eager["sel"] != 0).sum()) > 0
    # capture, after a warm run on the capture stream
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        step()
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        step()
    torch.cuda.synchronize()
    for rep in range(3):
        clear()
        ss.rope_lsh_encode(er, pl, out=out["codes"])  # other eager work on the same buffers
        torch.cuda.synchronize()
        graph.replay()
        got = snapshot()
        for k in eager:
            a, b = eager[k], got[k]
            same = torch.equal(a.view(torch.int16), b.view(torch.int16)) if a.dtype == bf else torch.equal(a, b)
            assert same, (rep, k)
    # and an eager run after the replays still gives the same results
    clear()
    step()
    again = snapshot()
    for k in eager:
        a, b = eager[k], again[k]
        assert (torch.equal(a.view(torch.int16), b.view(torch.int16)) if a.dtype == bf else torch.equal(a, b)), k
