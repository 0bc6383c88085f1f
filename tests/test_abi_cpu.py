"""The C-ABI library loads on a GPU-less host, exports every symbol the header
declares, and rejects bad arguments on the host before enqueuing anything
(no call here reaches a kernel launch).  CPU only."""
import ctypes
import os
import subprocess

import pytest

import paper_2509_24832_amd as ss
from paper_2509_24832_amd import semshare as b

FAKE = 0x1000  # never dereferenced: every call below fails validation first
FAKE_ODD = 0x1008  # 8-byte but not 16-byte aligned


@pytest.fixture(scope="module")
def lib():
    return ss.load()


def test_header_declares_the_five_calls():
    syms = ss.declared_symbols()
    for name in ("semshare_rope_embed", "semshare_lsh_encode", "semshare_match", "semshare_gather_kv",
                 "semshare_partial_prefill"):
        assert name in syms


def test_library_exports_every_declared_symbol(lib):
    out = subprocess.run(["nm", "-D", "--defined-only", b.LIB_PATH], capture_output=True, text=True, check=True).stdout
    exported = {line.split()[-1] for line in out.splitlines() if line.strip()}
    for name in ss.declared_symbols():
        assert name in exported, name
        assert getattr(lib, name) is not None


def test_library_targets_gfx950_only(tmp_path):
    fb = tmp_path / "fatbin.bin"
    # an explicit output file keeps objcopy from rewriting the library in place
    subprocess.run(["objcopy", "--dump-section", f".hip_fatbin={fb}", b.LIB_PATH, str(tmp_path / "copy.so")],
                   check=True)
    out = subprocess.run(["/opt/rocm/llvm/bin/clang-offload-bundler", "--list", "--type=o", f"--input={fb}"],
                         capture_output=True, text=True, check=True)
    targets = [t for t in out.stdout.split() if "amdgcn" in t]
    assert targets and all(t.endswith("gfx950") for t in targets)


def test_version(lib):
    assert ss.version() == 10000


def _st(fn, *args):
    return getattr(ss.load(), fn)(*args)


def test_rope_validation(lib):
    assert _st("semshare_rope_embed", FAKE, FAKE, 4, 7, 0, 1e4, 1, None) == b.E_INVAL  # odd dim
    assert "even" in ss.last_error()
    assert _st("semshare_rope_embed", FAKE, FAKE, 4, 8, 0, -1.0, 1, None) == b.E_INVAL  # base
    assert _st("semshare_rope_embed", FAKE, FAKE, 4, 8, -1, 1e4, 1, None) == b.E_INVAL  # pos0
    assert _st("semshare_rope_embed", FAKE, FAKE, 4, 8, 0, 1e4, 7, None) == b.E_INVAL  # dtype
    assert _st("semshare_rope_embed", None, None, 4, 8, 0, 1e4, 1, None) == b.E_INVAL  # null
    assert _st("semshare_rope_embed", None, None, 0, 8, 0, 1e4, 1, None) == b.OK  # empty
    assert ss.last_error() == ""


def test_lsh_validation(lib):
    assert _st("semshare_lsh_encode", FAKE, FAKE, FAKE, 10, 64, 96, 1, None) == b.E_INVAL  # n_bits
    assert _st("semshare_lsh_encode", FAKE, FAKE, FAKE, 10, 100, 64, 1, None) == b.E_UNSUPPORTED  # bf16 dim
    assert _st("semshare_lsh_encode", FAKE, FAKE, FAKE, 10, 6, 64, 0, None) == b.E_UNSUPPORTED  # fp32 dim
    assert _st("semshare_lsh_encode", FAKE_ODD, FAKE, FAKE, 10, 64, 64, 1, None) == b.E_INVAL  # alignment
    assert _st("semshare_lsh_encode", None, FAKE, FAKE, 10, 64, 64, 1, None) == b.E_INVAL
    assert _st("semshare_lsh_encode", None, None, None, 0, 64, 64, 1, None) == b.OK


def test_rope_lsh_encode_validation(lib):
    e = "semshare_rope_lsh_encode"
    assert _st(e, FAKE, FAKE, FAKE, 4, 4096, 128, 0, 10000.0, 0, None) == b.E_UNSUPPORTED  # fp32
    assert _st(e, FAKE, FAKE, FAKE, 4, 4096, 256, 0, 10000.0, 1, None) == b.E_UNSUPPORTED  # 256 bits
    assert _st(e, FAKE, FAKE, FAKE, 4, 4096, 96, 0, 10000.0, 1, None) == b.E_INVAL  # n_bits
    assert _st(e, FAKE, FAKE, FAKE, 4, 4095, 128, 0, 10000.0, 1, None) == b.E_INVAL  # odd dim
    assert _st(e, FAKE, FAKE, FAKE, 4, 4032 + 32, 128, 0, 10000.0, 1, None) == b.E_UNSUPPORTED  # dim % 64
    assert _st(e, FAKE, FAKE, FAKE, 4, 4096, 128, -1, 10000.0, 1, None) == b.E_INVAL  # pos0
    assert _st(e, FAKE, FAKE, FAKE, 4, 4096, 128, 0, float("nan"), 1, None) == b.E_INVAL  # base
    assert _st(e, FAKE, FAKE, None, 4, 4096, 128, 0, 10000.0, 1, None) == b.E_INVAL  # null codes
    assert _st(e, FAKE_ODD, FAKE, FAKE, 4, 4096, 128, 0, 10000.0, 1, None) == b.E_INVAL  # alignment
    assert _st(e, None, None, None, 0, 4096, 128, 0, 10000.0, 1, None) == b.OK


def test_attention_mass_and_dynamic_validation(lib):
    e = "semshare_attention_mass"
    ws = int(lib.semshare_attention_mass_workspace(100, 32))
    assert ws == 2 * 32 * 100 * 4
    assert _st(e, FAKE, FAKE, 100, 0, 32, 8, 128, 0.0, FAKE, FAKE, ws, 0, None) == b.E_UNSUPPORTED  # fp32
    assert _st(e, FAKE, FAKE, 100, 0, 32, 8, 64, 0.0, FAKE, FAKE, ws, 1, None) == b.E_UNSUPPORTED  # head_dim
    assert _st(e, FAKE, FAKE, 100, 0, 32, 6, 128, 0.0, FAKE, FAKE, ws, 1, None) == b.E_INVAL  # GQA
    assert _st(e, FAKE, FAKE, 100, 0, 32, 8, 128, -1.0, FAKE, FAKE, ws, 1, None) == b.E_INVAL  # scale
    assert _st(e, FAKE, FAKE, 100, 0, 32, 8, 128, 0.0, FAKE, FAKE, ws - 4, 1, None) == b.E_INVAL  # workspace
    assert _st(e, FAKE_ODD, FAKE, 100, 0, 32, 8, 128, 0.0, FAKE, FAKE, ws, 1, None) == b.E_INVAL  # alignment
    assert _st(e, FAKE, FAKE, 100, 0, 32, 8, 128, 0.0, None, FAKE, ws, 1, None) == b.E_INVAL  # null mass
    assert _st(e, None, None, 0, 0, 32, 8, 128, 0.0, None, None, 0, 1, None) == b.OK
    w = "semshare_attention_mass_window"  # same checks
    assert _st(w, FAKE, FAKE, 100, 100, 32, 8, 128, 0.0, FAKE, FAKE, ws, 1, None) == b.E_INVAL  # row_begin
    assert _st(w, FAKE, FAKE, 100, 0, 32, 8, 128, 0.0, FAKE, None, ws, 1, None) == b.E_INVAL  # null workspace
    assert _st(w, FAKE, FAKE, 100, 0, 32, 8, 128, 0.0, FAKE, FAKE, ws - 4, 1, None) == b.E_INVAL  # workspace
    assert _st(w, FAKE, FAKE, 100, 0, 32, 8, 64, 0.0, FAKE, FAKE, ws, 1, None) == b.E_UNSUPPORTED  # head_dim
    assert _st(w, None, None, 0, 0, 32, 8, 128, 0.0, None, None, 0, 1, None) == b.OK
    d = "semshare_dynamic_recompute"
    assert _st(d, FAKE, FAKE, 65537, 0.55, 0.5, 0.1, FAKE, FAKE, None) == b.E_UNSUPPORTED
    assert _st("semshare_retention", FAKE, FAKE, 65537, FAKE, FAKE, 0.8, FAKE, FAKE, FAKE, None) == b.E_UNSUPPORTED
    assert _st(d, FAKE, FAKE, -1, 0.55, 0.5, 0.1, FAKE, FAKE, None) == b.E_INVAL
    assert _st(d, FAKE, FAKE, 10, 1.5, 0.5, 0.1, FAKE, FAKE, None) == b.E_INVAL
    assert _st(d, FAKE, FAKE, 10, 0.55, float("nan"), 0.1, FAKE, FAKE, None) == b.E_INVAL
    assert _st(d, FAKE, FAKE, 10, 0.55, 0.5, 0.1, FAKE, None, None) == b.E_INVAL  # null counts
    assert _st(d, None, FAKE, 10, 0.55, 0.5, 0.1, FAKE, FAKE, None) == b.E_INVAL  # null mass


@pytest.mark.parametrize("entry", ["semshare_match", "semshare_match_mfma"])
def test_match_validation(lib, entry):
    assert _st(entry, FAKE, 4, FAKE, 4, 0, FAKE, None, None) == b.E_INVAL  # n_words
    assert _st(entry, FAKE, 4, FAKE, 4, 5, FAKE, None, None) == b.E_INVAL
    assert _st(entry, FAKE, 4, FAKE, 0, 2, FAKE, None, None) == b.E_INVAL  # empty reference
    assert _st(entry, FAKE, 4, FAKE, 1 << 23, 2, FAKE, None, None) == b.E_UNSUPPORTED
    assert _st(entry, FAKE, 4, FAKE, 4, 2, None, None, None) == b.E_INVAL  # null idx
    assert _st(entry, None, 0, None, 4, 2, None, None, None) == b.OK


def test_gather_except_validation(lib):
    e = "semshare_gather_kv_except"
    assert _st(e, FAKE, None, FAKE, 4, 4, FAKE, None, 2, 8, 128, 1, None, 1, None) == b.E_INVAL  # list missing
    assert _st(e, FAKE, None, FAKE, 4, 4, FAKE, None, 2, 8, 128, 1, FAKE, 5, None) == b.E_INVAL  # n_except > n_tgt
    assert _st(e, FAKE, None, FAKE, 4, 4, FAKE, None, 2, 8, 128, 1, FAKE, -1, None) == b.E_INVAL
    assert _st(e, FAKE, None, FAKE, 0, 4, FAKE, None, 2, 8, 128, 1, None, 0, None) == b.OK


def test_gather_validation(lib):
    args = dict(n_tgt=4, n_ref=4, L=2, h=8, d=128, dt=1)
    assert _st("semshare_gather_kv", FAKE, FAKE, FAKE, 4, 4, FAKE, None, 2, 8, 128, 1, None) == b.E_INVAL  # v pair
    assert _st("semshare_gather_kv", FAKE, None, FAKE, 4, 4, FAKE, None, 2, 1, 3, 1, None) == b.E_UNSUPPORTED  # 6 B rows
    assert _st("semshare_gather_kv", FAKE_ODD, None, FAKE, 4, 4, FAKE, None, 2, 8, 128, 1, None) == b.E_INVAL
    assert _st("semshare_gather_kv", FAKE, None, None, 4, 4, FAKE, None, 2, 8, 128, 1, None) == b.E_INVAL
    assert _st("semshare_gather_kv", FAKE, None, FAKE, 0, 4, FAKE, None, 2, 8, 128, 1, None) == b.OK
    assert _st("semshare_gather_kv", FAKE, None, FAKE, 4, 4, FAKE, None, 0, 8, 128, 1, None) == b.OK
    del args


def _pp(n_sel=8, n_tok=16, hidden=256, hq=8, hkv=2, d=128, base=1e4, scale=0.0, out=FAKE, dev=None,
        ws=FAKE, ws_bytes=1 << 30, dt=1, xsel=FAKE, pos=FAKE, wq=FAKE):
    return _st("semshare_partial_prefill", xsel, pos, n_sel, wq, FAKE, FAKE, FAKE, FAKE, n_tok, hidden, hq, hkv, d,
               base, scale, out, dev, ws, ws_bytes, dt, None)


def test_partial_prefill_validation(lib):
    assert _pp(n_sel=17, n_tok=16) == b.E_INVAL  # n_sel > n_tok
    assert _pp(hq=6, hkv=4) == b.E_INVAL  # heads not divisible
    assert _pp(d=96) == b.E_UNSUPPORTED  # bf16 head_dim
    assert _pp(d=7) == b.E_INVAL  # odd head_dim
    assert _pp(hidden=100) == b.E_UNSUPPORTED
    assert _pp(hq=3 * 2, hkv=2) == b.E_UNSUPPORTED  # G = 3 does not divide 128
    assert _pp(hkv=1, hq=1, d=64) == b.E_UNSUPPORTED  # kv row of 64 is not a 128-column tile
    assert _pp(d=256, dt=0) == b.E_UNSUPPORTED  # fp32 head_dim limit
    assert _pp(n_tok=9000, n_sel=8, dt=0) == b.E_UNSUPPORTED
    assert _pp(base=0.0) == b.E_INVAL
    assert _pp(scale=-1.0) == b.E_INVAL
    assert _pp(ws_bytes=16) == b.E_INVAL and "workspace" in ss.last_error()
    assert _pp(ws=FAKE + 16) == b.E_INVAL  # workspace alignment
    assert _pp(wq=None) == b.E_INVAL  # out requested without wq
    assert _pp(xsel=FAKE_ODD) == b.E_INVAL
    assert _pp(pos=None) == b.E_INVAL
    assert _pp(n_sel=0, xsel=None, pos=None) == b.OK


def test_partial_prefill_workspace_sizes(lib):
    W = ss.load().semshare_partial_prefill_workspace
    assert W(8, 16, 256, 8, 2, 128, 7) == 0 and W(8, 16, 256, 6, 4, 128, 1) == 0
    small = W(256, 1024, 4096, 32, 8, 128, 1)
    # q (256*32*128*2) + rope table + deviation + split-KV partials
    assert small >= 256 * 4096 * 2 + 256 * 64 * 8
    full = W(5120, 5120, 4096, 32, 8, 128, 1)
    assert full >= 5120 * 4096 * 2
    assert W(1280, 5120, 4096, 32, 8, 128, 1) > W(1280, 5120, 4096, 32, 8, 128, 1) - 1


def test_workspaces_grow_with_the_row_count(lib):
    """A workspace sized for n selected rows serves every call with fewer: the
    projection's deviation parts follow its tile width, which narrows when few
    rows are selected (here across 640 / 641 rows at 32 q / 8 kv heads), so its
    workspace reserves the narrow tiles' count; the attention mass workspace
    grows with the token count."""
    L = lib
    for heads in ((32, 8), (64, 8), (8, 8), (32, 4)):
        prev = 0
        for n in list(range(0, 2200, 1)) + [5120, 32768]:
            w = L.semshare_qkv_rope_workspace(n, heads[0], heads[1], 128, 1)
            assert w >= prev, (heads, n)
            prev = w
            wp = L.semshare_partial_prefill_workspace(n, 5120, 4096, heads[0], heads[1], 128, 1)
            assert wp >= w, (heads, n)
    prev = 0
    for t in (1, 33, 1000, 5120, 8192):
        w = L.semshare_attention_mass_workspace(t, 32)
        assert w >= prev and w >= 2 * 32 * t * 4
        prev = w


def test_select_validation(lib):
    assert _st("semshare_select_recompute", FAKE, 10, 11, FAKE, None) == b.E_INVAL
    assert _st("semshare_select_recompute", FAKE, (1 << 20) + 1, 5, FAKE, None) == b.E_UNSUPPORTED
    assert _st("semshare_select_recompute", FAKE, 10, 0, None, None) == b.OK


def test_binding_requires_device_tensors():
    import torch
    x = torch.zeros(4, 8)
    with pytest.raises(ValueError):
        ss.rope_embed(x)


def test_binding_fails_loudly_without_library(monkeypatch, tmp_path):
    monkeypatch.setattr(b, "_lib", None)
    monkeypatch.setattr(b, "LIB_PATH", str(tmp_path / "missing.so"))
    with pytest.raises(RuntimeError, match="not built"):
        b.load()


def test_product_package_never_imports_the_oracle():
    pkg = os.path.dirname(b.__file__)
    for root, _, files in os.walk(pkg):
        for f in files:
            if f.endswith((".py", ".hip", ".cpp", ".h")):
                text = open(os.path.join(root, f)).read()
                assert "import oracle" not in text and "from oracle" not in text and "orc_" not in text, f


def test_split_call_validation(lib):
    L = ss.load()
    assert L.semshare_qkv_rope(FAKE, FAKE, 8, FAKE, FAKE, FAKE, FAKE, FAKE, 4, 256, 8, 2, 128, 1e4, FAKE, None, FAKE,
                               1 << 30, 1, None) == b.E_INVAL  # n_sel > n_tok
    assert L.semshare_qkv_rope(FAKE, FAKE, 8, None, FAKE, FAKE, FAKE, FAKE, 16, 256, 8, 2, 128, 1e4, FAKE, None, FAKE,
                               1 << 30, 1, None) == b.E_INVAL  # q requested without wq
    assert L.semshare_qkv_rope(FAKE, FAKE, 8, FAKE, FAKE, FAKE, FAKE, FAKE, 16, 256, 8, 2, 128, 1e4, FAKE, None, FAKE,
                               0, 1, None) == b.E_INVAL  # workspace too small
    assert L.semshare_prefill_attention(FAKE, FAKE, 8, FAKE, FAKE, 16, 8, 2, 96, 0.0, FAKE, FAKE, 1 << 30, 1,
                                        None) == b.E_UNSUPPORTED
    assert L.semshare_prefill_attention(FAKE, FAKE, 8, FAKE, FAKE, 16, 8, 2, 128, -2.0, FAKE, FAKE, 1 << 30, 1,
                                        None) == b.E_INVAL
    assert L.semshare_prefill_attention(FAKE, FAKE, 8, FAKE, FAKE, 16, 8, 2, 128, 0.0, None, FAKE, 1 << 30, 1,
                                        None) == b.E_INVAL
    assert L.semshare_prefill_attention(None, None, 0, None, None, 16, 8, 2, 128, 0.0, None, None, 0, 1, None) == b.OK
    # composition: the partial-prefill workspace covers q plus both steps
    W = L.semshare_partial_prefill_workspace(1280, 5120, 4096, 32, 8, 128, 1)
    assert W >= 1280 * 32 * 128 * 2 + L.semshare_qkv_rope_workspace(1280, 32, 8, 128, 1) + \
        L.semshare_prefill_attention_workspace(1280, 5120, 32, 8, 128, 1)
    # bf16: the work plan plus partial-result slots for the cut row tiles, at
    # most 2 per workgroup (256 CUs / 8 kv heads = 32 per head) whatever the size
    slot = 256 * 128 * 2 + 256 * 8  # O / l in bf16, (m, l) in fp32
    for n_sel, n_tok in [(256, 256), (1280, 5120), (16384, 16384)]:
        ws = L.semshare_prefill_attention_workspace(n_sel, n_tok, 32, 8, 128, 1)
        assert 0 < ws <= 8 * 64 * slot + 4 * (4 + 5 * 32 + 8 * (n_sel // 64 + 1)) + 1024, (n_sel, n_tok, ws)
    assert L.semshare_prefill_attention_workspace(1280, 5120, 32, 8, 128, 1) >= 8 * 52 * slot  # 20 row tiles + 32
    assert L.semshare_prefill_attention_workspace(256, 256, 32, 8, 128, 0) == 0  # fp32 path: no workspace


def test_rope_table_validation(lib):
    L = ss.load()
    assert L.semshare_rope_table_bytes(1280, 128) == 1280 * 64 * 8
    assert L.semshare_rope_table_bytes(0, 128) == 0 and L.semshare_rope_table_bytes(8, 7) == 0
    assert L.semshare_rope_table(FAKE, 8, 16, 7, 1e4, FAKE, 1 << 20, None) == b.E_INVAL  # odd head_dim
    assert L.semshare_rope_table(FAKE, 8, 16, 128, 0.0, FAKE, 1 << 20, None) == b.E_INVAL  # rope_base
    assert L.semshare_rope_table(FAKE, 8, 16, 128, 1e4, FAKE, 8 * 64 * 8 - 1, None) == b.E_INVAL  # too small
    assert L.semshare_rope_table(FAKE, 8, 16, 128, 1e4, FAKE_ODD, 1 << 20, None) == b.E_INVAL  # alignment
    assert L.semshare_rope_table(None, 0, 16, 128, 1e4, None, 0, None) == b.OK
    # the projection with a table: its size and dtype, then the checks it shares with semshare_qkv_rope
    rest = (FAKE, FAKE, 8, FAKE, FAKE, FAKE, FAKE, FAKE, 16, 256, 8, 2, 128, FAKE, None, FAKE, 1 << 30)
    assert L.semshare_qkv_rope_tabled(FAKE, 8 * 64 * 8 - 1, *rest, 1, None) == b.E_INVAL
    assert L.semshare_qkv_rope_tabled(FAKE_ODD, 1 << 20, *rest, 1, None) == b.E_INVAL
    assert L.semshare_qkv_rope_tabled(None, 0, *rest, 1, None) == b.E_INVAL
    assert L.semshare_qkv_rope_tabled(FAKE, 1 << 20, *rest, 0, None) == b.E_UNSUPPORTED  # fp32 projection
    bad_n = (FAKE, FAKE, 8, FAKE, FAKE, FAKE, FAKE, FAKE, 4, 256, 8, 2, 128, FAKE, None, FAKE, 1 << 30)
    assert L.semshare_qkv_rope_tabled(FAKE, 1 << 20, *bad_n, 1, None) == b.E_INVAL  # n_sel > n_tok
    # the same with the rows read in place through x_rows: the row index and n_x, then the shared checks
    rows = L.semshare_qkv_rope_tabled_rows
    tail = (FAKE, FAKE, FAKE, FAKE, FAKE, 16, 256, 8, 2, 128, FAKE, None, FAKE, 1 << 30)
    assert rows(FAKE, 1 << 20, FAKE, 100, None, FAKE, 8, *tail, 1, None) == b.E_INVAL  # no x_rows
    assert rows(None, 0, FAKE, 100, FAKE, FAKE, 8, *tail, 1, None) == b.E_INVAL  # no table
    assert rows(FAKE, 1 << 20, FAKE, 0, FAKE, FAKE, 8, *tail, 1, None) == b.E_INVAL  # n_x = 0
    assert rows(FAKE, 1 << 20, FAKE, -1, FAKE, FAKE, 8, *tail, 1, None) == b.E_INVAL
    assert rows(FAKE, 1 << 20, FAKE, 1 << 22, FAKE, FAKE, 8, *tail, 1, None) == b.E_UNSUPPORTED  # x of 2 GiB
    assert rows(FAKE, 1 << 20, FAKE, 100, FAKE, FAKE, 8, *tail, 0, None) == b.E_UNSUPPORTED  # fp32
    assert rows(FAKE, 1 << 20, FAKE_ODD, 100, FAKE, FAKE, 8, *tail, 1, None) == b.E_INVAL  # x alignment
    assert rows(None, 0, None, 0, None, None, 0, *tail, 1, None) == b.OK  # nothing to do


def test_bank_similarity_validation(lib):
    L = ss.load()
    assert L.semshare_bank_similarity_workspace(4096, 16) == 32 * 16 * 8
    assert L.semshare_bank_similarity_workspace(0, 16) == 0 and L.semshare_bank_similarity_workspace(10, 0) == 0
    call = L.semshare_bank_similarity
    ok_args = dict(tgt=FAKE, n_tgt=100, ref=FAKE, n_ref=50, off=FAKE, n_prompts=3, n_words=2, dmin=0.0, dmax=30.0,
                   dsum=FAKE, sim=FAKE, ws=FAKE, ws_bytes=1 << 20)

    def st(**kw):
        a = dict(ok_args, **kw)
        return call(a["tgt"], a["n_tgt"], a["ref"], a["n_ref"], a["off"], a["n_prompts"], a["n_words"], a["dmin"],
                    a["dmax"], a["dsum"], a["sim"], a["ws"], a["ws_bytes"], None)
    assert st(n_words=0) == b.E_INVAL and st(n_words=5) == b.E_INVAL
    assert st(dmax=0.0) == b.E_INVAL and st(dmin=float("nan")) == b.E_INVAL
    assert st(n_prompts=70000) == b.E_UNSUPPORTED
    assert st(n_tgt=-1) == b.E_INVAL
    assert st(ws_bytes=8) == b.E_INVAL and "workspace" in ss.last_error()
    assert st(ws=FAKE + 4) == b.E_INVAL  # 8-byte alignment
    assert st(off=None) == b.E_INVAL and st(sim=None) == b.E_INVAL
    assert st(n_prompts=0, off=None, dsum=None, sim=None) == b.OK



def test_qkv_rope_dev_ref_validation(lib):
    L = ss.load()
    head = (FAKE, FAKE, 8, FAKE, FAKE, FAKE, FAKE, FAKE, 16, 256, 8, 2, 128, 1e4, FAKE)
    ws = (FAKE, 1 << 30)
    assert L.semshare_qkv_rope_dev_ref(*head, None, FAKE, FAKE, FAKE, 16, *ws, 1, None) == b.E_INVAL  # no deviation
    assert L.semshare_qkv_rope_dev_ref(*head, FAKE, None, FAKE, FAKE, 16, *ws, 1, None) == b.E_INVAL  # no ref_k
    assert L.semshare_qkv_rope_dev_ref(*head, FAKE, FAKE, FAKE, None, 16, *ws, 1, None) == b.E_INVAL  # no idx
    assert L.semshare_qkv_rope_dev_ref(*head, FAKE, FAKE_ODD, FAKE, FAKE, 16, *ws, 1, None) == b.E_INVAL  # alignment
    assert L.semshare_qkv_rope_dev_ref(*head, FAKE, FAKE, FAKE, FAKE, -1, *ws, 1, None) == b.E_INVAL  # n_ref
    assert L.semshare_qkv_rope_dev_ref(*head, FAKE, FAKE, FAKE, FAKE, 16, *ws, 0, None) == b.E_UNSUPPORTED  # fp32
    bad = (FAKE, FAKE, 8, FAKE, FAKE, FAKE, FAKE, FAKE, 4, 256, 8, 2, 128, 1e4, FAKE)
    assert L.semshare_qkv_rope_dev_ref(*bad, FAKE, FAKE, FAKE, FAKE, 16, *ws, 1, None) == b.E_INVAL  # n_sel > n_tok
    assert L.semshare_qkv_rope_dev_ref(*head, FAKE, FAKE, FAKE, FAKE, 16, FAKE, 0, 1, None) == b.E_INVAL  # workspace


def test_prefill_attention_noalloc_validation(lib):
    L = ss.load()
    args = (FAKE, FAKE, 8, FAKE, FAKE, 16, 8, 2, 128)
    assert L.semshare_prefill_attention_noalloc(*args, 0.0, None, 1, None) == b.E_INVAL  # no output
    assert L.semshare_prefill_attention_noalloc(*args, -1.0, FAKE, 1, None) == b.E_INVAL  # scale
    assert L.semshare_prefill_attention_noalloc(FAKE_ODD, FAKE, 8, FAKE, FAKE, 16, 8, 2, 128, 0.0, FAKE, 1,
                                                None) == b.E_INVAL  # alignment
    assert L.semshare_prefill_attention_noalloc(FAKE, FAKE, 8, FAKE, FAKE, 16, 8, 2, 96, 0.0, FAKE, 1,
                                                None) == b.E_UNSUPPORTED  # head_dim
    assert L.semshare_prefill_attention_noalloc(None, None, 0, None, None, 16, 8, 2, 128, 0.0, None, 1, None) == b.OK
    # 512 kv heads of head_dim 128 need 64 MiB of partial results: beyond the 40 MiB static scratch
    assert L.semshare_prefill_attention_noalloc(FAKE, FAKE, 64, FAKE, FAKE, 64, 512, 512, 128, 0.0, FAKE, 1,
                                                None) == b.E_UNSUPPORTED
    assert "scratch" in ss.last_error()
    # the headline shapes fit: the workspace the other call needs stays below 40 MiB
    for n_sel, n_tok in [(1280, 5120), (5120, 5120), (3277, 32768), (32768, 32768)]:
        assert L.semshare_prefill_attention_workspace(n_sel, n_tok, 32, 8, 128, 1) <= 40 << 20
