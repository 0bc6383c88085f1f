"""ctypes binding of libsemshare.so (include/semshare.h).

Argument marshalling only: torch provides device memory and the current HIP
stream; every step of the computation runs in the library's HIP kernels.
There is no fallback: if the library is missing or a call fails, an
exception is raised.
"""
from __future__ import annotations

import ctypes
import os
import re
from typing import List, Optional, Tuple

import torch  # loaded first so the library binds to the same HIP runtime

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG, "libsemshare.so")
HEADER_PATH = os.path.join(os.path.dirname(_PKG), "include", "semshare.h")

OK, E_INVAL, E_UNSUPPORTED, E_DEVICE = 0, -1, -2, -3
FP32, BF16 = 0, 1

_lib: Optional[ctypes.CDLL] = None


class SemShareError(RuntimeError):
    def __init__(self, status: int, message: str):
        super().__init__(f"semshare status {status}: {message}")
        self.status = status
        self.message = message


def declared_symbols() -> List[str]:
    """Every function the C header declares."""
    with open(HEADER_PATH) as f:
        text = f.read()
    return sorted(set(re.findall(r"^\s*(?:const\s+)?[\w]+\**\s+\**(semshare_\w+)\s*\(", text, re.M)))


def load() -> ctypes.CDLL:
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise RuntimeError(f"{LIB_PATH} is not built; run `python -m paper_2509_24832_amd.build` "
                           "(or __graft_entry__.build()) first")
    lib = ctypes.CDLL(LIB_PATH)
    P, I64, I32, F64, F32, SZ = (ctypes.c_void_p, ctypes.c_int64, ctypes.c_int32, ctypes.c_double,
                                 ctypes.c_float, ctypes.c_size_t)
    sig = {
        "semshare_last_error": (ctypes.c_char_p, []),
        "semshare_version": (I32, []),
        "semshare_rope_embed": (I32, [P, P, I64, I32, I64, F64, I32, P]),
        "semshare_lsh_encode": (I32, [P, P, P, I64, I32, I32, I32, P]),
        "semshare_rope_lsh_encode": (I32, [P, P, P, I64, I32, I32, I64, F64, I32, P]),
        "semshare_match": (I32, [P, I64, P, I64, I32, P, P, P]),
        "semshare_match_mfma": (I32, [P, I64, P, I64, I32, P, P, P]),
        "semshare_gather_kv": (I32, [P, P, P, I64, I64, P, P, I32, I32, I32, I32, P]),
        "semshare_gather_kv_except": (I32, [P, P, P, I64, I64, P, P, I32, I32, I32, I32, P, I64, P]),
        "semshare_partial_prefill": (I32, [P, P, I64, P, P, P, P, P, I64, I32, I32, I32, I32, F64, F32,
                                           P, P, P, SZ, I32, P]),
        "semshare_partial_prefill_workspace": (SZ, [I64, I64, I32, I32, I32, I32, I32]),
        "semshare_select_recompute": (I32, [P, I64, I64, P, P]),
        "semshare_select_recompute_nested": (I32, [P, P, I64, I64, P, P]),
        "semshare_retention_layer": (I32, [P, I32, I32, P, I32, P, P, P, P, P, P]),
        "semshare_attention_mass_workspace": (SZ, [I64, I32]),
        "semshare_attention_mass": (I32, [P, P, I64, I64, I32, I32, I32, F32, P, P, SZ, I32, P]),
        "semshare_attention_mass_window": (I32, [P, P, I64, I64, I32, I32, I32, F32, P, P, SZ, I32, P]),
        "semshare_retention": (I32, [P, P, I32, P, P, F64, P, P, P, P]),
        "semshare_dynamic_recompute": (I32, [P, P, I32, F64, F64, F64, P, P, P]),
        "semshare_qkv_rope": (I32, [P, P, I64, P, P, P, P, P, I64, I32, I32, I32, I32, F64, P, P, P, SZ, I32, P]),
        "semshare_qkv_rope_workspace": (SZ, [I64, I32, I32, I32, I32]),
        "semshare_prefill_attention_noalloc": (I32, [P, P, I64, P, P, I64, I32, I32, I32, F32, P, I32, P]),
        "semshare_qkv_rope_dev_ref": (I32, [P, P, I64, P, P, P, P, P, I64, I32, I32, I32, I32, F64, P, P, P, P, P,
                                            I64, P, SZ, I32, P]),
        "semshare_prefill_attention": (I32, [P, P, I64, P, P, I64, I32, I32, I32, F32, P, P, SZ, I32, P]),
        "semshare_prefill_attention_workspace": (SZ, [I64, I64, I32, I32, I32, I32]),
        "semshare_bank_similarity_workspace": (SZ, [I64, I32]),
        "semshare_bank_similarity": (I32, [P, I64, P, I64, P, I32, I32, F64, F64, P, P, P, SZ, P]),
        "semshare_rope_table_bytes": (SZ, [I64, I32]),
        "semshare_rope_table": (I32, [P, I64, I64, I32, F64, P, SZ, P]),
        "semshare_qkv_rope_tabled": (I32, [P, SZ, P, P, I64, P, P, P, P, P, I64, I32, I32, I32, I32, P, P, P, SZ,
                                           I32, P]),
        "semshare_qkv_rope_tabled_rows": (I32, [P, SZ, P, I64, P, P, I64, P, P, P, P, P, I64, I32, I32, I32, I32, P,
                                                P, P, SZ, I32, P]),
        "semshare_attention_plan_bytes": (SZ, [I64, I64, I32, I32, I32, I32]),
        "semshare_attention_plan": (I32, [P, I64, I64, I32, I32, I32, I32, P, SZ, P]),
        "semshare_prefill_attention_planned": (I32, [P, SZ, P, P, I64, P, P, I64, I32, I32, I32, F32, P, P, SZ,
                                                     I32, P]),
    }
    missing = set(declared_symbols()) - set(sig)
    if missing:  # an entry without argtypes would pass pointers and int64 sizes as 32-bit ints
        raise RuntimeError(f"no ctypes signature for {sorted(missing)}")
    for name, (res, args) in sig.items():
        fn = getattr(lib, name)
        fn.restype = res
        fn.argtypes = args
    _lib = lib
    return lib


def version() -> int:
    return int(load().semshare_version())


def last_error() -> str:
    return load().semshare_last_error().decode()


def _call(fn_name: str, *args) -> None:
    lib = load()
    st = getattr(lib, fn_name)(*args)
    if st != OK:
        raise SemShareError(int(st), lib.semshare_last_error().decode())


def _stream() -> int:
    return torch.cuda.current_stream().cuda_stream


def _ptr(t: Optional[torch.Tensor]) -> Optional[int]:
    return None if t is None else t.data_ptr()


def _dt(t: torch.Tensor) -> int:
    if t.dtype == torch.bfloat16:
        return BF16
    if t.dtype == torch.float32:
        return FP32
    raise TypeError(f"unsupported dtype {t.dtype}; use bfloat16 or float32")


def _dev(t: torch.Tensor, name: str, dtype=None) -> torch.Tensor:
    if not isinstance(t, torch.Tensor):
        raise TypeError(f"{name} must be a torch.Tensor")
    if t.device.type != "cuda":
        raise ValueError(f"{name} must be a device tensor (got {t.device})")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    if dtype is not None and t.dtype != dtype:
        raise TypeError(f"{name} must be {dtype} (got {t.dtype})")
    return t


# ----------------------------------------------------------------- the calls

def rope_embed(x: torch.Tensor, out: Optional[torch.Tensor] = None, pos0: int = 0,
               base: float = 10000.0) -> torch.Tensor:
    """RoPE of every row of x [n_tok, dim] (row r at position pos0 + r)."""
    _dev(x, "x")
    if x.dim() != 2:
        raise ValueError("x must be [n_tok, dim]")
    y = torch.empty_like(x) if out is None else _dev(out, "out", x.dtype)
    if y.shape != x.shape:
        raise ValueError("out shape mismatch")
    _call("semshare_rope_embed", _ptr(x), _ptr(y), x.shape[0], x.shape[1], int(pos0), float(base), _dt(x),
          _stream())
    return y


def lsh_encode(x: torch.Tensor, planes: torch.Tensor, out: Optional[torch.Tensor] = None) -> torch.Tensor:
    """Sign-bit LSH codes [n_tok, n_bits/64] (int64 tensor holding the u64 words)."""
    _dev(x, "x")
    _dev(planes, "planes", x.dtype)
    if x.dim() != 2 or planes.dim() != 2 or planes.shape[1] != x.shape[1]:
        raise ValueError("x [n_tok, dim] and planes [n_bits, dim] required")
    n_bits = planes.shape[0]
    codes = (torch.empty((x.shape[0], max(n_bits // 64, 1)), dtype=torch.int64, device=x.device)
             if out is None else _dev(out, "out", torch.int64))
    _call("semshare_lsh_encode", _ptr(x), _ptr(planes), _ptr(codes), x.shape[0], x.shape[1], n_bits, _dt(x),
          _stream())
    return codes


def rope_lsh_encode(x: torch.Tensor, planes: torch.Tensor, out: Optional[torch.Tensor] = None, pos0: int = 0,
                    base: float = 10000.0) -> torch.Tensor:
    """LSH codes of the RoPE-embedded rows of x (row r at position pos0 + r), in one pass."""
    _dev(x, "x")
    _dev(planes, "planes", x.dtype)
    if x.dim() != 2 or planes.dim() != 2 or planes.shape[1] != x.shape[1]:
        raise ValueError("x [n_tok, dim] and planes [n_bits, dim] required")
    n_bits = planes.shape[0]
    codes = (torch.empty((x.shape[0], max(n_bits // 64, 1)), dtype=torch.int64, device=x.device)
             if out is None else _dev(out, "out", torch.int64))
    _call("semshare_rope_lsh_encode", _ptr(x), _ptr(planes), _ptr(codes), x.shape[0], x.shape[1], n_bits,
          int(pos0), float(base), _dt(x), _stream())
    return codes


def attention_mass(q: torch.Tensor, k_cache: torch.Tensor, n_q_heads: int, n_kv_heads: int, sm_scale: float = 0.0,
                   mass: Optional[torch.Tensor] = None, workspace: Optional[torch.Tensor] = None,
                   row_begin: int = 0, reuse_normalisers: bool = False) -> torch.Tensor:
    """Average attention score per token over the query rows >= row_begin: q [T, Hq, D], k_cache [T, Hkv, D]
    -> mass [T] float32.  reuse_normalisers: semshare_attention_mass_window, which takes the row normalisers
    from `workspace` as a previous call over the same q and k_cache left them (workspace required)."""
    if reuse_normalisers and workspace is None:
        raise ValueError("reuse_normalisers needs the workspace of a previous attention_mass call")
    _dev(q, "q")
    _dev(k_cache, "k_cache", q.dtype)
    T = q.shape[0]
    d = q.shape[-1]
    if mass is None:
        mass = torch.empty(T, dtype=torch.float32, device=q.device)
    _dev(mass, "mass", torch.float32)
    need = int(load().semshare_attention_mass_workspace(T, n_q_heads))
    if workspace is None:
        workspace = torch.empty(max(need, 1), dtype=torch.uint8, device=q.device)
    _call("semshare_attention_mass_window" if reuse_normalisers else "semshare_attention_mass", _ptr(q),
          _ptr(k_cache), T, int(row_begin), n_q_heads, n_kv_heads, d,
          float(sm_scale), _ptr(mass),
          _ptr(workspace), workspace.numel() * workspace.element_size(), _dt(q), _stream())
    return mass


def dynamic_recompute(mass: torch.Tensor, sigma: torch.Tensor, thres: float = 0.55, w_hot: float = 0.5,
                      w_cold: float = 0.1, sel_pos: Optional[torch.Tensor] = None,
                      counts: Optional[torch.Tensor] = None) -> Tuple[torch.Tensor, torch.Tensor]:
    """Hot tokens by Attention Recovery and the recompute set: returns (sel_pos [T] int32 with the first
    counts[1] valid, counts [3] int32 = AR, number selected, hot among them), both on the device."""
    _dev(mass, "mass", torch.float32)
    _dev(sigma, "sigma", torch.float32)
    T = mass.shape[0]
    if sel_pos is None:
        sel_pos = torch.empty(max(T, 1), dtype=torch.int32, device=mass.device)
    if counts is None:
        counts = torch.empty(3, dtype=torch.int32, device=mass.device)
    _call("semshare_dynamic_recompute", _ptr(mass), _ptr(sigma), T, float(thres), float(w_hot), float(w_cold),
          _ptr(sel_pos), _ptr(counts), _stream())
    return sel_pos, counts


def retention(mass: torch.Tensor, score: torch.Tensor, sel_pos: torch.Tensor, counts: torch.Tensor,
              min_keep: float = 0.8) -> Tuple[torch.Tensor, torch.Tensor, torch.Tensor]:
    """First-layer retention: returns (rank [T], kept_pos [T] with the first n_kept valid, n_kept [1]), on the device."""
    _dev(mass, "mass", torch.float32)
    _dev(score, "score", torch.float32)
    _dev(sel_pos, "sel_pos", torch.int32)
    _dev(counts, "counts", torch.int32)
    T = mass.shape[0]
    rank = torch.empty(max(T, 1), dtype=torch.int32, device=mass.device)
    kept = torch.empty(max(T, 1), dtype=torch.int32, device=mass.device)
    n_kept = torch.empty(1, dtype=torch.int32, device=mass.device)
    _call("semshare_retention", _ptr(mass), _ptr(score), T, _ptr(sel_pos), _ptr(counts), float(min_keep), _ptr(rank),
          _ptr(kept), _ptr(n_kept), _stream())
    return rank, kept, n_kept


def _match(entry: str, tgt_codes, ref_codes, idx, dist, want_dist):
    _dev(tgt_codes, "tgt_codes", torch.int64)
    _dev(ref_codes, "ref_codes", torch.int64)
    if tgt_codes.dim() != 2 or ref_codes.dim() != 2 or tgt_codes.shape[1] != ref_codes.shape[1]:
        raise ValueError("codes must be [n, n_words] with equal n_words")
    n_tgt = tgt_codes.shape[0]
    if idx is None:
        idx = torch.empty(n_tgt, dtype=torch.int32, device=tgt_codes.device)
    _dev(idx, "idx", torch.int32)
    if want_dist and dist is None:
        dist = torch.empty(n_tgt, dtype=torch.int32, device=tgt_codes.device)
    if dist is not None:
        _dev(dist, "dist", torch.int32)
    _call(entry, _ptr(tgt_codes), n_tgt, _ptr(ref_codes), ref_codes.shape[0], tgt_codes.shape[1],
          _ptr(idx), _ptr(dist), _stream())
    return idx, dist


def match(tgt_codes: torch.Tensor, ref_codes: torch.Tensor, idx: Optional[torch.Tensor] = None,
          dist: Optional[torch.Tensor] = None, want_dist: bool = True) -> Tuple[torch.Tensor, Optional[torch.Tensor]]:
    """Top-1 Hamming match of target codes against reference codes."""
    return _match("semshare_match", tgt_codes, ref_codes, idx, dist, want_dist)


def match_mfma(tgt_codes: torch.Tensor, ref_codes: torch.Tensor, idx: Optional[torch.Tensor] = None,
               dist: Optional[torch.Tensor] = None,
               want_dist: bool = True) -> Tuple[torch.Tensor, Optional[torch.Tensor]]:
    """The same match computed as +-1 dot products on the int8 matrix cores."""
    return _match("semshare_match_mfma", tgt_codes, ref_codes, idx, dist, want_dist)


def gather_kv(ref_k: torch.Tensor, ref_v: Optional[torch.Tensor], idx: torch.Tensor,
              out_k: Optional[torch.Tensor] = None, out_v: Optional[torch.Tensor] = None,
              except_pos: Optional[torch.Tensor] = None, n_except: Optional[int] = None):
    """out[l][t] = ref[l][idx[t]]; ref_* [L, n_ref, Hkv, D] -> out_* [L, n_tgt, Hkv, D].  With except_pos
    (ascending int32 target rows, repeats allowed; the first n_except of it, 0 <= n_except <=
    min(except_pos.numel(), n_tgt))
    those rows are left as they are."""
    _dev(ref_k, "ref_k")
    _dev(idx, "idx", torch.int32)
    if ref_k.dim() != 4:
        raise ValueError("ref_k must be [L, n_ref, Hkv, D]")
    L, n_ref, hkv, d = ref_k.shape
    n_tgt = idx.shape[0]
    shape = (L, n_tgt, hkv, d)
    if out_k is None:
        out_k = torch.empty(shape, dtype=ref_k.dtype, device=ref_k.device)
    _dev(out_k, "out_k", ref_k.dtype)
    if ref_v is not None:
        _dev(ref_v, "ref_v", ref_k.dtype)
        if ref_v.shape != ref_k.shape:
            raise ValueError("ref_v shape mismatch")
        if out_v is None:
            out_v = torch.empty(shape, dtype=ref_k.dtype, device=ref_k.device)
        _dev(out_v, "out_v", ref_k.dtype)
    else:
        out_v = None
    if tuple(out_k.shape) != shape or (out_v is not None and tuple(out_v.shape) != shape):
        raise ValueError("output shape mismatch")
    if except_pos is None:
        _call("semshare_gather_kv", _ptr(ref_k), _ptr(ref_v), _ptr(idx), n_tgt, n_ref, _ptr(out_k), _ptr(out_v), L,
              hkv, d, _dt(ref_k), _stream())
    else:
        _dev(except_pos, "except_pos", torch.int32)
        ne = except_pos.shape[0] if n_except is None else int(n_except)
        if except_pos.dim() != 1 or not 0 <= ne <= except_pos.numel():
            raise ValueError(f"n_except must lie in [0, {except_pos.numel()}] (got {ne})")
        _call("semshare_gather_kv_except", _ptr(ref_k), _ptr(ref_v), _ptr(idx), n_tgt, n_ref, _ptr(out_k),
              _ptr(out_v), L, hkv, d, _dt(ref_k), _ptr(except_pos), ne, _stream())
    return out_k, out_v


def gather_rows(src: torch.Tensor, idx: torch.Tensor, out: Optional[torch.Tensor] = None) -> torch.Tensor:
    """Plain row gather out[t] = src[idx[t]] of a [n_ref, width] tensor."""
    _dev(src, "src")
    if src.dim() != 2:
        raise ValueError("src must be [n_ref, width]")
    if out is None:
        out = torch.empty((idx.shape[0], src.shape[1]), dtype=src.dtype, device=src.device)
    o, _ = gather_kv(src.view(1, src.shape[0], 1, src.shape[1]), None, idx,
                     out_k=out.view(1, idx.shape[0], 1, src.shape[1]))
    return out


def partial_prefill_workspace_bytes(n_sel: int, n_tok: int, hidden: int, n_q_heads: int, n_kv_heads: int,
                                    head_dim: int, dtype: torch.dtype) -> int:
    code = BF16 if dtype == torch.bfloat16 else FP32
    return int(load().semshare_partial_prefill_workspace(n_sel, n_tok, hidden, n_q_heads, n_kv_heads, head_dim,
                                                         code))


def partial_prefill(x_sel: torch.Tensor, sel_pos: torch.Tensor, wq: Optional[torch.Tensor], wk: torch.Tensor,
                    wv: torch.Tensor, k_cache: torch.Tensor, v_cache: torch.Tensor, n_q_heads: int,
                    n_kv_heads: int, rope_base: float = 10000.0, sm_scale: float = 0.0,
                    out: Optional[torch.Tensor] = None, want_out: bool = True,
                    deviation: Optional[torch.Tensor] = None, want_deviation: bool = False,
                    workspace: Optional[torch.Tensor] = None):
    """One layer of partial prefill; updates k_cache/v_cache rows sel_pos in place.
    Returns (out [n_sel, Hq, D] or None, deviation [n_sel] or None)."""
    _dev(x_sel, "x_sel")
    dt = x_sel.dtype
    _dev(sel_pos, "sel_pos", torch.int32)
    for name, t in (("wk", wk), ("wv", wv), ("k_cache", k_cache), ("v_cache", v_cache)):
        _dev(t, name, dt)
    n_sel, hidden = x_sel.shape
    n_tok = k_cache.shape[0]
    head_dim = k_cache.shape[-1]
    if k_cache.numel() != n_tok * n_kv_heads * head_dim or v_cache.shape != k_cache.shape:
        raise ValueError("caches must be [n_tok, n_kv_heads, head_dim]")
    if sel_pos.shape[0] != n_sel:
        raise ValueError("sel_pos length must equal x_sel rows")
    if want_out:
        if wq is None:
            raise ValueError("wq required for the attention output")
        _dev(wq, "wq", dt)
        if out is None:
            out = torch.empty((n_sel, n_q_heads, head_dim), dtype=dt, device=x_sel.device)
        _dev(out, "out", dt)
    else:
        out = None
    if want_deviation:
        if deviation is None:
            deviation = torch.empty(n_sel, dtype=torch.float32, device=x_sel.device)
        _dev(deviation, "deviation", torch.float32)
    else:
        deviation = None
    need = partial_prefill_workspace_bytes(n_sel, n_tok, hidden, n_q_heads, n_kv_heads, head_dim, dt)
    if workspace is None:
        workspace = torch.empty(max(need, 1), dtype=torch.uint8, device=x_sel.device)
    _dev(workspace, "workspace", torch.uint8)
    _call("semshare_partial_prefill", _ptr(x_sel), _ptr(sel_pos), n_sel, _ptr(wq) if want_out else None, _ptr(wk),
          _ptr(wv), _ptr(k_cache), _ptr(v_cache), n_tok, hidden, n_q_heads, n_kv_heads, head_dim,
          float(rope_base), float(sm_scale), _ptr(out), _ptr(deviation), _ptr(workspace), workspace.numel(),
          _dt(x_sel), _stream())
    return out, deviation


def qkv_rope_workspace_bytes(n_sel: int, n_q_heads: int, n_kv_heads: int, head_dim: int,
                             dtype: torch.dtype) -> int:
    return int(load().semshare_qkv_rope_workspace(n_sel, n_q_heads, n_kv_heads, head_dim,
                                                  BF16 if dtype == torch.bfloat16 else FP32))


def prefill_attention_workspace_bytes(n_sel: int, n_tok: int, n_q_heads: int, n_kv_heads: int, head_dim: int,
                                      dtype: torch.dtype) -> int:
    return int(load().semshare_prefill_attention_workspace(n_sel, n_tok, n_q_heads, n_kv_heads, head_dim,
                                                           BF16 if dtype == torch.bfloat16 else FP32))


def _workspace(need: int, given: Optional[torch.Tensor], like: torch.Tensor) -> Optional[torch.Tensor]:
    if given is not None:
        return _dev(given, "workspace", torch.uint8)
    if need == 0:
        return None
    return torch.empty(need, dtype=torch.uint8, device=like.device)


def qkv_rope(x_sel: torch.Tensor, sel_pos: torch.Tensor, wq: Optional[torch.Tensor], wk: torch.Tensor,
             wv: torch.Tensor, k_cache: torch.Tensor, v_cache: torch.Tensor, n_q_heads: int, n_kv_heads: int,
             rope_base: float = 10000.0, q_out: Optional[torch.Tensor] = None, want_q: bool = True,
             deviation: Optional[torch.Tensor] = None, want_deviation: bool = False,
             workspace: Optional[torch.Tensor] = None, rope_table: Optional[torch.Tensor] = None,
             x_rows: Optional[torch.Tensor] = None):
    """Projection + RoPE + deviation + cache scatter of the selected rows (with `rope_table` from
    rope_table(), bf16: its factors instead of rope_base).  With x_rows (int32 [n_sel], bf16 with a
    rope_table only): input row i is row x_rows[i] of x_sel, which then holds every row [n_x, hidden]
    (no gathered copy; the same results as gather_rows then qkv_rope).
    Returns (q [n_sel, Hq, D] or None, deviation [n_sel] or None)."""
    _dev(x_sel, "x_sel")
    dt = x_sel.dtype
    _dev(sel_pos, "sel_pos", torch.int32)
    for name, t in (("wk", wk), ("wv", wv), ("k_cache", k_cache), ("v_cache", v_cache)):
        _dev(t, name, dt)
    n_sel, hidden = x_sel.shape
    if x_rows is not None:
        _dev(x_rows, "x_rows", torch.int32)
        if rope_table is None:
            raise ValueError("x_rows needs a rope_table")
        n_sel = x_rows.numel()
        if sel_pos.numel() < n_sel:
            raise ValueError("sel_pos shorter than x_rows")
    n_tok, head_dim = k_cache.shape[0], k_cache.shape[-1]
    if k_cache.numel() != n_tok * n_kv_heads * head_dim or v_cache.shape != k_cache.shape:
        raise ValueError("caches must be [n_tok, n_kv_heads, head_dim]")
    if want_q:
        _dev(wq, "wq", dt)
        if q_out is None:
            q_out = torch.empty((n_sel, n_q_heads, head_dim), dtype=dt, device=x_sel.device)
        _dev(q_out, "q_out", dt)
    else:
        q_out = None
    if want_deviation and deviation is None:
        deviation = torch.empty(n_sel, dtype=torch.float32, device=x_sel.device)
    if not want_deviation:
        deviation = None
    ws = _workspace(qkv_rope_workspace_bytes(n_sel, n_q_heads, n_kv_heads, head_dim, dt), workspace, x_sel)
    if x_rows is not None:
        _dev(rope_table, "rope_table", torch.uint8)
        _call("semshare_qkv_rope_tabled_rows", _ptr(rope_table), rope_table.numel(), _ptr(x_sel), x_sel.shape[0],
              _ptr(x_rows), _ptr(sel_pos), n_sel, _ptr(wq) if want_q else None, _ptr(wk), _ptr(wv), _ptr(k_cache),
              _ptr(v_cache), n_tok, hidden, n_q_heads, n_kv_heads, head_dim, _ptr(q_out), _ptr(deviation),
              _ptr(ws), 0 if ws is None else ws.numel(), _dt(x_sel), _stream())
        return q_out, deviation
    if rope_table is not None:
        _dev(rope_table, "rope_table", torch.uint8)
        _call("semshare_qkv_rope_tabled", _ptr(rope_table), rope_table.numel(), _ptr(x_sel), _ptr(sel_pos), n_sel,
              _ptr(wq) if want_q else None, _ptr(wk), _ptr(wv), _ptr(k_cache), _ptr(v_cache), n_tok, hidden,
              n_q_heads, n_kv_heads, head_dim, _ptr(q_out), _ptr(deviation), _ptr(ws),
              0 if ws is None else ws.numel(), _dt(x_sel), _stream())
        return q_out, deviation
    _call("semshare_qkv_rope", _ptr(x_sel), _ptr(sel_pos), n_sel, _ptr(wq) if want_q else None, _ptr(wk), _ptr(wv),
          _ptr(k_cache), _ptr(v_cache), n_tok, hidden, n_q_heads, n_kv_heads, head_dim, float(rope_base),
          _ptr(q_out), _ptr(deviation), _ptr(ws), 0 if ws is None else ws.numel(), _dt(x_sel), _stream())
    return q_out, deviation


def qkv_rope_dev_ref(x_sel: torch.Tensor, sel_pos: torch.Tensor, wq: Optional[torch.Tensor], wk: torch.Tensor,
                     wv: torch.Tensor, k_cache: torch.Tensor, v_cache: torch.Tensor, n_q_heads: int, n_kv_heads: int,
                     ref_k: torch.Tensor, ref_v: torch.Tensor, idx: torch.Tensor, rope_base: float = 10000.0,
                     q_out: Optional[torch.Tensor] = None, want_q: bool = True,
                     deviation: Optional[torch.Tensor] = None, workspace: Optional[torch.Tensor] = None):
    """qkv_rope (bf16) whose deviation compares each recomputed row p with the matched reference row
    ref[idx[p]] (ref_* [n_ref, Hkv, D], one layer; idx [n_tok] int32), as gather_kv then qkv_rope would.
    Returns (q [n_sel, Hq, D] or None, deviation [n_sel])."""
    _dev(x_sel, "x_sel")
    dt = x_sel.dtype
    _dev(sel_pos, "sel_pos", torch.int32)
    _dev(idx, "idx", torch.int32)
    for name, t in (("wk", wk), ("wv", wv), ("k_cache", k_cache), ("v_cache", v_cache), ("ref_k", ref_k),
                    ("ref_v", ref_v)):
        _dev(t, name, dt)
    n_sel, hidden = x_sel.shape
    n_tok, head_dim = k_cache.shape[0], k_cache.shape[-1]
    if k_cache.numel() != n_tok * n_kv_heads * head_dim or v_cache.shape != k_cache.shape:
        raise ValueError("caches must be [n_tok, n_kv_heads, head_dim]")
    n_ref = ref_k.shape[0]
    if ref_k.numel() != n_ref * n_kv_heads * head_dim or ref_v.shape != ref_k.shape:
        raise ValueError("reference caches must be [n_ref, n_kv_heads, head_dim]")
    if idx.dim() != 1 or idx.numel() < n_tok:
        raise ValueError("idx must hold one entry per cache row")
    if want_q:
        _dev(wq, "wq", dt)
        if q_out is None:
            q_out = torch.empty((n_sel, n_q_heads, head_dim), dtype=dt, device=x_sel.device)
        _dev(q_out, "q_out", dt)
    else:
        q_out = None
    if deviation is None:
        deviation = torch.empty(n_sel, dtype=torch.float32, device=x_sel.device)
    _dev(deviation, "deviation", torch.float32)
    ws = _workspace(qkv_rope_workspace_bytes(n_sel, n_q_heads, n_kv_heads, head_dim, dt), workspace, x_sel)
    _call("semshare_qkv_rope_dev_ref", _ptr(x_sel), _ptr(sel_pos), n_sel, _ptr(wq) if want_q else None, _ptr(wk),
          _ptr(wv), _ptr(k_cache), _ptr(v_cache), n_tok, hidden, n_q_heads, n_kv_heads, head_dim, float(rope_base),
          _ptr(q_out), _ptr(deviation), _ptr(ref_k), _ptr(ref_v), _ptr(idx), n_ref, _ptr(ws),
          0 if ws is None else ws.numel(), _dt(x_sel), _stream())
    return q_out, deviation


def bank_similarity(tgt_codes: torch.Tensor, ref_codes: torch.Tensor, ref_offsets: torch.Tensor,
                    dmin: float = 0.0, dmax: float = 30.0, workspace: Optional[torch.Tensor] = None):
    """Per reference prompt of a bank (codes [ref_offsets[b], ref_offsets[b+1]) of ref_codes): the sum of
    the target tokens' top-1 Hamming distances within it and the similarity score.
    Returns (dist_sum int64 [n_prompts], similarity float64 [n_prompts])."""
    for name, t in (("tgt_codes", tgt_codes), ("ref_codes", ref_codes)):
        if t.dim() != 2:
            raise ValueError(f"{name} must be [n, n_words]")
        _dev(t, name, torch.int64)
    _dev(ref_offsets, "ref_offsets", torch.int64)
    n_tgt, n_words = tgt_codes.shape
    n_ref = ref_codes.shape[0]
    if ref_codes.shape[1] != n_words:
        raise ValueError("codes must have equal n_words")
    n_prompts = ref_offsets.numel() - 1
    if n_prompts < 0:
        raise ValueError("ref_offsets needs n_prompts + 1 entries")
    dist_sum = torch.empty(n_prompts, dtype=torch.int64, device=tgt_codes.device)  # every entry is written
    sim = torch.empty(n_prompts, dtype=torch.float64, device=tgt_codes.device)
    need = int(load().semshare_bank_similarity_workspace(n_tgt, n_prompts))
    ws = workspace if workspace is not None else (torch.empty(need, dtype=torch.uint8, device=tgt_codes.device)
                                                  if need else None)
    _call("semshare_bank_similarity", _ptr(tgt_codes), n_tgt, _ptr(ref_codes), n_ref, _ptr(ref_offsets), n_prompts,
          n_words, float(dmin), float(dmax), _ptr(dist_sum), _ptr(sim), _ptr(ws), 0 if ws is None else ws.numel(),
          _stream())
    return dist_sum, sim


def rope_table_bytes(n_sel: int, head_dim: int) -> int:
    return int(load().semshare_rope_table_bytes(n_sel, head_dim))


def rope_table(sel_pos: torch.Tensor, n_tok: int, head_dim: int, rope_base: float = 10000.0,
               out: Optional[torch.Tensor] = None) -> torch.Tensor:
    """RoPE factors of qkv_rope for these selected positions (reusable across layers), as bytes."""
    _dev(sel_pos, "sel_pos", torch.int32)
    n_sel = sel_pos.numel()
    need = rope_table_bytes(n_sel, head_dim)
    if out is None:
        out = torch.empty(max(need, 16), dtype=torch.uint8, device=sel_pos.device)
    _dev(out, "rope_table", torch.uint8)
    _call("semshare_rope_table", _ptr(sel_pos), n_sel, n_tok, head_dim, float(rope_base), _ptr(out), out.numel(),
          _stream())
    return out


def attention_plan_bytes(n_sel: int, n_tok: int, n_q_heads: int, n_kv_heads: int, head_dim: int,
                         dtype: torch.dtype = torch.bfloat16) -> int:
    return int(load().semshare_attention_plan_bytes(n_sel, n_tok, n_q_heads, n_kv_heads, head_dim,
                                                    BF16 if dtype == torch.bfloat16 else FP32))


def attention_plan(sel_pos: torch.Tensor, n_tok: int, n_q_heads: int, n_kv_heads: int, head_dim: int,
                   dtype: torch.dtype = torch.bfloat16, out: Optional[torch.Tensor] = None) -> torch.Tensor:
    """Work plan of prefill_attention for these selected positions (reusable across layers)."""
    _dev(sel_pos, "sel_pos", torch.int32)
    n_sel = sel_pos.numel()
    need = attention_plan_bytes(n_sel, n_tok, n_q_heads, n_kv_heads, head_dim, dtype)
    if out is None:
        out = torch.empty(max(need, 1), dtype=torch.uint8, device=sel_pos.device)
    _dev(out, "plan", torch.uint8)
    _call("semshare_attention_plan", _ptr(sel_pos), n_sel, n_tok, n_q_heads, n_kv_heads, head_dim, BF16 if dtype == torch.bfloat16 else FP32,
          _ptr(out), out.numel(), _stream())
    return out


def prefill_attention(q: torch.Tensor, sel_pos: torch.Tensor, k_cache: torch.Tensor, v_cache: torch.Tensor,
                      n_kv_heads: int, sm_scale: float = 0.0, out: Optional[torch.Tensor] = None,
                      workspace: Optional[torch.Tensor] = None, plan: Optional[torch.Tensor] = None) -> torch.Tensor:
    """Causal GQA attention of the selected rows (q [n_sel, Hq, D]) over the cache (with `plan` from
    attention_plan for the same positions and sizes: the plan step is skipped)."""
    _dev(q, "q")
    dt = q.dtype
    _dev(sel_pos, "sel_pos", torch.int32)
    _dev(k_cache, "k_cache", dt)
    _dev(v_cache, "v_cache", dt)
    n_sel, n_q_heads, head_dim = q.shape
    n_tok = k_cache.shape[0]
    if out is None:
        out = torch.empty_like(q)
    _dev(out, "out", dt)
    ws = _workspace(prefill_attention_workspace_bytes(n_sel, n_tok, n_q_heads, n_kv_heads, head_dim, dt),
                    workspace, q)
    if plan is None:
        _call("semshare_prefill_attention", _ptr(q), _ptr(sel_pos), n_sel, _ptr(k_cache), _ptr(v_cache), n_tok,
              n_q_heads, n_kv_heads, head_dim, float(sm_scale), _ptr(out), _ptr(ws), 0 if ws is None else ws.numel(),
              _dt(q), _stream())
    else:
        _dev(plan, "plan", torch.uint8)
        _call("semshare_prefill_attention_planned", _ptr(plan), plan.numel(), _ptr(q), _ptr(sel_pos), n_sel,
              _ptr(k_cache), _ptr(v_cache), n_tok, n_q_heads, n_kv_heads, head_dim, float(sm_scale), _ptr(out),
              _ptr(ws), 0 if ws is None else ws.numel(), _dt(q), _stream())
    return out


def prefill_attention_noalloc(q: torch.Tensor, sel_pos: torch.Tensor, k_cache: torch.Tensor, v_cache: torch.Tensor,
                              n_kv_heads: int, sm_scale: float = 0.0,
                              out: Optional[torch.Tensor] = None) -> torch.Tensor:
    """prefill_attention with no workspace: the library's static device scratch holds the plan and the
    partial results (calls on one GPU must not overlap)."""
    _dev(q, "q")
    dt = q.dtype
    _dev(sel_pos, "sel_pos", torch.int32)
    _dev(k_cache, "k_cache", dt)
    _dev(v_cache, "v_cache", dt)
    n_sel, n_q_heads, head_dim = q.shape
    n_tok = k_cache.shape[0]
    if k_cache.numel() != n_tok * n_kv_heads * head_dim or v_cache.shape != k_cache.shape:
        raise ValueError("caches must be [n_tok, n_kv_heads, head_dim]")
    if out is None:
        out = torch.empty_like(q)
    _dev(out, "out", dt)
    _call("semshare_prefill_attention_noalloc", _ptr(q), _ptr(sel_pos), n_sel, _ptr(k_cache), _ptr(v_cache), n_tok,
          n_q_heads, n_kv_heads, head_dim, float(sm_scale), _ptr(out), _dt(q), _stream())
    return out


def select_recompute_nested(sigma: torch.Tensor, cand_pos: torch.Tensor, n_sel: int,
                            out: Optional[torch.Tensor] = None) -> torch.Tensor:
    """The n_sel candidates (positions cand_pos, deviations sigma) of largest deviation (ties: lower
    position), their positions ascending: a later layer's recompute set drawn from the previous one's."""
    _dev(sigma, "sigma", torch.float32)
    _dev(cand_pos, "cand_pos", torch.int32)
    if cand_pos.numel() != sigma.numel():
        raise ValueError("sigma and cand_pos must have one entry per candidate")
    if out is None:
        out = torch.empty(n_sel, dtype=torch.int32, device=sigma.device)
    _dev(out, "out", torch.int32)
    _call("semshare_select_recompute_nested", _ptr(sigma), _ptr(cand_pos), sigma.numel(), int(n_sel), _ptr(out),
          _stream())
    return out


def retention_layer(rank: torch.Tensor, n_retain: int, sel_pos: torch.Tensor, idx: Optional[torch.Tensor] = None):
    """Kept positions of a later layer (rank < n_retain, plus the recomputed sel_pos), ascending; the
    reference row each compacted row copies (with idx); the recomputed tokens' rows in the compacted cache.
    Returns (kept_pos [n_tok] (first n_kept valid), src_idx [n_tok] or None, sel_rows [n_sel], n_kept [1]),
    all on the device."""
    _dev(rank, "rank", torch.int32)
    _dev(sel_pos, "sel_pos", torch.int32)
    n_tok, n_sel = rank.numel(), sel_pos.numel()
    kept = torch.empty(max(n_tok, 1), dtype=torch.int32, device=rank.device)
    src = None
    if idx is not None:
        _dev(idx, "idx", torch.int32)
        if idx.numel() < n_tok:
            raise ValueError("idx needs one entry per position")
        src = torch.empty(max(n_tok, 1), dtype=torch.int32, device=rank.device)
    rows = torch.empty(max(n_sel, 1), dtype=torch.int32, device=rank.device)
    n_kept = torch.empty(1, dtype=torch.int32, device=rank.device)
    _call("semshare_retention_layer", _ptr(rank), n_tok, int(n_retain), _ptr(sel_pos), n_sel, _ptr(idx), _ptr(kept),
          _ptr(src), _ptr(rows), _ptr(n_kept), _stream())
    return kept, src, rows[:n_sel], n_kept


def select_recompute(sigma: torch.Tensor, n_sel: int, out: Optional[torch.Tensor] = None) -> torch.Tensor:
    """The n_sel positions of largest deviation (ties: lower position), ascending."""
    _dev(sigma, "sigma", torch.float32)
    if out is None:
        out = torch.empty(n_sel, dtype=torch.int32, device=sigma.device)
    _dev(out, "out", torch.int32)
    _call("semshare_select_recompute", _ptr(sigma), sigma.numel(), int(n_sel), _ptr(out), _stream())
    return out
