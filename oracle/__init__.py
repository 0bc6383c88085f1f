"""CPU oracle of the SemShareKV hot path -- TEST INFRASTRUCTURE ONLY.

Python face of ``oracle.c`` (plain C, fp64, optional OpenMP over rows).  Only
the test suite, ``__graft_entry__.smoke()`` and the benchmark's CPU-baseline
leg may import this package.  The product library never calls it and shares
no code with it.

Every function takes numpy arrays holding exact storage-dtype values (float32
arrays are fine: they are widened to fp64 without change) and returns fp64
arrays whose values are rounded to ``dtype`` where the product path stores
them ("bf16", "fp32", or "f64" for no rounding).
"""
from __future__ import annotations

import ctypes
import os
import subprocess
from fractions import Fraction
from typing import Optional, Tuple

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "oracle.c")
_LIB_PATH = os.path.join(_HERE, "liboracle.so")
_DT = {"fp32": 0, "bf16": 1, "f64": 2}

_lib: Optional[ctypes.CDLL] = None


def build(verbose: bool = False) -> str:
    """Compile oracle.c into liboracle.so next to it (gcc, IEEE fp64, no FMA
    contraction, OpenMP)."""
    cmd = ["gcc", "-O2", "-std=c11", "-fPIC", "-shared", "-fopenmp", "-ffp-contract=off",
           "-fno-fast-math", "-Wall", "-Wextra", "-o", _LIB_PATH + ".tmp", _SRC, "-lm"]
    if verbose:
        print(" ".join(cmd))
    subprocess.run(cmd, check=True)
    os.replace(_LIB_PATH + ".tmp", _LIB_PATH)
    return _LIB_PATH


def _load() -> ctypes.CDLL:
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(_LIB_PATH) or os.path.getmtime(_LIB_PATH) < os.path.getmtime(_SRC):
        build()
    lib = ctypes.CDLL(_LIB_PATH)
    P = ctypes.c_void_p
    I64, I32, F64, INT = ctypes.c_int64, ctypes.c_int32, ctypes.c_double, ctypes.c_int
    sig = {
        "orc_round_array": (None, [P, P, I64, INT]),
        "orc_rope_embed": (None, [P, P, I64, I32, I64, F64, INT]),
        "orc_lsh_project": (None, [P, P, P, I64, I32, I32]),
        "orc_lsh_encode": (None, [P, P, P, I64, I32, I32]),
        "orc_match": (None, [P, I64, P, I64, I32, P, P]),
        "orc_gather_rows": (None, [P, P, I64, I64, P, I32, I64]),
        "orc_qkv_rows": (None, [P, P, I64, P, P, P, I32, I32, I32, I32, F64, P, P, P, INT]),
        "orc_deviation": (None, [P, P, P, I64, P, P, I32, P]),
        "orc_attention_rows": (None, [P, P, I64, P, I64, P, P, I32, I32, I32, F64, P, INT, P]),
        "orc_partial_prefill": (None, [P, P, I64, P, P, P, P, P, I64, I32, I32, I32, I32, F64, F64,
                                       P, P, INT]),
        "orc_select_recompute": (None, [P, I64, I64, P]),
        "orc_attention_mass": (None, [P, P, I64, I32, I32, I32, F64, I64, P, I64, P]),
        "orc_similarity": (F64, [P, I64, F64, F64]),
        "orc_bank_similarity": (None, [P, I64, P, P, INT, INT, F64, F64, P, P]),
        "orc_num_threads": (INT, []),
        "orc_set_num_threads": (None, [INT]),
    }
    for name, (res, args) in sig.items():
        fn = getattr(lib, name)
        fn.restype = res
        fn.argtypes = args
    _lib = lib
    return lib


def _f64(a) -> np.ndarray:
    return np.ascontiguousarray(a, dtype=np.float64)


def _ptr(a: Optional[np.ndarray]):
    return None if a is None else a.ctypes.data_as(ctypes.c_void_p)


def num_threads() -> int:
    return int(_load().orc_num_threads())


def set_num_threads(n: int) -> None:
    _load().orc_set_num_threads(int(n))


def round_to(x, dtype: str) -> np.ndarray:
    x = _f64(x)
    y = np.empty_like(x)
    _load().orc_round_array(_ptr(x), _ptr(y), x.size, _DT[dtype])
    return y


def rope_embed(x, pos0: int = 0, base: float = 10000.0, dtype: str = "f64") -> np.ndarray:
    """RoPE of every row of x [n_tok, d]; row r sits at position pos0 + r."""
    x = _f64(x)
    n, d = x.shape
    if d % 2:
        raise ValueError("dim must be even")
    y = np.empty_like(x)
    _load().orc_rope_embed(_ptr(x), _ptr(y), n, d, int(pos0), float(base), _DT[dtype])
    return y


def lsh_project(x, planes) -> np.ndarray:
    x, planes = _f64(x), _f64(planes)
    n, d = x.shape
    nb = planes.shape[0]
    p = np.empty((n, nb), dtype=np.float64)
    _load().orc_lsh_project(_ptr(x), _ptr(planes), _ptr(p), n, d, nb)
    return p


def lsh_encode(x, planes) -> np.ndarray:
    """Sign-bit codes [n_tok, n_bits/64] uint64."""
    x, planes = _f64(x), _f64(planes)
    n, d = x.shape
    nb = planes.shape[0]
    if nb % 64:
        raise ValueError("n_bits must be a multiple of 64")
    c = np.empty((n, nb // 64), dtype=np.uint64)
    _load().orc_lsh_encode(_ptr(x), _ptr(planes), _ptr(c), n, d, nb)
    return c


def match(tgt_codes, ref_codes) -> Tuple[np.ndarray, np.ndarray]:
    """Top-1 Hamming match: (idx int32 [n_tgt], dist int32 [n_tgt])."""
    t = np.ascontiguousarray(tgt_codes, dtype=np.uint64)
    r = np.ascontiguousarray(ref_codes, dtype=np.uint64)
    if t.ndim != 2 or r.ndim != 2 or t.shape[1] != r.shape[1]:
        raise ValueError("codes must be [n, n_words] with equal n_words")
    idx = np.empty(t.shape[0], dtype=np.int32)
    dist = np.empty(t.shape[0], dtype=np.int32)
    _load().orc_match(_ptr(t), t.shape[0], _ptr(r), r.shape[0], t.shape[1], _ptr(idx), _ptr(dist))
    return idx, dist


def gather_rows(src: np.ndarray, idx) -> np.ndarray:
    """src [L, n_ref, ...] -> [L, n_tgt, ...] with row t = src[:, idx[t]] (bytewise)."""
    src = np.ascontiguousarray(src)
    idx = np.ascontiguousarray(idx, dtype=np.int32)
    L, n_ref = src.shape[:2]
    row_bytes = src[0, 0].nbytes if n_ref else 0
    if idx.size and (idx.min() < 0 or idx.max() >= n_ref):
        raise ValueError("index out of range")
    dst = np.empty((L, idx.size) + src.shape[2:], dtype=src.dtype)
    _load().orc_gather_rows(_ptr(src), _ptr(idx), idx.size, n_ref, _ptr(dst), L, row_bytes)
    return dst


def qkv_rows(x_sel, sel_pos, wq, wk, wv, n_q_heads: int, n_kv_heads: int, head_dim: int,
             base: float = 10000.0, dtype: str = "f64", want_q: bool = True, want_kv: bool = True):
    """Recomputed (q, k, v) rows; q or (k, v) is None when not wanted."""
    x = _f64(x_sel)
    pos = np.ascontiguousarray(sel_pos, dtype=np.int32)
    wq = _f64(wq) if want_q else None
    wk, wv = (_f64(wk), _f64(wv)) if want_kv else (None, None)
    n, hidden = x.shape
    q = np.empty((n, n_q_heads * head_dim)) if want_q else None
    k = np.empty((n, n_kv_heads * head_dim)) if want_kv else None
    v = np.empty((n, n_kv_heads * head_dim)) if want_kv else None
    _load().orc_qkv_rows(_ptr(x), _ptr(pos), n, _ptr(wq), _ptr(wk), _ptr(wv), hidden, n_q_heads,
                         n_kv_heads, head_dim, float(base), _ptr(q), _ptr(k), _ptr(v), _DT[dtype])
    return q, k, v


def deviation(k_cache, v_cache, sel_pos, k_new, v_new) -> np.ndarray:
    kc, vc = _f64(k_cache), _f64(v_cache)
    kn, vn = _f64(k_new), _f64(v_new)
    pos = np.ascontiguousarray(sel_pos, dtype=np.int32)
    row = kn.shape[1]
    sig = np.empty(pos.size)
    _load().orc_deviation(_ptr(kc), _ptr(vc), _ptr(pos), pos.size, _ptr(kn), _ptr(vn), row, _ptr(sig))
    return sig


def attention_rows(q, sel_pos, k_cache, v_cache, n_q_heads: int, n_kv_heads: int, head_dim: int,
                   scale: float = 0.0, dtype: str = "f64", rows=None, keep=None) -> np.ndarray:
    """Causal attention of selected rows over a cache [n_tok, Hkv*D].
    Returns [n_sel, Hq*D]; with ``rows`` only those rows are computed (others NaN).
    With ``keep`` (bool per cache position) only kept positions are attended
    (the cache after retention, Section 4.3.4)."""
    q = _f64(q)
    pos = np.ascontiguousarray(sel_pos, dtype=np.int32)
    kc = _f64(k_cache).reshape(-1, n_kv_heads * head_dim)
    vc = _f64(v_cache).reshape(-1, n_kv_heads * head_dim)
    if scale <= 0:
        scale = 1.0 / np.sqrt(head_dim)
    out = np.full((pos.size, n_q_heads * head_dim), np.nan)
    r = None if rows is None else np.ascontiguousarray(rows, dtype=np.int64)
    kp = None
    if keep is not None:
        kp = np.ascontiguousarray(keep, dtype=np.uint8)
        if kp.size != kc.shape[0]:
            raise ValueError("keep needs one entry per cache position")
    _load().orc_attention_rows(_ptr(q), _ptr(pos), pos.size, _ptr(r), 0 if r is None else r.size,
                               _ptr(kc), _ptr(vc), n_q_heads, n_kv_heads, head_dim, float(scale),
                               _ptr(out), _DT[dtype], _ptr(kp))
    return out


def partial_prefill(x_sel, sel_pos, wq, wk, wv, k_cache, v_cache, n_q_heads: int, n_kv_heads: int,
                    head_dim: int, base: float = 10000.0, scale: float = 0.0, dtype: str = "f64",
                    want_out: bool = True, want_sigma: bool = False):
    """One layer of partial prefill.  k_cache/v_cache [n_tok, Hkv*D] (or
    [n_tok, Hkv, D]) are not modified; the updated caches are returned.
    Returns (out [n_sel, Hq*D] or None, sigma [n_sel] or None, k_cache', v_cache')."""
    x = _f64(x_sel)
    pos = np.ascontiguousarray(sel_pos, dtype=np.int32)
    wq, wk, wv = _f64(wq), _f64(wk), _f64(wv)
    kc = _f64(k_cache).reshape(-1, n_kv_heads * head_dim).copy()
    vc = _f64(v_cache).reshape(-1, n_kv_heads * head_dim).copy()
    n, hidden = x.shape
    out = np.empty((n, n_q_heads * head_dim)) if want_out else None
    sig = np.empty(n) if want_sigma else None
    _load().orc_partial_prefill(_ptr(x), _ptr(pos), n, _ptr(wq), _ptr(wk), _ptr(wv), _ptr(kc),
                                _ptr(vc), kc.shape[0], hidden, n_q_heads, n_kv_heads, head_dim,
                                float(base), float(scale), _ptr(out), _ptr(sig), _DT[dtype])
    return out, sig, kc, vc


def select_recompute(sigma, n_sel: int) -> np.ndarray:
    s = _f64(sigma)
    if not 0 <= n_sel <= s.size:
        raise ValueError("n_sel out of range")
    pos = np.empty(n_sel, dtype=np.int32)
    _load().orc_select_recompute(_ptr(s), s.size, n_sel, _ptr(pos))
    return pos


def select_recompute_nested(sigma, cand_pos, n_sel: int) -> np.ndarray:
    """A later layer's recompute set drawn from the previous layer's (Section
    4.3.3, Appendix A.5): of the candidates cand_pos (ascending positions) with
    deviations sigma, the n_sel of largest deviation, lower position first on
    ties; their positions ascending."""
    cand = np.ascontiguousarray(cand_pos, dtype=np.int64)
    if cand.size != np.size(sigma):
        raise ValueError("one deviation per candidate")
    return cand[select_recompute(sigma, n_sel)].astype(np.int32)


def retention_layer(rank, n_retain: int, sel_pos, idx=None):
    """Retention on a later layer (Section 4.3.4, Appendix A.6): the positions
    with first-layer rank below n_retain plus the recomputed sel_pos (never
    evicted), ascending; the reference rows they copy (idx[kept]); the rows of
    sel_pos in the compacted cache.  Returns (kept, src_idx or None, sel_rows)."""
    rank = np.asarray(rank, dtype=np.int64)
    keep = (rank >= 0) & (rank < n_retain)
    sel = np.asarray(sel_pos, dtype=np.int64)
    keep[sel[(sel >= 0) & (sel < rank.size)]] = True
    kept = np.flatnonzero(keep)
    row_of = np.full(rank.size, -1, dtype=np.int64)
    row_of[kept] = np.arange(kept.size)
    rows = np.array([row_of[p] if 0 <= p < rank.size else -1 for p in sel], dtype=np.int64)
    src = None if idx is None else np.asarray(idx, dtype=np.int64)[kept]
    return kept, src, rows


def bank_similarity(tgt_codes, ref_codes, offsets, dmin: float = 0.0, dmax: float = 30.0):
    """Per reference prompt of a bank (codes [offsets[b], offsets[b+1]) of ref_codes): the sum of the
    target tokens' top-1 Hamming distances within that prompt (int64) and its similarity score (fp64)."""
    t = np.ascontiguousarray(tgt_codes, dtype=np.uint64)
    r = np.ascontiguousarray(ref_codes, dtype=np.uint64)
    off = np.ascontiguousarray(offsets, dtype=np.int64)
    if t.ndim != 2 or r.ndim != 2 or t.shape[1] != r.shape[1]:
        raise ValueError("codes must be [n, n_words] with equal n_words")
    n_prompts = off.size - 1
    if n_prompts < 0 or (n_prompts > 0 and (off[0] < 0 or off[-1] > r.shape[0] or np.any(np.diff(off) < 0))):
        raise ValueError("offsets must ascend within the bank")
    dsum = np.empty(max(n_prompts, 0), dtype=np.int64)
    sim = np.empty(max(n_prompts, 0), dtype=np.float64)
    _load().orc_bank_similarity(_ptr(t), t.shape[0], _ptr(r), _ptr(off), n_prompts, t.shape[1], float(dmin),
                                float(dmax), _ptr(dsum), _ptr(sim))
    return dsum, sim


def similarity(dist, dmin: float = 0.0, dmax: float = 30.0) -> float:
    d = np.ascontiguousarray(dist, dtype=np.int32)
    return float(_load().orc_similarity(_ptr(d), d.size, float(dmin), float(dmax)))


def attention_mass(q, k_cache, n_q_heads: int, n_kv_heads: int, head_dim: int, sm_scale: float = 0.0,
                   row_begin: int = 0) -> np.ndarray:
    """Average attention score of every token at a fully computed layer
    (Section 3, Insight 2): the causal softmax attention of each head, averaged
    over the heads and then over the query rows (the first dimension) from
    row_begin on (Section 4.3.4 ranks retention by the last rows).  fp64; one
    T x T score matrix per head (numpy matmul as the product step)."""
    q = _f64(q).reshape(q.shape[0], n_q_heads, head_dim)
    k = _f64(k_cache).reshape(k_cache.shape[0], n_kv_heads, head_dim)
    T = q.shape[0]
    scale = sm_scale if sm_scale else 1.0 / np.sqrt(head_dim)
    G = n_q_heads // n_kv_heads
    causal = np.tril(np.ones((T, T), dtype=bool))
    total = np.zeros(T)
    for h in range(n_q_heads):
        s = (q[:, h, :] @ k[:, h // G, :].T) * scale
        s = np.where(causal, s, -np.inf)
        p = np.exp(s - s.max(axis=1, keepdims=True))
        p /= p.sum(axis=1, keepdims=True)
        total += p[row_begin:].sum(axis=0)
    return total / (n_q_heads * (T - row_begin))


def attention_mass_cols(q, k_cache, n_q_heads: int, n_kv_heads: int, head_dim: int, sm_scale: float = 0.0,
                        row_begin: int = 0, cols=None) -> np.ndarray:
    """attention_mass (same definition, plain C loops in fp64) for the key
    columns ``cols`` only (all keys when None): every row's softmax
    normaliser first, then the requested column sums."""
    T = q.shape[0]
    q = _f64(q).reshape(T, n_q_heads * head_dim)
    k = _f64(k_cache).reshape(T, n_kv_heads * head_dim)
    scale = sm_scale if sm_scale else 1.0 / np.sqrt(head_dim)
    if not 0 <= row_begin < max(T, 1):
        raise ValueError("row_begin must lie in [0, T)")
    c = None if cols is None else np.ascontiguousarray(cols, dtype=np.int64)
    if c is not None and c.size and (c.min() < 0 or c.max() >= T):
        raise ValueError("column out of range")
    out = np.empty(T if c is None else c.size)
    _load().orc_attention_mass(_ptr(q), _ptr(k), T, n_q_heads, n_kv_heads, head_dim, float(scale), int(row_begin),
                               _ptr(c), 0 if c is None else c.size, _ptr(out))
    return out


def _exact_units(m32: np.ndarray) -> list:
    """Every fp32 value is an integer multiple of 2^-149 (the smallest
    subnormal); these integers make every sum of masses exact."""
    out = []
    for v in m32.tolist():
        num, den = float(v).as_integer_ratio()
        out.append(num * ((1 << 149) // den))
    return out


def attention_recovery(mass, thres: float = 0.55) -> Tuple[int, np.ndarray]:
    """Attention Recovery (Section 3, Insight 2 equation): the tokens ordered by
    mass, largest first (lower position first on ties); AR is the smallest k >= 1
    whose top-k mass reaches thres of the total.  The sums and the comparison
    are exact (integers in units of 2^-149 and the exact rational value of
    thres), so the answer is the plain definition on the given fp32 masses.
    Masses must be finite and in [0, 1] (averages of probabilities).
    Returns (AR, order)."""
    m32 = np.asarray(mass, dtype=np.float32)
    n = m32.shape[0]
    if n == 0:
        return 0, np.zeros(0, dtype=np.int64)
    if not np.all(np.isfinite(m32)) or np.any(m32 < 0) or np.any(m32 > 1):
        raise ValueError("masses must be finite and lie in [0, 1]")
    order = np.array(sorted(range(n), key=lambda j: (-float(m32[j]), j)), dtype=np.int64)
    units = _exact_units(m32)
    p, q = Fraction(thres).as_integer_ratio()
    total = sum(units)
    run = 0
    for k, j in enumerate(order.tolist(), start=1):
        run += units[j]
        if run * q >= p * total:  # run >= thres * total, exactly
            return k, order
    return n, order


def dynamic_recompute(mass, sigma, thres: float = 0.55, w_hot: float = 0.5,
                      w_cold: float = 0.1, ar: Optional[int] = None) -> Tuple[int, np.ndarray, int]:
    """Dynamic recompute set (Section 4.3.3): the AR first tokens by mass are
    hot, the rest cold; floor(w_hot AR + 1/2) hot and floor(w_cold (T - AR) + 1/2)
    cold tokens with the largest deviation (lower position first on ties) are
    recomputed.  ``ar`` replaces the computed AR (to follow another valid
    reading of a tie at the threshold).  Returns (AR, selected positions
    ascending, hot count chosen)."""
    ar_exact, order = attention_recovery(mass, thres)
    ar = ar_exact if ar is None else int(ar)
    n = len(order)
    sig = np.maximum(np.asarray(sigma, dtype=np.float32), np.float32(0))
    hot = set(int(j) for j in order[:ar])
    n_hot = int(np.floor(w_hot * ar + 0.5))
    n_cold = int(np.floor(w_cold * (n - ar) + 0.5))
    by_sigma = lambda js: sorted(js, key=lambda j: (-float(sig[j]), j))
    chosen = by_sigma([j for j in range(n) if j in hot])[:n_hot] + by_sigma([j for j in range(n) if j not in hot])[:n_cold]
    return ar, np.array(sorted(chosen), dtype=np.int64), n_hot


def retention(mass, score, ar: int, sel_pos, min_keep: float = 0.8) -> Tuple[np.ndarray, np.ndarray, int]:
    """First-layer retention (Section 4.3.4): hot tokens (the ar first by mass)
    and recomputed tokens are never evicted and rank first in position order;
    the others follow by score, largest first (lower position first on ties).
    The first max(floor(max(min_keep, ar / T) T + 1/2), never-evicted) are kept.
    Returns (rank of every position, kept positions ascending, count kept)."""
    n = len(mass)
    _, order = attention_recovery(mass)
    forced = set(int(j) for j in order[:ar]) | set(int(j) for j in sel_pos)
    sc = np.maximum(np.asarray(score, dtype=np.float32), np.float32(0))
    rest = sorted((j for j in range(n) if j not in forced), key=lambda j: (-float(sc[j]), j))
    ranking = sorted(forced) + rest
    ratio = ar / n if n and ar / n > min_keep else min_keep
    keep = min(max(int(np.floor(ratio * n + 0.5)), len(forced)), n)
    rank = np.empty(n, dtype=np.int64)
    rank[np.array(ranking, dtype=np.int64)] = np.arange(n)
    return rank, np.array(sorted(ranking[:keep]), dtype=np.int64), keep
