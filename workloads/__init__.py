"""Seeded synthetic inputs shaped like the paper's workloads.

This module only draws random numbers and lays them out.  It holds none of
the method's arithmetic: no RoPE, no hashing, no matching, no attention.  Both
the CPU oracle and the HIP path are fed from here, so that each side receives
the same bits.

Recipe (the paper's datasets -- MultiNews and friends, Section 5.1 -- are not
available, so these prompts stand in for its "semantically similar prompt
pairs", Section 3 and Appendix B):

* Reference embeddings E_ref ~ N(0, 1), shape [T_ref, d].
* Target embeddings: round(rho_fresh * T) positions, chosen uniformly without
  replacement, are fresh N(0, 1) rows.  Every other row t copies
  E_ref[pi(t)] and adds noise (sigma * ||E_ref[pi(t)]|| / sqrt(d)) * z with
  z ~ N(0, I); pi shuffles uniformly within each aligned window of 16 tokens
  (the last, possibly shorter, window is shuffled within itself).
* Random hyperplanes for the sign-bit LSH: N(0, 1) entries scaled by
  d**-0.5, so every plane has norm close to 1.
* Per-layer projection weights Wq, Wk, Wv ~ N(0, 0.02) in nn.Linear layout
  [out_features, in_features].
* bf16 configurations round every generated array to bf16 (round to nearest
  even) before either side sees it; arrays are returned as float32 numpy
  arrays whose values are exactly representable in the storage dtype.

Seeds: numpy PCG64 seeded with [1000 + config id, stream tag]; every array
has its own stream tag, so arrays are independent of each other and of the
order in which they are drawn.
"""
from __future__ import annotations

import dataclasses
import math
from typing import Dict, List, Optional, Tuple

import numpy as np

# Stream tags (one independent PCG64 stream per array kind).
_TAG_REF = 1
_TAG_PERM = 2
_TAG_FRESH_POS = 3
_TAG_NOISE = 4
_TAG_FRESH_VAL = 5
_TAG_PLANES = 6
_TAG_CACHE = 7
_TAG_SEL = 8
_TAG_X = 9
_TAG_BANK = 10
_TAG_WEIGHTS = 1000  # + layer index


@dataclasses.dataclass(frozen=True)
class Config:
    """One workload shape. Field names follow the paper's notation."""

    cid: int
    name: str
    dtype: str  # "fp32" | "bf16"
    n_tok: int  # tokens in the target prompt (and in each reference prompt)
    dim: int  # embedding dim d (= hidden size of the attention layer)
    n_bits: int  # LSH code length
    n_layers: int
    n_q_heads: int
    n_kv_heads: int
    head_dim: int
    recompute_fracs: Tuple[float, ...]
    noise_sigma: float
    fresh_frac: float
    n_refs: int = 1  # reference prompts in the bank
    bank_sigmas: Tuple[float, ...] = ()
    window: int = 16
    rope_base: float = 10000.0

    @property
    def n_words(self) -> int:
        return self.n_bits // 64

    @property
    def group(self) -> int:
        return self.n_q_heads // self.n_kv_heads

    def n_sel(self, frac: float) -> int:
        """Number of recomputed tokens: floor(f * T + 1/2)."""
        return int(math.floor(frac * self.n_tok + 0.5))

    def seed(self, tag: int) -> np.random.Generator:
        return np.random.default_rng([1000 + self.cid, tag])


CONFIGS: Dict[int, Config] = {
    0: Config(0, "tiny-fp32", "fp32", 512, 256, 64, 2, 4, 4, 64, (0.20,), 0.3, 0.20),
    1: Config(1, "llama3-8b-1layer-1k", "bf16", 1024, 4096, 128, 1, 32, 8, 128, (0.25,), 0.3, 0.20),
    2: Config(2, "llama3-8b-32layer-5k", "bf16", 5120, 4096, 128, 32, 32, 8, 128, (0.10, 0.25, 0.50), 0.3, 0.15),
    3: Config(3, "bank-16x4k", "bf16", 4096, 4096, 256, 32, 32, 8, 128, (), 0.0, 0.0,
              n_refs=16, bank_sigmas=(0.2, 0.4, 0.6)),
    4: Config(4, "llama3-8b-32layer-32k", "bf16", 32768, 4096, 128, 32, 32, 8, 128, (0.10,), 0.3, 0.20),
}


def round_bf16(a: np.ndarray) -> np.ndarray:
    """Round float32 values to the nearest bf16 (ties to even); float32 out."""
    a = np.ascontiguousarray(a, dtype=np.float32)
    u = a.view(np.uint32).astype(np.uint64)
    u = ((u + np.uint64(0x7FFF) + ((u >> np.uint64(16)) & np.uint64(1))) >> np.uint64(16)) << np.uint64(16)
    return u.astype(np.uint32).view(np.float32).reshape(a.shape)


def to_storage(a: np.ndarray, dtype: str) -> np.ndarray:
    if dtype == "bf16":
        return round_bf16(a)
    if dtype == "fp32":
        return np.ascontiguousarray(a, dtype=np.float32)
    raise ValueError(f"unknown dtype {dtype!r}")


def _normal(rng: np.random.Generator, shape) -> np.ndarray:
    return rng.standard_normal(size=shape, dtype=np.float32)


def window_permutation(n: int, window: int, rng: np.random.Generator) -> np.ndarray:
    """pi: a uniform shuffle inside each aligned window of `window` positions."""
    pi = np.arange(n, dtype=np.int64)
    for w0 in range(0, n, window):
        w1 = min(n, w0 + window)
        pi[w0:w1] = w0 + rng.permutation(w1 - w0)
    return pi


@dataclasses.dataclass
class PromptPair:
    e_ref: np.ndarray  # [T_ref, d] float32 (storage-dtype values)
    e_tgt: np.ndarray  # [T_tgt, d]
    pi: np.ndarray  # [T_tgt] int64: source reference row of each copied token (-1 if fresh)


def make_prompt_pair(cfg: Config, n_tok: Optional[int] = None, dim: Optional[int] = None,
                     noise_sigma: Optional[float] = None, fresh_frac: Optional[float] = None) -> PromptPair:
    """Reference/target embedding pair per the module recipe."""
    T = cfg.n_tok if n_tok is None else n_tok
    d = cfg.dim if dim is None else dim
    sigma = cfg.noise_sigma if noise_sigma is None else noise_sigma
    rho = cfg.fresh_frac if fresh_frac is None else fresh_frac
    e_ref = _normal(cfg.seed(_TAG_REF), (T, d))
    pi = window_permutation(T, cfg.window, cfg.seed(_TAG_PERM))
    n_fresh = int(round(rho * T))
    fresh = cfg.seed(_TAG_FRESH_POS).choice(T, size=n_fresh, replace=False)
    src = e_ref[pi]
    scale = sigma * np.linalg.norm(src, axis=1, keepdims=True) / np.float32(math.sqrt(d))
    e_tgt = src + scale.astype(np.float32) * _normal(cfg.seed(_TAG_NOISE), (T, d))
    if n_fresh:
        e_tgt[fresh] = _normal(cfg.seed(_TAG_FRESH_VAL), (n_fresh, d))
    pi_out = pi.copy()
    pi_out[fresh] = -1
    return PromptPair(to_storage(e_ref, cfg.dtype), to_storage(e_tgt, cfg.dtype), pi_out)


@dataclasses.dataclass
class Bank:
    e_refs: np.ndarray  # [n_refs * T, d]: the bank, reference b occupying rows [b*T, (b+1)*T)
    e_tgt: np.ndarray  # [T, d]
    sigmas: List[float]


def make_bank(cfg: Config, n_tok: Optional[int] = None, dim: Optional[int] = None,
              n_refs: Optional[int] = None) -> Bank:
    """Many-reference bank: a common sequence C ~ N(0,1); reference b is C plus
    relative noise of sigma_b = bank_sigmas[b mod 3]; the target is C itself."""
    T = cfg.n_tok if n_tok is None else n_tok
    d = cfg.dim if dim is None else dim
    nb = cfg.n_refs if n_refs is None else n_refs
    c = _normal(cfg.seed(_TAG_REF), (T, d))
    norm = np.linalg.norm(c, axis=1, keepdims=True) / np.float32(math.sqrt(d))
    refs = np.empty((nb * T, d), dtype=np.float32)
    sig = []
    for b in range(nb):
        s = cfg.bank_sigmas[b % len(cfg.bank_sigmas)]
        sig.append(s)
        z = _normal(cfg.seed(_TAG_BANK + 100 * (b + 1)), (T, d))
        refs[b * T:(b + 1) * T] = c + (np.float32(s) * norm) * z
    return Bank(to_storage(refs, cfg.dtype), to_storage(c, cfg.dtype), sig)


def make_planes(cfg: Config, n_bits: Optional[int] = None, dim: Optional[int] = None) -> np.ndarray:
    """Random hyperplanes [n_bits, d] (row j = plane j), entries N(0,1)/sqrt(d)."""
    nb = cfg.n_bits if n_bits is None else n_bits
    d = cfg.dim if dim is None else dim
    r = _normal(cfg.seed(_TAG_PLANES), (nb, d)) * np.float32(1.0 / math.sqrt(d))
    return to_storage(r, cfg.dtype)


@dataclasses.dataclass
class LayerWeights:
    wq: np.ndarray  # [Hq*D, hidden]
    wk: np.ndarray  # [Hkv*D, hidden]
    wv: np.ndarray  # [Hkv*D, hidden]


def make_weights(cfg: Config, layer: int, hidden: Optional[int] = None, n_q_heads: Optional[int] = None,
                 n_kv_heads: Optional[int] = None, head_dim: Optional[int] = None,
                 std: float = 0.02) -> LayerWeights:
    h = cfg.dim if hidden is None else hidden
    hq = cfg.n_q_heads if n_q_heads is None else n_q_heads
    hkv = cfg.n_kv_heads if n_kv_heads is None else n_kv_heads
    dd = cfg.head_dim if head_dim is None else head_dim
    rng = cfg.seed(_TAG_WEIGHTS + layer)
    wq = _normal(rng, (hq * dd, h)) * np.float32(std)
    wk = _normal(rng, (hkv * dd, h)) * np.float32(std)
    wv = _normal(rng, (hkv * dd, h)) * np.float32(std)
    return LayerWeights(to_storage(wq, cfg.dtype), to_storage(wk, cfg.dtype), to_storage(wv, cfg.dtype))


def make_cache(cfg: Config, n_layers: int, n_tok: int, n_kv_heads: Optional[int] = None,
               head_dim: Optional[int] = None, tag: int = 0, scale: float = 1.0) -> Tuple[np.ndarray, np.ndarray]:
    """A synthetic post-RoPE K/V cache [L, T, Hkv, D] (N(0, scale^2) values),
    standing in for a reference prompt's cache where its exact origin is
    irrelevant to the step under test."""
    hkv = cfg.n_kv_heads if n_kv_heads is None else n_kv_heads
    dd = cfg.head_dim if head_dim is None else head_dim
    rng = cfg.seed(_TAG_CACHE + 100 * (tag + 1))
    k = _normal(rng, (n_layers, n_tok, hkv, dd)) * np.float32(scale)
    v = _normal(rng, (n_layers, n_tok, hkv, dd)) * np.float32(scale)
    return to_storage(k, cfg.dtype), to_storage(v, cfg.dtype)


def make_rows(cfg: Config, n_rows: int, width: int, tag: int = 0, scale: float = 1.0) -> np.ndarray:
    """Generic N(0, scale^2) rows in the config's storage dtype."""
    x = _normal(cfg.seed(_TAG_X + 100 * (tag + 1)), (n_rows, width)) * np.float32(scale)
    return to_storage(x, cfg.dtype)


def make_sel_pos(cfg: Config, n_tok: int, n_sel: int, tag: int = 0, include_ends: bool = True) -> np.ndarray:
    """A strictly ascending set of n_sel positions in [0, n_tok) (int32)."""
    if n_sel > n_tok:
        raise ValueError("n_sel > n_tok")
    rng = cfg.seed(_TAG_SEL + 100 * (tag + 1))
    if n_sel == n_tok:
        return np.arange(n_tok, dtype=np.int32)
    if include_ends and n_sel >= 2:
        inner = rng.choice(np.arange(1, n_tok - 1), size=n_sel - 2, replace=False)
        pos = np.concatenate([[0, n_tok - 1], inner])
    else:
        pos = rng.choice(n_tok, size=n_sel, replace=False)
    return np.sort(pos).astype(np.int32)


def make_codes(cfg: Config, n_rows: int, n_words: int, tag: int = 0) -> np.ndarray:
    """Uniformly random u64 code words [n_rows, n_words]."""
    rng = cfg.seed(_TAG_X + 100 * (tag + 1) + 7)
    return rng.integers(0, 2**64, size=(n_rows, n_words), dtype=np.uint64)
