"""Shared helpers for the GPU parity tests: moving generator/oracle values
to and from device tensors, and the comparison rules."""
from __future__ import annotations

import sys

import numpy as np
import torch

TORCH_DT = {"bf16": torch.bfloat16, "fp32": torch.float32}


def announce(msg: str) -> None:
    """Name the case before a GPU step, flushed, so a crash log shows it."""
    print(f"[gpu-case] {msg}", file=sys.stderr, flush=True)


def dev(a: np.ndarray, dtype: str) -> torch.Tensor:
    """float32 numpy array of storage-dtype values -> contiguous device tensor (exact)."""
    return torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).to("cuda").to(TORCH_DT[dtype]).contiguous()


def dev_i32(a) -> torch.Tensor:
    return torch.from_numpy(np.ascontiguousarray(a, dtype=np.int32)).to("cuda")


def dev_codes(c: np.ndarray) -> torch.Tensor:
    return torch.from_numpy(np.ascontiguousarray(c, dtype=np.uint64).view(np.int64)).to("cuda")


def host(t: torch.Tensor) -> np.ndarray:
    """Device tensor -> float64 numpy (exact for bf16 / fp32)."""
    torch.cuda.synchronize()
    return t.detach().float().cpu().numpy().astype(np.float64)


def host_codes(t: torch.Tensor) -> np.ndarray:
    torch.cuda.synchronize()
    return t.detach().cpu().numpy().view(np.uint64)


def bf16_ulp_distance(a: np.ndarray, b: np.ndarray) -> np.ndarray:
    """Distance in bf16 ulps between bf16-representable values (same sign ordering)."""
    def key(x):
        u = (np.asarray(x, dtype=np.float32).view(np.uint32) >> 16).astype(np.int64)
        return np.where(u & 0x8000, -(u & 0x7FFF), u)
    return np.abs(key(a) - key(b))


def fp32_ulp_distance(a: np.ndarray, b: np.ndarray) -> np.ndarray:
    def key(x):
        u = np.asarray(x, dtype=np.float32).view(np.uint32).astype(np.int64)
        return np.where(u & 0x80000000, -(u & 0x7FFFFFFF), u)
    return np.abs(key(a) - key(b))


def code_mismatch_ok(gpu: np.ndarray, ref: np.ndarray, proj: np.ndarray, x: np.ndarray,
                     planes: np.ndarray, rel: float = 1e-5):
    """LSH codes agree bit for bit except where the fp64 projection is within
    rel * ||x|| * ||r_j|| of zero.  Returns (n_flips, n_flips_outside_band)."""
    n, nb = proj.shape
    bits_g = np.unpackbits(gpu.view(np.uint8), axis=1, bitorder="little")[:, :nb]
    bits_r = np.unpackbits(ref.view(np.uint8), axis=1, bitorder="little")[:, :nb]
    diff = bits_g != bits_r
    band = rel * np.linalg.norm(x, axis=1)[:, None] * np.linalg.norm(planes, axis=1)[None, :]
    outside = diff & (np.abs(proj) >= band)
    return int(diff.sum()), int(outside.sum())


def bf16_ulp(ref: np.ndarray) -> np.ndarray:
    """Spacing of bf16 values at |ref| (8 significant bits; subnormal floor)."""
    a = np.abs(np.asarray(ref, dtype=np.float64))
    e = np.floor(np.log2(np.where(a > 0, a, 1.0)))
    return np.where(a > 0, np.exp2(np.maximum(e, -126) - 7), 2.0 ** -133)


def fp32_dot_error_bound(x: np.ndarray, w: np.ndarray) -> np.ndarray:
    """Worst-case error of fp32 dot products x_i . w_j in any summation order:
    gamma_K * sum_k |x_ik| |w_jk|, gamma_K = K u / (1 - K u), u = 2^-24."""
    K = x.shape[1]
    u = 2.0 ** -24
    gamma = K * u / (1 - K * u)
    return gamma * (np.abs(x.astype(np.float64)) @ np.abs(w.astype(np.float64)).T)


def rotated_pair_bound(b: np.ndarray, head_dim: int) -> np.ndarray:
    """A RoPE'd element mixes both members of its pair: bound_2k = bound_2k+1 =
    bound of the first plus bound of the second member (|cos|, |sin| <= 1)."""
    pair = b[:, 0::2] + b[:, 1::2]
    return np.repeat(pair, 2, axis=1)


def check_cache_rows(dt, got, ref, before, sel, x_sel, w, rotated):
    """Selected rows within the derived bound of the oracle; other rows untouched."""
    n_tok = got.shape[0]
    got = got.reshape(n_tok, -1)
    ref = ref.reshape(n_tok, -1)
    before = before.reshape(n_tok, -1)
    keep = np.ones(n_tok, bool)
    keep[sel] = False
    assert np.array_equal(got[keep], before[keep])
    b = fp32_dot_error_bound(x_sel, w)
    if rotated:
        b = rotated_pair_bound(b, 0) + 1e-6 * np.abs(ref[sel])
    spacing = bf16_ulp(ref[sel]) if dt == "bf16" else 2.0 ** -23 * np.abs(ref[sel])
    err = np.abs(got[sel] - ref[sel])
    assert np.all(err <= spacing + b), f"max excess {(err - spacing - b).max()}"
    if dt == "bf16":
        assert (bf16_ulp_distance(got[sel], ref[sel]) > 1).mean() < 1e-3


# ---- integer decisions taken on floating-point values that each side
# computes itself (GPU in fp32, oracle in fp64): equal, or, where the two
# differ, valid for the oracle's values within the float tolerance tol

def topk_valid(ref_keys: np.ndarray, chosen: np.ndarray, tol) -> bool:
    """A set chosen as the k largest: no unchosen key exceeds a chosen one by more than tol."""
    ref_keys = np.asarray(ref_keys, dtype=np.float64)
    mask = np.zeros(ref_keys.size, bool)
    mask[np.asarray(chosen, dtype=np.int64)] = True
    if mask.all() or not mask.any():
        return True
    t = np.broadcast_to(np.asarray(tol, dtype=np.float64), ref_keys.shape)
    return bool(ref_keys[mask].min() >= (ref_keys[~mask] - t[~mask] - t[mask].max()).max())


def order_valid(ref_keys: np.ndarray, order: np.ndarray, tol) -> bool:
    """An order by descending key: every key is at least every later key minus tol."""
    k = np.asarray(ref_keys, dtype=np.float64)[np.asarray(order, dtype=np.int64)]
    t = np.broadcast_to(np.asarray(tol, dtype=np.float64), np.shape(ref_keys))[np.asarray(order, dtype=np.int64)]
    suffix_max = np.maximum.accumulate((k - t)[::-1])[::-1]
    return bool(np.all(k[:-1] + t[:-1] >= suffix_max[1:])) if k.size > 1 else True


def recovery_valid(ref_mass: np.ndarray, order: np.ndarray, ar: int, thres: float, tol_sum: float) -> bool:
    """An AR taken on masses within tol of ref_mass: the first ar tokens of `order` reach thres of the
    total within tol_sum, the first ar - 1 do not exceed it by more than tol_sum."""
    m = np.asarray(ref_mass, dtype=np.float64)
    tot = m.sum()
    s = np.cumsum(m[np.asarray(order, dtype=np.int64)])
    ok_hi = s[ar - 1] >= thres * tot - tol_sum
    ok_lo = ar == 1 or s[ar - 2] < thres * tot + tol_sum
    return bool(ok_hi and ok_lo)
