"""Seeded synthetic inputs for the routed mixture-of-head attention layer.

This module only draws and formats random inputs; it holds none of the
layer's arithmetic (no selection, no ranks, no rotation, no softmax).  Both
the GPU library's callers (tests, benchmark) and the CPU oracle's callers take
their inputs from here, so the two sides always see identical bytes.

Recipe (every tensor is drawn independently):

* generator: numpy ``PCG64`` seeded with ``[seed, tensor_id, b, h]``
  (``h`` = 0 for tensors that are not per-head), ``seed = 260938832 + workload
  index`` for the named workloads;
* tensor ids: logits 0, q 1, k 2, v 3, decode-cache keys 4, decode-cache
  values 5, decode new-token q/k/v 6/7/8, prior-history routing 9; for the
  layer with projections: token inputs x 10, per-head projection weights
  W_QKV 11 and W_O 12 (x N(0,1), W_QKV N(0,1)/sqrt(d_model), W_O
  N(0,1)/sqrt(d), all bf16);
* draws: ``standard_normal`` in float32, multiplied by the float32 scale, then
  rounded to bfloat16 (round to nearest even) for bf16 tensors;
* logits: float32 N(0,1); the skewed workload adds the per-head bias
  ``1.5*ln(1/(h+1))`` in float64 and rounds once to float32.

The shapes and distributions follow the paper's workloads: the layer's head
count / active-head count / head width of the pretraining setup (Sec. 4.1),
long-context lengths (Sec. 4.3) and a Zipf-like skewed routing case; the
paper's text corpora are not available, and these seeded draws stand in for
them.
"""
from __future__ import annotations

import concurrent.futures as cf
import math
import os
from dataclasses import dataclass, replace
from typing import Optional

import numpy as np

BASE_SEED = 260938832

TID_LOGITS, TID_Q, TID_K, TID_V = 0, 1, 2, 3
TID_KCACHE, TID_VCACHE = 4, 5
TID_DEC_Q, TID_DEC_K, TID_DEC_V = 6, 7, 8
TID_PRIOR = 9
TID_X, TID_WQKV, TID_WO = 10, 11, 12


@dataclass(frozen=True)
class Workload:
    """One layer invocation: sizes, dtype, distributions and RoPE base."""
    name: str
    B: int
    T: int              # prefill: sequence length; decode: 1
    H: int
    K: int
    d: int
    dtype: str          # "f32" or "bf16"
    qkv_scale: float
    rope_base: float
    zipf_bias: float = 0.0       # logits += zipf_bias * ln(1/(h+1))
    prior: int = 0               # decode: routed prior tokens per sequence
    seed: int = BASE_SEED
    decode: bool = False
    d_model: int = 0             # > 0: the layer with its per-head projections

    def with_(self, **kw) -> "Workload":
        return replace(self, **kw)


WORKLOADS = {
    1: Workload("tiny_fp32_B1_T512_H8_K2_d32", B=1, T=512, H=8, K=2, d=32,
                dtype="f32", qkv_scale=1 / math.sqrt(32), rope_base=1e4,
                seed=BASE_SEED + 1),
    2: Workload("balanced_bf16_B4_T4096_H32_K8_d64", B=4, T=4096, H=32, K=8,
                d=64, dtype="bf16", qkv_scale=1 / 8, rope_base=1e4,
                seed=BASE_SEED + 2),
    3: Workload("head_scaling_bf16_B1_T32768_H64_K8_d128", B=1, T=32768, H=64,
                K=8, d=128, dtype="bf16", qkv_scale=1 / math.sqrt(128),
                rope_base=5e5, seed=BASE_SEED + 3),
    4: Workload("skewed_bf16_B2_T16384_H32_K4_d128", B=2, T=16384, H=32, K=4,
                d=128, dtype="bf16", qkv_scale=1 / math.sqrt(128),
                rope_base=1e4, zipf_bias=1.5, seed=BASE_SEED + 4),
    5: Workload("decode_bf16_B64_prior131072_H64_K8_d128", B=64, T=1, H=64,
                K=8, d=128, dtype="bf16", qkv_scale=1 / math.sqrt(128),
                rope_base=5e5, prior=131072, seed=BASE_SEED + 5, decode=True),
    # the balanced prefill shape with the paper's model width (Sec. 4.1:
    # d_model 2048, head width 64, 32 heads with 8 active): routed Q/K/V
    # projections, attention, routed output projections
    6: Workload("layer_bf16_B4_T4096_H32_K8_d64_dm2048", B=4, T=4096, H=32, K=8,
                d=64, dtype="bf16", qkv_scale=1 / 8, rope_base=1e4,
                seed=BASE_SEED + 6, d_model=2048),
}


# ----------------------------------------------------------------------------
# number formats

def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """float32 -> bfloat16 bit pattern (uint16), round to nearest even.

    Inputs are finite draws; NaN handling is not needed here.
    """
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    r = (u + np.uint32(0x7FFF) + ((u >> np.uint32(16)) & np.uint32(1))) >> np.uint32(16)
    return r.astype(np.uint16)


def bf16_bits_to_f32(bits: np.ndarray) -> np.ndarray:
    """bfloat16 bit pattern -> float32 (exact)."""
    return (np.asarray(bits, dtype=np.uint16).astype(np.uint32) << np.uint32(16)).view(np.float32)


def as_float64(x: np.ndarray, dtype: str) -> np.ndarray:
    """Exact float64 view of a stored tensor (uint16 bf16 bits or float32)."""
    if dtype == "bf16":
        return bf16_bits_to_f32(x).astype(np.float64)
    return np.asarray(x, dtype=np.float32).astype(np.float64)


# ----------------------------------------------------------------------------
# primitive draws

def _rng(seed: int, tid: int, b: int = 0, h: int = 0) -> np.random.Generator:
    return np.random.Generator(np.random.PCG64([seed, tid, b, h]))


def normal_block(seed: int, tid: int, b: int, h: int, shape, scale: float,
                 dtype: str) -> np.ndarray:
    """One independently seeded block: float32 N(0,1)*scale, then bf16 bits
    (uint16) for ``dtype == 'bf16'`` or float32 otherwise."""
    z = _rng(seed, tid, b, h).standard_normal(shape, dtype=np.float32)
    z *= np.float32(scale)
    if dtype == "bf16":
        return f32_to_bf16_bits(z)
    return z


def storage_dtype(dtype: str):
    return np.uint16 if dtype == "bf16" else np.float32


# ----------------------------------------------------------------------------
# prefill inputs

def prefill_logits(w: Workload) -> np.ndarray:
    """Router logits float32 [B, T, H]."""
    out = np.empty((w.B, w.T, w.H), dtype=np.float32)
    for b in range(w.B):
        z = _rng(w.seed, TID_LOGITS, b, 0).standard_normal((w.T, w.H), dtype=np.float32)
        if w.zipf_bias:
            bias = w.zipf_bias * np.log(1.0 / (np.arange(w.H, dtype=np.float64) + 1.0))
            out[b] = (z.astype(np.float64) + bias[None, :]).astype(np.float32)
        else:
            out[b] = z
    return out


def _workers() -> int:
    return max(1, min(16, len(os.sched_getaffinity(0))))


def prefill_qkv(w: Workload, which: str) -> np.ndarray:
    """Dense per-head tensor [B, H, T, d] for which in {'q','k','v'}.

    bf16 tensors are returned as uint16 bit patterns, f32 as float32.  Blocks
    are drawn in parallel threads (each block has its own seeded generator,
    so the result does not depend on the thread count).
    """
    tid = {"q": TID_Q, "k": TID_K, "v": TID_V}[which]
    out = np.empty((w.B, w.H, w.T, w.d), dtype=storage_dtype(w.dtype))

    def fill(bh):
        b, h = divmod(bh, w.H)
        out[b, h] = normal_block(w.seed, tid, b, h, (w.T, w.d), w.qkv_scale, w.dtype)

    with cf.ThreadPoolExecutor(_workers()) as ex:
        list(ex.map(fill, range(w.B * w.H)))
    return out


def prefill_inputs(w: Workload) -> dict:
    return {"logits": prefill_logits(w), "q": prefill_qkv(w, "q"),
            "k": prefill_qkv(w, "k"), "v": prefill_qkv(w, "v")}


def projection_inputs(w: Workload) -> dict:
    """Token inputs x [B, T, d_model] and the per-head weights stored as
    linear maps (out x in): w_qkv [H, 3, d, d_model] (query, key, value rows)
    and w_o [H, d_model, d]; all bf16 bit patterns (uint16)."""
    dm = w.d_model
    x = np.empty((w.B, w.T, dm), dtype=np.uint16)
    for b in range(w.B):
        x[b] = normal_block(w.seed, TID_X, b, 0, (w.T, dm), 1.0, "bf16")
    w_qkv = np.empty((w.H, 3, w.d, dm), dtype=np.uint16)
    w_o = np.empty((w.H, dm, w.d), dtype=np.uint16)
    for h in range(w.H):
        w_qkv[h] = normal_block(w.seed, TID_WQKV, 0, h, (3, w.d, dm), 1.0 / math.sqrt(dm), "bf16")
        w_o[h] = normal_block(w.seed, TID_WO, 0, h, (dm, w.d), 1.0 / math.sqrt(w.d), "bf16")
    return {"logits": prefill_logits(w), "x": x, "w_qkv": w_qkv, "w_o": w_o}


# ----------------------------------------------------------------------------
# decode inputs

def decode_prior_lengths(w: Workload) -> np.ndarray:
    """Head history lengths int32 [B, H] after ``w.prior`` earlier tokens.

    Each earlier token joins ``K`` distinct heads drawn uniformly at random
    (by symmetry this is how i.i.d. N(0,1) router logits distribute tokens
    over heads); the draw is the first ``K`` of a uniformly random ordering of
    the heads, taken from float32 uniforms.
    """
    out = np.zeros((w.B, w.H), dtype=np.int64)
    chunk = 1 << 15

    def count(b):
        g = _rng(w.seed, TID_PRIOR, b, 0)
        left = w.prior
        while left > 0:
            m = min(chunk, left)
            u = g.random((m, w.H), dtype=np.float32)
            pick = np.argpartition(u, w.K - 1, axis=1)[:, :w.K]
            out[b] += np.bincount(pick.ravel(), minlength=w.H)
            left -= m

    with cf.ThreadPoolExecutor(_workers()) as ex:
        list(ex.map(count, range(w.B)))
    return out.astype(np.int32)


def decode_step_inputs(w: Workload) -> dict:
    """New-token logits f32 [B, H] and q/k/v [B, H, d] (bf16 bits or f32)."""
    logits = np.empty((w.B, w.H), dtype=np.float32)
    q = np.empty((w.B, w.H, w.d), dtype=storage_dtype(w.dtype))
    k = np.empty_like(q)
    v = np.empty_like(q)
    for b in range(w.B):
        logits[b] = _rng(w.seed, TID_LOGITS, b, 0).standard_normal(w.H, dtype=np.float32)
        for h in range(w.H):
            q[b, h] = normal_block(w.seed, TID_DEC_Q, b, h, (w.d,), w.qkv_scale, w.dtype)
            k[b, h] = normal_block(w.seed, TID_DEC_K, b, h, (w.d,), w.qkv_scale, w.dtype)
            v[b, h] = normal_block(w.seed, TID_DEC_V, b, h, (w.d,), w.qkv_scale, w.dtype)
    return {"logits": logits, "q": q, "k": k, "v": v}


def decode_cache_block(w: Workload, b: int, h: int, rows: int, which: str) -> np.ndarray:
    """Rows ``[0, rows)`` of head ``h``'s cached keys ('k', taken as already
    rotated) or values ('v') for sequence ``b``: [rows, d] bf16 bits / f32."""
    tid = TID_KCACHE if which == "k" else TID_VCACHE
    return normal_block(w.seed, tid, b, h, (rows, w.d), w.qkv_scale, w.dtype)


def decode_cache_capacity(lengths: np.ndarray, steps: int = 64) -> int:
    """Cache capacity: longest history plus room for ``steps`` appends,
    rounded up to a multiple of 256 rows."""
    need = int(lengths.max()) + steps
    return (need + 255) // 256 * 256


# ----------------------------------------------------------------------------
# small derived sizes used by reports (pure counting, no layer arithmetic)

def dense_bytes(w: Workload) -> int:
    esz = 2 if w.dtype == "bf16" else 4
    return 3 * w.B * w.H * w.T * w.d * esz
