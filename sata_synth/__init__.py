"""Seeded synthetic inputs shared by the tests, the benchmark and the smoke check.

This module holds no arithmetic of the attention method: it only draws
i.i.d. N(0, 1) queries, keys and values (the paper's synthetic protocol,
App. A3) and rounds them to the storage precision.

Recipe.  Every (workload, batch b, head h, tensor) gets its own stream
``numpy.random.default_rng([SEED, workload, b, h, tensor])`` so that any head
can be regenerated alone.  Values are drawn in float64, rounded to float32
(round to nearest even) and, for bf16 workloads, from float32 to bfloat16
(round to nearest even).  The arrays returned are float32 holding exactly the
values that the GPU receives, so the oracle sees the same inputs bit for bit.

Long sequences (``long_head``, up to 10^8 tokens) are drawn faster: float32
N(0, 1) values straight from the generator, in blocks of 2^20 tokens, each
block from its own stream ``default_rng([SEED, workload, LONG, block,
tensor])``, so that the blocks can be drawn in parallel threads and any
prefix of the sequence is the same whatever its length.
"""
from __future__ import annotations

import numpy as np

SEED = 260200294
TENSOR_Q, TENSOR_K, TENSOR_V = 0, 1, 2
LONG = 1 << 20  # stream-key tag of the long-sequence generator
LONG_BLOCK = 1 << 20  # tokens per block

__all__ = ["SEED", "round_to_bf16", "bf16_bits", "head_stream", "make_qkv", "make_head", "long_head"]


def round_to_bf16(x) -> np.ndarray:
    """float32 -> nearest bfloat16 value (ties to even), returned as float32.

    NaN and infinities never occur in these inputs and are not treated specially.
    """
    x = np.ascontiguousarray(x, dtype=np.float32)
    bits = x.view(np.uint32).astype(np.uint64)
    lsb = (bits >> 16) & 1
    rounded = ((bits + 0x7FFF + lsb) >> 16) << 16
    return rounded.astype(np.uint32).view(np.float32).reshape(x.shape)


def bf16_bits(x) -> np.ndarray:
    """Upper 16 bits of float32 values that are already bfloat16-representable."""
    x = np.ascontiguousarray(x, dtype=np.float32)
    return (x.view(np.uint32) >> 16).astype(np.uint16)


def head_stream(workload: int, b: int, h: int, tensor: int, shape, dtype: str = "f32") -> np.ndarray:
    """One tensor of one head: N(0,1) of the given shape, rounded to ``dtype``."""
    rng = np.random.default_rng([SEED, int(workload), int(b), int(h), int(tensor)])
    x = rng.standard_normal(shape).astype(np.float32)
    if dtype == "bf16":
        x = round_to_bf16(x)
    elif dtype != "f32":
        raise ValueError(f"unknown dtype {dtype!r}")
    return x


def make_head(workload: int, b: int, h: int, n: int, d_k: int, d_v: int, dtype: str = "f32"):
    """(q [n, d_k], k [n, d_k], v [n, d_v]) for one head."""
    return (head_stream(workload, b, h, TENSOR_Q, (n, d_k), dtype),
            head_stream(workload, b, h, TENSOR_K, (n, d_k), dtype),
            head_stream(workload, b, h, TENSOR_V, (n, d_v), dtype))


def make_qkv(workload: int, B: int, H: int, n: int, d_k: int, d_v: int, dtype: str = "f32"):
    """(q [B,H,n,d_k], k [B,H,n,d_k], v [B,H,n,d_v]) as float32 arrays."""
    q = np.empty((B, H, n, d_k), np.float32)
    k = np.empty((B, H, n, d_k), np.float32)
    v = np.empty((B, H, n, d_v), np.float32)
    for b in range(B):
        for h in range(H):
            q[b, h], k[b, h], v[b, h] = make_head(workload, b, h, n, d_k, d_v, dtype)
    return q, k, v


def long_head(workload: int, n: int, d_k: int, d_v: int, threads: int = 16):
    """(q [n, d_k], k [n, d_k], v [n, d_v]) float32 N(0, 1) for one long head;
    blocks of LONG_BLOCK tokens drawn in parallel threads."""
    from concurrent.futures import ThreadPoolExecutor
    out = [np.empty((n, d_k), np.float32), np.empty((n, d_k), np.float32), np.empty((n, d_v), np.float32)]
    jobs = [(t, b) for t in range(3) for b in range((n + LONG_BLOCK - 1) // LONG_BLOCK)]

    def fill(job):
        t, b = job
        r0, r1 = b * LONG_BLOCK, min(n, (b + 1) * LONG_BLOCK)
        rng = np.random.default_rng([SEED, int(workload), LONG, b, t])
        out[t][r0:r1] = rng.standard_normal((r1 - r0, out[t].shape[1]), dtype=np.float32)

    with ThreadPoolExecutor(max(1, threads)) as ex:
        list(ex.map(fill, jobs))
    return tuple(out)
