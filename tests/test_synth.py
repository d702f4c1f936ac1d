"""The seeded input generators: reproducible, independent per key, and (for
the long-sequence generator) prefix-stable across lengths and block edges."""
import numpy as np

import sata_synth as syn


def test_head_stream_reproducible_and_rounded():
    a = syn.head_stream(3, 1, 2, syn.TENSOR_Q, (64, 8), "bf16")
    b = syn.head_stream(3, 1, 2, syn.TENSOR_Q, (64, 8), "bf16")
    c = syn.head_stream(3, 1, 3, syn.TENSOR_Q, (64, 8), "bf16")
    assert np.array_equal(a, b) and not np.array_equal(a, c)
    assert np.array_equal(syn.round_to_bf16(a), a)  # already bf16 values


def test_long_head_prefix_stable_across_block_edges():
    n = syn.LONG_BLOCK + 1000  # one full block and a partial one
    q, k, v = syn.long_head(9, n, 4, 6, threads=4)
    assert q.dtype == np.float32 and q.shape == (n, 4) and v.shape == (n, 6)
    q2, k2, v2 = syn.long_head(9, syn.LONG_BLOCK - 5, 4, 6, threads=1)
    assert np.array_equal(q2, q[: syn.LONG_BLOCK - 5]) and np.array_equal(v2, v[: syn.LONG_BLOCK - 5])
    # tensors and blocks are distinct streams
    assert not np.array_equal(q[:100], k[:100])
    assert not np.array_equal(q[:100], q[syn.LONG_BLOCK:syn.LONG_BLOCK + 100])


def test_long_head_is_standard_normal():
    q, _, _ = syn.long_head(10, 400_000, 8, 8)
    x = q.astype(np.float64).ravel()
    assert abs(x.mean()) < 0.005 and abs(x.std() - 1.0) < 0.005
