"""GPU parity of the backward (sata_backward): dL/dq, dL/dk, dL/dv against the
float64 oracle's gradients of the causal output (oracle.taylor_attention_backward,
pinned by finite differences).  Per head, each gradient must be within the
tolerance in the Frobenius sense, ||g_gpu - g|| / ||g||; the arithmetic is
float32, so 1e-4 for float32 inputs and 2^-8 for bfloat16 inputs and outputs
(whose storage rounding is 2^-9 per element).  Inputs are chosen with no
cancelling denominator (kappa <= 100 on every row), which the test asserts."""
import sys

import numpy as np
import pytest

import oracle
import sata_synth as syn
from gpu_util import to_dev, to_host
from oracle.metrics import KAPPA_MAX, y_tol

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


@pytest.fixture(scope="module")
def sata():
    if not torch.cuda.is_available():
        pytest.fail("no GPU visible")
    import paper_2602_00294_amd as m
    m.load_library()
    return m


def _say(msg):
    print(msg, file=sys.stderr, flush=True)


def _rel(a, b):
    return float(np.linalg.norm(a - b) / np.linalg.norm(b))


@pytest.mark.parametrize("B,H,n,dk,dv,P,chunk,dtype", [
    (1, 1, 130, 8, 8, 4, 64, "f32"),      # ragged last chunk
    (2, 2, 97, 16, 16, 3, 32, "f32"),
    (1, 2, 64, 4, 6, 5, 16, "f32"),
    (1, 1, 200, 32, 32, 4, 64, "bf16"),   # the benchmark's head shape
    (1, 1, 45, 5, 3, 1, 16, "f32"),       # P = 1: no gradient for q and k
    (1, 1, 300, 8, 8, 2, 64, "f32"),
    (1, 1, 150, 4, 4, 6, 64, "f32"),      # degrees above 3 (the full product rule)
    (1, 1, 100, 64, 64, 3, 64, "bf16"),   # the largest head, five column tiles in the forward readout
])
def test_backward_matches_oracle(sata, B, H, n, dk, dv, P, chunk, dtype):
    _say(f"backward B={B} H={H} n={n} dk={dk} dv={dv} P={P} chunk={chunk} {dtype}")
    q, k, v = syn.make_qkv(160 + dk, B, H, n, dk, dv, dtype)
    dy = syn.make_qkv(170 + dk, B, H, n, dv, dv, dtype)[2]
    g = sata.backward(*(to_dev(a, dtype) for a in (q, k, v, dy)), P, chunk)
    torch.cuda.synchronize()
    got = [to_host(x) for x in g]
    tol = y_tol("f32", dtype)
    for b in range(B):
        for h in range(H):
            _, _, kap = oracle.taylor_attention(q[b, h], k[b, h], v[b, h], P)
            assert kap.max() <= KAPPA_MAX
            want = oracle.taylor_attention_backward(q[b, h], k[b, h], v[b, h], dy[b, h], P)
            for name, gg, ww in zip(("dq", "dk", "dv"), got, want):
                if P == 1 and name != "dv":
                    assert np.all(gg[b, h] == 0), name
                    continue
                err = _rel(gg[b, h], ww)
                _say(f"  b{b} h{h} {name}: {err:.3e}")
                assert err <= tol, f"b{b} h{h} {name}: {err:.3e}"


def test_backward_chunk_invariance(sata):
    q, k, v = syn.make_qkv(180, 1, 1, 150, 8, 8, "f32")
    dy = syn.make_qkv(181, 1, 1, 150, 8, 8, "f32")[2]
    args = [to_dev(a, "f32") for a in (q, k, v, dy)]
    outs = [[to_host(x) for x in sata.backward(*args, 4, c)] for c in (16, 32, 64)]
    torch.cuda.synchronize()
    for o in outs[1:]:
        for a, b in zip(o, outs[0]):
            assert _rel(a, b) < 1e-5
