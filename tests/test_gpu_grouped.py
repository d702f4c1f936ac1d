"""GPU parity of the grouped-query decode (sata_decode_step_grouped): each
key/value head keeps one state and serves G query heads.  The reference is
the float64 oracle applied per query head to its key/value head's tokens
(query head g + G h reads key/value head h); the state must equal the
oracle's state of the key/value head."""
import sys

import numpy as np
import pytest

import oracle
import sata_synth as syn
from gpu_util import check_rows, check_state, operands, to_dev, to_host, torch_dtype, y_tol

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


def _inputs(wid, B, Hkv, G, n, d, dtype):
    q, _, _ = syn.make_qkv(wid, B, Hkv * G, n, d, d, dtype)
    _, k, v = syn.make_qkv(wid + 1, B, Hkv, n, d, d, dtype)
    return q, k, v


def _state_after_prefill(sata, k, v, n1, P, dtype):
    B, Hkv, _, d = k.shape
    if n1 == 0:
        return torch.zeros(B, Hkv, oracle.feature_count(d, P), v.shape[-1] + 1, device="cuda")
    kk = to_dev(k[:, :, :n1], dtype)
    _, S = sata.prefill(kk, kk, to_dev(v[:, :, :n1], dtype), P, 32)  # the state does not depend on q
    return S


@pytest.mark.parametrize("B,Hkv,G,n1,n2,d,P,dtype", [
    (1, 2, 4, 40, 3, 8, 4, "f32"),     # small heads: one 256-thread workgroup per head
    (2, 3, 2, 70, 2, 16, 4, "bf16"),
    (1, 2, 8, 30, 2, 32, 4, "bf16"),   # the benchmark's head size, several pieces per head
    (1, 1, 4, 20, 2, 64, 4, "f32"),    # D = 47905: many pieces per head
    (1, 2, 2, 0, 3, 5, 3, "f32"),      # empty prefill; rows of 6 floats, heads not 16-byte aligned
    (2, 4, 4, 10, 2, 7, 5, "f32"),
])
def test_grouped_decode_matches_oracle(sata, B, Hkv, G, n1, n2, d, P, dtype):
    _say(f"grouped decode B={B} H_kv={Hkv} G={G} n1={n1} n2={n2} d={d} P={P} {dtype}")
    q, k, v = _inputs(80 + d, B, Hkv, G, n1 + n2, d, dtype)
    S = _state_after_prefill(sata, k, v, n1, P, dtype)
    ops = operands(sata, dtype, B, Hkv, n1, d, d, P, 32) if n1 > 0 else "f32"
    ys = []
    for t in range(n1, n1 + n2):
        ys.append(to_host(sata.decode_step_grouped(S, to_dev(q[:, :, t].copy(), dtype), to_dev(k[:, :, t].copy(), dtype),
                                                   to_dev(v[:, :, t].copy(), dtype), P)))
    torch.cuda.synchronize()
    S_host = to_host(S)
    for b in range(B):
        for hq in range(Hkv * G):
            h = hq // G
            yr, _, kap = oracle.taylor_attention_rows(q[b, hq], k[b, h], v[b, h], P, list(range(n1, n1 + n2)))
            got = np.stack([yy[b, hq] for yy in ys])
            check_rows(got, yr, kap, y_tol(ops, dtype), P, f"b{b} query head {hq}")
        for h in range(Hkv):
            check_state(S_host[b, h], k[b, h], v[b, h], P, ops, n1, 32, f"state b{b} h{h}", steps=n2)


def test_grouped_decode_deterministic_and_g1_is_decode_step(sata):
    """Repeated calls give identical bits; G = 1 is the single-query decode."""
    B, Hkv, G, n, d, P = 1, 2, 4, 50, 32, 4
    q, k, v = _inputs(90, B, Hkv, G, n + 1, d, "bf16")
    S0 = _state_after_prefill(sata, k, v, n, P, "bf16")
    step = [to_dev(a[:, :, n].copy(), "bf16") for a in (q, k, v)]
    S1, S2 = S0.clone(), S0.clone()
    y1 = sata.decode_step_grouped(S1, *step, P)
    y2 = sata.decode_step_grouped(S2, *step, P)
    torch.cuda.synchronize()
    assert torch.equal(y1, y2) and torch.equal(S1, S2)
    q1 = step[0][:, ::G].contiguous()  # one query head per key/value head
    S3, S4 = S0.clone(), S0.clone()
    ya = sata.decode_step_grouped(S3, q1, step[1], step[2], P)
    yb = sata.decode_step(S4, q1, step[1], step[2], P)
    torch.cuda.synchronize()
    assert torch.equal(ya, yb) and torch.equal(S3, S4)


@pytest.mark.parametrize("B,Hkv,G,n,d,P,chunk,dtype", [
    (1, 2, 4, 150, 32, 4, 64, "bf16"),   # the d = 32 matrix-core kernel
    (2, 2, 2, 97, 16, 4, 32, "bf16"),    # the per-block matrix-core kernel
    (1, 3, 2, 100, 8, 3, 64, "bf16"),    # the generated-feature matrix-core kernel
    (1, 3, 2, 70, 8, 4, 64, "f32"),      # the float32 kernel
    (1, 1, 8, 40, 5, 3, 16, "f32"),
    (1, 1, 2, 4096, 8, 3, 64, "f32"),    # the generated-feature kernel, sequence in 4 parts
])
def test_grouped_prefill_matches_oracle(sata, B, Hkv, G, n, d, P, chunk, dtype):
    """Every query head's rows against the oracle applied to its own queries and
    its key/value head's tokens; each member of a group bitwise equal to the
    single-head prefill of its queries; the states equal to the plain prefill's
    (they depend on the keys and values only); then a grouped decode step."""
    _say(f"grouped prefill B={B} H_kv={Hkv} G={G} n={n} d={d} P={P} chunk={chunk} {dtype}")
    q, k, v = _inputs(140 + d, B, Hkv, G, n + 1, d, dtype)
    dev = lambda a: to_dev(np.ascontiguousarray(a), dtype)
    qd, kd, vd = dev(q[:, :, :n]), dev(k[:, :, :n]), dev(v[:, :, :n])
    y, S = sata.prefill_grouped(qd, kd, vd, P, chunk)
    torch.cuda.synchronize()
    ops = operands(sata, dtype, B, Hkv, n, d, d, P, chunk)
    if n >= 4096:
        assert sata.prefill_parts(torch_dtype(dtype), B, Hkv, n, d, d, P, chunk) == 4
    yh = to_host(y)
    for b in range(B):
        for hq in range(Hkv * G):
            h = hq // G
            yr, _, kap = oracle.taylor_attention(q[b, hq, :n], k[b, h, :n], v[b, h, :n], P)
            check_rows(yh[b, hq], yr, kap, y_tol(ops, dtype), P, f"b{b} query head {hq}")
    for g in range(G):
        yg, Sg = sata.prefill(qd[:, g::G].contiguous(), kd, vd, P, chunk)
        torch.cuda.synchronize()
        assert torch.equal(yg, y[:, g::G]), f"member {g}"
        assert torch.equal(Sg, S)
    for b in range(B):
        for h in range(Hkv):
            check_state(to_host(S[b, h]), k[b, h, :n], v[b, h, :n], P, ops, n, chunk, f"state b{b} h{h}")
    yd = to_host(sata.decode_step_grouped(S, dev(q[:, :, n]), dev(k[:, :, n]), dev(v[:, :, n]), P)) \
        if S.data_ptr() % 16 == 0 else None
    torch.cuda.synchronize()
    if yd is not None:
        for b in range(B):
            for hq in range(Hkv * G):
                h = hq // G
                yr, _, kap = oracle.taylor_attention_rows(q[b, hq], k[b, h], v[b, h], P, [n])
                check_rows(yd[b, hq][None], yr, kap, y_tol(ops, dtype), P, f"decode b{b} query head {hq}")
