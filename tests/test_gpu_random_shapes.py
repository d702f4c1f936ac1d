"""GPU parity over seeded draws of shapes: prefill (output and state), then
a few decode steps that continue it, each against the float64 oracle; and
the same for grouped query heads (prefill and decode of G query heads per
key/value head).

The fixed cases of the other files pin one kernel family each; this draw
mixes the arguments they leave uncrossed (d_k != d_v, every chunk size,
ragged lengths, P = 1..7, both input types, lengths long enough for the
sequence to run in parts) so that a planner decision no fixed case reaches
is still compared with the oracle.  The draw is seeded: every run sees the
same shapes, and each case prints its arguments before it starts.
"""
import sys
from math import comb

import numpy as np
import pytest

import oracle
import sata_synth as syn
from gpu_util import check_prefill_head, check_rows, check_state, operands, to_dev, to_host, torch_dtype, y_tol

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


def _draw_cases(seed=2602, count=32):
    """(workload, B, H, n, d_k, d_v, P, chunk, dtype) tuples; the oracle's
    state check (a [n][D] feature matrix per head) is kept under ~2e7 entries."""
    rng = np.random.default_rng(seed)
    cases = []
    while len(cases) < count:
        chunk = int(rng.choice([16, 32, 64, 64, 128]))
        dmax = 32 if chunk == 128 else (96 if chunk <= 32 else 64)
        dk = int(rng.integers(1, dmax + 1))
        dv = int(rng.integers(1, dmax + 1))
        P = int(rng.integers(1, 8))
        D = comb(dk + P - 1, P - 1)
        if D > 60000:
            continue
        long_seq = rng.random() < 0.25
        n = int(rng.integers(2048, 4500)) if long_seq else int(rng.integers(1, 700))
        if n * D * max(P - 1, 1) > 2e7:
            continue
        B = int(rng.integers(1, 3))
        H = 1 if long_seq else int(rng.integers(1, 4))
        dtype = "bf16" if rng.random() < 0.5 else "f32"
        cases.append((200 + len(cases), B, H, n, dk, dv, P, chunk, dtype))
    return cases


CASES = _draw_cases()


@pytest.fixture(scope="module")
def sata():
    if not torch.cuda.is_available():
        pytest.fail("no GPU visible")
    import paper_2602_00294_amd as m
    m.load_library()
    return m


@pytest.mark.parametrize("case", CASES, ids=lambda c: "w{}_B{}H{}n{}dk{}dv{}P{}C{}_{}".format(*c))
def test_prefill_then_decode_matches_oracle(sata, case):
    workload, B, H, n, dk, dv, P, chunk, dtype = case
    steps = 3
    parts = sata.prefill_parts(torch_dtype(dtype), B, H, n, dk, dv, P, chunk)
    print(f"random shape {case} D={comb(dk + P - 1, P - 1)} parts={parts}", file=sys.stderr, flush=True)
    q, k, v = syn.make_qkv(workload, B, H, n + steps, dk, dv, dtype)
    dev = lambda a: to_dev(a, dtype)
    ops = operands(sata, dtype, B, H, n, dk, dv, P, chunk)
    y, S = sata.prefill(dev(q[:, :, :n]), dev(k[:, :, :n]), dev(v[:, :, :n]), P, chunk)
    torch.cuda.synchronize()
    y_host = to_host(y)
    for b in range(B):
        for h in range(H):
            check_prefill_head(y_host[b, h], to_host(S[b, h]), q[b, h, :n], k[b, h, :n], v[b, h, :n], P, ops, dtype,
                               chunk, f"{case} {ops} b{b} h{h}")
    ys = []
    for t in range(n, n + steps):
        ys.append(to_host(sata.decode_step(S, dev(q[:, :, t].copy()), dev(k[:, :, t].copy()),
                                           dev(v[:, :, t].copy()), P)))
    torch.cuda.synchronize()
    S_host = to_host(S)
    for b in range(B):
        for h in range(H):
            yr, _, kap = oracle.taylor_attention_rows(q[b, h], k[b, h], v[b, h], P, list(range(n, n + steps)))
            got = np.stack([yy[b, h] for yy in ys])
            rho = oracle.term_scale(q[b, h], k[b, h], v[b, h], P, rows=list(range(n, n + steps)))
            check_rows(got, yr, kap, y_tol(ops, dtype), P, f"{case} decode b{b} h{h}", rho)
            check_state(S_host[b, h], k[b, h], v[b, h], P, ops, n, chunk, f"{case} decoded state b{b} h{h}",
                        steps=steps)


def _draw_grouped_cases(seed=2603, count=12):
    """(workload, B, H_kv, G, n, d_k, d_v, P, chunk, dtype) tuples for the
    grouped prefill and decode, under the same oracle budget."""
    rng = np.random.default_rng(seed)
    cases = []
    while len(cases) < count:
        chunk = int(rng.choice([16, 32, 64, 64]))
        dk = int(rng.integers(1, 65))
        dv = int(rng.integers(1, 65))
        P = int(rng.integers(1, 7))
        D = comb(dk + P - 1, P - 1)
        if D > 60000:
            continue
        long_seq = rng.random() < 0.25
        n = int(rng.integers(2048, 4200)) if long_seq else int(rng.integers(1, 500))
        if n * D * max(P - 1, 1) > 2e7:
            continue
        G = int(rng.choice([2, 4, 8]))
        Hkv = 1 if long_seq else int(rng.integers(1, 3))
        B = int(rng.integers(1, 3))
        dtype = "bf16" if rng.random() < 0.5 else "f32"
        cases.append((300 + len(cases), B, Hkv, G, n, dk, dv, P, chunk, dtype))
    return cases


GROUPED_CASES = _draw_grouped_cases()


@pytest.mark.parametrize("case", GROUPED_CASES, ids=lambda c: "w{}_B{}Hkv{}G{}n{}dk{}dv{}P{}C{}_{}".format(*c))
def test_grouped_prefill_then_decode_matches_oracle(sata, case):
    """Query head g + G h against the oracle on its own queries and key/value
    head h's tokens, through the grouped prefill and two grouped decode steps."""
    workload, B, Hkv, G, n, dk, dv, P, chunk, dtype = case
    steps = 2
    print(f"random grouped shape {case} D={comb(dk + P - 1, P - 1)}", file=sys.stderr, flush=True)
    q, _, _ = syn.make_qkv(workload, B, Hkv * G, n + steps, dk, dv, dtype)
    _, k, v = syn.make_qkv(workload + 1000, B, Hkv, n + steps, dk, dv, dtype)
    dev = lambda a: to_dev(np.ascontiguousarray(a), dtype)
    ops = operands(sata, dtype, B, Hkv, n, dk, dv, P, chunk)
    y, S = sata.prefill_grouped(dev(q[:, :, :n]), dev(k[:, :, :n]), dev(v[:, :, :n]), P, chunk)
    torch.cuda.synchronize()
    yh = to_host(y)
    ys = [to_host(sata.decode_step_grouped(S, dev(q[:, :, t]), dev(k[:, :, t]), dev(v[:, :, t]), P))
          for t in range(n, n + steps)]
    torch.cuda.synchronize()
    S_host = to_host(S)
    tol = y_tol(ops, dtype)
    for b in range(B):
        for hq in range(Hkv * G):
            h = hq // G
            label = f"{case} b{b} query head {hq}"
            yr, _, kap = oracle.taylor_attention(q[b, hq, :n], k[b, h, :n], v[b, h, :n], P)
            check_rows(yh[b, hq], yr, kap, tol, P, label, oracle.term_scale(q[b, hq, :n], k[b, h, :n], v[b, h, :n], P))
            rows = list(range(n, n + steps))
            yr, _, kap = oracle.taylor_attention_rows(q[b, hq], k[b, h], v[b, h], P, rows)
            got = np.stack([yy[b, hq] for yy in ys])
            check_rows(got, yr, kap, tol, P, label + " decode", oracle.term_scale(q[b, hq], k[b, h], v[b, h], P, rows))
        for h in range(Hkv):
            check_state(S_host[b, h], k[b, h], v[b, h], P, ops, n, chunk, f"{case} state b{b} h{h}", steps=steps)
