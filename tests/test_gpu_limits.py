"""GPU parity at the limits the C ABI accepts: the largest head dimension,
the highest Taylor order and the most heads per call, each through prefill and
decode against the float64 oracle (same tolerances as the other parity tests).
"""
import sys

import numpy as np
import pytest

import oracle
import sata_synth as syn
from gpu_util import check_prefill_head, check_rows, check_state, operands, to_dev, to_host, y_tol

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


def _prefill_then_decode(sata, q, k, v, n, P, chunk, dtype, heads):
    """Prefill tokens [0, n), decode the rest one step at a time; check the
    listed (b, h) heads: every prefill row, every decoded row and both states."""
    dev = lambda a: to_dev(a, dtype)
    B, H = q.shape[:2]
    d = q.shape[-1]
    ops = operands(sata, dtype, B, H, n, d, v.shape[-1], P, chunk)
    y, S = sata.prefill(dev(q[:, :, :n]), dev(k[:, :, :n]), dev(v[:, :, :n]), P, chunk)
    torch.cuda.synchronize()
    for b, h in heads:
        check_prefill_head(to_host(y[b, h]), to_host(S[b, h]), q[b, h, :n], k[b, h, :n], v[b, h, :n], P,
                           ops, dtype, chunk, f"prefill b{b} h{h}")
    del y
    steps = q.shape[2] - n
    ys = []
    for t in range(n, n + steps):
        ys.append(sata.decode_step(S, dev(q[:, :, t].copy()), dev(k[:, :, t].copy()), dev(v[:, :, t].copy()), P))
    torch.cuda.synchronize()
    for b, h in heads:
        yr, _, kap = oracle.taylor_attention_rows(q[b, h], k[b, h], v[b, h], P, list(range(n, n + steps)))
        got = np.stack([to_host(yy[b, h]) for yy in ys])
        check_rows(got, yr, kap, y_tol(ops, dtype), P, f"decode b{b} h{h}")
        check_state(to_host(S[b, h]), k[b, h], v[b, h], P, ops, n, chunk, f"decode state b{b} h{h}", steps=steps)
    return S


def test_largest_head_dim(sata):
    """d_k = d_v = 255, the largest accepted, at P = 2 (D = 256): float32
    prefill in chunks of 16 over a ragged 40 tokens, then 2 decode steps."""
    d, P, n, steps = 255, 2, 40, 2
    _say(f"limits: d={d} P={P} n={n} decode {steps}")
    q, k, v = syn.make_qkv(60, 1, 1, n + steps, d, d, "f32")
    _prefill_then_decode(sata, q, k, v, n, P, 16, "f32", [(0, 0)])


def test_largest_head_dim_chunk_refused_untouched(sata):
    """At d = 255 the 64-token chunk's tiles do not fit on chip: the call is
    refused as unsupported and writes neither output."""
    d, P, n = 255, 2, 8
    q, k, v = syn.make_qkv(61, 1, 1, n, d, d, "f32")
    dev = lambda a: to_dev(a, "f32")
    y = torch.full((1, 1, n, d), 7.0, device="cuda")
    S = torch.full((1, 1, oracle.feature_count(d, P), d + 1), 7.0, device="cuda")
    with pytest.raises(sata.SataError) as err:
        sata.prefill(dev(q), dev(k), dev(v), P, 64, y=y, S=S)
    assert err.value.status == -2
    torch.cuda.synchronize()
    assert bool((y == 7.0).all()) and bool((S == 7.0).all())


@pytest.mark.parametrize("B,H,n,steps,d,P,chunk,dtype", [
    (1, 2, 70, 3, 3, 8, 32, "f32"),    # D = 120, 7 factors per feature
    (1, 1, 45, 2, 4, 8, 16, "bf16"),   # D = 330
])
def test_highest_order(sata, B, H, n, steps, d, P, chunk, dtype):
    """P = 8, the highest accepted order (features of degree up to 7)."""
    _say(f"limits: P={P} d={d} n={n} {dtype}")
    q, k, v = syn.make_qkv(62 + d, B, H, n + steps, d, d, dtype)
    _prefill_then_decode(sata, q, k, v, n, P, chunk, dtype, [(b, h) for b in range(B) for h in range(H)])


def test_most_heads(sata):
    """B*H = 65535, the most accepted, on the benchmark's kernels (bf16,
    d = 32, P = 4, chunk 64; 56.6 GB of state): a ragged 70-token prefill and
    one decode step, checked on heads at both ends, at batch boundaries and
    at random."""
    B, H, n, steps, d, P = 5, 13107, 70, 1, 32, 4
    _say(f"limits: B={B} H={H} n={n} d={d} P={P} bf16")
    q, k, v = syn.make_qkv(63, B, H, n + steps, d, d, "bf16")
    rng = np.random.default_rng(63)
    heads = [(0, 0), (0, 1), (0, H - 1), (1, 0), (2, H // 2), (B - 1, H - 1)]
    heads += [(int(rng.integers(B)), int(rng.integers(H))) for _ in range(3)]
    S = _prefill_then_decode(sata, q, k, v, n, P, 64, "bf16", heads)
    del S
    torch.cuda.empty_cache()


def test_long_call_keeps_workspace_bounded(sata):
    """bf16, P = 4, d = 32, chunk 64, 4 heads of 2^21 tokens: the tuned d = 32
    kernel would hold 576 bytes of partial readouts per head-token (4.8 GB), so
    the call takes the segmented matrix-core kernel (at most 512 MB of partial
    sums per segment).  Sampled rows of two heads against the oracle."""
    H, n, d, P = 4, 1 << 21, 32, 4
    _say(f"long bf16 call H={H} n={n}: generate inputs")
    heads = [tuple(syn.round_to_bf16(a) for a in syn.long_head(720 + h, n, d, d)) for h in range(H)]
    qd, kd, vd = (torch.stack([torch.from_numpy(hd[i]) for hd in heads]).view(1, H, n, d).to("cuda")
                  .to(torch.bfloat16) for i in range(3))
    assert operands(sata, "bf16", 1, H, n, d, d, P, 64) == "bf16"
    _say("prefill")
    y, _ = sata.prefill(qd, kd, vd, P, 64, want_state=False)
    torch.cuda.synchronize()
    rows = [0, 63, 64, 4097, n // 3, n - 65, n - 1]
    for h in (0, H - 1):
        _say(f"oracle rows head {h}")
        q, k, v = (a.astype(np.float64) for a in heads[h])
        yr, _, kap = oracle.taylor_attention_rows(q, k, v, P, rows)
        got = y[0, h, rows].float().cpu().numpy().astype(np.float64)
        check_rows(got, yr, kap, y_tol("bf16", "bf16"), P, f"long call head {h}")
