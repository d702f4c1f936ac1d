"""GPU parity of the compensated decode (sata_decode_step_compensated): the
method's constant cost per token holds however long the context (Sec. 1,
Sec. 3.2), and with the compensated entries its outputs also keep float32
accuracy past 2^24 tokens, where a plain float32 normaliser stops counting.

* Small shapes (every decode kernel layout: one workgroup per head, two and
  many pieces per head): rows against the float64 oracle, the state element
  by element, and the residuals within float32 roundoff of the state.
* d = 8, P = 4, float32, one head: a prefill of 2^24 + 64 tokens, then 4096
  decode steps; sampled decoded rows against the oracle within 1e-4.
"""
import sys
import time

import numpy as np
import pytest

import oracle
import sata_synth as syn
from gpu_util import check_rows, check_state, operands, to_dev, to_host, y_tol

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
    print(f"[{time.strftime('%H:%M:%S')}] {msg}", file=sys.stderr, flush=True)


@pytest.mark.parametrize("B,H,n1,n2,d,P,dtype", [
    (2, 2, 40, 5, 8, 4, "f32"),      # small heads, one 256-thread workgroup each
    (1, 3, 64, 4, 16, 4, "bf16"),
    (1, 2, 70, 3, 32, 4, "bf16"),    # two pieces per head
    (1, 1, 20, 2, 64, 4, "f32"),     # many pieces per head
    (1, 2, 0, 4, 5, 3, "f32"),       # from an empty state; rows of 6 floats
    (2, 2, 33, 3, 7, 5, "bf16"),
])
def test_compensated_decode_matches_oracle(sata, B, H, n1, n2, d, P, dtype):
    _say(f"compensated decode B={B} H={H} n1={n1} n2={n2} d={d} P={P} {dtype}")
    q, k, v = syn.make_qkv(120 + d, B, H, n1 + n2, d, d, dtype)
    dev = lambda a: to_dev(np.ascontiguousarray(a), dtype)
    D = oracle.feature_count(d, P)
    if n1 > 0:
        _, S = sata.prefill(dev(q[:, :, :n1]), dev(k[:, :, :n1]), dev(v[:, :, :n1]), P, 32)
        ops = operands(sata, dtype, B, H, n1, d, d, P, 32)
    else:
        S = torch.zeros(B, H, D, d + 1, device="cuda")
        ops = "f32"
    R = torch.zeros(B, H, sata.residual_elems(d, d, P), device="cuda")
    S_plain = S.clone()
    ys, ys_plain = [], []
    for t in range(n1, n1 + n2):
        args = [dev(a[:, :, t]) for a in (q, k, v)]
        ys.append(to_host(sata.decode_step_compensated(S, R, *args, P)))
        ys_plain.append(to_host(sata.decode_step(S_plain, *args, P)))
    torch.cuda.synchronize()
    Sh, Rh = to_host(S), to_host(R)
    for b in range(B):
        for h in range(H):
            yr, _, kap = oracle.taylor_attention_rows(q[b, h], k[b, h], v[b, h], P, list(range(n1, n1 + n2)))
            got = np.stack([yy[b, h] for yy in ys])
            check_rows(got, yr, kap, y_tol(ops, dtype), P, f"b{b} h{h}")
            # over a short context the residuals change nothing beyond float32
            # rounding (and at most one step of the bfloat16 output rounding)
            plain = np.stack([yy[b, h] for yy in ys_plain])
            same = 1e-5 if dtype == "f32" else 2.0 ** -7
            assert np.max(oracle.row_rel_error(got, plain)) < same
            check_state(Sh[b, h], k[b, h], v[b, h], P, ops, n1, 32, f"state b{b} h{h}", steps=n2)
            # a residual is at most half an ulp of its entry (plus what it carries from the last step)
            z = Sh[b, h][:, d]
            assert np.all(np.abs(Rh[b, h][:D]) <= 2.0 ** -23 * np.abs(z) + 1e-30)
            pre = Sh[b, h][: d + 1, :d].reshape(-1)
            assert np.all(np.abs(Rh[b, h][D:]) <= 2.0 ** -23 * np.abs(pre) + 1e-30)


def test_compensated_decode_refuses_unaligned_state(sata):
    d, P = 8, 4
    D = oracle.feature_count(d, P)
    flat = torch.zeros(D * (d + 1) + 1, device="cuda")
    S = flat[1:].view(1, 1, D, d + 1)
    R = torch.zeros(1, 1, sata.residual_elems(d, d, P), device="cuda")
    x = torch.zeros(1, 1, d, device="cuda")
    with pytest.raises(sata.SataError) as err:
        sata.decode_step_compensated(S, R, x, x, x, P)
    assert err.value.status == -2


def test_compensated_decode_after_2_pow_24_tokens(sata):
    """One float32 head (d = 8, P = 4): a prefill of 2^24 + 64 tokens, where the
    float32 token count has an ulp of 2, then 4096 decode steps.  Decoded rows
    spread over the steps match the float64 oracle within 1e-4 with the
    compensated call; the plain call's error is reported beside it (every one
    of its 4096 count increments is lost)."""
    n, steps, d, P = (1 << 24) + 64, 4096, 8, 4
    _say(f"long decode: generate {n + steps} tokens")
    q, k, v = syn.long_head(709, n + steps, d, d)
    dev = [torch.from_numpy(a[:n]).to("cuda").view(1, 1, n, d) for a in (q, k, v)]
    _say("prefill")
    _, S = sata.prefill(*dev, P, 64)
    torch.cuda.synchronize()
    del dev
    S_plain = S.clone()
    R = torch.zeros(1, 1, sata.residual_elems(d, d, P), device="cuda")
    dq, dk_, dv_ = (torch.from_numpy(np.ascontiguousarray(a[n:])).to("cuda") for a in (q, k, v))
    y = torch.empty(steps, d, device="cuda")
    y_plain = torch.empty(steps, d, device="cuda")
    _say(f"decode {steps} steps, compensated and plain")
    for t in range(steps):
        a = [dq[t].view(1, 1, d), dk_[t].view(1, 1, d), dv_[t].view(1, 1, d)]
        sata.decode_step_compensated(S, R, *a, P, y=y[t].view(1, 1, d))
        sata.decode_step(S_plain, *a, P, y=y_plain[t].view(1, 1, d))
    torch.cuda.synchronize()
    sample = [0, 1, 255, 1024, 2047, 3071, 4094, 4095]
    _say("oracle rows")
    yr, _, kap = oracle.taylor_attention_rows(q, k, v, P, [n + t for t in sample])
    got = y.cpu().numpy().astype(np.float64)[sample]
    err, _ = check_rows(got, yr, kap, y_tol("f32", "f32"), P, "compensated")
    err_plain = float(np.max(oracle.row_rel_error(y_plain.cpu().numpy().astype(np.float64)[sample], yr)))
    _say(f"after {n} + {steps} tokens: compensated row error {err:.3e}, plain {err_plain:.3e}")
    count = float(S[0, 0, 0, d].item()) + float(R[0, 0, 0].item())
    assert count == n + steps, count             # the degree-0 normaliser is the exact token count
    assert float(S_plain[0, 0, 0, d].item()) == n  # (the plain one stopped counting)
