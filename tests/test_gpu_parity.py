"""GPU parity: every hot-path call through the C ABI against the float64 oracle.

Inputs are the seeded synthetic N(0,1) tensors of sata_synth.  Per query row,
||y - y_ref|| / ||y_ref|| must be within 2e-2 where the state contractions take
bfloat16 operands, 1e-4 with float32 arithmetic and output, 2^-8 with float32
arithmetic and a bfloat16 output, over rows whose denominator does not cancel
(kappa <= 100; none may be left out at odd P).  States are compared element
by element against the bound that the path's arithmetic allows
(oracle.metrics.state_tol).
"""
import sys

import numpy as np
import pytest

import oracle
import sata_synth as syn
from gpu_util import (check_prefill_head, check_rows, check_state, check_state_against, operands, to_dev, to_host,
                      torch_dtype, y_tol)
from oracle.metrics import max_row_rel_error

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


# ------------------------------------------------------------------ feature map

@pytest.mark.parametrize("d,P,rows,dtype", [
    (8, 4, 37, "f32"), (16, 4, 100, "bf16"), (3, 7, 19, "f32"), (32, 4, 65, "bf16"),
    (1, 1, 5, "f32"), (5, 2, 1, "f32"), (64, 3, 33, "f32"),
    # the largest d, degrees above 3 over several row blocks, and more rows
    # than one launch takes (65535 blocks of 32 rows)
    (255, 2, 40, "bf16"), (16, 6, 3000, "f32"), (1, 2, 2_100_001, "f32")])
def test_feature_map(sata, d, P, rows, dtype):
    _say(f"feature_map d={d} P={P} rows={rows} {dtype}")
    x = syn.head_stream(100, d, P, 0, (rows, d), dtype)
    phi = to_host(sata.feature_map(to_dev(x, dtype), P))
    ref = oracle.phi_ref(x, P)
    assert phi.shape == ref.shape
    np.testing.assert_allclose(phi, ref, rtol=2e-6, atol=1e-30)


def test_feature_map_many_row_blocks_and_feature_blocks(sata):
    """Several feature blocks per row (D = 561) over more row blocks than one
    launch takes (65535 blocks of 32 rows): the XCD-ordered tiles of every
    launch cover each output once.  Sampled rows: the first, those around the
    launch boundary (row 65535 * 32) and the last."""
    d, P, rows = 32, 3, 2_100_000
    D = oracle.feature_count(d, P)
    x = syn.head_stream(102, d, P, 0, (rows, d), "f32")
    phi = sata.feature_map(to_dev(x, "f32"), P)
    torch.cuda.synchronize()
    b = 65535 * 32
    idx = np.r_[0:40, b - 40:b + 40, rows - 40:rows]
    got = to_host(phi[torch.from_numpy(idx).cuda()])
    np.testing.assert_allclose(got, oracle.phi_ref(x[idx], P), rtol=2e-6, atol=1e-30)
    assert bool(torch.isfinite(phi).all())


def test_feature_map_unaligned_output(sata):
    """An output pointer that is not 16-byte aligned (the C ABI allows any
    float pointer) takes element stores; the elements around it stay untouched."""
    import ctypes
    d, P, rows = 6, 4, 50
    D = oracle.feature_count(d, P)
    x = syn.head_stream(101, d, P, 0, (rows, d), "f32")
    xd = to_dev(x, "f32")
    buf = torch.full((rows * D + 8,), -7.0, device="cuda")
    lib = sata.load_library()
    st = lib.sata_feature_map(ctypes.c_void_p(xd.data_ptr()), 0, rows, d, P, ctypes.c_void_p(buf.data_ptr() + 4),
                              ctypes.c_void_p(torch.cuda.current_stream().cuda_stream))
    torch.cuda.synchronize()
    assert st == 0
    b = to_host(buf)
    assert b[0] == -7.0 and np.all(b[1 + rows * D:] == -7.0)
    np.testing.assert_allclose(b[1:1 + rows * D].reshape(rows, D), oracle.phi_ref(x, P), rtol=2e-6, atol=1e-30)


# ------------------------------------------------------------------ prefill

def _run_prefill(sata, workload, B, H, n, dk, dv, P, chunk, dtype, want_state=True):
    q, k, v = syn.make_qkv(workload, B, H, n, dk, dv, dtype)
    y, S = sata.prefill(to_dev(q, dtype), to_dev(k, dtype), to_dev(v, dtype), P, chunk, want_state=want_state)
    torch.cuda.synchronize()
    return q, k, v, to_host(y), (to_host(S) if S is not None else None)


PREFILL_CASES = [
    # workload, B, H, n, d_k, d_v, P, chunk, dtype
    (1, 1, 1, 256, 8, 8, 4, 64, "f32"),       # the single-head n=256 d=8 P=4 case
    (11, 1, 2, 77, 5, 3, 3, 16, "f32"),
    (12, 2, 1, 130, 4, 7, 5, 32, "f32"),
    (13, 1, 1, 1, 8, 8, 4, 64, "f32"),
    (14, 1, 1, 200, 16, 16, 6, 128, "f32"),
    (15, 1, 1, 50, 4, 4, 1, 16, "f32"),
    (16, 2, 2, 65, 8, 8, 2, 64, "bf16"),
    (17, 1, 3, 129, 16, 16, 4, 64, "bf16"),
    (18, 1, 2, 300, 32, 32, 4, 64, "bf16"),
    (19, 1, 1, 97, 2, 9, 7, 32, "f32"),
    # bf16, P = 4, d in {16, 32}: the matrix-core path
    (22, 2, 2, 100, 16, 16, 4, 32, "bf16"),
    (23, 1, 2, 257, 32, 32, 4, 128, "bf16"),
    (24, 1, 1, 5, 32, 32, 4, 64, "bf16"),
    (25, 3, 1, 64, 16, 16, 4, 64, "bf16"),
    (26, 1, 1, 1, 16, 16, 4, 32, "bf16"),
    (27, 2, 3, 191, 32, 32, 4, 64, "bf16"),
]


@pytest.mark.parametrize("case", PREFILL_CASES, ids=lambda c: "w{}_B{}H{}n{}dk{}dv{}P{}C{}_{}".format(*c))
def test_prefill_matches_oracle(sata, case):
    workload, B, H, n, dk, dv, P, chunk, dtype = case
    _say(f"prefill {case}")
    ops = operands(sata, dtype, B, H, n, dk, dv, P, chunk)
    q, k, v, y, S = _run_prefill(sata, *case)
    for b in range(B):
        for h in range(H):
            check_prefill_head(y[b, h], S[b, h], q[b, h], k[b, h], v[b, h], P, ops, dtype, chunk,
                               f"{case} {ops} b{b} h{h}")


# Shapes without a dedicated kernel: the matrix-core kernel that generates
# every feature from its monomial (any P >= 2, d_k and d_v up to 64, chunk 64;
# bf16 inputs as bf16 operands, float32 inputs as split hi + lo operands).
# The cases cover one to five column tiles of 16 (d_v + 1 up to 65), P = 2..7,
# several feature slices per head, ragged last chunks and single tokens.
FEATURE_KERNEL_CASES = [
    # workload, B, H, n, d_k, d_v, P, chunk, dtype
    (30, 1, 2, 200, 8, 8, 3, 64, "bf16"),
    (31, 1, 1, 130, 16, 16, 5, 64, "bf16"),
    (32, 1, 1, 97, 32, 32, 3, 64, "bf16"),
    (33, 1, 1, 70, 32, 32, 5, 64, "bf16"),
    (34, 1, 2, 129, 24, 48, 4, 64, "bf16"),
    (35, 1, 1, 130, 64, 64, 4, 64, "bf16"),
    (36, 2, 1, 64, 64, 64, 3, 64, "bf16"),
    (37, 2, 1, 1, 5, 3, 6, 64, "bf16"),
    # (d_v = 2 rather than 1: a one-element row is a single weighted mean of
    # N(0,1) values, which lands near zero somewhere in 300 rows, and there a
    # relative error measures the bf16 rounding of the other terms, not the kernel)
    (38, 1, 1, 300, 7, 2, 6, 64, "bf16"),
    (39, 1, 1, 65, 64, 16, 2, 64, "bf16"),
    (40, 1, 1, 90, 3, 64, 7, 64, "bf16"),
    # float32 inputs: split operands (16-byte vector loads where d_k and d_v
    # are multiples of 4, element loads otherwise)
    (41, 1, 2, 200, 8, 8, 3, 64, "f32"),
    (42, 1, 1, 130, 16, 16, 5, 64, "f32"),
    (43, 1, 1, 97, 32, 32, 4, 64, "f32"),
    (44, 1, 2, 129, 24, 48, 4, 64, "f32"),
    (45, 1, 1, 130, 64, 64, 3, 64, "f32"),
    (46, 2, 1, 1, 5, 3, 6, 64, "f32"),
    (47, 1, 1, 300, 7, 2, 6, 64, "f32"),
    (48, 1, 1, 90, 3, 64, 7, 64, "f32"),
]


@pytest.mark.parametrize("case", FEATURE_KERNEL_CASES, ids=lambda c: "w{}_B{}H{}n{}dk{}dv{}P{}C{}_{}".format(*c))
def test_prefill_generated_features_matches_oracle(sata, case):
    workload, B, H, n, dk, dv, P, chunk, dtype = case
    _say(f"prefill (generated features) {case}")
    ops = operands(sata, dtype, B, H, n, dk, dv, P, chunk)
    assert ops == ("bf16" if dtype == "bf16" else "split"), "expected on the matrix cores"
    q, k, v, y, S = _run_prefill(sata, *case)
    for b in range(B):
        for h in range(H):
            check_prefill_head(y[b, h], S[b, h], q[b, h], k[b, h], v[b, h], P, ops, dtype, chunk,
                               f"{case} b{b} h{h}")


# Few heads with few features over a long sequence: the sequence is cut into
# parts that run side by side, each starting from the summed state increments
# of the parts before it (sata_prefill_parts); every row and the final state
# against the oracle.
SPLIT_CASES = [
    # workload, B, H, n, d_k, d_v, P, chunk, dtype, parts
    (55, 1, 2, 8192, 8, 8, 3, 64, "f32", 8),
    (56, 1, 1, 4150, 16, 16, 2, 64, "bf16", 4),
    (57, 2, 1, 3000, 5, 3, 4, 64, "f32", 2),
    (58, 1, 1, 2100, 24, 48, 3, 64, "bf16", 2),
]


@pytest.mark.parametrize("case", SPLIT_CASES, ids=lambda c: "w{}_B{}H{}n{}dk{}dv{}P{}C{}_{}_parts{}".format(*c))
def test_prefill_split_sequence_matches_oracle(sata, case):
    *args, parts = case
    workload, B, H, n, dk, dv, P, chunk, dtype = args
    _say(f"prefill (sequence in parts) {case}")
    assert sata.prefill_parts(torch_dtype(dtype), B, H, n, dk, dv, P, chunk) == parts
    ops = operands(sata, dtype, B, H, n, dk, dv, P, chunk)
    q, k, v, y, S = _run_prefill(sata, *args)
    for b in range(B):
        for h in range(H):
            check_prefill_head(y[b, h], S[b, h], q[b, h], k[b, h], v[b, h], P, ops, dtype, chunk,
                               f"{case} b{b} h{h}")


# Many heads and features: the wide slices (more feature tiles per wave) that
# the kernel takes when they still give at least two workgroups per compute
# unit; one case per column-tile count and input type, sampled heads.
WIDE_CASES = [
    # workload, d_k, d_v, P
    (50, 32, 8, 4), (51, 16, 16, 5), (52, 32, 40, 4), (53, 24, 48, 4), (54, 16, 64, 4),
]


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
@pytest.mark.parametrize("case", WIDE_CASES, ids=lambda c: "w{}_dk{}dv{}P{}".format(*c))
def test_prefill_generated_features_wide_slices(sata, case, dtype):
    workload, dk, dv, P = case
    B, H, n = 1, 256, 40
    _say(f"prefill (generated features, wide slices) {case} {dtype}")
    ops = operands(sata, dtype, B, H, n, dk, dv, P, 64)
    assert ops == ("bf16" if dtype == "bf16" else "split")
    q, k, v, y, S = _run_prefill(sata, workload, B, H, n, dk, dv, P, 64, dtype)
    for h in (0, 85, 170, 255):
        check_prefill_head(y[0, h], S[0, h] if h in (0, 255) else None, q[0, h], k[0, h], v[0, h], P, ops, dtype, 64,
                           f"{case} {dtype} h{h}")


def test_prefill_empty_sequence_zeroes_state(sata):
    S = torch.full((1, 2, oracle.feature_count(4, 3), 6), 7.0, device="cuda")
    q = torch.empty(1, 2, 0, 4, device="cuda")
    v = torch.empty(1, 2, 0, 5, device="cuda")
    y, S2 = sata.prefill(q, q, v, 3, 32, S=S)
    torch.cuda.synchronize()
    assert y.numel() == 0 and float(S2.abs().max()) == 0.0


def test_prefill_deterministic(sata):
    q, k, v = syn.make_qkv(20, 1, 2, 333, 16, 16, "bf16")
    args = [to_dev(a, "bf16") for a in (q, k, v)]
    y1, S1 = sata.prefill(*args, 4, 64)
    y2, S2 = sata.prefill(*args, 4, 64)
    torch.cuda.synchronize()
    assert torch.equal(y1, y2) and torch.equal(S1, S2)


def test_prefill_chunk_invariance(sata):
    """The chunk size changes only the rounding: float32 inputs, d = 8.  Chunks
    16, 32 and 128 run in float32 arithmetic; chunk 64 on the matrix cores with
    split operands, held to that arithmetic's bounds against chunk 16."""
    q, k, v = syn.make_qkv(21, 1, 1, 300, 8, 8, "f32")
    chunks = (16, 32, 64, 128)
    ops = {c: operands(sata, "f32", 1, 1, 300, 8, 8, 4, c) for c in chunks}
    assert ops == {16: "f32", 32: "f32", 64: "split", 128: "f32"}
    outs = {c: sata.prefill(*(to_dev(a, "f32") for a in (q, k, v)), 4, c) for c in chunks}
    torch.cuda.synchronize()
    y0, S0 = to_host(outs[16][0]), to_host(outs[16][1])
    S_abs = oracle.state_abs_ref(k[0, 0], v[0, 0], 4)
    for c in (32, 128):
        assert max_row_rel_error(to_host(outs[c][0])[0, 0], y0[0, 0])[0] < 1e-5
        check_state_against(to_host(outs[c][1])[0, 0], S0[0, 0], S_abs, 2e-5, f"chunk {c}")
    assert max_row_rel_error(to_host(outs[64][0])[0, 0], y0[0, 0])[0] < y_tol("split", "f32")
    check_state_against(to_host(outs[64][1])[0, 0], S0[0, 0], S_abs,
                        oracle.state_tol("split", 300, 64, 4) + oracle.state_tol("f32", 300, 16, 4), "chunk 64")


@pytest.mark.parametrize("d", [16, 32])
def test_prefill_chunk_invariance_matrix_cores(sata, d):
    """bf16, P = 4 on the matrix-core kernels: chunks 32, 64 and 128 (served by
    different kernel variants) each match the oracle, and agree with each
    other within the bfloat16-operand bounds."""
    B, H, n, P = 1, 2, 300, 4
    q, k, v = syn.make_qkv(28 + d, B, H, n, d, d, "bf16")
    res = {}
    for c in (32, 64, 128):
        ops = operands(sata, "bf16", B, H, n, d, d, P, c)
        assert ops == "bf16", f"chunk {c} is expected on the matrix cores"
        y, S = sata.prefill(*(to_dev(a, "bf16") for a in (q, k, v)), P, c)
        torch.cuda.synchronize()
        res[c] = (to_host(y), to_host(S))
        for h in range(H):
            check_prefill_head(res[c][0][0, h], res[c][1][0, h], q[0, h], k[0, h], v[0, h], P, ops, "bf16", c,
                               f"d{d} chunk {c} h{h}")
    for h in range(H):
        S_abs = oracle.state_abs_ref(k[0, h], v[0, h], P)
        for c in (32, 128):
            assert max_row_rel_error(res[c][0][0, h], res[64][0][0, h])[0] < 2 * y_tol("bf16", "bf16")
            check_state_against(res[c][1][0, h], res[64][1][0, h], S_abs, 2 * oracle.state_tol("bf16", n, c, P),
                                f"d{d} chunk {c} vs 64 h{h}")


def test_prefill_rejects_bad_chunk(sata):
    x = torch.zeros(1, 1, 4, 4, device="cuda")
    with pytest.raises(sata.SataError):
        sata.prefill(x, x, x, 3, 48)


# ------------------------------------------------------------------ decode

@pytest.mark.parametrize("B,H,n1,n2,d,P,dtype", [
    (2, 2, 40, 9, 8, 4, "f32"), (1, 3, 64, 5, 16, 4, "bf16"), (1, 1, 0, 6, 4, 3, "f32"),
    (1, 2, 70, 4, 32, 4, "bf16"), (1, 1, 20, 3, 5, 6, "f32")])
def test_decode_continues_prefill(sata, B, H, n1, n2, d, P, dtype):
    _say(f"decode B={B} H={H} n1={n1} n2={n2} d={d} P={P} {dtype}")
    q, k, v = syn.make_qkv(30 + d, B, H, n1 + n2, d, d, dtype)
    dev = lambda a: to_dev(a, dtype)
    D = oracle.feature_count(d, P)
    if n1 > 0:
        _, S = sata.prefill(dev(q[:, :, :n1]), dev(k[:, :, :n1]), dev(v[:, :, :n1]), P, 32)
    else:
        S = torch.zeros(B, H, D, d + 1, device="cuda")
    ops = operands(sata, dtype, B, H, max(n1, 1), d, d, P, 32) if n1 > 0 else "f32"
    ys = []
    for t in range(n1, n1 + n2):
        ys.append(to_host(sata.decode_step(S, dev(q[:, :, t].copy()), dev(k[:, :, t].copy()),
                                           dev(v[:, :, t].copy()), P)))
    torch.cuda.synchronize()
    S_host = to_host(S)
    for b in range(B):
        for h in range(H):
            yr, _, kap = oracle.taylor_attention_rows(q[b, h], k[b, h], v[b, h], P, list(range(n1, n1 + n2)))
            got = np.stack([yy[b, h] for yy in ys])
            check_rows(got, yr, kap, y_tol(ops, dtype), P, f"b{b} h{h}")
            check_state(S_host[b, h], k[b, h], v[b, h], P, ops, n1, 32, f"state b{b} h{h}", steps=n2)


def test_decode_large_state_slices(sata):
    """A state large enough to be split over several workgroups per head."""
    d, P, B, H = 32, 4, 1, 2
    q, k, v = syn.make_qkv(40, B, H, 8, d, d, "f32")
    D = oracle.feature_count(d, P)
    rng = np.random.default_rng(5)
    S0 = rng.standard_normal((B, H, D, d + 1)).astype(np.float32)
    S0[..., d] = np.abs(S0[..., d]) + 50.0       # a comfortably positive normaliser
    S = torch.from_numpy(S0).cuda()
    y = to_host(sata.decode_step(S, to_dev(q[:, :, 0].copy(), "f32"), to_dev(k[:, :, 0].copy(), "f32"),
                                 to_dev(v[:, :, 0].copy(), "f32"), P))
    torch.cuda.synchronize()
    for h in range(H):
        yr, Sr = oracle.decode_ref(S0[0, h], q[0, h, :1], k[0, h, :1], v[0, h, :1], P)
        assert max_row_rel_error(y[0, h][None], yr)[0] < 1e-4
        _check_decoded_state(to_host(S)[0, h], S0[0, h], Sr, k[0, h, :1], v[0, h, :1], P, f"h{h}")


def _check_decoded_state(S_gpu, S0, Sr, k, v, P, label):
    """A state that started from S0 (not a sum of tokens) and took len(k)
    decode steps: each entry is off by at most a few float32 roundings of
    |S0| plus the magnitudes of the added terms."""
    S_abs = np.abs(np.asarray(S0, np.float64)) + oracle.state_abs_ref(k, v, P)
    check_state_against(S_gpu, Sr, S_abs, oracle.state_tol("f32", 0, 1, P, steps=len(k)), label)


def _random_state(rng, B, H, D, dv):
    S0 = rng.standard_normal((B, H, D, dv + 1)).astype(np.float32)
    S0[..., dv] = np.abs(S0[..., dv]) + 50.0       # a comfortably positive normaliser
    return S0


def test_decode_shapes_interleaved_on_one_stream(sata):
    """Decode calls of different B*H and d on one stream: the work-queue kernel's
    counters (shared between calls) must be back at zero after every call."""
    rng = np.random.default_rng(11)
    P = 4
    cases = [(1, 3, 32, "bf16"), (2, 40, 16, "bf16"), (1, 3, 32, "bf16"), (3, 5, 8, "f32"), (2, 40, 16, "bf16")]
    for i, (B, H, d, dtype) in enumerate(cases):
        _say(f"interleaved decode {i}: B={B} H={H} d={d} {dtype}")
        D = oracle.feature_count(d, P)
        S0 = _random_state(rng, B, H, D, d)
        q, k, v = syn.make_qkv(50 + i, B, H, 1, d, d, dtype)
        S = torch.from_numpy(S0).cuda()
        y = to_host(sata.decode_step(S, to_dev(q[:, :, 0].copy(), dtype), to_dev(k[:, :, 0].copy(), dtype),
                                     to_dev(v[:, :, 0].copy(), dtype), P))
        torch.cuda.synchronize()
        S_host = to_host(S)
        for b in range(B):
            for h in range(H):
                yr, Sr = oracle.decode_ref(S0[b, h], q[b, h, :1], k[b, h, :1], v[b, h, :1], P)
                assert max_row_rel_error(y[b, h][None], yr)[0] < y_tol("f32", dtype), f"case {i} b{b} h{h}"
                _check_decoded_state(S_host[b, h], S0[b, h], Sr, k[b, h, :1], v[b, h, :1], P,
                                     f"case {i} state b{b} h{h}")


def test_decode_unaligned_state(sata):
    """A state tensor that is not 16-byte aligned takes the row-wise kernel."""
    rng = np.random.default_rng(12)
    B, H, d, P = 1, 4, 16, 4
    D = oracle.feature_count(d, P)
    S0 = _random_state(rng, B, H, D, d)
    flat = torch.zeros(S0.size + 1, device="cuda")
    S = flat[1:].view(S0.shape)                    # offset by one float
    S.copy_(torch.from_numpy(S0).cuda())
    assert S.data_ptr() % 16 != 0
    q, k, v = syn.make_qkv(60, B, H, 1, d, d, "f32")
    y = to_host(sata.decode_step(S, to_dev(q[:, :, 0].copy(), "f32"), to_dev(k[:, :, 0].copy(), "f32"),
                                 to_dev(v[:, :, 0].copy(), "f32"), P))
    torch.cuda.synchronize()
    for h in range(H):
        yr, Sr = oracle.decode_ref(S0[0, h], q[0, h, :1], k[0, h, :1], v[0, h, :1], P)
        assert max_row_rel_error(y[0, h][None], yr)[0] < 1e-4
        _check_decoded_state(to_host(S)[0, h], S0[0, h], Sr, k[0, h, :1], v[0, h, :1], P, f"h{h}")


def test_decode_unaligned_large_state(sata):
    """A large head (d=64, feature values beyond LDS) whose state is not
    16-byte aligned takes the row-wise kernel in feature slices plus the
    launch that adds their sums."""
    rng = np.random.default_rng(13)
    B, H, d, P = 1, 2, 64, 4
    D = oracle.feature_count(d, P)
    S0 = _random_state(rng, B, H, D, d)
    flat = torch.zeros(S0.size + 1, device="cuda")
    S = flat[1:].view(S0.shape)                    # offset by one float
    S.copy_(torch.from_numpy(S0).cuda())
    assert S.data_ptr() % 16 != 0
    q, k, v = syn.make_qkv(61, B, H, 1, d, d, "f32")
    y = to_host(sata.decode_step(S, to_dev(q[:, :, 0].copy(), "f32"), to_dev(k[:, :, 0].copy(), "f32"),
                                 to_dev(v[:, :, 0].copy(), "f32"), P))
    torch.cuda.synchronize()
    Sh = to_host(S)
    for h in range(H):
        yr, Sr = oracle.decode_ref(S0[0, h], q[0, h, :1], k[0, h, :1], v[0, h, :1], P)
        assert max_row_rel_error(y[0, h][None], yr)[0] < 1e-4
        _check_decoded_state(Sh[0, h], S0[0, h], Sr, k[0, h, :1], v[0, h, :1], P, f"h{h}")


def test_decode_many_pieces_per_head(sata):
    """Few large heads: each is streamed by several pieces (d=64: D=47905,
    12.5 MB of state per head), bf16 inputs, two steps in a row."""
    rng = np.random.default_rng(14)
    B, H, d, P = 1, 3, 64, 4
    D = oracle.feature_count(d, P)
    S0 = _random_state(rng, B, H, D, d)
    S = torch.from_numpy(S0).cuda()
    q, k, v = syn.make_qkv(62, B, H, 2, d, d, "bf16")
    ys = []
    for t in range(2):
        ys.append(to_host(sata.decode_step(S, to_dev(q[:, :, t].copy(), "bf16"), to_dev(k[:, :, t].copy(), "bf16"),
                                           to_dev(v[:, :, t].copy(), "bf16"), P)))
    torch.cuda.synchronize()
    Sh = to_host(S)
    for h in range(H):
        yr, Sr = oracle.decode_ref(S0[0, h], q[0, h, :2], k[0, h, :2], v[0, h, :2], P)
        got = np.stack([yy[0, h] for yy in ys])
        assert max_row_rel_error(got, yr)[0] < y_tol("f32", "bf16")
        _check_decoded_state(Sh[0, h], S0[0, h], Sr, k[0, h, :2], v[0, h, :2], P, f"h{h}")


def test_state_host_round_trip_resumes_bit_identically(sata, tmp_path):
    """Checkpoint and resume: a prefill's state copied to host memory, written
    to a file, read back and copied to a new device tensor continues the
    decode with bitwise the same outputs and states as the original."""
    B, H, n, steps, d, P = 1, 3, 130, 3, 32, 4
    q, k, v = syn.make_qkv(70, B, H, n + steps, d, d, "bf16")
    dev = lambda a: to_dev(np.ascontiguousarray(a), "bf16")
    _, S = sata.prefill(dev(q[:, :, :n]), dev(k[:, :, :n]), dev(v[:, :, :n]), P, 64)
    torch.cuda.synchronize()
    path = tmp_path / "state.npy"
    np.save(path, S.cpu().numpy())
    S2 = torch.from_numpy(np.load(path)).cuda()
    assert torch.equal(S, S2)
    for t in range(n, n + steps):
        args = [dev(a[:, :, t]) for a in (q, k, v)]
        y1 = sata.decode_step(S, *args, P)
        y2 = sata.decode_step(S2, *args, P)
        torch.cuda.synchronize()
        assert torch.equal(y1, y2) and torch.equal(S, S2), f"step {t}"
