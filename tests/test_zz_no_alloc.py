"""The allocation-free decode entry point (sata_decode_step_noalloc) against
sata_decode_step through the C ABI: bitwise the same outputs and states on two
calls in a row, the second with a smaller input, both using the static
scratch (split heads with partial sums and arrival counters).  Also its
refusals: a (d_k, P) with no feature table on the device yet, and partial
sums beyond the scratch."""
import ctypes

import numpy as np
import pytest

import oracle
import sata_synth as syn
from gpu_util import to_dev

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


@pytest.fixture(scope="module")
def lib():
    if not torch.cuda.is_available():
        pytest.fail("no GPU visible")
    from paper_2602_00294_amd import _binding
    return _binding.load_library()


def _ptr(t):
    return ctypes.c_void_p(t.data_ptr())


def _stream():
    return ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)


def _call(fn, S, q, k, v, y, code, d, P):
    B, H = q.shape[:2]
    return fn(_ptr(S), _ptr(q), _ptr(k), _ptr(v), code, B, H, d, d, P, _ptr(y), _stream())


def test_noalloc_decode_matches_decode_step(lib):
    P = 4
    # first call: 96 heads of d = 32 (two pieces per head: partial sums and
    # counters in the scratch); second call: fewer heads, then a small-head shape
    for i, (B, H, d, dtype) in enumerate([(2, 48, 32, "bf16"), (1, 5, 32, "bf16"), (1, 3, 8, "f32")]):
        rng = np.random.default_rng(200 + i)
        D = oracle.feature_count(d, P)
        S0 = rng.standard_normal((B, H, D, d + 1)).astype(np.float32)
        S0[..., d] = np.abs(S0[..., d]) + 50.0
        q, k, v = (to_dev(a[:, :, 0].copy(), dtype) for a in syn.make_qkv(210 + i, B, H, 1, d, d, dtype))
        code = 1 if dtype == "bf16" else 0
        S_ref = torch.from_numpy(S0).cuda()
        y_ref = torch.empty(B, H, d, dtype=q.dtype, device="cuda")
        assert _call(lib.sata_decode_step, S_ref, q, k, v, y_ref, code, d, P) == 0
        # twice on the same input: the scratch keeps the last call's contents,
        # which the repeat must not see
        for rep in range(2):
            S_new = torch.from_numpy(S0).cuda()
            y_new = torch.full_like(y_ref, 7.0)
            assert _call(lib.sata_decode_step_noalloc, S_new, q, k, v, y_new, code, d, P) == 0, \
                lib.sata_last_error().decode()
            torch.cuda.synchronize()
            assert torch.equal(y_new, y_ref), f"call {i} repeat {rep}"
            assert torch.equal(S_new, S_ref), f"call {i} repeat {rep}"


def test_noalloc_refusals(lib):
    # (d_k, P) = (13, 2) is used by no other test: no table exists for it yet
    x = torch.zeros(1, 1, 13, device="cuda")
    y = torch.empty(1, 1, 13, device="cuda")
    S = torch.zeros(1, 1, oracle.feature_count(13, 2), 14, device="cuda")
    S[..., 13] = 1.0
    st = _call(lib.sata_decode_step_noalloc, S, x, x, x, y, 0, 13, 2)
    assert st in (0, -2)
    if st == -2:
        assert "table" in lib.sata_last_error().decode()
        assert _call(lib.sata_decode_step, S.clone(), x, x, x, y, 0, 13, 2) == 0
        assert _call(lib.sata_decode_step_noalloc, S, x, x, x, y, 0, 13, 2) == 0
    # 16000 heads of d = 32 need 2 * 16000 * 33 floats of partial sums: more than the scratch
    fake = ctypes.c_void_p(0x1000)  # never dereferenced: refused before any launch
    st = lib.sata_decode_step_noalloc(fake, fake, fake, fake, 1, 1, 16000, 32, 32, 4, fake, None)
    assert st == -3 and "scratch" in lib.sata_last_error().decode()
    torch.cuda.synchronize()
