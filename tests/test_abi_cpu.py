"""CPU-side checks of the C ABI: the library loads, exports every declared
symbol, and its host-only calls and argument validation behave as documented.
No compute call reaches a GPU here."""
import ctypes
import itertools
import math

import pytest

import oracle
from paper_2602_00294_amd import _binding as bnd


@pytest.fixture(scope="module")
def lib():
    return bnd.load_library()


def test_exports_every_declared_symbol(lib):
    names = bnd.header_functions()
    assert {"sata_feature_map", "sata_prefill", "sata_decode_step"} <= set(names)
    for name in names:
        assert hasattr(lib, name), name


def test_feature_and_state_counts(lib):
    for d in (1, 2, 8, 16, 32, 64):
        for P in range(1, 8):
            assert lib.sata_feature_count(d, P) == oracle.feature_count(d, P)
            assert lib.sata_state_elems(d, 5, P) == oracle.state_elems(d, 5, P)
    assert lib.sata_feature_count(0, 4) == -1
    assert lib.sata_feature_count(4, 0) == -1


@pytest.mark.parametrize("d,P", [(1, 5), (2, 3), (3, 4), (8, 4), (5, 7), (16, 3)])
def test_feature_order_matches_oracle(d, P):
    want = oracle.multi_indices(d, P)
    got = [bnd.feature_index(d, P, f) for f in range(len(want))]
    assert got == want


def test_feature_index_spot_checks_large():
    # last feature of degree P-1 is (d-1, ..., d-1); the first of degree 2 is (0, 0)
    for d, P in ((32, 4), (64, 4), (16, 6)):
        D = oracle.feature_count(d, P)
        assert bnd.feature_index(d, P, D - 1) == (d - 1,) * (P - 1)
        assert bnd.feature_index(d, P, 1 + d) == (0, 0)
        assert bnd.feature_index(d, P, d) == (d - 1,)


def test_feature_index_rejects_out_of_range(lib):
    deg = ctypes.c_int(0)
    idx = (ctypes.c_int * 8)()
    assert lib.sata_feature_index(4, 3, 14, ctypes.byref(deg), idx) == bnd.SATA_OK
    assert deg.value == 2 and (idx[0], idx[1]) == (3, 3)
    assert lib.sata_feature_index(4, 3, 15, ctypes.byref(deg), idx) == -1
    assert lib.sata_feature_index(4, 3, -1, ctypes.byref(deg), idx) == -1
    assert lib.sata_feature_index(4, 3, 0, None, idx) == -1


NULL = ctypes.c_void_p(None)
FAKE = ctypes.c_void_p(0x1000)  # never dereferenced: validation fails first


@pytest.mark.parametrize("args,code", [
    # (dtype, B, H, n, dk, dv, P, chunk, ptr)
    ((7, 1, 1, 8, 4, 4, 4, 64, FAKE), -1),       # bad dtype
    ((0, 0, 1, 8, 4, 4, 4, 64, FAKE), -1),       # B = 0
    ((0, 1, 1, -1, 4, 4, 4, 64, FAKE), -1),      # n < 0
    ((0, 1, 1, 8, 0, 4, 4, 64, FAKE), -1),       # d_k = 0
    ((0, 1, 1, 8, 4, 0, 4, 64, FAKE), -1),       # d_v = 0
    ((0, 1, 1, 8, 4, 4, 9, 64, FAKE), -1),       # P > 8
    ((0, 1, 1, 8, 4, 4, 4, 48, FAKE), -2),       # unsupported chunk
    ((0, 1, 1, 8, 200, 4, 8, 64, FAKE), -3),     # feature count too large
    ((0, 1, 1, 8, 256, 4, 2, 64, FAKE), -1),     # d_k > 255
    ((0, 1, 1, 8, 4, 256, 2, 64, FAKE), -1),     # d_v > 255
    ((0, 2, 32768, 8, 4, 4, 4, 64, FAKE), -3),   # B*H = 65536 > 65535
    ((1, 1, 65536, 8, 4, 4, 4, 64, FAKE), -3),   # B*H = 65536 > 65535
    ((0, 1, 1, 8, 4, 4, 4, 64, NULL), -1),       # null tensors
])
def test_prefill_validation(lib, args, code):
    dt, B, H, n, dk, dv, P, chunk, ptr = args
    st = lib.sata_prefill(ptr, ptr, ptr, dt, B, H, n, dk, dv, P, chunk, ptr, NULL, NULL)
    assert st == code
    assert lib.sata_last_error().decode() != ""


def test_decode_and_feature_map_validation(lib):
    assert lib.sata_decode_step(NULL, FAKE, FAKE, FAKE, 0, 1, 1, 4, 4, 4, FAKE, NULL) == -1
    assert lib.sata_decode_step(FAKE, FAKE, FAKE, FAKE, 3, 1, 1, 4, 4, 4, FAKE, NULL) == -1
    assert lib.sata_decode_step(FAKE, FAKE, FAKE, FAKE, 0, 1, 1, 4, 4, 0, FAKE, NULL) == -1
    assert lib.sata_decode_step(FAKE, FAKE, FAKE, FAKE, 0, 1, 1, 256, 4, 2, FAKE, NULL) == -1
    assert lib.sata_decode_step(FAKE, FAKE, FAKE, FAKE, 0, 1, 1, 4, 256, 2, FAKE, NULL) == -1
    assert lib.sata_decode_step(FAKE, FAKE, FAKE, FAKE, 0, 256, 256, 4, 4, 4, FAKE, NULL) == -3
    assert lib.sata_feature_map(FAKE, 0, 3, 256, 2, FAKE, NULL) == -1
    # grouped decode: (S, q, k, v, dtype, B, H_kv, G, d_k, d_v, P, y, stream)
    g = lib.sata_decode_step_grouped
    assert g(FAKE, FAKE, FAKE, FAKE, 0, 1, 1, 0, 4, 4, 4, FAKE, NULL) == -1       # G = 0
    assert g(NULL, FAKE, FAKE, FAKE, 0, 1, 1, 4, 4, 4, 4, FAKE, NULL) == -1       # null state
    assert g(FAKE, FAKE, FAKE, FAKE, 0, 1, 1, 3, 4, 4, 4, FAKE, NULL) == -2       # G = 3
    assert g(FAKE, FAKE, FAKE, FAKE, 0, 1, 1, 16, 4, 4, 4, FAKE, NULL) == -2      # G = 16
    assert g(ctypes.c_void_p(0x1004), FAKE, FAKE, FAKE, 0, 1, 1, 4, 4, 4, 4, FAKE, NULL) == -2  # unaligned
    assert g(FAKE, FAKE, FAKE, FAKE, 0, 1, 1, 4, 4, 200, 4, FAKE, NULL) == -2     # d_v = 200: no plan
    assert g(FAKE, FAKE, FAKE, FAKE, 0, 64, 128, 8, 4, 4, 4, FAKE, NULL) == -3    # B*H_kv*G = 65536
    assert lib.sata_feature_map(FAKE, 0, -5, 4, 3, FAKE, NULL) == -1
    assert lib.sata_feature_map(FAKE, 0, 0, 4, 3, FAKE, NULL) == 0   # rows = 0: no-op
    assert lib.sata_feature_map(NULL, 0, 3, 4, 3, FAKE, NULL) == -1


def test_prefill_grouped_validation(lib):
    # (q, k, v, dtype, B, H_kv, G, n, d_k, d_v, P, chunk, y, S_out, stream)
    g = lib.sata_prefill_grouped
    assert g(FAKE, FAKE, FAKE, 0, 1, 1, 0, 8, 4, 4, 4, 64, FAKE, NULL, NULL) == -1      # G = 0
    assert g(FAKE, FAKE, FAKE, 0, 1, 4096, 16, 8, 4, 4, 4, 64, FAKE, NULL, NULL) == -3  # B*H_kv*G = 65536
    assert g(FAKE, FAKE, FAKE, 0, 1, 1, 2, 8, 4, 4, 4, 48, FAKE, NULL, NULL) == -2      # chunk
    assert g(NULL, FAKE, FAKE, 0, 1, 1, 2, 8, 4, 4, 4, 64, FAKE, NULL, NULL) == -1      # null q
    assert g(FAKE, FAKE, FAKE, 5, 1, 1, 2, 8, 4, 4, 4, 64, FAKE, NULL, NULL) == -1      # dtype


def test_backward_validation(lib):
    # (q, k, v, dy, dtype, B, H, n, d_k, d_v, P, chunk, dq, dk, dv, stream)
    b = lib.sata_backward
    assert b(FAKE, FAKE, FAKE, FAKE, 0, 1, 1, 8, 4, 4, 4, 128, FAKE, FAKE, FAKE, NULL) == -2   # chunk 128
    assert b(FAKE, FAKE, FAKE, FAKE, 0, 1, 1, 8, 65, 4, 2, 64, FAKE, FAKE, FAKE, NULL) == -2   # d_k = 65
    assert b(FAKE, FAKE, FAKE, FAKE, 0, 1, 1, 8, 4, 4, 9, 64, FAKE, FAKE, FAKE, NULL) == -1    # P = 9
    assert b(FAKE, FAKE, FAKE, NULL, 0, 1, 1, 8, 4, 4, 4, 64, FAKE, FAKE, FAKE, NULL) == -1    # null dy
    assert b(FAKE, FAKE, FAKE, FAKE, 0, 1, 1, 0, 4, 4, 4, 64, FAKE, FAKE, FAKE, NULL) == 0     # n = 0


def test_status_strings(lib):
    for code in (0, -1, -2, -3, -4):
        assert lib.sata_status_string(code)


def test_prefill_operands_query(lib):
    out = ctypes.c_int(-1)
    # chunk 64 and d <= 64: the matrix cores, float32 inputs as split (hi + lo
    # bfloat16) operands; other chunks of float32 inputs: float32 products
    assert lib.sata_prefill_operands(0, 8, 32, 8192, 32, 32, 4, 64, ctypes.byref(out)) == 0 and out.value == 2
    assert lib.sata_prefill_operands(1, 8, 32, 8192, 32, 32, 4, 64, ctypes.byref(out)) == 0 and out.value == 1
    assert lib.sata_prefill_operands(0, 1, 64, 65536, 16, 16, 6, 64, ctypes.byref(out)) == 0 and out.value == 2
    assert lib.sata_prefill_operands(0, 1, 1, 100, 8, 8, 4, 32, ctypes.byref(out)) == 0 and out.value == 0
    assert lib.sata_prefill_operands(1, 1, 1, 100, 8, 8, 4, 32, ctypes.byref(out)) == 0 and out.value == 0
    assert lib.sata_prefill_operands(1, 1, 1, 100, 8, 8, 3, 64, ctypes.byref(out)) == 0 and out.value == 1
    # d_k above 64, and P = 1 (a single feature): float32 products
    assert lib.sata_prefill_operands(1, 1, 1, 100, 65, 8, 2, 64, ctypes.byref(out)) == 0 and out.value == 0
    assert lib.sata_prefill_operands(1, 1, 1, 100, 8, 8, 1, 64, ctypes.byref(out)) == 0 and out.value == 0
    # the same validation as the prefill itself
    assert lib.sata_prefill_operands(1, 1, 1, 8, 32, 32, 4, 48, ctypes.byref(out)) == -2
    assert lib.sata_prefill_operands(7, 1, 1, 8, 32, 32, 4, 64, ctypes.byref(out)) == -1
    assert lib.sata_prefill_operands(1, 1, 1, 8, 32, 32, 4, 64, None) == -1
    torch = pytest.importorskip("torch")
    assert bnd.prefill_operands(torch.float32, 1, 1, 100, 8, 8, 4, 64) == "split"
    assert bnd.prefill_operands(torch.float32, 1, 1, 100, 8, 8, 4, 16) == "f32"
    assert bnd.prefill_operands(torch.bfloat16, 1, 1, 100, 8, 8, 4, 64) == "bf16"


def test_prefill_parts_query(lib):
    out = ctypes.c_int(-1)
    # the float32 sweep at P = 2 and 3 (64 heads of 17 / 153 features, one
    # workgroup each): four parts of 16384 tokens fill the 256 compute units
    assert lib.sata_prefill_parts(0, 1, 64, 65536, 16, 16, 2, 64, ctypes.byref(out)) == 0 and out.value == 4
    assert lib.sata_prefill_parts(0, 1, 64, 65536, 16, 16, 3, 64, ctypes.byref(out)) == 0 and out.value == 4
    # enough workgroups already (4 slices x 64 heads; 94 x 16 at d = 64): one scan
    assert lib.sata_prefill_parts(0, 1, 64, 65536, 16, 16, 4, 64, ctypes.byref(out)) == 0 and out.value == 1
    assert lib.sata_prefill_parts(1, 2, 8, 4096, 64, 64, 4, 64, ctypes.byref(out)) == 0 and out.value == 1
    # parts keep at least 1024 tokens: two heads of 8192 tokens take 8, of 4096
    # take 4, of 2047 two (1024 + 1023), of 1500 none
    assert lib.sata_prefill_parts(0, 1, 2, 8192, 8, 8, 3, 64, ctypes.byref(out)) == 0 and out.value == 8
    assert lib.sata_prefill_parts(1, 1, 2, 4096, 8, 8, 3, 64, ctypes.byref(out)) == 0 and out.value == 4
    assert lib.sata_prefill_parts(1, 1, 2, 2047, 8, 8, 3, 64, ctypes.byref(out)) == 0 and out.value == 2
    assert lib.sata_prefill_parts(1, 1, 2, 1500, 8, 8, 3, 64, ctypes.byref(out)) == 0 and out.value == 1
    # one head, long sequence: at most 16 parts
    assert lib.sata_prefill_parts(0, 1, 1, 1 << 20, 8, 8, 3, 64, ctypes.byref(out)) == 0 and out.value == 16
    # other paths scan in one pass
    assert lib.sata_prefill_parts(1, 1, 1, 8192, 32, 32, 4, 64, ctypes.byref(out)) == 0 and out.value == 1
    assert lib.sata_prefill_parts(0, 1, 1, 8192, 8, 8, 4, 32, ctypes.byref(out)) == 0 and out.value == 1
    assert lib.sata_prefill_parts(1, 1, 1, 8, 32, 32, 4, 48, ctypes.byref(out)) == -2
    assert lib.sata_prefill_parts(1, 1, 1, 8, 32, 32, 4, 64, None) == -1
    torch = pytest.importorskip("torch")
    assert bnd.prefill_parts(torch.float32, 1, 64, 65536, 16, 16, 2) == 4


class TestBindingRejectsBeforeLaunch:
    """The tensor wrappers check dtypes and shapes before anything reaches the
    library, so a mismatched output or input is refused instead of being
    written or read past its end.  (CPU tensors: the checks come before the
    device check.)"""

    @pytest.fixture(autouse=True)
    def _torch(self):
        self.torch = pytest.importorskip("torch")

    def t(self, *shape, dtype=None):
        return self.torch.zeros(*shape, dtype=dtype or self.torch.float32)

    def test_feature_map_output(self):
        x = self.t(5, 3)                                      # D = 10 at d=3, P=3
        with pytest.raises(TypeError):
            bnd.feature_map(x, 3, phi=self.t(5, 10, dtype=self.torch.bfloat16))
        with pytest.raises(ValueError):
            bnd.feature_map(x, 3, phi=self.t(5, 9))

    def test_prefill(self):
        bf = self.torch.bfloat16
        q, k, v = self.t(1, 2, 8, 4), self.t(1, 2, 8, 4), self.t(1, 2, 8, 3)
        with pytest.raises(TypeError):
            bnd.prefill(q, k.to(bf), v, 3)
        with pytest.raises(TypeError):
            bnd.prefill(q, k, v.to(bf), 3)
        with pytest.raises(ValueError):
            bnd.prefill(q, self.t(1, 2, 7, 4), v, 3)          # short k
        with pytest.raises(ValueError):
            bnd.prefill(q, k, self.t(1, 2, 7, 3), 3)          # short v
        with pytest.raises(TypeError):
            bnd.prefill(q, k, v, 3, y=self.t(1, 2, 8, 3, dtype=bf))
        with pytest.raises(ValueError):
            bnd.prefill(q, k, v, 3, y=self.t(1, 2, 8, 2))
        with pytest.raises(ValueError):
            bnd.prefill(q, k, v, 3, S=self.t(1, 2, 14, 4))     # D = 15 at d=4, P=3
        with pytest.raises(TypeError):
            bnd.prefill(q, k, v, 3, S=self.t(1, 2, 15, 4, dtype=bf))
        with pytest.raises(ValueError, match="GPU"):
            bnd.prefill(q, k, v, 3)                           # consistent, but not on a GPU

    def test_decode(self):
        bf = self.torch.bfloat16
        S, q, k, v = self.t(2, 3, 15, 6), self.t(2, 3, 4), self.t(2, 3, 4), self.t(2, 3, 5)
        with pytest.raises(TypeError):
            bnd.decode_step(S, q, k.to(bf), v, 3)
        with pytest.raises(TypeError):
            bnd.decode_step(S, q, k, v.to(bf), 3)
        with pytest.raises(ValueError):
            bnd.decode_step(S, q, self.t(2, 3, 3), v, 3)      # k of the wrong width
        with pytest.raises(ValueError):
            bnd.decode_step(S, q, k, self.t(2, 2, 5), 3)      # v of too few heads
        with pytest.raises(TypeError):
            bnd.decode_step(S, q, k, v, 3, y=self.t(2, 3, 5, dtype=bf))
        with pytest.raises(ValueError):
            bnd.decode_step(S, q, k, v, 3, y=self.t(2, 3, 4))
        with pytest.raises(ValueError):
            bnd.decode_step(self.t(2, 3, 15, 5), q, k, v, 3)
        with pytest.raises(ValueError, match="GPU"):
            bnd.decode_step(S, q, k, v, 3)

    def test_decode_grouped(self):
        bf = self.torch.bfloat16
        S, q, k, v = self.t(1, 2, 15, 6), self.t(1, 8, 4), self.t(1, 2, 4), self.t(1, 2, 5)
        with pytest.raises(TypeError):
            bnd.decode_step_grouped(S, q, k.to(bf), v, 3)
        with pytest.raises(ValueError):
            bnd.decode_step_grouped(S, self.t(1, 7, 4), k, v, 3)   # 7 query heads over 2 key/value heads
        with pytest.raises(ValueError):
            bnd.decode_step_grouped(S, q, k, self.t(1, 3, 5), 3)
        with pytest.raises(TypeError):
            bnd.decode_step_grouped(S, q, k, v, 3, y=self.t(1, 8, 5, dtype=bf))
        with pytest.raises(ValueError):
            bnd.decode_step_grouped(S, q, k, v, 3, y=self.t(1, 2, 5))
        with pytest.raises(ValueError, match="GPU"):
            bnd.decode_step_grouped(S, q, k, v, 3)


def test_missing_library_fails_loudly(tmp_path):
    """No fallback: without the built library the binding raises before any work."""
    with pytest.raises(RuntimeError, match="missing"):
        bnd.load_library(str(tmp_path / "libsata.so"))


def test_product_path_does_not_touch_the_oracle():
    """The package's Python and HIP sources never import, load or name the
    oracle: every result comes from the library's kernels."""
    import pathlib
    import re
    pkg = pathlib.Path(bnd.__file__).resolve().parent
    sources = [p for p in pkg.rglob("*") if p.suffix in (".py", ".hip", ".hpp", ".h", ".cpp")]
    assert sources
    for p in sources:
        text = p.read_text()
        assert not re.search(r"\boracle\b", text), f"{p} names the oracle"
