"""Pins of the fp64 GEMM oracle and its error metrics (Sec. II-B, C = A B)."""
import math

import numpy as np
import pytest

import workloads as W
from oracle import gemm as O


def test_decode_matches_bf16_definition():
    # 1.0 = 0x3F80, -2.0 = 0xC000, 0.5 = 0x3F00, smallest normal 2^-126 = 0x0080
    bits = np.array([0x3F80, 0xC000, 0x3F00, 0x0080, 0x0000, 0x8000], dtype=np.uint16)
    assert list(O.decode_bf16(bits)) == [1.0, -2.0, 0.5, 2.0 ** -126, 0.0, -0.0]


@pytest.mark.parametrize("M,N,K", [(256, 512, 256), (37, 19, 256), (128, 128, 1), (64, 64, 64)])
def test_ternary_inputs_match_exact_integer_product(M, N, K):
    A = W.draw_array(11, M, K, "ternary")
    B = W.draw_array(12, K, N, "ternary")
    Ai = O.decode_bf16(A).astype(np.int64)
    Bi = O.decode_bf16(B).astype(np.int64)
    C = O.gemm_fp64(A, B)
    assert np.array_equal(C, (Ai @ Bi).astype(np.float64))


def test_identity_b_returns_a():
    A = W.draw_array(3, 64, 96, "normal", 1.0)
    I = W.round_to_bf16_bits(np.eye(96, dtype=np.float32))
    assert np.array_equal(O.gemm_fp64(A, I), O.decode_bf16(A))


def test_entries_match_fsum_definition():
    A = W.draw_array(4, 40, 300, "normal", 1.0)
    B = W.draw_array(5, 300, 50, "normal", 0.02)
    C = O.gemm_fp64(A, B)
    a, b = O.decode_bf16(A), O.decode_bf16(B)
    rng = np.random.default_rng(0)
    rows = rng.integers(0, 40, 25)
    cols = rng.integers(0, 50, 25)
    for r, c in zip(rows, cols):
        exact = math.fsum(a[r, k] * b[k, c] for k in range(300))
        assert abs(C[r, c] - exact) <= 1e-12 * (1 + abs(exact))


def test_error_metrics_on_known_perturbation():
    rng = np.random.default_rng(1)
    ref = rng.standard_normal((30, 20))
    err = O.errors(ref * (1 + 1e-3), ref)
    assert math.isclose(err["rel_fro"], 1e-3, rel_tol=1e-9)
    assert math.isclose(err["max_abs"], 1e-3 * np.abs(ref).max(), rel_tol=1e-9)
    assert O.within_tolerance(err)
    bad = ref.copy()
    bad[3, 4] += 0.5 * np.abs(ref).max()
    e2 = O.errors(bad, ref)
    assert e2["max_abs"] > 1e-2 * e2["max_ref"] and not O.within_tolerance(e2)


def test_inner_dimension_mismatch_raises():
    with pytest.raises(ValueError):
        O.gemm_fp64(np.zeros((2, 3)), np.zeros((4, 2)))


def test_scaled_gemm_on_integers_is_exact():
    """alpha A B + beta C on ternary inputs, against exact integer arithmetic
    (alpha, beta powers of two, so every value is exact in float64)."""
    A = W.draw_array(71, 64, 96, "ternary")
    B = W.draw_array(72, 96, 80, "ternary")
    C = W.draw_array(73, 64, 80, "ternary")
    ai = O.decode_bf16(A).astype(np.int64)
    bi = O.decode_bf16(B).astype(np.int64)
    ci = O.decode_bf16(C).astype(np.int64)
    for alpha, beta in ((1.0, 0.0), (0.5, 2.0), (-2.0, -1.0), (0.0, 4.0)):
        exact = alpha * (ai @ bi).astype(np.float64) + beta * ci.astype(np.float64)
        assert np.array_equal(O.gemm_scaled_fp64(A, B, C, alpha, beta), exact)


def test_scaled_gemm_beta_zero_ignores_c():
    A = W.draw_array(74, 32, 48)
    B = W.draw_array(75, 48, 16)
    C = np.full((32, 16), 0x7FC0, dtype=np.uint16)          # bf16 NaN everywhere
    out = O.gemm_scaled_fp64(A, B, C, 1.5, 0.0)
    assert np.all(np.isfinite(out))
    assert np.array_equal(out, 1.5 * O.gemm_fp64(A, B))


def test_scaled_gemm_identity_a():
    """A = I: alpha B + beta C elementwise."""
    B = W.draw_array(76, 64, 32)
    C = W.draw_array(77, 64, 32)
    eye = np.eye(64)
    got = O.gemm_scaled_fp64(eye, B, C, 0.25, -3.0)
    assert np.array_equal(got, 0.25 * O.decode_bf16(B) - 3.0 * O.decode_bf16(C))


def test_fp8_decode_hand_values():
    # 1.0 = 0.0111.000, -2.0 = 1.1000.000, 448 = 0.1111.110 (largest),
    # 2^-6 = 0.0001.000 (smallest normal), 2^-9 = 0.0000.001 (smallest subnormal),
    # 0.875 * 2^-6 = 0.0000.111, 1.125 = 0.0111.001
    bits = np.array([0x38, 0xC0, 0x7E, 0x08, 0x01, 0x07, 0x39, 0x00, 0x80], dtype=np.uint8)
    want = [1.0, -2.0, 448.0, 2.0 ** -6, 2.0 ** -9, 7 * 2.0 ** -9, 1.125, 0.0, -0.0]
    got = O.decode_fp8_e4m3(bits)
    assert list(got) == want
    assert np.signbit(got[-1])
    assert np.isnan(O.decode_fp8_e4m3(np.array([0x7F, 0xFF], dtype=np.uint8))).all()


def test_fp8_decode_matches_torch_for_every_pattern():
    torch = pytest.importorskip("torch")
    bits = np.arange(256, dtype=np.uint8)
    want = torch.from_numpy(bits).view(torch.float8_e4m3fn).to(torch.float64).numpy()
    got = O.decode_fp8_e4m3(bits)
    both_nan = np.isnan(want) & np.isnan(got)
    assert np.array_equal(got[~both_nan], want[~both_nan])
    assert np.array_equal(np.isnan(got), np.isnan(want))


def test_fp8_gemm_on_integers_is_exact():
    A = W.draw_array_fp8(91, 48, 128, "ternary")
    B = W.draw_array_fp8(92, 128, 40, "ternary")
    ai = O.decode_fp8_e4m3(A).astype(np.int64)
    bi = O.decode_fp8_e4m3(B).astype(np.int64)
    assert set(np.unique(ai)) <= {-1, 0, 1}
    assert np.array_equal(O.gemm_fp64(A, B), (ai @ bi).astype(np.float64))


@pytest.mark.parametrize("block", [1, 7, 64, 200])
def test_error_accumulator_over_row_blocks_equals_errors(block):
    """The block-wise form gives errors()'s values for any row blocking, and
    still sees a single planted outlier."""
    rng = np.random.default_rng(2)
    ref = rng.standard_normal((200, 37))
    test = ref + 1e-4 * rng.standard_normal((200, 37))
    test[123, 5] += 0.3
    acc = O.ErrorAccumulator()
    for r0 in range(0, 200, block):
        acc.add(test[r0:r0 + block], ref[r0:r0 + block])
    got, want = acc.result(), O.errors(test, ref)
    assert acc.count == ref.size
    for key in ("rel_fro", "max_abs", "max_ref"):
        assert math.isclose(got[key], want[key], rel_tol=1e-12), key
    assert math.isclose(got["max_abs"], abs(test[123, 5] - ref[123, 5]), rel_tol=1e-12)


def test_error_accumulator_rejects_mismatched_blocks():
    acc = O.ErrorAccumulator()
    with pytest.raises(ValueError):
        acc.add(np.zeros((2, 3)), np.zeros((3, 2)))
    acc.add(np.zeros((0, 4)), np.zeros((0, 4)))
    assert acc.result() == {"rel_fro": 0.0, "max_abs": 0.0, "max_ref": 0.0}
