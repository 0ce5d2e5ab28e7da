"""Pins for the oracle's transformed quantization and SmoothQuant calibration.

The rows quantized here are v[k] = T(x[k]) * c[k]: T the identity or GELU (the input of
the MLP down-projection), c the per-input-channel multiplier that SmoothQuant applies to
the activations at run time (Section 3, "The quantization recipe (reused)": per-channel
int8 weights, per-token dynamic int8 activations, SmoothQuant with alpha = 0.5). Each
pin rests on something other than the oracle's own formula: textbook values of the
normal CDF, closed forms, identities, exact power-of-two scalings, or brute force.
"""
import math

import numpy as np
import pytest

import oracle
import synth_inputs as si

# Standard normal CDF at a few points (published tables).
PHI = {0.5: 0.6914624612740131, 1.0: 0.8413447460685429, 2.0: 0.9772498680518208,
       3.0: 0.9986501019683699, -5.0: 2.8665157187919391e-07,
       -6.0: 9.865876450376946e-10, -10.0: 7.6198530241605261e-24}


def _bf16(vals):
    a = np.asarray(vals, np.float32)
    return oracle.f32_to_bf16(a).reshape(a.shape)


def test_gelu_textbook_values():
    xs = np.array(sorted(PHI), np.float64)
    got = oracle.gelu_f64(xs)
    for x, g in zip(xs, got):
        want = x * PHI[float(x)]
        assert g == pytest.approx(want, rel=1e-12), x
    # negative points through Phi(-x) = 1 - Phi(x)
    for x in (0.5, 1.0, 2.0, 3.0):
        assert oracle.gelu_f64(np.array([-x]))[0] == pytest.approx(-x * (1 - PHI[x]), rel=1e-12)


def test_gelu_matches_library_cdf():
    import scipy.special
    x = np.linspace(-12, 12, 4801)
    want = x * scipy.special.ndtr(x)
    np.testing.assert_allclose(oracle.gelu_f64(x), want, rtol=1e-11, atol=1e-300)


def test_gelu_odd_part_is_identity():
    # Phi(x) + Phi(-x) = 1, so GELU(x) - GELU(-x) = x for every x.
    x = np.random.default_rng(3).standard_normal(2000) * 4
    d = oracle.gelu_f64(x) - oracle.gelu_f64(-x)
    np.testing.assert_allclose(d, x, rtol=1e-14, atol=1e-15)


def test_colmul_of_ones_is_the_plain_rule():
    x, _, _ = si.make_inputs((9, 256, 1), seed=5)
    q0, s0 = oracle.quantize_rows(x)
    q1, s1 = oracle.quantize_rows(x, col_mul=np.ones(256, np.float32))
    np.testing.assert_array_equal(q0, q1)
    np.testing.assert_array_equal(s0, s1)


def test_colmul_power_of_two_equals_prescaled_input():
    # Multiplying by 2^e is exact in float32 and in bf16 (no overflow/underflow here),
    # so quantizing x * 2^e[k] with the multiplier must equal quantizing the
    # pre-scaled bf16 matrix with the plain rule. A multiplier indexed by row instead of
    # column, or applied after the absmax, fails this.
    rng = np.random.default_rng(11)
    x, _, _ = si.make_inputs((7, 96, 1), seed=6)
    e = rng.integers(-6, 7, size=96)
    cm = np.ldexp(np.float32(1.0), e).astype(np.float32)
    pre = _bf16(oracle.bf16_to_f32(x) * cm[None, :])
    np.testing.assert_array_equal(oracle.bf16_to_f32(pre), oracle.bf16_to_f32(x) * cm)
    q0, s0 = oracle.quantize_rows(pre)
    q1, s1 = oracle.quantize_rows(x, col_mul=cm)
    np.testing.assert_array_equal(q0, q1)
    np.testing.assert_array_equal(s0, s1)


def test_colmul_worked_row():
    # x = [1, -2, 3, 0.5], c = [1, 0.5, 2, 4] -> v = [1, -1, 6, 2]; a = 6,
    # 127/6 = 21.1667: codes rne(21.17) = 21, -21, 127, rne(42.33) = 42; s = 6/127.
    q, s = oracle.quantize_rows(_bf16([[1, -2, 3, 0.5]]),
                                col_mul=np.array([1, 0.5, 2, 4], np.float32))
    assert q.tolist() == [[21, -21, 127, 42]]
    assert s[0] == np.float32(6) / np.float32(127)


def test_gelu_worked_row():
    # v = x * Phi(x) for x = [1, -2, 3, 0.5] from the table: [0.84134, -0.04550, 2.99595,
    # 0.34573]; a = 2.99595, 127/a = 42.3905: codes 35.67 -> 36, -1.93 -> -2, 127,
    # 14.66 -> 15 (no value near a rounding tie).
    q, s = oracle.quantize_rows(_bf16([[1, -2, 3, 0.5]]), act="gelu")
    assert q.tolist() == [[36, -2, 127, 15]]
    a = 3 * PHI[3.0]
    assert s[0] == pytest.approx(a / 127, rel=1e-7)


def test_gelu_left_tail_row():
    # GELU(-5) = -5 Phi(-5) = -1.43326e-6 and GELU(-6) = -5.91953e-9: the row's absmax
    # is the tail value at -5 and the -6 entry is 127 * 0.0041302 = 0.5245 steps -> -1.
    # A GELU that loses the left tail (1 + erf cancelling in single precision) gets
    # neither right.
    q, s = oracle.quantize_rows(_bf16([[-5, -6]]), act="gelu")
    assert q.tolist() == [[-127, -1]]
    assert s[0] == pytest.approx(5 * PHI[-5.0] / 127, rel=1e-6)


def _transformed_f32(x_bits, act, cm):
    v = oracle.bf16_to_f32(x_bits).astype(np.float32)
    if act == "gelu":
        v = oracle.gelu_f64(v.astype(np.float64)).astype(np.float32)
    if cm is not None:
        v = (v * cm[None, :]).astype(np.float32)
    return v


@pytest.mark.parametrize("act", ["none", "gelu"])
@pytest.mark.parametrize("with_cm", [False, True])
def test_transformed_rows_invariants(act, with_cm):
    rng = np.random.default_rng(21)
    x = _bf16(rng.standard_normal((40, 320)).astype(np.float32) * 3)
    cm = rng.uniform(0.05, 8, 320).astype(np.float32) if with_cm else None
    q, s = oracle.quantize_rows(x, act=act, col_mul=cm)
    v = _transformed_f32(x, act, cm)
    assert q.min() >= -127 and q.max() <= 127
    for r in range(40):
        assert np.abs(q[r]).max() == 127
        rec = s[r].astype(np.float64) * q[r]
        assert np.all(np.abs(rec - v[r]) <= 0.5 * s[r] * (1 + 1e-4))
    # the row scale is max|v| / 127
    np.testing.assert_array_equal(s, (np.abs(v).max(axis=1) / np.float32(127)).astype(np.float32))


def test_transformed_zero_and_tiny_rows():
    x = np.zeros((3, 64), np.uint16)
    x[1] = _bf16(np.linspace(-1, 1, 64))
    x[2] = _bf16(np.linspace(-1, 1, 64))
    cm = np.full(64, 1e-38, np.float32)      # row maxima fall below ~3.7e-37: zero rows
    q, s = oracle.quantize_rows(x, act="gelu")
    assert s[0] == 0 and not q[0].any()       # GELU(0) = 0
    q2, s2 = oracle.quantize_rows(x, act="gelu", col_mul=cm)
    assert np.all(s2 == 0) and not q2.any()


def test_col_absmax_brute_force():
    rng = np.random.default_rng(8)
    x = _bf16(rng.standard_normal((6, 5)).astype(np.float32) * 2)
    xf = oracle.bf16_to_f32(x)
    for act in ("none", "gelu"):
        got = oracle.col_absmax(x, act=act)
        for k in range(5):
            best = 0.0
            for r in range(6):
                v = float(xf[r, k])
                if act == "gelu":
                    v = float(np.float32(v * PHI_fn(v)))
                best = max(best, abs(v))
            assert got[k] == np.float32(best), (act, k)


def PHI_fn(v):
    return 0.5 * math.erfc(-v / math.sqrt(2.0))


def test_smooth_factors_closed_forms():
    ax = np.array([4, 9, 2, 1, 0, 5, 2.0 ** -60], np.float32)
    aw = np.array([1, 4, 2, 4, 3, 0, 2.0 ** 60], np.float32)
    s, si_ = oracle.smooth_factors(ax, aw, 0.5)
    np.testing.assert_array_equal(s, np.array([2, 1.5, 1, 0.5, 1, 1, 2.0 ** -60], np.float32))
    np.testing.assert_array_equal(si_, (np.float32(1) / s).astype(np.float32))
    # alpha = 1: s = ax; alpha = 0: s = 1 / aw; alpha = 1/4 with ax = aw = 16: 2 / 8
    s1, _ = oracle.smooth_factors(np.array([3.0], np.float32), np.array([7.0], np.float32), 1.0)
    assert s1[0] == np.float32(3.0)
    s0, _ = oracle.smooth_factors(np.array([3.0], np.float32), np.array([8.0], np.float32), 0.0)
    assert s0[0] == np.float32(0.125)
    sq, _ = oracle.smooth_factors(np.array([16.0], np.float32), np.array([16.0], np.float32), 0.25)
    assert sq[0] == np.float32(0.25)
    with pytest.raises(oracle.OracleError):
        oracle.smooth_factors(ax, aw, 1.5)


def test_smooth_factors_balance_the_channel_maxima():
    # With alpha = 0.5 the smoothed maxima meet in the middle: max|X_k| / s_k and
    # max|W_k| * s_k both equal sqrt(ax_k * aw_k). A swapped pair or a wrong exponent
    # breaks the equality.
    rng = np.random.default_rng(4)
    ax = rng.uniform(0.01, 80, 500).astype(np.float32)
    aw = rng.uniform(1e-3, 0.5, 500).astype(np.float32)
    s, _ = oracle.smooth_factors(ax, aw, 0.5)
    lhs = ax.astype(np.float64) / s
    rhs = aw.astype(np.float64) * s
    np.testing.assert_allclose(lhs, rhs, rtol=3e-7)
    np.testing.assert_allclose(lhs, np.sqrt(ax.astype(np.float64) * aw), rtol=3e-7)


def test_smoothing_preserves_the_product():
    rng = np.random.default_rng(12)
    x = rng.standard_normal((16, 48))
    w = rng.standard_normal((24, 48))
    s, si_ = oracle.smooth_factors(np.abs(x).max(0).astype(np.float32),
                                   np.abs(w).max(0).astype(np.float32), 0.5)
    y0 = x @ w.T
    y1 = (x * si_.astype(np.float64)) @ (w * s.astype(np.float64)).T
    np.testing.assert_allclose(y1, y0, rtol=1e-5, atol=1e-5)


def _w8a8_error(x, w, b, s=None, s_inv=None):
    wq, sw = oracle.quantize_rows(w, col_mul=s)
    xq, sx = oracle.quantize_rows(x, col_mul=s_inv)
    y = oracle.bf16_to_f32(oracle.epilogue(oracle.gemm_acc(xq, wq), sx, sw, b))
    ref = (oracle.bf16_to_f32(x).astype(np.float64) @ oracle.bf16_to_f32(w).astype(np.float64).T
           + oracle.bf16_to_f32(b))
    return float(np.linalg.norm(y - ref) / np.linalg.norm(ref))


def test_smoothing_reduces_error_on_outlier_channels():
    # Inputs with two x20 outlier input channels: per-token scales are set by the
    # outliers and the other channels lose resolution. Smoothing (calibrated on other
    # batches of the same distribution) must bring the W8A8 error down.
    x, w, b = si.make_inputs((64, 256, 128), seed=20260)
    calib = [si.make_inputs((64, 256, 128), seed=7000 + i)[0] for i in range(4)]
    ax = np.max([oracle.col_absmax(c) for c in calib], axis=0)
    aw = oracle.col_absmax(w)
    s, s_inv = oracle.smooth_factors(ax, aw, 0.5)
    e_plain = _w8a8_error(x, w, b)
    e_smooth = _w8a8_error(x, w, b, s, s_inv)
    assert e_smooth < 0.8 * e_plain, (e_plain, e_smooth)
