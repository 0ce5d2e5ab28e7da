"""Pins for the CPU oracle (no GPU).

Each test ties the oracle to something other than itself: hand-worked cases from the
definitions, brute force on tiny inputs, an independent library route, closed forms
and invariants of symmetric absmax quantization. The plausible mistakes each one
catches are named in its docstring.
"""
from fractions import Fraction

import numpy as np
import pytest
import torch

import oracle
import synth_inputs as si

pytestmark = pytest.mark.filterwarnings("ignore::RuntimeWarning")


def bits(vals):
    """bf16 bits of values that are exactly representable in bf16."""
    t = torch.tensor(vals, dtype=torch.float32)
    b = t.to(torch.bfloat16)
    assert torch.equal(b.to(torch.float32), t), "value not bf16-exact"
    return b.view(torch.int16).numpy().view(np.uint16).copy()


def torch_bf16(f32):
    t = torch.from_numpy(np.ascontiguousarray(f32, dtype=np.float32))
    return t.to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)


# ---------------------------------------------------------------- bf16 conversions

def test_bf16_rounding_matches_library():
    """The oracle's own float32 -> bf16 RNE against torch's dtype conversion.
    Catches: truncation instead of rounding, ties away from zero, a missed carry into
    the exponent, NaN made signalling."""
    rng = np.random.default_rng(0)
    u = rng.integers(0, 2**32, size=200_000, dtype=np.uint64).astype(np.uint32)
    # force exact ties and near-ties in a third of them
    u[::3] = (u[::3] & 0xFFFF0000) | 0x8000
    u[1::7] = (u[1::7] & 0xFFFF0000) | 0x7FFF
    f = u.view(np.float32)
    special = np.array([0.0, -0.0, 1.0, -1.0, np.inf, -np.inf, 3.3895314e38, 3.4028235e38,
                        1e-45, -1e-45, 1.1754942e-38, 16003.5, 65504.0], np.float32)
    f = np.concatenate([f, special])
    mine = oracle.f32_to_bf16(f)
    ref = torch_bf16(f)
    nan = np.isnan(f)
    assert np.array_equal(mine[~nan], ref[~nan])
    # NaN stays NaN with the quiet bit set
    assert np.all((mine[nan] & 0x7F80) == 0x7F80) and np.all(mine[nan] & 0x0040)


def test_bf16_widening_exact():
    b = np.arange(0, 2**16, dtype=np.uint32).astype(np.uint16)
    f = oracle.bf16_to_f32(b)
    back = torch.from_numpy(b.view(np.int16)).view(torch.bfloat16).to(torch.float32).numpy()
    ok = ~np.isnan(back)
    assert np.array_equal(f[ok].view(np.uint32), back[ok].view(np.uint32))


def _round_fraction_to_bf16_value(fr: Fraction) -> Fraction:
    """Exact nearest-even rounding of a rational to the bf16 grid (brute force)."""
    if fr == 0:
        return Fraction(0)
    sgn = -1 if fr < 0 else 1
    a = abs(fr)
    e = a.numerator.bit_length() - a.denominator.bit_length()
    while Fraction(2) ** e > a:
        e -= 1
    while Fraction(2) ** (e + 1) <= a:
        e += 1
    e = max(e, -126)
    q = Fraction(2) ** (e - 7)
    n = a / q
    fl = n.numerator // n.denominator
    rem = n - fl
    if rem > Fraction(1, 2) or (rem == Fraction(1, 2) and fl % 2 == 1):
        fl += 1
    return sgn * fl * q


def test_f64_to_bf16_single_rounding_brute_force():
    """Diagnostic double -> bf16 rounding against exact rational rounding.
    Catches: double rounding through float32, wrong subnormal quantum."""
    rng = np.random.default_rng(1)
    vals = np.concatenate([rng.standard_normal(3000) * 10.0 ** rng.integers(-40, 30, 3000),
                           np.array([1.0 + 2**-8, 1.0 + 2**-8 + 2**-30, -(1.0 + 3 * 2**-8),
                                     2.0**-133, 3 * 2.0**-134, 2.0**-135])])
    mine = oracle.f64_to_bf16(vals)
    for v, b in zip(vals, mine):
        exact = _round_fraction_to_bf16_value(Fraction(float(v)))
        got = Fraction(float(oracle.bf16_to_f32(np.array([b]))[0]))
        assert got == exact, (v, b)


# ---------------------------------------------------------------- quantization

def test_quant_worked_case_exact_scale():
    """a = 127 gives 127/a = 1 and s = 1, so the codes are the RNE integers of the row.
    62.5 -> 62, 0.5 -> 0, -0.5 -> -0, 1.5 -> 2, 2.5 -> 2, -2.5 -> -2, -63.5 -> -64.
    Catches: ties away from zero (62.5 -> 63, 0.5 -> 1, 2.5 -> 3), truncation (1.5 -> 1)."""
    row = bits([127.0, -63.5, 62.5, 0.5, -0.5, 1.5, 2.5, -2.5]).reshape(1, -1)
    q, s = oracle.quantize_rows(row)
    assert q.tolist() == [[127, -64, 62, 0, 0, 2, 2, -2]]
    assert s.tolist() == [1.0]


def test_quant_worked_case_half_step():
    """a = 254: 127/a = 0.5, s = 2. 3*0.5 = 1.5 -> 2, 5*0.5 = 2.5 -> 2, +-1*0.5 -> 0.
    Reconstruction s*q = [254, 4, 4, 0, 0] misses by exactly s/2 = 1 on the ties.
    Catches: scale a*127 or 1/a, per-element division by a."""
    row = bits([254.0, 3.0, 5.0, -1.0, 1.0]).reshape(1, -1)
    q, s = oracle.quantize_rows(row)
    assert q.tolist() == [[127, 2, 2, 0, 0]]
    assert s.tolist() == [2.0]
    recon = s[0] * q[0].astype(np.float32)
    assert recon.tolist() == [254.0, 4.0, 4.0, 0.0, 0.0]


def test_quant_negative_max_and_clamp():
    """The row maximum magnitude may be negative: it maps to -127 (never -128)."""
    row = bits([-3.0, 1.5, 0.75, -0.0]).reshape(1, -1)
    q, s = oracle.quantize_rows(row)
    # 127/3 = 42.33333... ; 1.5*that = 63.5 (rounded float) ; 0.75*that = 31.75
    assert q[0, 0] == -127
    assert q.min() >= -127
    assert s[0] == np.float32(3.0) / np.float32(127.0)
    assert q[0, 3] == 0


@pytest.mark.parametrize("dist", ["outlier", "gelu", "student_t"])
def test_quant_invariants(dist):
    """Closed properties of symmetric absmax quantization, on the synthetic
    distributions: codes in [-127, 127]; every nonzero row reaches |q| = 127 at its
    absmax; |s*q - v| <= s/2 (half a step, slack for the float32 roundings of 127/a and
    a/127); s = a/127 exactly as a float32 division.
    Catches: wrong clamp, wrong scale (e.g. a/128, a/255), wrong axis."""
    x, _, _ = si.make_inputs((96, 520, 8), seed=7, dist=dist)
    q, s = oracle.quantize_rows(x)
    v = oracle.bf16_to_f32(x)
    a = np.abs(v).max(axis=1)
    assert q.dtype == np.int8 and q.min() >= -127 and q.max() <= 127
    assert np.all(np.abs(q).max(axis=1) == 127)
    assert np.array_equal(s, (a / np.float32(127.0)).astype(np.float32))
    err = np.abs(s[:, None].astype(np.float64) * q - v.astype(np.float64))
    assert np.all(err <= 0.5 * s[:, None] * (1 + 1e-4))
    # the absmax element itself reconstructs exactly up to float32 scale rounding
    am = np.abs(v).argmax(axis=1)
    assert np.all(np.abs(q[np.arange(len(am)), am]) == 127)


def test_quant_zero_and_tiny_rows():
    """Row of zeros, and a row whose 127/a overflows float32 (a < ~3.7e-37), are zero
    rows: s = 0 and q = 0. A row at a ~ 1e-36 (127/a finite) keeps its subnormal
    entries, which quantize to nonzero codes."""
    z = np.zeros((1, 16), np.uint16)
    tiny = torch_bf16(np.full((1, 16), 1e-38, np.float32) * np.linspace(-1, 1, 16, dtype=np.float32))
    small = torch_bf16(np.array([[1e-36, 5e-39, -1e-38, 0.0]], np.float32))
    q, s = oracle.quantize_rows(np.concatenate([z, tiny]))
    assert np.all(q == 0) and np.all(s == 0)
    q2, s2 = oracle.quantize_rows(small)
    assert s2[0] > 0 and q2[0, 0] == 127
    assert q2[0, 2] != 0  # a subnormal input that must not be flushed


def test_quant_constant_row():
    """A constant row v gives 127/v * v ~= 127 -> all codes 127, s = v/127."""
    row = bits([0.3125] * 40).reshape(1, -1)
    q, s = oracle.quantize_rows(row)
    assert np.all(q == 127)


def test_quant_reading_multiply_by_reciprocal():
    """Reading (recorded in the design doc): codes are rne(v * fl(127/a)), not rne(v / fl(a/127)).
    The two differ at near-ties; this case is found by search and must follow the
    multiply form."""
    rng = np.random.default_rng(3)
    for _ in range(200):
        a = np.float32(rng.uniform(0.5, 50.0))
        a = oracle.bf16_to_f32(torch_bf16(np.array([a])))[0]
        inv = np.float32(127.0) / a
        s = a / np.float32(127.0)
        vals = oracle.bf16_to_f32(np.arange(0x3C00, 0x4300, dtype=np.uint16))
        vals = vals[vals < a]
        mul = np.rint(vals * inv)
        div = np.rint(vals / s)
        diff = np.nonzero(mul != div)[0]
        if diff.size:
            v = vals[diff[0]]
            row = torch_bf16(np.array([[a, v]], np.float32))
            q, _ = oracle.quantize_rows(row)
            assert q[0, 1] == mul[diff[0]] != div[diff[0]]
            return
    pytest.skip("no differing case found")


def test_quant_rejects_nonfinite():
    row = bits([1.0, 2.0]).reshape(1, -1)
    row[0, 1] = 0x7F80  # +inf
    with pytest.raises(oracle.OracleError):
        oracle.quantize_rows(row)


# ---------------------------------------------------------------- integer product

def test_acc_brute_force_tiny_config():
    """Pure-Python integer loops over the 64x256x128 workload (2.1 M MACs).
    Catches: transposed operand, wrong K stride, sign errors, int8 wrap."""
    shp = si.WORKLOADS[0][0]
    x, w, _ = si.make_inputs(shp)
    xq, _ = oracle.quantize_rows(x)
    wq, _ = oracle.quantize_rows(w)
    acc = oracle.gemm_acc(xq, wq)
    xl = xq.astype(int).tolist()
    wl = wq.astype(int).tolist()
    for m in range(shp.M):
        xr = xl[m]
        for n in range(shp.N):
            wr = wl[n]
            assert acc[m, n] == sum(a * b for a, b in zip(xr, wr))


def test_acc_against_numpy_int64():
    """Independent library route: numpy int64 matmul on a ragged 257x1000x131 case."""
    rng = np.random.default_rng(5)
    xq = rng.integers(-127, 128, size=(257, 1000), dtype=np.int64).astype(np.int8)
    wq = rng.integers(-127, 128, size=(131, 1000), dtype=np.int64).astype(np.int8)
    acc = oracle.gemm_acc(xq, wq)
    ref = xq.astype(np.int64) @ wq.astype(np.int64).T
    assert np.array_equal(acc.astype(np.int64), ref)


def test_acc_extremes_and_overflow_guard():
    """|acc| <= 127^2 K fits int32 up to K = 133144; one more overflows and the
    oracle reports it."""
    K = 133144
    xq = np.full((1, K), 127, np.int8)
    wq = np.full((2, K), -127, np.int8)
    wq[1] = 127
    acc = oracle.gemm_acc(xq, wq)
    assert acc[0, 0] == -16129 * K and acc[0, 1] == 16129 * K
    with pytest.raises(oracle.OracleError):
        oracle.gemm_acc(np.full((1, K + 1), 127, np.int8), np.full((1, K + 1), 127, np.int8))


def test_empty_shapes():
    acc = oracle.gemm_acc(np.zeros((0, 8), np.int8), np.zeros((3, 8), np.int8))
    assert acc.shape == (0, 3)
    acc = oracle.gemm_acc(np.zeros((2, 0), np.int8), np.zeros((3, 0), np.int8))
    assert np.all(acc == 0)


# ---------------------------------------------------------------- epilogue

def test_worked_gemm_and_epilogue():
    """K = 4, xq = [127, -64, 62, 0], wq = [127, 1, -1, 2]:
    acc = 16129 - 64 - 62 + 0 = 16003. sx = sw = 1, b = 0.5: y32 = 16003.5 and the
    bf16 grid in [8192, 16384) has spacing 64, so y = 16000 (16003.5/64 = 250.05).
    Catches: a dropped bias (16003 -> 16000 too, so the second case differs), a bias
    added after rounding, truncating conversion."""
    xq = np.array([[127, -64, 62, 0]], np.int8)
    wq = np.array([[127, 1, -1, 2]], np.int8)
    acc = oracle.gemm_acc(xq, wq)
    assert acc.tolist() == [[16003]]
    one = np.ones(1, np.float32)
    y = oracle.epilogue(acc, one, one, bits([0.5]))
    assert oracle.bf16_to_f32(y).tolist() == [[16000.0]]
    # b = 40: 16043 / 64 = 250.67 -> 251 * 64 = 16064; without bias -> 16000.
    y = oracle.epilogue(acc, one, one, bits([40.0]))
    assert oracle.bf16_to_f32(y).tolist() == [[16064.0]]
    # scales: sx = 0.5, sw = 0.25 -> 16003 * 0.125 = 2000.375 -> grid 8 in [1024,2048)
    y = oracle.epilogue(acc, np.array([0.5], np.float32), np.array([0.25], np.float32), None)
    assert oracle.bf16_to_f32(y).tolist() == [[2000.0]]


def _f32_round(fr: Fraction) -> Fraction:
    """Exact nearest-even rounding of a rational to float32 (normal range)."""
    if fr == 0:
        return Fraction(0)
    sgn = -1 if fr < 0 else 1
    a = abs(fr)
    e = a.numerator.bit_length() - a.denominator.bit_length()
    while Fraction(2) ** e > a:
        e -= 1
    while Fraction(2) ** (e + 1) <= a:
        e += 1
    e = max(e, -126)
    q = Fraction(2) ** (e - 23)
    n = a / q
    fl = n.numerator // n.denominator
    rem = n - fl
    if rem > Fraction(1, 2) or (rem == Fraction(1, 2) and fl % 2 == 1):
        fl += 1
    return sgn * fl * q


def test_epilogue_brute_force_exact_arithmetic():
    """Each float32 step of the epilogue redone in exact rationals with explicit
    nearest-even rounding: float(acc), sx*sw, the fused multiply-add (one rounding),
    then bf16. Catches: a non-fused multiply-add, a different order, a missing bias,
    scale indices swapped (sx[n] / sw[m])."""
    rng = np.random.default_rng(11)
    M, N = 6, 5
    acc = rng.integers(-(2**30), 2**30, size=(M, N)).astype(np.int32)
    acc[0, :] = rng.integers(-5000, 5000, size=N)
    sx = (rng.uniform(0.001, 0.1, M)).astype(np.float32)
    sw = (rng.uniform(1e-5, 1e-3, N)).astype(np.float32)
    b = torch_bf16(rng.standard_normal(N).astype(np.float32) * 3)
    y = oracle.epilogue(acc, sx, sw, b)
    bf = oracle.bf16_to_f32(b)
    for m in range(M):
        for n in range(N):
            a32 = _f32_round(Fraction(int(acc[m, n])))
            s32 = _f32_round(Fraction(float(sx[m])) * Fraction(float(sw[n])))
            y32 = _f32_round(a32 * s32 + Fraction(float(bf[n])))
            want = torch_bf16(np.array([float(y32)], np.float32))[0]
            assert y[m, n] == want, (m, n)


def test_epilogue_no_bias_equals_zero_bias():
    rng = np.random.default_rng(2)
    acc = rng.integers(-10**6, 10**6, size=(7, 9)).astype(np.int32)
    sx = rng.uniform(0, 1, 7).astype(np.float32)
    sw = rng.uniform(0, 1, 9).astype(np.float32)
    assert np.array_equal(oracle.epilogue(acc, sx, sw, None),
                          oracle.epilogue(acc, sx, sw, np.zeros(9, np.uint16)))


def test_epilogue_within_one_ulp_of_exact():
    """The float32 epilogue against the double-precision dequantization rounded once:
    at most 1 bf16 ulp apart, cosine >= 0.99999, on the tiny workload."""
    x, w, b = si.make_inputs(si.WORKLOADS[0][0])
    wq, sw = oracle.quantize_rows(w)
    y, xq, sx, acc = oracle.linear(x, wq, sw, b)
    y64 = oracle.epilogue_f64(acc, sx, sw, b)
    assert ulp_distance(y, y64).max() <= 1
    assert cosine(y, y64) >= 0.99999


def ulp_distance(a_bits, b_bits):
    def ordered(u):
        u = u.astype(np.int32)
        return np.where(u & 0x8000, -(u & 0x7FFF), u)
    return np.abs(ordered(a_bits) - ordered(b_bits))


def cosine(a_bits, b_bits):
    a = oracle.bf16_to_f32(a_bits).astype(np.float64).ravel()
    b = oracle.bf16_to_f32(b_bits).astype(np.float64).ravel()
    return float(a @ b / (np.linalg.norm(a) * np.linalg.norm(b)))


# ---------------------------------------------------------------- closed forms

def test_identity_weight_closed_form():
    """W = c*I (N = K, c = 0.5): every weight row has a = c, so sw = c/127 and
    Wq = 127*I; then acc = 127*Xq exactly, and Y is within 1 bf16 ulp of c times the
    dequantized X (sx*Xq). Catches: weight rows and columns swapped, per-tensor instead
    of per-channel scale."""
    K = 64
    x, _, _ = si.make_inputs((16, K, K), seed=9)
    w = bits((0.5 * np.eye(K, dtype=np.float32)).ravel().tolist()).reshape(K, K)
    wq, sw = oracle.quantize_rows(w)
    assert np.array_equal(wq, 127 * np.eye(K, dtype=np.int8))
    assert np.all(sw == np.float32(0.5) / np.float32(127))
    y, xq, sx, acc = oracle.linear(x, wq, sw, None)
    assert np.array_equal(acc, 127 * xq.astype(np.int32))
    deq = 0.5 * sx[:, None].astype(np.float64) * xq
    assert ulp_distance(y, oracle.f64_to_bf16(deq).reshape(y.shape)).max() <= 1


def test_constant_activation_row_closed_form():
    """A token whose activations are all equal quantizes to all-127, so
    acc[m, n] = 127 * sum_k Wq[n, k]."""
    K, N = 48, 10
    _, w, _ = si.make_inputs((1, K, N), seed=4)
    x = bits([-1.25] * K).reshape(1, K)
    wq, sw = oracle.quantize_rows(w)
    y, xq, sx, acc = oracle.linear(x, wq, sw, None)
    assert np.all(xq == -127)
    assert np.array_equal(acc[0], -127 * wq.astype(np.int32).sum(axis=1))


def test_zero_token_gives_bias_exactly():
    """A zero token row has s = 0 and q = 0, so its output row is exactly bf16(b)."""
    x, w, b = si.make_inputs((4, 96, 12), seed=8)
    x[2] = 0
    wq, sw = oracle.quantize_rows(w)
    y, _, sx, _ = oracle.linear(x, wq, sw, b)
    assert sx[2] == 0 and np.array_equal(y[2], b)
