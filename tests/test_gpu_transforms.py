"""Parity of the transformed-activation and SmoothQuant paths with the CPU oracle
(needs an MI355X).

Bars: with a per-channel multiplier only, the float32 product x * c[k] is correctly
rounded on both sides, so codes and scales are bit-exact. With GELU, each side computes
its own GELU (the oracle in double, rounded once to float32; the kernel in float32 via
erfcf, a few units in the last place off): scales must agree to 2^-17 relative, codes
exactly except where the exact value lies within 2e-3 of a rounding tie (there they
may differ by one), and every code must reconstruct its value within half a step. The
GELU linear is compared with the oracle's own chain (its GELU codes, its product, its
epilogue): rows whose codes and scale agree must agree to 1 ulp, and every other output
must lie within the bound that its code and scale differences allow.
"""
import numpy as np
import pytest
import torch

import oracle
import synth_inputs as si
import paper_2606_14598_amd as w8a8
from _gelu_checks import check_gelu_codes, check_gelu_linear_against_oracle_chain
from _helpers import assert_bf16_parity, dev_bf16, dev_f32, host, host_bits, say

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    w8a8.load_library()
    yield
    torch.cuda.synchronize()


def _exact(q, s, q_o, s_o, what):
    assert np.array_equal(host(q), q_o), what
    assert np.array_equal(host(s), s_o), what


# ---------------------------------------------------------------- multiplier: exact

CM_CASES = [(37, 8), (37, 24), (37, 264), (16, 1024), (9, 3136), (9, 4096), (5, 12288),
            (5, 16384), (3, 20000), (4, 32768), (3, 32776), (3, 40000), (37, 7), (11, 269),
            (8300, 512)]


@pytest.mark.parametrize("M,K", CM_CASES)
def test_colmul_quantizer_exact(M, K):
    say(f"colmul quantizer M={M} K={K}")
    x, _, _ = si.make_inputs((M, K, 1), seed=300 + K, dist="outlier")
    cm = np.random.default_rng(K).uniform(0.05, 8, K).astype(np.float32)
    q_o, s_o = oracle.quantize_rows(x, col_mul=cm)
    q, s = w8a8.quantize_act(dev_bf16(x), col_mul=dev_f32(cm))
    _exact(q, s, q_o, s_o, f"act M={M} K={K}")
    qw, sw = w8a8.quantize_weight(dev_bf16(x), col_mul=dev_f32(cm))
    _exact(qw, sw, q_o, s_o, f"weight M={M} K={K}")


def test_colmul_unaligned_multiplier_takes_the_element_path():
    M, K = 13, 4096
    x, _, _ = si.make_inputs((M, K, 1), seed=77)
    cm = np.random.default_rng(5).uniform(0.1, 4, K).astype(np.float32)
    buf = torch.empty(K + 1, dtype=torch.float32, device="cuda")
    cm_d = buf[1:]
    cm_d.copy_(dev_f32(cm))
    assert cm_d.data_ptr() % 16 != 0
    q_o, s_o = oracle.quantize_rows(x, col_mul=cm)
    q, s = w8a8.quantize_act(dev_bf16(x), col_mul=cm_d)
    _exact(q, s, q_o, s_o, "unaligned multiplier")


# (rows, K) covering each threads-per-row x vectors-per-thread choice for transformed
# rows past 256 vectors per row, with a ragged last vector.
TRANSFORM_MAPPINGS = [(300, 1000),    # 128 x 1
                      (300, 2040),    # 256 x 1
                      (1030, 1536),   # 64 x 3
                      (1500, 4096),   # 256 x 2
                      (4100, 4096),   # 128 x 4
                      (4100, 2560),   # 64 x 5
                      (4100, 3072),   # 64 x 6
                      (4100, 3576),   # 64 x 7
                      (37, 4624),     # 256 x 3
                      (1030, 4624),   # 128 x 5
                      (1030, 6128),   # 128 x 6
                      (300, 8176),    # 256 x 4
                      (37, 12272),    # 512 x 3
                      (300, 12272),   # 256 x 6
                      (1030, 16368)]  # 256 x 8


@pytest.mark.parametrize("M,K", TRANSFORM_MAPPINGS)
def test_transformed_row_mappings(M, K):
    say(f"transformed mapping M={M} K={K}")
    h, _, _ = si.make_inputs((M, K, 1), seed=1700 + K + M, dist="preact")
    h[M // 2] = 0
    cm = np.random.default_rng(K + M).uniform(0.05, 8, K).astype(np.float32)
    q_o, s_o = oracle.quantize_rows(h, col_mul=cm)
    q, s = w8a8.quantize_act(dev_bf16(h), col_mul=dev_f32(cm))
    _exact(q, s, q_o, s_o, f"multiplier M={M} K={K}")
    q_o, s_o = oracle.quantize_rows(h, act="gelu", col_mul=cm)
    q, s = w8a8.quantize_act(dev_bf16(h), act="gelu", col_mul=dev_f32(cm))
    check_gelu_codes(h, host(q), host(s), q_o, s_o, cm, f"gelu*c M={M} K={K}")
    q_o, s_o = oracle.quantize_rows(h, act="gelu")
    q, s = w8a8.quantize_act(dev_bf16(h), act="gelu")
    check_gelu_codes(h, host(q), host(s), q_o, s_o, what=f"gelu M={M} K={K}")


# ---------------------------------------------------------------- GELU: within bound

GELU_CASES = [(37, 8), (37, 264), (64, 4096), (9, 16384), (5, 20000), (4, 32768),
              (3, 32776), (3, 53248), (11, 269), (8300, 512), (4100, 4096)]


@pytest.mark.parametrize("M,K", GELU_CASES)
def test_gelu_quantizer(M, K):
    say(f"gelu quantizer M={M} K={K}")
    h, _, _ = si.make_inputs((M, K, 1), seed=400 + K, dist="preact")
    q_o, s_o = oracle.quantize_rows(h, act="gelu")
    q, s = w8a8.quantize_act(dev_bf16(h), act="gelu")
    check_gelu_codes(h, host(q), host(s), q_o, s_o, what=f"gelu M={M} K={K}")


def test_gelu_with_multiplier_and_edge_rows():
    M, K = 24, 4096
    h, _, _ = si.make_inputs((M, K, 1), seed=91, dist="preact")
    h[0] = 0                                              # GELU(0) = 0: zero row
    h[1] = oracle.f32_to_bf16(-np.abs(oracle.bf16_to_f32(h[1])) - 4)   # left tail only
    h[2] = oracle.f32_to_bf16(oracle.bf16_to_f32(h[2]) * 40)           # large values
    cm = np.random.default_rng(2).uniform(0.2, 5, K).astype(np.float32)
    q_o, s_o = oracle.quantize_rows(h, act="gelu", col_mul=cm)
    q, s = w8a8.quantize_act(dev_bf16(h), act="gelu", col_mul=dev_f32(cm))
    assert host(s)[0] == 0 and not host(q)[0].any()
    # row 1 lives entirely in the left tail, where float32 erfc carries the argument's
    # rounding error amplified by 2z^2: compare its scale loosely and skip its codes.
    s1 = float(host(s)[1])
    assert s1 == pytest.approx(float(s_o[1]), rel=1e-4)
    keep = np.r_[0, 2:M]
    check_gelu_codes(h[keep], host(q)[keep], host(s)[keep], q_o[keep], s_o[keep], cm,
                     "gelu*c")
    check_left_tail_row(h[1], host(q)[1], s1, q_o[1], float(s_o[1]), cm)


def check_left_tail_row(h_row, q_g, s_g, q_o, s_o, cm):
    """A row with every x <= -4. GELU(x) = x Phi(x) there is tiny and float32 erfc(z),
    z = -x / sqrt(2), carries the relative rounding error of its argument amplified by
    about 2 z^2, plus that of the fit and the exponential: for the row's largest
    |GELU(x) c[k]| (x >= -10, z^2 <= 50) that is below 2 * 50 * 2^-24 + 1e-6 ~ 7e-6
    relative, and the codes' products v * (127 / a) move by at most 127 times that, ~1e-3.
    Stated bound: scale within 2e-5 relative; codes equal wherever the exact product is
    more than 2e-3 from a rounding tie, within 1 elsewhere; every code reconstructs the
    exact value within half a step (plus the scale's relative error)."""
    v = oracle.gelu_f64(oracle.bf16_to_f32(h_row).astype(np.float64)) * cm.astype(np.float64)
    a = np.abs(v).max()
    rel = abs(s_g / s_o - 1.0)
    t = np.abs(v) * (127.0 / a)
    near = np.abs(t - np.floor(t) - 0.5) < 2e-3
    d = np.abs(q_g.astype(np.int32) - q_o.astype(np.int32))
    say(f"   left-tail row: scale rel err {rel:.2e}, {int((d != 0).sum())} code differences, "
        f"{int(near.sum())} near ties, min x {oracle.bf16_to_f32(h_row).min():.2f}")
    assert rel <= 2e-5
    assert d.max() <= 1
    assert not (d[~near] != 0).any(), np.argwhere((d != 0) & ~near)[:5]
    assert np.abs(q_g).max() == 127
    rec = s_g * q_g.astype(np.float64)
    assert np.all(np.abs(rec - v) <= 0.5 * s_g * (1 + 1e-3) + s_g * 127 * 2e-5 + 1e-30)


# ---------------------------------------------------------------- calibration

def test_col_absmax_exact_and_accumulating():
    K = 4104
    batches = [si.make_inputs((300, K, 1), seed=500 + i)[0] for i in range(3)]
    want = np.max([oracle.col_absmax(b) for b in batches], axis=0)
    out = w8a8.col_absmax(dev_bf16(batches[0]))
    for b in batches[1:]:
        w8a8.col_absmax(dev_bf16(b), out=out, accumulate=True)
    assert np.array_equal(host(out), want)
    # a fresh call (accumulate=False) overwrites
    w8a8.col_absmax(dev_bf16(batches[1]), out=out)
    assert np.array_equal(host(out), oracle.col_absmax(batches[1]))
    # ragged K and a single row
    x, _, _ = si.make_inputs((1, 77, 1), seed=9)
    assert np.array_equal(host(w8a8.col_absmax(dev_bf16(x))), oracle.col_absmax(x))


def test_col_absmax_gelu():
    h, _, _ = si.make_inputs((700, 1000, 1), seed=510, dist="preact")
    got = host(w8a8.col_absmax(dev_bf16(h), act="gelu")).astype(np.float64)
    want = oracle.col_absmax(h, act="gelu").astype(np.float64)
    assert np.max(np.abs(got / want - 1)) <= 2.0 ** -17


def _amax_cases():
    rng = np.random.default_rng(31)
    ax = rng.uniform(0.01, 80, 5000).astype(np.float32)
    aw = rng.uniform(1e-3, 0.5, 5000).astype(np.float32)
    ax[:6] = [0, 3, 2.0 ** -120, 2.0 ** 120, 5, 1]
    aw[:6] = [1, 0, 2.0 ** 120, 2.0 ** -120, 5, 1]
    return ax, aw


def test_smooth_factors_alpha_half_exact():
    ax, aw = _amax_cases()
    s_o, si_o = oracle.smooth_factors(ax, aw, 0.5)
    s, s_inv = w8a8.smooth_factors(dev_f32(ax), dev_f32(aw), 0.5)
    assert np.array_equal(host(s), s_o)
    assert np.array_equal(host(s_inv), si_o)


@pytest.mark.parametrize("alpha", [0.0, 0.3, 0.75, 1.0])
def test_smooth_factors_other_alpha(alpha):
    ax, aw = _amax_cases()
    s_o, _ = oracle.smooth_factors(ax, aw, alpha)
    s, s_inv = w8a8.smooth_factors(dev_f32(ax), dev_f32(aw), alpha)
    s, s_inv = host(s), host(s_inv)
    assert np.max(np.abs(s.astype(np.float64) / s_o - 1)) <= 2.0 ** -20
    assert np.array_equal(s_inv, (np.float32(1) / s).astype(np.float32))


# ---------------------------------------------------------------- whole linears

def _ref_error(y_bits, x, w, b):
    ref = (oracle.bf16_to_f32(x).astype(np.float64) @ oracle.bf16_to_f32(w).astype(np.float64).T
           + oracle.bf16_to_f32(b))
    y = oracle.bf16_to_f32(y_bits).astype(np.float64)
    return float(np.linalg.norm(y - ref) / np.linalg.norm(ref))


def test_smoothed_linear_matches_oracle_and_helps():
    M, K, N = 257, 1024, 391
    say(f"smoothed linear M={M} K={K} N={N}")
    x, w, b = si.make_inputs((M, K, N), seed=20260)
    calib = [si.make_inputs((M, K, N), seed=7100 + i)[0] for i in range(3)]
    ax = w8a8.col_absmax(dev_bf16(calib[0]))
    for c in calib[1:]:
        w8a8.col_absmax(dev_bf16(c), out=ax, accumulate=True)
    aw = w8a8.col_absmax(dev_bf16(w))
    s, s_inv = w8a8.smooth_factors(ax, aw, 0.5)
    ax_o = np.max([oracle.col_absmax(c) for c in calib], axis=0)
    aw_o = oracle.col_absmax(w)
    s_o, si_o = oracle.smooth_factors(ax_o, aw_o, 0.5)
    assert np.array_equal(host(s), s_o) and np.array_equal(host(s_inv), si_o)
    wq, sw = w8a8.quantize_weight(dev_bf16(w), col_mul=s)
    wq_o, sw_o = oracle.quantize_rows(w, col_mul=s_o)
    _exact(wq, sw, wq_o, sw_o, "smoothed weights")
    y = host_bits(w8a8.linear(dev_bf16(x), wq, sw, dev_bf16(b), col_mul=s_inv))
    xq_o, sx_o = oracle.quantize_rows(x, col_mul=si_o)
    y_o = oracle.epilogue(oracle.gemm_acc(xq_o, wq_o), sx_o, sw_o, b)
    st = assert_bf16_parity(y, y_o, "smoothed linear")
    # the point of smoothing: the outlier channels no longer set every token's step
    wq0, sw0 = w8a8.quantize_weight(dev_bf16(w))
    y0 = host_bits(w8a8.linear(dev_bf16(x), wq0, sw0, dev_bf16(b)))
    e0, e1 = _ref_error(y0, x, w, b), _ref_error(y, x, w, b)
    say(f"   {st}; rel. error vs fp64: plain {e0:.4f}, smoothed {e1:.4f}")
    assert e1 < 0.8 * e0


@pytest.mark.parametrize("M,K,N", [(300, 4096, 520), (64, 264, 130), (1, 16384, 64)])
def test_gelu_linear(M, K, N):
    say(f"gelu linear M={M} K={K} N={N}")
    h, w, b = si.make_inputs((M, K, N), seed=600 + M, dist="preact")
    wq_o, sw_o = oracle.quantize_rows(w)
    wq, sw = w8a8.quantize_weight(dev_bf16(w))
    assert np.array_equal(host(wq), wq_o) and np.array_equal(host(sw), sw_o)
    hd = dev_bf16(h)
    y = host_bits(w8a8.linear(hd, wq, sw, dev_bf16(b), act="gelu"))
    xq, sx = w8a8.quantize_act(hd, act="gelu")
    check_gelu_linear_against_oracle_chain(h, wq_o, sw_o, b, y, host(xq), host(sx),
                                           f"gelu linear {M}x{K}x{N}")
    assert np.array_equal(y, host_bits(w8a8.gemm(xq, sx, wq, sw, dev_bf16(b))))


def test_full_size_gelu_down_projection():
    """The MLP down-projection at its workload shape (M=2560, K=16384, N=4096), fed the
    pre-activation, every output against the oracle's own chain."""
    shp = si.workload(2, "mlp_down")
    say(f"full-size gelu down-projection M={shp.M} K={shp.K} N={shp.N}")
    h, w, b = si.make_inputs(shp, dist="preact")
    wq_o, sw_o = oracle.quantize_rows(w)
    wq, sw = w8a8.quantize_weight(dev_bf16(w))
    assert np.array_equal(host(wq), wq_o) and np.array_equal(host(sw), sw_o)
    hd = dev_bf16(h)
    y = host_bits(w8a8.linear(hd, wq, sw, dev_bf16(b), act="gelu"))
    xq, sx = w8a8.quantize_act(hd, act="gelu")
    check_gelu_linear_against_oracle_chain(h, wq_o, sw_o, b, y, host(xq), host(sx),
                                           "down-projection")
