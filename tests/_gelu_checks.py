"""Bounds for GELU rows, shared by the GPU tests (comparison only: the arithmetic they
compare against is the oracle's).

Each side computes its own GELU in front of the quantizer (the oracle in double, rounded
once to float32; the kernel in float32 through an erfc fit, a few units in the last
place off), so for GELU rows the scales agree to 2^-17 relative, codes agree exactly
except near rounding ties, and a linear's outputs differ by at most what those code and
scale differences allow.
"""
import numpy as np

import oracle
from _helpers import assert_bf16_parity, say


def check_gelu_codes(h_bits, q_g, s_g, q_o, s_o, cm=None, what=""):
    """GELU rows: scales to 2^-17, codes exact away from rounding ties, +-1 near them."""
    q_g = np.asarray(q_g).astype(np.int32)
    s_g = np.asarray(s_g)
    v = oracle.gelu_f64(oracle.bf16_to_f32(h_bits).astype(np.float64))
    if cm is not None:
        v = v * cm.astype(np.float64)[None, :]
    a = np.abs(v).max(axis=1)
    live = s_o > 0
    assert np.array_equal(live, s_g > 0), what
    rel = np.abs(s_g[live].astype(np.float64) / s_o[live] - 1)
    assert rel.size == 0 or rel.max() <= 2.0 ** -17, (what, rel.max())
    t = np.zeros_like(v)
    t[live] = np.abs(v[live]) * (127.0 / a[live, None])
    frac = t - np.floor(t)
    near = np.abs(frac - 0.5) < 2e-3
    d = np.abs(q_g - q_o.astype(np.int32))
    assert d.max(initial=0) <= 1, what
    assert not (d[~near] != 0).any(), (what, np.argwhere((d != 0) & ~near)[:5])
    assert np.all(np.abs(q_g[live]).max(axis=1) == 127), what
    # every code reconstructs its value within half a step (slack for both roundings)
    rec = s_g[:, None].astype(np.float64) * q_g
    assert np.all(np.abs(rec - v) <= 0.5 * s_g[:, None] * (1 + 1e-3) + 1e-30), what
    say(f"   {what}: {int((d != 0).sum())} code differences, {int(near.sum())} near ties, "
        f"scale rel err {rel.max(initial=0):.2e}")


def check_gelu_linear_against_oracle_chain(h, wq_o, sw_o, b, y, xq_g, sx_g, what):
    """The GELU linear's output y against the oracle's own chain: GELU codes and scales
    from the oracle's quantizer, its exact product, its epilogue. Rows whose codes and
    scale agree must agree to 1 ulp. On any other row an output may differ by what its
    code and scale differences allow,
      |dy| <= sw[n] (|sx_g - sx_o| |acc_o| + sx_g |acc_g - acc_o|) + ulp(y_g) + ulp(y_o),
    where |acc_g - acc_o| <= 127 * (number of differing codes in the row). The number of
    differing codes is bounded too: at most 0.1% of the row's codes."""
    q_o, s_o = oracle.quantize_rows(h, act="gelu")
    acc_o = oracle.gemm_acc(q_o, wq_o)
    y_o = oracle.epilogue(acc_o, s_o, sw_o, b)
    check_gelu_codes(h, xq_g, sx_g, q_o, s_o, what=f"{what} codes")
    dq = xq_g.astype(np.int32) != q_o.astype(np.int32)
    same = ~dq.any(axis=1) & (sx_g.view(np.uint32) == s_o.view(np.uint32))
    assert dq.sum() <= max(2, dq.size // 1000), (what, int(dq.sum()))
    st = assert_bf16_parity(y[same], y_o[same], f"{what}: rows with equal codes")
    other = np.flatnonzero(~same)
    if other.size:
        yg = oracle.bf16_to_f32(y[other]).astype(np.float64)
        yo = oracle.bf16_to_f32(y_o[other]).astype(np.float64)
        ndiff = dq[other].sum(axis=1).astype(np.float64)
        bound = sw_o.astype(np.float64)[None, :] * (
            np.abs(sx_g[other].astype(np.float64) - s_o[other])[:, None]
            * np.abs(acc_o[other].astype(np.float64))
            + sx_g[other].astype(np.float64)[:, None] * 127.0 * ndiff[:, None])
        ulp = lambda v: np.spacing(np.abs(v).astype(np.float32)).astype(np.float64) * 65536
        assert np.all(np.abs(yg - yo) <= bound + ulp(yg) + ulp(yo)), what
    say(f"   {what}: {int(same.sum())}/{len(same)} rows with equal codes, {st}; "
        f"{int(dq.sum())} code differences")
