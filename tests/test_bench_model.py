"""The benchmark's algorithmic byte/op model, pinned to the paper (no GPU).

The paper classifies its five DiT GEMM shapes as compute-bound with arithmetic
intensities of 768 to 6337 ops/byte over token counts 512..16384 (fixture
tests/golden/arith_intensity.txt). With int8 operands read once and a bf16 output
written once, 2MNK / (MK + NK + 2MN) reproduces both ends of that range; a byte model
that counted bf16 operands, an fp32 output, or dropped the output would not.
"""
import os

import bench

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "arith_intensity.txt")


def load_golden():
    shapes, vals = [], {}
    for line in open(GOLDEN):
        line = line.strip()
        if not line or line.startswith("#"):
            continue
        parts = line.split()
        if parts[0] == "shape":
            shapes.append((parts[1], int(parts[2]), int(parts[3])))
        else:
            vals[parts[0]] = [int(p) for p in parts[1:]]
    return shapes, vals


def intensity(M, N, K):
    return bench.gemm_ops(M, N, K) / bench.gemm_bytes(M, N, K, with_vectors=False)


def test_paper_intensity_range_reproduced():
    shapes, vals = load_golden()
    m_lo, m_hi = vals["m_range"]
    lo = min(intensity(m_lo, N, K) for _, N, K in shapes)
    hi = max(intensity(m_hi, N, K) for _, N, K in shapes)
    assert round(lo) == vals["intensity_min"][0]
    assert round(hi) == vals["intensity_max"][0]
    # every shape and token count in the range stays above the MI355X ridge point
    # (5033 TOP/s / 8 TB/s ~ 629 ops/byte) at M >= 512
    for _, N, K in shapes:
        for M in (m_lo, 1024, 4110, m_hi):
            assert intensity(M, N, K) > 629


def test_wrong_models_fail():
    shapes, vals = load_golden()
    m_lo = vals["m_range"][0]
    # bf16 operands instead of int8: the low end moves
    lo_bf16 = min(bench.gemm_ops(m_lo, N, K) / (2 * m_lo * K + 2 * N * K + 2 * m_lo * N)
                  for _, N, K in shapes)
    assert round(lo_bf16) != vals["intensity_min"][0]
    # output dropped: the low end moves
    lo_noout = min(bench.gemm_ops(m_lo, N, K) / (m_lo * K + N * K) for _, N, K in shapes)
    assert round(lo_noout) != vals["intensity_min"][0]


def test_full_byte_model_adds_scales_and_bias():
    M, N, K = 2560, 4096, 4096
    assert bench.gemm_bytes(M, N, K) == M * K + N * K + 2 * M * N + 4 * M + 4 * N + 2 * N
    assert bench.quant_bytes(M, K) == 3 * M * K + 4 * M
