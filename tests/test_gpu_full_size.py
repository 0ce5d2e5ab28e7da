"""Full-tensor parity at the production shapes (needs an MI355X).

Every element of Xq, sx, the int32 accumulator and the bf16 output is compared with the
CPU oracle on the same seeded inputs, through the entry points and tiles the benchmark
times:
  * all workload shapes (the tiny linear, the 768px attention projection and QKV, the
    768px MLP, the four 1024px linears, the skinny and odd shapes);
  * the paper's five model shapes at its in-model token count M = 4110 (Section 5, "The
    kernel is exact and the GEMMs are compute-bound": bit-exact on all five shapes),
    and one token bucket for every other tile the table selects for them (the
    96-channel tiles, the split-K tiles at K = 53248, the 256-row tiles);
  * the two table tiles that serve only M >= 12289 run, forced through w8a8_gemm_ex,
    at a smaller M with their shapes' own N and K.
Bars: codes, scale bits and the accumulator exact; bf16 within 1 ulp with cosine >=
0.99999 (both sides evaluate the epilogue in the same order, so the outputs are in fact
identical and the mismatch count is printed)."""
import numpy as np
import pytest
import torch

import oracle
import synth_inputs as si
import paper_2606_14598_amd as w8a8
from _helpers import assert_bf16_parity, dev_bf16, host, host_bits, say

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    w8a8.load_library()
    yield
    torch.cuda.synchronize()


def _full_compare(shp, tile=None):
    """Quantize W on both sides, run the product path on the GPU (w8a8_linear, or
    w8a8_gemm_ex with a forced tile) and the oracle's chain on the CPU, and compare every
    element."""
    M, K, N = shp.M, shp.K, shp.N
    chosen = w8a8.select_tile(M, N, K) if tile is None else tile
    say(f"full {shp.name}: M={M} K={K} N={N} dist={shp.dist} seed={shp.seed} "
        f"tile={w8a8.tile_name(chosen)}{' (forced)' if tile is not None else ''}")
    x, w, b = si.make_inputs(shp)
    wq_o, sw_o = oracle.quantize_rows(w)
    wq, sw = w8a8.quantize_weight(dev_bf16(w))
    assert np.array_equal(host(wq), wq_o), "weight codes"
    assert np.array_equal(host(sw).view(np.uint32), sw_o.view(np.uint32)), "weight scales"
    del w
    xd, bd = dev_bf16(x), dev_bf16(b)
    xq, sx = w8a8.quantize_act(xd)
    if tile is None:
        y = host_bits(w8a8.linear(xd, wq, sw, bd))
    else:
        y = host_bits(w8a8.gemm(xq, sx, wq, sw, bd, tile=tile))
    acc = host(w8a8.gemm_acc_i32(xq, wq))
    xq_h, sx_h = host(xq), host(sx)
    del xd, xq, wq
    torch.cuda.empty_cache()
    y_o, xq_o, sx_o, acc_o = oracle.linear(x, wq_o, sw_o, b)
    assert np.array_equal(xq_h, xq_o), "activation codes"
    assert np.array_equal(sx_h.view(np.uint32), sx_o.view(np.uint32)), "activation scales"
    bad = np.argwhere(acc != acc_o)
    assert bad.size == 0, f"{len(bad)} accumulators differ, first at {bad[:3].tolist()}"
    st = assert_bf16_parity(y, y_o, shp.name)
    say(f"   exact codes/scales/acc over {M}x{N}; bf16 {st}")


WORKLOAD_SHAPES = [(c, s.name) for c in sorted(si.WORKLOADS) for s in si.WORKLOADS[c]]


@pytest.mark.parametrize("config,name", WORKLOAD_SHAPES)
def test_workload_full_tensors(config, name):
    _full_compare(si.workload(config, name))


# The paper's shapes at M = 4110, then a bucket for each other tile the table selects:
# 96-channel tiles (attn_out / ffn_down at 512 and 1024 tokens), split-K tiles (llm_proj
# at 512 and 1024, K = 53248), 256 x 128 (qkv at 512), 256 x 256 eight-wavefront (qkv at
# 1024).
PAPER_CASES = [(p[0], 4110) for p in si.PAPER_SHAPES] + [
    ("attn_out", 512), ("attn_out", 1024), ("ffn_down", 512), ("ffn_down", 1024),
    ("llm_proj", 512), ("llm_proj", 1024), ("qkv", 512), ("qkv", 1024)]


@pytest.mark.parametrize("name,M", PAPER_CASES)
def test_paper_shape_full_tensors(name, M):
    _full_compare(si.paper_shape(name, M))


# Tiles the table picks only for M >= 12289 (ffn_down: m256n256k128w2x2s2, llm_proj:
# m128n256k128w2x2s3), forced at a smaller, ragged M with the shape's N and K.
FORCED = [("ffn_down", 2001, "m256n256k128w2x2s2"), ("llm_proj", 1000, "m128n256k128w2x2s3")]


@pytest.mark.parametrize("name,M,tile_name", FORCED)
def test_large_token_tiles_full_tensors(name, M, tile_name):
    ids = [t for t in range(w8a8.tile_count()) if w8a8.tile_name(t) == tile_name]
    assert len(ids) == 1
    big = si.paper_shape(name, 16384)
    assert w8a8.select_tile(big.M, big.N, big.K) == ids[0], "the table's tile changed"
    _full_compare(si.paper_shape(name, M), tile=ids[0])
