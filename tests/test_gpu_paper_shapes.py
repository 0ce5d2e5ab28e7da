"""The paper's five model GEMM shapes (Section 3, "Target architecture") at its in-model
token count M = 4110 (Section 5), through the product path, against the CPU oracle on
sampled rows and columns (needs an MI355X). M = 4110 fits no tile height, so every
shape also runs a ragged last row of tiles; K = 53248 (the LLM projection) takes the
quantizer's 1024-thread rows and the longest accumulation (|acc| up to 8.6e8). The
N = 4608 shapes also run at 512 and 1024 tokens, where the table picks the 96-channel
tiles."""
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


def _sample(n, rng, extra=()):
    base = {0, 1, 127, 128, 255, 256, n - 2, n - 1, *extra}
    base |= set(rng.integers(0, n, size=4).tolist())
    return np.array(sorted(i for i in base if 0 <= i < n))


CASES = [(p[0], 4110) for p in si.PAPER_SHAPES] + [
    ("attn_out", 512), ("attn_out", 1024), ("ffn_down", 512), ("ffn_down", 1024)]


@pytest.mark.parametrize("name,M", CASES)
def test_paper_shape_at_in_model_tokens(name, M):
    shp = si.paper_shape(name, M)
    say(f"paper shape {name}: M={shp.M} K={shp.K} N={shp.N} tile="
        f"{w8a8.tile_name(w8a8.select_tile(shp.M, shp.N, shp.K))}")
    x, w, b = si.make_inputs(shp)
    wq_o, sw_o = oracle.quantize_rows(w)
    wq, sw = w8a8.quantize_weight(dev_bf16(w))
    assert np.array_equal(host(wq), wq_o) and np.array_equal(host(sw), sw_o)
    xd = dev_bf16(x)
    y = host_bits(w8a8.linear(xd, wq, sw, dev_bf16(b)))
    xq, sx = w8a8.quantize_act(xd)
    acc = host(w8a8.gemm_acc_i32(xq, wq))
    rng = np.random.default_rng(shp.seed)
    rows = _sample(shp.M, rng, extra=(4095, 4096, 4103))
    cols = _sample(shp.N, rng)
    y_r, xq_r, sx_r, acc_r = oracle.linear(x[rows], wq_o, sw_o, b)
    assert np.array_equal(host(xq)[rows], xq_r)
    assert np.array_equal(host(sx)[rows], sx_r)
    assert np.array_equal(acc[rows], acc_r)
    st = assert_bf16_parity(y[rows], y_r, f"{name} rows")
    y_c, _, _, acc_c = oracle.linear(x, wq_o[cols], sw_o[cols], b[cols])
    assert np.array_equal(acc[:, cols], acc_c)
    st2 = assert_bf16_parity(y[:, cols], y_c, f"{name} cols")
    say("   rows", st, "cols", st2)
