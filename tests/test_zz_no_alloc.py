"""w8a8_linear_noalloc, the entry point for callers that cannot allocate: through the C
ABI, against w8a8_linear_ex with a caller-allocated workspace (the same kernels, so the
outputs must be identical bit for bit), on calls in a row whose sizes shrink, so the
shared device scratch holds the previous call's contents."""
import ctypes

import numpy as np
import pytest
import torch

import synth_inputs as si
import paper_2606_14598_amd as w8a8
from _helpers import dev_bf16, host_bits, say

pytestmark = pytest.mark.gpu

P = ctypes.c_void_p
ACT = {"none": 0, "gelu": 1}


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    lib = w8a8.load_library()
    f = lib.w8a8_linear_noalloc
    f.argtypes = [P, ctypes.c_int, P, P, P, P, P, ctypes.c_int64, ctypes.c_int64,
                  ctypes.c_int64, P]
    f.restype = ctypes.c_int
    yield
    torch.cuda.synchronize()


def _ptr(t):
    return None if t is None else P(t.data_ptr())


def _case(M, K, N, dist, seed, act, with_cm):
    x, w, b = si.make_inputs((M, K, N), seed=seed, dist=dist)
    xd, bd = dev_bf16(x), dev_bf16(b)
    wq, sw = w8a8.quantize_weight(dev_bf16(w))
    cm = None
    if with_cm:
        g = torch.Generator(device="cpu").manual_seed(seed)
        cm = (torch.rand(K, generator=g) * 4 + 0.25).cuda()
    return xd, wq, sw, bd, cm


def _noalloc(xd, wq, sw, bd, cm, act):
    lib = w8a8.load_library()
    M, K = xd.shape
    N = wq.shape[0]
    y = torch.empty((M, N), dtype=torch.bfloat16, device="cuda")
    st = lib.w8a8_linear_noalloc(_ptr(xd), ACT[act], _ptr(cm), _ptr(wq), _ptr(sw), _ptr(bd),
                                 _ptr(y), M, N, K,
                                 P(torch.cuda.current_stream().cuda_stream))
    assert st == 0, lib.w8a8_status_string(st)
    return y


def _with_workspace(xd, wq, sw, bd, cm, act):
    lib = w8a8.load_library()
    M, K = xd.shape
    N = wq.shape[0]
    y = torch.empty((M, N), dtype=torch.bfloat16, device="cuda")
    nws = w8a8.linear_workspace_bytes(M, N, K)
    ws = torch.empty(nws, dtype=torch.uint8, device="cuda")
    st = lib.w8a8_linear_ex(_ptr(xd), ACT[act], _ptr(cm), _ptr(wq), _ptr(sw), _ptr(bd),
                            _ptr(y), M, N, K, _ptr(ws), nws,
                            P(torch.cuda.current_stream().cuda_stream))
    assert st == 0, lib.w8a8_status_string(st)
    return y


# Pairs of calls, the second smaller than the first: the attention projection then a
# ragged smaller linear; the LLM projection with split-K partials in the scratch (512
# tokens, K = 53248) then a shorter one; GELU with the SmoothQuant multiplier.
SEQUENCES = [
    [((2560, 4096, 4096), "outlier", "none", False), ((1000, 4096, 391), "student_t", "none", False)],
    [((512, 53248, 4608), "outlier", "none", False), ((300, 4112, 1000), "outlier", "none", False)],
    [((700, 4096, 2048), "preact", "gelu", True), ((257, 1040, 264), "preact", "gelu", True)],
]


@pytest.mark.parametrize("seq", range(len(SEQUENCES)))
def test_noalloc_matches_workspace_entry_point(seq):
    for i, ((M, K, N), dist, act, cm) in enumerate(SEQUENCES[seq]):
        say(f"noalloc seq {seq} call {i}: M={M} K={K} N={N} act={act} col_mul={cm}")
        args = _case(M, K, N, dist, 40 + 7 * seq + i, act, cm)
        want = host_bits(_with_workspace(*args, act))
        got = host_bits(_noalloc(*args, act))
        assert np.array_equal(got, want), (seq, i)


def test_noalloc_rejects_problems_beyond_its_scratch():
    lib = w8a8.load_library()
    limit = 128 << 20
    M, N, K = 8192, 64, 16384           # Xq alone is 128 MiB; sx pushes it over
    assert w8a8.linear_workspace_bytes(M, N, K) > limit
    fake = P(256)                        # never dereferenced: rejected before any launch
    assert lib.w8a8_linear_noalloc(fake, 0, None, fake, fake, None, fake, M, N, K,
                                   None) == 7
