"""Parity of the HIP path with the CPU oracle (needs an MI355X).

Every comparison is against the oracle run on the same seeded inputs; nothing the GPU
produces feeds the oracle. Bars: int8 codes, float32 scales and the int32 accumulator
bit-exact; bf16 outputs within 1 ulp, all finite, cosine >= 0.99999 (the float32
epilogue runs in the same order on both sides, so they are in fact expected to match
bit for bit -- the mismatch count is printed).
"""
import numpy as np
import pytest
import torch

import oracle
import synth_inputs as si
import paper_2606_14598_amd as w8a8
from _helpers import assert_bf16_parity

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    w8a8.load_library()
    yield
    torch.cuda.synchronize()


def dev_bf16(bits: np.ndarray) -> torch.Tensor:
    return torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).view(torch.bfloat16).cuda()


def host_bits(t: torch.Tensor) -> np.ndarray:
    return t.contiguous().view(torch.int16).cpu().numpy().view(np.uint16)


def host(t: torch.Tensor) -> np.ndarray:
    return t.cpu().numpy()


def say(*a):
    print(*a, flush=True)


# ---------------------------------------------------------------- quantizer

QUANT_K = [1, 3, 7, 8, 16, 24, 264, 512, 520, 1024, 2048, 3136, 4096, 4104, 8192, 16384,
           16392, 20000, 32768, 32776, 53248, 65536, 65544, 65538]


@pytest.mark.parametrize("K", QUANT_K)
def test_quantizer_bytes_and_scales_exact(K):
    """Codes and scale bits equal the oracle's for every kernel variant (register-resident
    rows of one wavefront up to a 1024-thread block, K <= 65536; looped rows beyond;
    scalar rows for K % 8 != 0)."""
    say(f"quantizer K={K}")
    x, _, _ = si.make_inputs((37, K, 1), seed=100 + K, dist="student_t")
    if K >= 4:
        x[3] = 0                                                   # zero row
        x[5] = si.bf16_bits_from_f32(oracle.bf16_to_f32(x[5]) * np.float32(1e-38))
        x[6] = si.bf16_bits_from_f32(np.where(np.arange(K) % 3 == 0, 1e-36, 7e-39).astype(np.float32))
        x[7] = si.bf16_bits_from_f32(-np.abs(oracle.bf16_to_f32(x[7])))
    q_o, s_o = oracle.quantize_rows(x)
    q, s = w8a8.quantize_act(dev_bf16(x))
    torch.cuda.synchronize()
    assert np.array_equal(host(q), q_o)
    assert np.array_equal(host(s).view(np.uint32), s_o.view(np.uint32))
    qw, sw = w8a8.quantize_weight(dev_bf16(x))
    assert np.array_equal(host(qw), q_o) and np.array_equal(host(sw).view(np.uint32),
                                                             s_o.view(np.uint32))


@pytest.mark.parametrize("K", [2056, 3136, 4096])
def test_quantizer_many_rows_exact(K):
    """At 4096 rows and more, K in (2048, 4096] takes one wavefront per row (fewer rows
    take two wavefronts per row, two rows per block): both variants against the oracle."""
    x, _, _ = si.make_inputs((4200, K, 1), seed=700 + K, dist="student_t")
    x[4099] = 0
    q_o, s_o = oracle.quantize_rows(x)
    q, s = w8a8.quantize_act(dev_bf16(x))
    assert np.array_equal(host(q), q_o) and np.array_equal(host(s), s_o)
    q2, s2 = w8a8.quantize_act(dev_bf16(x[:4095]))
    assert np.array_equal(host(q2), q_o[:4095]) and np.array_equal(host(s2), s_o[:4095])


# (rows, K) covering each threads-per-row x vectors-per-thread choice of the plain rule
# past 256 vectors per row, with a ragged last vector; K % 16 == 8 takes 8-byte stores,
# K % 16 == 0 the 16-byte streaming stores (with an odd vector count, the last vector's
# pair is stored by the even lane).
ROW_MAPPINGS = [(37, 4096),     # 512 x 1
                (300, 4104),    # 256 x 3, 8-byte stores
                (37, 4624),     # 256 x 3
                (1500, 4096),   # 128 x 4
                (1030, 4624),   # 128 x 5
                (1030, 4616),   # 128 x 5, 8-byte stores
                (1030, 6128),   # 128 x 6
                (300, 8176),    # 256 x 4
                (4100, 8176),   # 128 x 8
                (300, 12272),   # 256 x 6
                (1030, 16368),  # 256 x 8
                (2050, 16368),  # 1024 x 2
                (1030, 2568),   # 64 x 5, 8-byte stores
                (4100, 2560),   # 64 x 5
                (1030, 3072),   # 64 x 6
                (4100, 3584),   # 64 x 7
                (4100, 3568),   # 64 x 7, ragged last vector
                (300, 1000),    # 128 x 1
                (1030, 1016),   # 64 x 2
                (300, 2040),    # 256 x 1
                (1030, 1536),   # 64 x 3
                (1030, 1544),   # 64 x 4, 8-byte stores
                (37, 504),      # 64 x 1
                (200, 12272),   # 512 x 3
                (255, 16368)]   # 512 x 4


@pytest.mark.parametrize("M,K", ROW_MAPPINGS)
def test_quantizer_row_mappings(M, K):
    say(f"quantizer mapping M={M} K={K}")
    x, _, _ = si.make_inputs((M, K, 1), seed=1300 + K + M, dist="student_t")
    x[M // 2] = 0
    q_o, s_o = oracle.quantize_rows(x)
    q, s = w8a8.quantize_act(dev_bf16(x))
    assert np.array_equal(host(q), q_o)
    assert np.array_equal(host(s).view(np.uint32), s_o.view(np.uint32))


@pytest.mark.parametrize("M,K", [(1100, 40000), (600, 24576)])
def test_quantizer_long_rows_many_blocks(M, K):
    """Rows of a 1024-thread block, more rows than the persistent grid's 512 blocks: each
    block walks several rows with the next one prefetched; the zero row sits in a block's
    second round."""
    say(f"quantizer long rows M={M} K={K}")
    x, _, _ = si.make_inputs((M, K, 1), seed=900 + K, dist="student_t")
    x[M - 3] = 0
    q_o, s_o = oracle.quantize_rows(x)
    q, s = w8a8.quantize_act(dev_bf16(x))
    assert np.array_equal(host(q), q_o)
    assert np.array_equal(host(s).view(np.uint32), s_o.view(np.uint32))


def test_quantizer_more_rows_than_looped_grid():
    """K % 8 != 0 takes the looped kernel, whose grid stops at 65536 blocks: every block
    then takes a second row (or more), after the shared row maximum is reused."""
    M, K = 70001, 5
    x, _, _ = si.make_inputs((M, K, 1), seed=4242, dist="student_t")
    x[65536] = 0
    q_o, s_o = oracle.quantize_rows(x)
    q, s = w8a8.quantize_act(dev_bf16(x))
    assert np.array_equal(host(q), q_o)
    assert np.array_equal(host(s).view(np.uint32), s_o.view(np.uint32))


def test_quantizer_unaligned_pointers():
    K = 256
    x, _, _ = si.make_inputs((20, K + 1, 1), seed=3)
    buf = dev_bf16(x.ravel())
    view = buf[1:1 + 19 * K].view(19, K)     # 2-byte offset: not 16-byte aligned
    q_o, s_o = oracle.quantize_rows(x.ravel()[1:1 + 19 * K].reshape(19, K))
    q, s = w8a8.quantize_act(view)
    assert np.array_equal(host(q), q_o)
    assert np.array_equal(host(s), s_o)


# ---------------------------------------------------------------- int32 accumulator

ACC_SHAPES = [(64, 128, 256), (257, 391, 384), (300, 520, 1040), (1, 1, 16), (33, 65, 4096),
              (130, 17, 3136), (5, 300, 128), (513, 260, 512)]
GENERIC_SHAPES = [(45, 77, 269), (3, 5, 1), (70, 140, 264 + 8)]


def _acc_case(M, N, K, seed):
    x, w, _ = si.make_inputs((M, K, N), seed=seed)
    xq_o, _ = oracle.quantize_rows(x)
    wq_o, _ = oracle.quantize_rows(w)
    return xq_o, wq_o, oracle.gemm_acc(xq_o, wq_o)


# The library's tile count; test_tile_count_matches keeps it honest.
NUM_TILES = 40


def test_tile_count_matches():
    assert w8a8.tile_count() == NUM_TILES


@pytest.mark.parametrize("tile", range(NUM_TILES))
def test_acc_exact_every_tile(tile):
    """Every tile configuration gives the exact accumulator on ragged shapes (M, N not
    multiples of the tile, K tails, single rows/columns)."""
    for (M, N, K) in ACC_SHAPES + GENERIC_SHAPES:
        say(f"acc tile={tile} ({w8a8.tile_name(tile)}) M={M} N={N} K={K}")
        xq_o, wq_o, acc_o = _acc_case(M, N, K, seed=M * 7 + N * 3 + K)
        acc = w8a8.gemm_acc_i32(torch.from_numpy(xq_o).cuda(), torch.from_numpy(wq_o).cuda(),
                                tile=tile)
        assert np.array_equal(host(acc), acc_o), (tile, M, N, K)


def test_acc_unaligned_pointers_generic_path():
    M, N, K = 40, 50, 256
    xq_o, wq_o, acc_o = _acc_case(M, N, K, seed=77)
    xb = torch.zeros(M * K + 3, dtype=torch.int8, device="cuda")
    wb = torch.zeros(N * K + 5, dtype=torch.int8, device="cuda")
    xb[3:].copy_(torch.from_numpy(xq_o.ravel()))
    wb[5:].copy_(torch.from_numpy(wq_o.ravel()))
    acc = w8a8.gemm_acc_i32(xb[3:].view(M, K), wb[5:].view(N, K))
    assert np.array_equal(host(acc), acc_o)


def test_acc_extreme_values_at_max_k():
    """|acc| reaches 127^2 * K at K = 133144 without wrapping."""
    K = w8a8.MAX_K
    xq = torch.full((3, K), 127, dtype=torch.int8, device="cuda")
    xq[1] = -127
    wq = torch.full((5, K), 127, dtype=torch.int8, device="cuda")
    wq[2] = -127
    acc = host(w8a8.gemm_acc_i32(xq, wq))
    want = np.outer([127, -127, 127], [127, 127, -127, 127, 127]).astype(np.int64) * K
    assert np.array_equal(acc.astype(np.int64), want)


def test_acc_against_torch_int_mm():
    """The paper's own reference routine (a library int8 matmul), where ROCm has it."""
    M, N, K = 256, 384, 512
    xq_o, wq_o, acc_o = _acc_case(M, N, K, seed=5)
    xq, wq = torch.from_numpy(xq_o).cuda(), torch.from_numpy(wq_o).cuda()
    acc = host(w8a8.gemm_acc_i32(xq, wq))
    assert np.array_equal(acc, acc_o)
    try:
        ref = torch._int_mm(xq, wq.t().contiguous())
    except Exception as e:  # noqa: BLE001
        pytest.skip(f"torch._int_mm unavailable: {e}")
    assert np.array_equal(acc, host(ref))


# ---------------------------------------------------------------- bf16 output

LINEAR_SMALL = [(64, 256, 128, "outlier"), (257, 384, 391, "student_t"),
                (130, 3136, 260, "gelu"), (1, 4096, 130, "outlier"), (77, 264, 64, "outlier"),
                (45, 269, 77, "student_t"), (300, 512, 200, "outlier"),
                # few tokens on a long K: the fallback splits K in four inside w8a8_linear
                (40, 8192, 4096, "student_t"), (100, 8192, 3072, "outlier")]


@pytest.mark.parametrize("M,K,N,dist", LINEAR_SMALL)
def test_linear_full_compare_small(M, K, N, dist):
    say(f"linear small M={M} K={K} N={N} {dist}")
    x, w, b = si.make_inputs((M, K, N), seed=M + K + N, dist=dist)
    wq_o, sw_o = oracle.quantize_rows(w)
    y_o, xq_o, sx_o, acc_o = oracle.linear(x, wq_o, sw_o, b)
    wq, sw = w8a8.quantize_weight(dev_bf16(w))
    assert np.array_equal(host(wq), wq_o) and np.array_equal(host(sw), sw_o)
    y = w8a8.linear(dev_bf16(x), wq, sw, dev_bf16(b))
    st = assert_bf16_parity(host_bits(y), y_o, f"linear {M}x{K}x{N}")
    say("  ", st)
    # gemm on the oracle-checked quantized activations, every tile
    xq, sx = w8a8.quantize_act(dev_bf16(x))
    for t in range(w8a8.tile_count()):
        y2 = w8a8.gemm(xq, sx, wq, sw, dev_bf16(b), tile=t)
        assert np.array_equal(host_bits(y2), host_bits(y)), t
    # without bias
    y_nb = w8a8.gemm(xq, sx, wq, sw, None)
    assert_bf16_parity(host_bits(y_nb), oracle.epilogue(acc_o, sx_o, sw_o, None), "no bias")


def test_linear_k_zero_gives_bias():
    M, N = 9, 33
    _, _, b = si.make_inputs((1, 8, N), seed=1)
    x = torch.empty((M, 0), dtype=torch.bfloat16, device="cuda")
    wq = torch.empty((N, 0), dtype=torch.int8, device="cuda")
    sw = torch.zeros(N, dtype=torch.float32, device="cuda")
    y = w8a8.linear(x, wq, sw, dev_bf16(b))
    assert np.array_equal(host_bits(y), np.broadcast_to(b, (M, N)))


def test_empty_shapes():
    x = torch.empty((0, 64), dtype=torch.bfloat16, device="cuda")
    wq = torch.zeros((8, 64), dtype=torch.int8, device="cuda")
    sw = torch.ones(8, dtype=torch.float32, device="cuda")
    assert w8a8.linear(x, wq, sw).shape == (0, 8)
    q, s = w8a8.quantize_act(x)
    assert q.shape == (0, 64) and s.shape == (0,)


def test_zero_and_tiny_tokens_give_bias():
    """Token 0 is zero and token 1 has a ~ 4e-39 (127/a overflows): both are zero rows and
    give the bias exactly. Token 2 has a ~ 1e-36: a subnormal scale a/127, kept (not
    flushed) on both sides."""
    M, K, N = 40, 512, 96
    x, w, b = si.make_inputs((M, K, N), seed=21)
    x[0] = 0
    x[1] = si.bf16_bits_from_f32(oracle.bf16_to_f32(x[1]) * np.float32(1e-40))
    r2 = oracle.bf16_to_f32(x[2]).astype(np.float64)
    x[2] = si.bf16_bits_from_f32((r2 * (1e-36 / np.abs(r2).max())).astype(np.float32))
    wq_o, sw_o = oracle.quantize_rows(w)
    y_o, _, sx_o, _ = oracle.linear(x, wq_o, sw_o, b)
    assert sx_o[0] == 0 and sx_o[1] == 0
    assert 0 < sx_o[2] < np.finfo(np.float32).tiny
    wq, sw = w8a8.quantize_weight(dev_bf16(w))
    y = host_bits(w8a8.linear(dev_bf16(x), wq, sw, dev_bf16(b)))
    assert np.array_equal(y[0], b) and np.array_equal(y[1], b)
    assert_bf16_parity(y, y_o, "zero/tiny tokens")


def test_guard_bands_untouched():
    """Canary elements around the output and the quantized activations stay intact."""
    M, K, N = 131, 1040, 262
    x, w, b = si.make_inputs((M, K, N), seed=31)
    wq, sw = w8a8.quantize_weight(dev_bf16(w))
    pad = 4096
    ybuf = torch.full((M * N + 2 * pad,), 1.5, dtype=torch.bfloat16, device="cuda")
    y = ybuf[pad:pad + M * N].view(M, N)
    w8a8.linear(dev_bf16(x), wq, sw, dev_bf16(b), out=y)
    qbuf = torch.full((M * K + 2 * pad,), 99, dtype=torch.int8, device="cuda")
    sbuf = torch.full((M + 2 * pad,), -3.0, dtype=torch.float32, device="cuda")
    lib = w8a8.load_library()
    import ctypes
    st = lib.w8a8_quantize_act(ctypes.c_void_p(dev_bf16(x).data_ptr()), M, K,
                               ctypes.c_void_p(qbuf[pad:].data_ptr()),
                               ctypes.c_void_p(sbuf[pad:].data_ptr()),
                               ctypes.c_void_p(torch.cuda.current_stream().cuda_stream))
    torch.cuda.synchronize()
    assert st == 0
    yb = ybuf.float().cpu().numpy()
    assert np.all(yb[:pad] == 1.5) and np.all(yb[pad + M * N:] == 1.5)
    qb = host(qbuf)
    assert np.all(qb[:pad] == 99) and np.all(qb[pad + M * K:] == 99)
    sb = host(sbuf)
    assert np.all(sb[:pad] == -3.0) and np.all(sb[pad + M:] == -3.0)


def test_deterministic_and_stream_independent():
    shp = si.workload(1, "attn_proj")
    x, w, b = si.make_inputs(shp)
    xd, bd = dev_bf16(x), dev_bf16(b)
    wq, sw = w8a8.quantize_weight(dev_bf16(w))
    y0 = host_bits(w8a8.linear(xd, wq, sw, bd))
    for _ in range(5):
        assert np.array_equal(host_bits(w8a8.linear(xd, wq, sw, bd)), y0)
    s = torch.cuda.Stream()
    with torch.cuda.stream(s):
        y1 = w8a8.linear(xd, wq, sw, bd)
    s.synchronize()
    assert np.array_equal(host_bits(y1), y0)


# ---------------------------------------------------------------- HIP graphs

@pytest.mark.parametrize("act,with_cm", [("none", False), ("gelu", True)])
def test_graph_replays_match_eager(act, with_cm):
    """The entry points allocate nothing and record no memset, so a captured linear
    replays correctly: several replays, with eager work and synchronizations between
    them, each equal bit for bit to the eager result."""
    M, K, N = 2560, 4096, 4096
    x, w, b = si.make_inputs((M, K, N), seed=20360)
    xd, bd = dev_bf16(x), dev_bf16(b)
    wq, sw = w8a8.quantize_weight(dev_bf16(w))
    cm = torch.rand(K, device="cuda") + 0.5 if with_cm else None
    y = torch.empty((M, N), dtype=torch.bfloat16, device="cuda")
    ws = torch.empty(w8a8.linear_workspace_bytes(M, N, K), dtype=torch.uint8, device="cuda")
    want = host_bits(w8a8.linear(xd, wq, sw, bd, act=act, col_mul=cm))
    g = torch.cuda.CUDAGraph()
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        with torch.cuda.graph(g, stream=s):
            w8a8.linear(xd, wq, sw, bd, act=act, col_mul=cm, out=y, workspace=ws)
    torch.cuda.current_stream().wait_stream(s)
    other = torch.empty_like(y)
    for r in range(4):
        y.zero_()
        ws.fill_(0x5A)
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        assert np.array_equal(host_bits(y), want), f"replay {r}"
        # eager work between replays, through the same workspace
        w8a8.linear(xd[: M // 2], wq, sw, None, out=other[: M // 2], workspace=ws)
        torch.cuda.synchronize()


# ---------------------------------------------------------------- split-K tiles

SPLIT_SHAPES = [(333, 512, 4096), (77, 520, 3136), (300, 391, 4112), (64, 256, 256),
                (129, 384, 128)]


@pytest.mark.parametrize("M,N,K", SPLIT_SHAPES)
def test_split_k_tiles_exact(M, N, K):
    """Every split-K tile through w8a8_gemm_ex: the int32 partials of the K-ranges are
    summed in a second kernel, so the bf16 output equals the oracle's bit for bit
    (several splits, a ragged last panel, K short enough for one or two splits, N not a
    multiple of 4 for the scalar reduction)."""
    x, w, b = si.make_inputs((M, K, N), seed=900 + K)
    xq_o, sx_o = oracle.quantize_rows(x)
    wq_o, sw_o = oracle.quantize_rows(w)
    y_o = oracle.epilogue(oracle.gemm_acc(xq_o, wq_o), sx_o, sw_o, b)
    xq, sx = w8a8.quantize_act(dev_bf16(x))
    wq, sw = w8a8.quantize_weight(dev_bf16(w))
    bd = dev_bf16(b)
    split_ids = [t for t in range(w8a8.tile_count()) if "_k" in w8a8.tile_name(t)]
    assert split_ids
    for t in split_ids:
        y = host_bits(w8a8.gemm(xq, sx, wq, sw, bd, tile=t))
        assert np.array_equal(y, y_o), w8a8.tile_name(t)
        acc = host(w8a8.gemm_acc_i32(xq, wq, tile=t))   # runs unsplit
        assert np.array_equal(acc, oracle.gemm_acc(xq_o, wq_o)), w8a8.tile_name(t)


# ---------------------------------------------------------------- measurement aid

def _ceiling_checksums(xq, wq, iters):
    """Per-wavefront sum of accumulators of the ceiling kernel, from its definition:
    iters * sum over K-steps s and k < 32 of (sum of the wavefront's 64 weight rows at
    k_s + k) * (sum of its 160 token rows at k_s + k), modulo 2^32."""
    M, K = xq.shape
    N = wq.shape[0]
    x64, w64 = xq.astype(np.int64), wq.astype(np.int64)
    out = np.zeros(1024, dtype=np.int64)
    for b in range(256):
        tm, tn = b // 16, b % 16
        ks = [((b * 8 + s) % (K // 32)) * 32 for s in range(8)]
        rows_m = [(tm * 160 + r) % M for r in range(160)]
        colx = x64[rows_m].sum(axis=0)
        for w in range(4):
            rows_n = [(tn * 256 + w * 64 + r) % N for r in range(64)]
            colw = w64[rows_n].sum(axis=0)
            tot = sum(int((colw[k:k + 32] * colx[k:k + 32]).sum()) for k in ks)
            out[b * 4 + w] = (iters * tot) % (1 << 32)
    return out


@pytest.mark.parametrize("M,N,K", [(2560, 4096, 4096), (77, 130, 96)])
def test_mfma_ceiling_checksums(M, N, K):
    """The matrix-core ceiling probe computes what it claims: its per-wavefront
    accumulator sums equal the closed form on the same codes (so the timed MFMAs are
    real work on the given operands)."""
    say(f"mfma ceiling M={M} N={N} K={K}")
    rng = np.random.default_rng(M + N + K)
    xq = rng.integers(-127, 128, size=(M, K), dtype=np.int8)
    wq = rng.integers(-127, 128, size=(N, K), dtype=np.int8)
    base = _ceiling_checksums(xq, wq, 1)
    for iters in (1, 3):
        sums = w8a8.mfma_ceiling(torch.from_numpy(xq).cuda(), torch.from_numpy(wq).cuda(), iters)
        got = host(sums).astype(np.int64) % (1 << 32)
        assert np.array_equal(got, (iters * base) % (1 << 32)), iters


@pytest.mark.parametrize("nbytes", [16 * 2048, 16 * 2048 * 37, 4096 * 4096])
def test_read_ceiling_checksums(nbytes):
    """The read-ceiling probe reads every byte it is given: workgroup b's checksum is the
    XOR of the 32-bit words of the b-th contiguous chunk."""
    say(f"read ceiling {nbytes} bytes")
    rng = np.random.default_rng(nbytes)
    words = rng.integers(0, 1 << 32, size=nbytes // 4, dtype=np.uint64).astype(np.uint32)
    sums = host(w8a8.read_ceiling(torch.from_numpy(words.view(np.int32)).cuda()))
    want = np.bitwise_xor.reduce(words.reshape(w8a8.READ_BLOCKS, -1), axis=1)
    assert np.array_equal(sums.view(np.uint32), want)


# ---------------------------------------------------------------- small fused linear

# (M, K, N, fused): few tokens whose tile streams the weight run quantizer and GEMM in
# one launch (the workspace stays untouched); the rest keep the two-launch path: a tile
# that does not stream the weight (M = 77, 2560; M = 4, N = 16384), a token block over
# the LDS budget (64 x 4112 on the register-staged streaming tiles), more than 7
# vectors per lane to quantize there (M = 64, K = 4096), more bf16 token bytes than
# weight bytes per workgroup on the token-block-in-LDS tiles (13 or 16 tokens on 16
# channels), K % 16 != 0 (264). Up to 8 tokens the token block sits in LDS: one row
# quantized by 8, 4 or 2 wavefronts (M = 1, 2, 3), one per wavefront (7, 8), with K
# tails (528, 3088) and ragged channel blocks (300, 520).
SMALL_FUSED = [(64, 256, 128, True), (1, 4096, 4096, True), (1, 4096, 16384, True),
               (1, 3136, 4096, True), (5, 1024, 520, True), (16, 2048, 4096, False),
               (4, 4096, 16384, False), (8, 3088, 80, True), (13, 3088, 80, False),
               (64, 4112, 80, False), (77, 3136, 4096, False),
               (2560, 256, 64, False), (3, 264, 64, False), (2, 16, 40, True),
               (3, 528, 300, True), (7, 4096, 64, True), (16, 1024, 48, False),
               (64, 4096, 128, False), (1, 16384, 4096, True),
               # codes + scales fit 48 KB, yet not one launch (they once overflowed LDS
               # beside a 128 KB reduction array)
               (64, 512, 4096, False), (48, 768, 4096, False),
               # the swept few-token rules: register-staged streaming tile, token block in
               # LDS over several token blocks
               (32, 512, 4096, True), (24, 4096, 4096, False), (100, 1024, 520, True),
               (80, 512, 2048, True), (128, 3136, 520, False)]


@pytest.mark.parametrize("M,K,N,fused", SMALL_FUSED)
def test_small_fused_linear(M, K, N, fused):
    """The one-launch linear for few tokens gives the two-launch path's bits (codes,
    scales and accumulator exact, so the same bf16 output) and the oracle's."""
    say(f"small fused linear M={M} K={K} N={N} fused={fused}")
    x, w, b = si.make_inputs((M, K, N), seed=3 * M + K + N, dist="student_t")
    wq_o, sw_o = oracle.quantize_rows(w)
    y_o, _, _, _ = oracle.linear(x, wq_o, sw_o, b)
    xd, bd = dev_bf16(x), dev_bf16(b)
    wq, sw = w8a8.quantize_weight(dev_bf16(w))
    nws = w8a8.linear_workspace_bytes(M, N, K)
    ws = torch.full((nws,), 0x5A, dtype=torch.uint8, device="cuda")
    y = w8a8.linear(xd, wq, sw, bd, workspace=ws)
    torch.cuda.synchronize()
    untouched = bool((ws == 0x5A).all().item())
    assert untouched == fused, (M, K, N, untouched)
    assert w8a8.linear_one_launch(M, N, K) == fused
    xq, sx = w8a8.quantize_act(xd)
    y2 = w8a8.gemm(xq, sx, wq, sw, bd)
    assert np.array_equal(host_bits(y), host_bits(y2))
    assert_bf16_parity(host_bits(y), y_o, f"small fused {M}x{K}x{N}")
    # the same without bias
    y3 = w8a8.linear(xd, wq, sw, None)
    y4 = w8a8.gemm(xq, sx, wq, sw, None)
    assert np.array_equal(host_bits(y3), host_bits(y4))


def test_small_fused_linear_zero_and_tiny_rows():
    """Zero and tiny token rows in the fused path: codes and scales 0, so y = bias."""
    M, K, N = 4, 512, 256
    x, w, b = si.make_inputs((M, K, N), seed=11)
    x = x.copy()
    x[0] = 0                                  # a zero row
    x[1] = 0x0080                             # tiny positive values (bf16 1.2e-38): 127/a overflows
    wq, sw = w8a8.quantize_weight(dev_bf16(w))
    y = w8a8.linear(dev_bf16(x), wq, sw, dev_bf16(b))
    wq_o, sw_o = oracle.quantize_rows(w)
    y_o, _, sx_o, _ = oracle.linear(x, wq_o, sw_o, b)
    assert sx_o[0] == 0 and sx_o[1] == 0
    assert np.array_equal(host_bits(y)[:2], np.stack([b, b]))
    assert_bf16_parity(host_bits(y), y_o, "fused zero/tiny rows")


# ---------------------------------------------------------------- seeded random shapes

def _random_shapes(n=24, seed=20261202):
    """Shapes across the default tile rules: few tokens (the token-block and streaming
    kernels, the deep-ring tiles, split-K on long K), a few hundred and more tokens
    (the cost model), aligned and unaligned K. A fixed seed: the same shapes every run."""
    rng = np.random.default_rng(seed)
    out = []
    for i in range(n):
        M = int(rng.choice([1, 2, 5, 13, 16, 17, 31, 40, 64, 77, 100, 128, 129, 200, 333, 517]))
        N = int(rng.integers(1, 5200)) if i % 3 else int(rng.choice([1024, 2048, 4096, 8192]))
        K = int(rng.choice([16, 48, 272, 1040, 2048, 3136, 4096, 8192]))
        if i % 5 == 4:
            K += 8                                       # K % 16 != 0: the generic path
        while M * N * K > 1_500_000_000:
            N = max(1, N // 2)
        out.append((M, K, N))
    return out


@pytest.mark.parametrize("M,K,N", _random_shapes())
def test_random_shapes_against_oracle(M, K, N):
    """w8a8_linear on the default tile of each shape against the oracle's linear: codes
    and scales exact, the int32 accumulator exact through the debug path, the bf16
    output within the bf16 gate."""
    say(f"random shape M={M} K={K} N={N} tile={w8a8.tile_name(w8a8.select_tile(M, N, K))}")
    x, w, b = si.make_inputs((M, K, N), seed=M * 31 + K * 7 + N, dist="student_t")
    wq_o, sw_o = oracle.quantize_rows(w)
    y_o, xq_o, sx_o, acc_o = oracle.linear(x, wq_o, sw_o, b)
    wq, sw = w8a8.quantize_weight(dev_bf16(w))
    assert np.array_equal(host(wq), wq_o) and np.array_equal(host(sw), sw_o)
    y = w8a8.linear(dev_bf16(x), wq, sw, dev_bf16(b))
    assert_bf16_parity(host_bits(y), y_o, f"random {M}x{K}x{N}")
    xq, sx = w8a8.quantize_act(dev_bf16(x))
    assert np.array_equal(host(xq), xq_o) and np.array_equal(host(sx), sx_o)
    acc = w8a8.gemm_acc_i32(xq, wq)
    assert np.array_equal(host(acc), acc_o)


EXTREME_SHAPES = [(1, 4096, 40000), (65536, 64, 40), (3, 133136, 8), (2, 133136, 300),
                  (70000, 16, 1)]


@pytest.mark.parametrize("M,K,N", EXTREME_SHAPES)
def test_extreme_aspect_shapes_against_oracle(M, K, N):
    """A wide weight at one token (2500 workgroups), many tokens on a tiny weight, K near
    its maximum on tiny M and N: every output against the oracle's linear."""
    say(f"extreme shape M={M} K={K} N={N} tile={w8a8.tile_name(w8a8.select_tile(M, N, K))}")
    x, w, b = si.make_inputs((M, K, N), seed=M + 3 * K + 7 * N, dist="outlier")
    wq_o, sw_o = oracle.quantize_rows(w)
    y_o, xq_o, sx_o, acc_o = oracle.linear(x, wq_o, sw_o, b)
    wq, sw = w8a8.quantize_weight(dev_bf16(w))
    assert np.array_equal(host(wq), wq_o) and np.array_equal(host(sw), sw_o)
    y = w8a8.linear(dev_bf16(x), wq, sw, dev_bf16(b))
    assert_bf16_parity(host_bits(y), y_o, f"extreme {M}x{K}x{N}")
    xq, sx = w8a8.quantize_act(dev_bf16(x))
    assert np.array_equal(host(w8a8.gemm_acc_i32(xq, wq)), acc_o)
