"""The C ABI without a GPU: the library loads, exports every function include/w8a8.h
declares, and rejects bad arguments before anything is launched."""
import ctypes
import os
import re

import pytest

import paper_2606_14598_amd as w8a8

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "w8a8.h")

OK, ERR_NULL, ERR_SHAPE, ERR_K, ERR_HIP, ERR_WS, ERR_ARG = range(7)


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    names = re.findall(r"\b(w8a8_[a-z0-9_]+)\s*\(", text)
    return sorted(set(names))


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(w8a8.library_path()):
        pytest.fail("libw8a8.so is not built (run python -m paper_2606_14598_amd.build)")
    return w8a8.load_library()


def test_header_declares_the_entry_points():
    names = declared_functions()
    for must in ("w8a8_quantize_weight", "w8a8_quantize_act", "w8a8_gemm", "w8a8_linear",
                 "w8a8_gemm_acc_i32"):
        assert must in names


def test_every_declared_symbol_is_exported(lib):
    raw = ctypes.CDLL(w8a8.library_path())
    for name in declared_functions():
        assert hasattr(raw, name), f"{name} not exported"


def test_no_internal_symbols_exported():
    import subprocess
    out = subprocess.run(["nm", "-D", "--defined-only", w8a8.library_path()],
                         capture_output=True, text=True, check=True).stdout
    funcs = [l.split()[-1] for l in out.splitlines() if " T " in l]
    assert funcs and all(f.startswith("w8a8_") for f in funcs), funcs


def test_status_strings(lib):
    for st in range(8):
        assert lib.w8a8_status_string(st)
    assert lib.w8a8_status_string(99) == b"unknown status"


def test_validation_before_launch(lib):
    P = ctypes.c_void_p
    fake = P(256)  # never dereferenced: validation fails first
    # negative sizes
    assert lib.w8a8_gemm(fake, fake, fake, fake, None, fake, -1, 8, 8, None, 0, None) == ERR_SHAPE
    assert lib.w8a8_quantize_act(fake, 4, -3, fake, fake, None) == ERR_SHAPE
    assert lib.w8a8_linear(fake, fake, fake, None, fake, 4, -8, 8, fake, 1 << 20, None) == ERR_SHAPE
    # K too large for an int32 accumulator
    assert lib.w8a8_gemm_acc_i32(fake, fake, fake, 4, 4, w8a8.MAX_K + 1, None) == ERR_K
    assert lib.w8a8_gemm(fake, fake, fake, fake, None, fake, 4, 4, w8a8.MAX_K + 1, None, 0,
                         None) == ERR_K
    # NULL pointers
    assert lib.w8a8_gemm(None, fake, fake, fake, None, fake, 4, 4, 16, None, 0, None) == ERR_NULL
    assert lib.w8a8_gemm(fake, None, fake, fake, None, fake, 4, 4, 16, None, 0, None) == ERR_NULL
    assert lib.w8a8_gemm(fake, fake, fake, fake, None, None, 4, 4, 16, None, 0, None) == ERR_NULL
    assert lib.w8a8_quantize_weight(fake, 4, 16, None, fake, None) == ERR_NULL
    assert lib.w8a8_quantize_weight(fake, 4, 16, fake, None, None) == ERR_NULL
    assert lib.w8a8_gemm_acc_i32(fake, fake, None, 4, 4, 16, None) == ERR_NULL
    # workspace
    assert lib.w8a8_linear(fake, fake, fake, None, fake, 4, 8, 16, None, 0, None) == ERR_WS
    need = lib.w8a8_linear_workspace_bytes(4, 8, 16)
    assert lib.w8a8_linear(fake, fake, fake, None, fake, 4, 8, 16, fake, need - 1, None) == ERR_WS
    assert lib.w8a8_linear(fake, fake, fake, None, fake, 4, 8, 16, P(256 + 8), need, None) == ERR_WS
    # unknown tile
    n = lib.w8a8_tile_count()
    assert lib.w8a8_gemm_ex(fake, fake, fake, fake, None, fake, 4, 4, 16, None, 0, n,
                            None) == ERR_ARG
    assert lib.w8a8_gemm_acc_i32_ex(fake, fake, fake, 4, 4, 16, -2, None) == ERR_ARG


def test_empty_is_a_no_op(lib):
    # M == 0 or N == 0: valid and nothing is launched (works without a GPU)
    assert lib.w8a8_gemm(None, None, None, None, None, None, 0, 8, 16, None, 0, None) == OK
    assert lib.w8a8_gemm(None, None, None, None, None, None, 8, 0, 16, None, 0, None) == OK
    assert lib.w8a8_gemm_acc_i32(None, None, None, 0, 0, 0, None) == OK
    assert lib.w8a8_linear(None, None, None, None, None, 0, 8, 16, None, 0, None) == OK
    assert lib.w8a8_quantize_act(None, 0, 16, None, None, None) == OK


def test_tile_table_host_logic(lib):
    n = lib.w8a8_tile_count()
    assert n >= 4
    names = [lib.w8a8_tile_name(i).decode() for i in range(n)]
    assert len(set(names)) == n
    assert lib.w8a8_tile_name(n) is None
    for M, N, K in [(1, 4096, 4096), (77, 16384, 4096), (2560, 4096, 4096),
                    (4608, 12288, 4096), (4625, 4096, 3136), (64, 128, 256)]:
        t = lib.w8a8_select_tile(M, N, K)
        assert 0 <= t < n
    assert lib.w8a8_select_tile(0, 8, 8) == -1


def test_workspace_queries(lib):
    M, N, K = 2560, 4096, 4096
    need = lib.w8a8_linear_workspace_bytes(M, N, K)
    assert need >= M * K + 4 * M
    assert need % 256 == 0 or lib.w8a8_gemm_workspace_bytes(M, N, K) % 256 != 0
    assert lib.w8a8_linear_workspace_bytes(0, N, K) == 0


def test_python_binding_rejects_cpu_tensors():
    import torch
    x = torch.zeros(4, 16, dtype=torch.bfloat16)
    with pytest.raises(ValueError):
        w8a8.quantize_act(x)
    with pytest.raises(TypeError):
        w8a8.quantize_act(x.float())


def test_transform_and_smoothing_validation(lib):
    P = ctypes.c_void_p
    fake = P(256)
    # unknown activation transform
    assert lib.w8a8_quantize_act_ex(fake, 4, 16, 2, None, fake, fake, None) == ERR_ARG
    assert lib.w8a8_quantize_act_ex(fake, 4, 16, -1, None, fake, fake, None) == ERR_ARG
    assert lib.w8a8_linear_ex(fake, 7, None, fake, fake, None, fake, 4, 8, 16, fake, 1 << 20,
                              None) == ERR_ARG
    assert lib.w8a8_col_absmax(fake, 4, 16, 3, fake, 0, None) == ERR_ARG
    # shapes and pointers
    assert lib.w8a8_quantize_act_ex(fake, -4, 16, 1, None, fake, fake, None) == ERR_SHAPE
    assert lib.w8a8_quantize_weight_ex(fake, 4, 16, fake, None, fake, None) == ERR_NULL
    assert lib.w8a8_col_absmax(fake, -1, 16, 0, fake, 0, None) == ERR_SHAPE
    assert lib.w8a8_col_absmax(fake, 4, 16, 0, None, 0, None) == ERR_NULL
    assert lib.w8a8_col_absmax(None, 4, 16, 0, fake, 0, None) == ERR_NULL
    # alpha must lie in [0, 1]
    for alpha in (-0.1, 1.5, float("nan")):
        assert lib.w8a8_smooth_factors(fake, fake, 16, alpha, fake, fake, None) == ERR_ARG
    assert lib.w8a8_smooth_factors(fake, None, 16, 0.5, fake, fake, None) == ERR_NULL
    assert lib.w8a8_smooth_factors(fake, fake, -1, 0.5, fake, fake, None) == ERR_SHAPE
    # empty problems are no-ops
    assert lib.w8a8_smooth_factors(None, None, 0, 0.5, None, None, None) == OK
    assert lib.w8a8_col_absmax(None, 0, 0, 1, None, 0, None) == OK
    assert lib.w8a8_quantize_act_ex(None, 0, 16, 1, None, None, None, None) == OK
    assert lib.w8a8_linear_ex(None, 1, None, None, None, None, None, 0, 8, 16, None, 0,
                              None) == OK


def test_python_binding_checks_transform_arguments():
    import torch
    x = torch.zeros(4, 16, dtype=torch.bfloat16)
    with pytest.raises(ValueError):
        w8a8.quantize_act(x, act="relu")
    with pytest.raises(ValueError):
        w8a8.col_absmax(x, accumulate=True)


def _table_costs():
    path = os.path.join(ROOT, "paper_2606_14598_amd", "csrc", "tile_table.inc")
    text = open(path).read()
    body = text[text.index("kTileCost[] = {"):]
    body = body[:body.index("};")]
    return [(float(c), float(d)) for c, d in re.findall(r"\{([-0-9.e+]+), ([-0-9.e+]+)\}", body)]


def test_default_tile_follows_the_wave_cost_model(lib):
    costs = _table_costs()
    n = lib.w8a8_tile_count()
    assert len(costs) == n
    dims = []
    for i in range(n):
        m = re.match(r"m(\d+)n(\d+)", lib.w8a8_tile_name(i).decode())
        dims.append((int(m.group(1)), int(m.group(2))) if m else None)
    for M, N, K in [(129, 4096, 4096), (333, 16384, 4096), (512, 4608, 4608),
                    (2560, 4096, 4096), (4110, 13824, 4608), (5000, 7000, 4096),
                    (16384, 4608, 53248), (300, 5000, 2048)]:
        best, cost = None, None
        for i in range(n):
            c, d = costs[i]
            if d <= 0:
                continue
            tm, tn = dims[i]
            rounds = -(-(-(-M // tm) * -(-N // tn)) // 256)
            est = rounds * (c + d * K * tm * tn * 1e-9)
            if cost is None or est < cost:
                best, cost = i, est
        assert lib.w8a8_default_tile(M, N, K) == best, (M, N, K)
    # few tokens: the swept rules (M, N, K) -> tile
    rules = {(1, 128, 4096): "wsx_m16n16w8d4", (16, 4096, 4096): "wsx_m16n16w8d4",
             (8, 16384, 4096): "m64n64k128w2x2s8", (1, 16384, 4096): "wsx_m16n16w8d4",
             (64, 128, 4096): "wsx_m16n16w8d4", (128, 2048, 4096): "wsx_m16n32w8d4",
             (40, 4096, 16384): "m32n128k128w1x4s6_k4", (100, 4096, 8192): "m64n128k128w1x4s6_k4",
             (40, 16384, 4096): "m32n128k128w1x4s6", (128, 8192, 4096): "m64n128k128w1x4s6",
             (17, 4096, 4096): "skinny_m32n16w16", (32, 3072, 1024): "skinny_m32n16w16",
             (33, 4096, 4096): "wsx_m32n32w8d2", (64, 4096, 1024): "wsx_m32n32w8d2",
             (65, 4096, 4096): "m64n64k128w2x2s8", (128, 4096, 2048): "m64n64k128w2x2s8"}
    for (M, N, K), want in rules.items():
        assert lib.w8a8_tile_name(lib.w8a8_default_tile(M, N, K)).decode() == want, (M, N, K)
    assert lib.w8a8_default_tile(0, 8, 8) == -1


def test_mfma_ceiling_validation(lib):
    P = ctypes.c_void_p
    fake = P(256)  # never dereferenced: validation fails first
    assert lib.w8a8_mfma_ceiling(None, fake, 4, 4, 64, 1, fake, None) == ERR_NULL
    assert lib.w8a8_mfma_ceiling(fake, fake, 4, 4, 64, 1, None, None) == ERR_NULL
    assert lib.w8a8_mfma_ceiling(fake, fake, 4, 4, 48, 1, fake, None) == ERR_SHAPE   # K % 32
    assert lib.w8a8_mfma_ceiling(fake, fake, 0, 4, 64, 1, fake, None) == ERR_SHAPE
    assert lib.w8a8_mfma_ceiling(fake, fake, 4, 4, 64, 0, fake, None) == ERR_ARG
    assert lib.w8a8_mfma_ceiling(P(264), fake, 4, 4, 64, 1, fake, None) == ERR_ARG  # alignment
    # ops of one launch: 256 workgroups x 4 wavefronts x 8 K-steps x 10 MFMAs x 65536 ops
    assert lib.w8a8_mfma_ceiling_ops(3) == 256 * 4 * 3 * 8 * 10 * 65536
    assert lib.w8a8_mfma_ceiling_ops(0) == -1


def test_read_ceiling_validation(lib):
    P = ctypes.c_void_p
    fake = P(256)  # never dereferenced: validation fails first
    unit = 16 * 2048
    assert lib.w8a8_read_ceiling(None, unit, fake, None) == ERR_NULL
    assert lib.w8a8_read_ceiling(fake, unit, None, None) == ERR_NULL
    assert lib.w8a8_read_ceiling(fake, 0, fake, None) == ERR_SHAPE
    assert lib.w8a8_read_ceiling(fake, unit + 16, fake, None) == ERR_SHAPE
    assert lib.w8a8_read_ceiling(P(264), unit, fake, None) == ERR_ARG
    assert lib.w8a8_read_ceiling(fake, unit, P(258), None) == ERR_ARG


def _skinny_static_lds(name: str) -> int:
    """Static LDS of a weight-streaming tile, from its name skinny_m<M>n<C>w<NW>: the
    cross-wavefront reduction array holds NW x (C/16) x (M/16) x 64 lanes x 16 bytes."""
    m = re.match(r"skinny_m(\d+)n(\d+)w(\d+)$", name)
    assert m, name
    tm, tn, nw = (int(g) for g in m.groups())
    return nw * (tn // 16) * (tm // 16) * 64 * 16


def _wsx_lds(name: str, rows: int, K: int) -> int:
    """LDS of the one-launch linear on a token-block-in-LDS tile wsx_m<M>n<C>w<NW>d<D>:
    M/16 x 16 scales and NW maxima (4 bytes each) rounded up to 256 bytes, then the
    larger of (code rows of ceil(K / 1024) KiB + 16 bytes and bf16 rows of
    ceil(2K / 1024) KiB) and the reduction array of NW x (C/16) x (M/16) x 1 KiB, which
    reuses the rows' space once the main loop is done."""
    m = re.match(r"wsx_m(\d+)n(\d+)w(\d+)d(\d+)$", name)
    assert m, name
    tm, tn, nw, _ = (int(g) for g in m.groups())
    rows_bytes = rows * (-(-K // 1024) * 1024 + 16) + rows * (-(-2 * K // 1024) * 1024)
    head = -(-(4 * tm + 4 * nw) // 256) * 256
    return head + max(rows_bytes, nw * (tn // 16) * (tm // 16) * 1024)


def test_one_launch_linear_fits_the_workgroup_lds(lib):
    """Wherever w8a8_linear takes the one-launch path, the tile's LDS fits gfx950's
    160 KiB: on the register-staged streaming tiles the token block's codes (rows of
    K + 16 bytes) and scales plus the static reduction array; on the tiles that keep
    the token block in LDS, the whole layout of bf16 rows, codes and reduction array."""
    budget = 160 * 1024
    seen = {"skinny": 0, "wsx": 0}
    for M in list(range(1, 129)):
        for K in (16, 256, 512, 768, 1024, 2048, 3136, 4096, 8192, 16384):
            for N in (64, 520, 4096, 16384):
                if not lib.w8a8_linear_one_launch(M, N, K):
                    continue
                name = lib.w8a8_tile_name(lib.w8a8_select_tile(M, N, K)).decode()
                if name.startswith("wsx"):
                    seen["wsx"] += 1
                    tm = int(re.match(r"wsx_m(\d+)", name).group(1))
                    assert _wsx_lds(name, min(M, tm), K) <= budget, (M, N, K, name)
                    continue
                seen["skinny"] += 1
                tm = int(re.match(r"skinny_m(\d+)", name).group(1))
                rows = min(M, tm)
                dyn = rows * (K + 16) + rows * 4
                assert dyn <= 48 * 1024, (M, N, K, name)
                assert dyn + _skinny_static_lds(name) <= budget, (M, N, K, name)
    assert seen["skinny"] > 50 and seen["wsx"] > 50, seen
    # a token block too large for LDS does not take the one-launch path
    assert not lib.w8a8_linear_one_launch(16, 64, 16384)
    assert lib.w8a8_linear_one_launch(1, 4096, 16384)
    # shapes that once passed the dynamic check alone but overflow the total
    assert not lib.w8a8_linear_one_launch(64, 4096, 512)
    assert not lib.w8a8_linear_one_launch(48, 4096, 768)
    # and shapes that do take the path
    assert lib.w8a8_linear_one_launch(64, 128, 256)
    assert lib.w8a8_linear_one_launch(1, 4096, 3136)
    assert not lib.w8a8_linear_one_launch(0, 4096, 3136)
    assert not lib.w8a8_linear_one_launch(16, 4096, 264)     # K % 16 != 0


def test_python_binding_checks_out_and_workspace():
    """A caller's out tensor must have the dtype, shape and device the kernels write: an
    undersized or mistyped out is rejected before any launch (fake tensors stand in for
    device memory, so this runs without a GPU)."""
    import torch
    from torch._subclasses.fake_tensor import FakeTensorMode
    with FakeTensorMode():
        M, K, N = 33, 256, 64
        x = torch.empty(M, K, dtype=torch.bfloat16, device="cuda")
        wq = torch.empty(N, K, dtype=torch.int8, device="cuda")
        sw = torch.empty(N, dtype=torch.float32, device="cuda")
        xq = torch.empty(M, K, dtype=torch.int8, device="cuda")
        sx = torch.empty(M, dtype=torch.float32, device="cuda")
        bad_outs = [torch.empty(M, N - 1, dtype=torch.bfloat16, device="cuda"),
                    torch.empty(M - 1, N, dtype=torch.bfloat16, device="cuda"),
                    torch.empty(M * N, dtype=torch.bfloat16, device="cuda"),
                    torch.empty(M, N, dtype=torch.float32, device="cuda"),
                    torch.empty(N, M, dtype=torch.bfloat16, device="cuda").t(),
                    torch.empty(M, N, dtype=torch.bfloat16, device="cpu")]
        for out in bad_outs:
            with pytest.raises((ValueError, TypeError)):
                w8a8.linear(x, wq, sw, out=out)
            with pytest.raises((ValueError, TypeError)):
                w8a8.gemm(xq, sx, wq, sw, out=out)
        for out in (torch.empty(M, N - 1, dtype=torch.int32, device="cuda"),
                    torch.empty(M, N, dtype=torch.bfloat16, device="cuda")):
            with pytest.raises((ValueError, TypeError)):
                w8a8.gemm_acc_i32(xq, wq, out=out)
        need = w8a8.linear_workspace_bytes(M, N, K)
        with pytest.raises(ValueError):
            w8a8.linear(x, wq, sw, workspace=torch.empty(need - 1, dtype=torch.uint8,
                                                          device="cuda"))
        with pytest.raises(ValueError):
            w8a8.linear(x, wq, sw, workspace=torch.empty(need, dtype=torch.uint8))


def test_noalloc_validation_before_any_device_call(lib):
    """w8a8_linear_noalloc validates like w8a8_linear_ex and rejects problems beyond its
    128 MiB scratch before it looks up the device array (so this runs without a GPU)."""
    P = ctypes.c_void_p
    fake = P(256)
    f = lib.w8a8_linear_noalloc
    f.argtypes = [P, ctypes.c_int, P, P, P, P, P, ctypes.c_int64, ctypes.c_int64,
                  ctypes.c_int64, P]
    f.restype = ctypes.c_int
    assert f(fake, 0, None, fake, fake, None, fake, 8192, 64, 16384, None) == 7
    assert lib.w8a8_status_string(7)
    assert f(fake, 5, None, fake, fake, None, fake, 4, 8, 16, None) == ERR_ARG
    assert f(fake, 0, None, fake, fake, None, fake, -4, 8, 16, None) == ERR_SHAPE
    assert f(fake, 0, None, fake, fake, None, fake, 4, 8, w8a8.MAX_K + 1, None) == ERR_K
    assert f(fake, 0, None, fake, None, None, fake, 4, 8, 16, None) == ERR_NULL
    assert f(None, 0, None, None, None, None, None, 0, 8, 16, None) == OK
