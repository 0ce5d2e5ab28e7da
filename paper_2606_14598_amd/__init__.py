"""Fused W8A8 quantized linear for MI355X (gfx950): Python binding of libw8a8.so.

The arithmetic all runs in the library's HIP kernels; this module only checks
arguments, allocates outputs with torch and passes raw device pointers and torch's
current HIP stream through ctypes. Entry points mirror the C ABI in include/w8a8.h:

  quantize_weight(w)                 -> (wq int8 [N,K], w_scale fp32 [N])
  quantize_act(x)                    -> (xq int8 [M,K], x_scale fp32 [M])
  gemm(xq, x_scale, wq, w_scale, b)  -> y bf16 [M,N]
  linear(x, wq, w_scale, b)          -> y bf16 [..., N]   (x [..., K])
  gemm_acc_i32(xq, wq)               -> acc int32 [M,N]   (debug, no epilogue)
  col_absmax(v, act=)                -> amax fp32 [K]     (calibration)
  smooth_factors(x_amax, w_amax)     -> (s, s_inv) fp32 [K] (SmoothQuant, alpha = 0.5)

quantize_act and linear take act="gelu" (quantize GELU(x), exact erf, instead of x) and
col_mul (a per-input-channel float32 multiplier: SmoothQuant's 1/s); quantize_weight
takes col_mul (SmoothQuant's s, folded into W before quantization).

The method is Section 3 of the paper ("The quantization recipe (reused)", "The fused
kernel"): per-channel int8 weights, per-token dynamic int8 activations, an int8 x int8
-> int32 product, and an epilogue that applies sx[m] * sw[n] and the bias off the
int32 accumulator. If the library is missing, every call raises: there is no fallback.
"""
from __future__ import annotations

import ctypes
import os

import torch

__all__ = ["quantize_weight", "quantize_act", "gemm", "linear", "gemm_acc_i32",
           "col_absmax", "smooth_factors", "ACTS",
           "tile_count", "tile_name", "select_tile", "default_tile", "gemm_workspace_bytes",
           "linear_workspace_bytes", "linear_one_launch", "library_path", "load_library", "W8A8Error",
           "MAX_K", "version", "mfma_ceiling", "mfma_ceiling_ops", "read_ceiling",
           "READ_BLOCKS"]

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libw8a8.so")
MAX_K = 133144

_lib = None


class W8A8Error(RuntimeError):
    def __init__(self, func: str, status: int, msg: str):
        super().__init__(f"{func} failed with status {status}: {msg}")
        self.status = status


def library_path() -> str:
    return LIB_PATH


def load_library():
    """Load libw8a8.so (built in-tree by paper_2606_14598_amd.build). Raises if absent."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise RuntimeError(
            f"{LIB_PATH} is missing: build it with `python -m paper_2606_14598_amd.build` "
            "(the W8A8 path has no fallback)")
    lib = ctypes.CDLL(LIB_PATH)
    P, I64, SZ, INT = ctypes.c_void_p, ctypes.c_int64, ctypes.c_size_t, ctypes.c_int
    sigs = {
        "w8a8_quantize_weight": ([P, I64, I64, P, P, P], INT),
        "w8a8_quantize_act": ([P, I64, I64, P, P, P], INT),
        "w8a8_quantize_weight_ex": ([P, I64, I64, P, P, P, P], INT),
        "w8a8_quantize_act_ex": ([P, I64, I64, INT, P, P, P, P], INT),
        "w8a8_linear_ex": ([P, INT, P, P, P, P, P, I64, I64, I64, P, SZ, P], INT),
        "w8a8_col_absmax": ([P, I64, I64, INT, P, INT, P], INT),
        "w8a8_smooth_factors": ([P, P, I64, ctypes.c_float, P, P, P], INT),
        "w8a8_gemm": ([P, P, P, P, P, P, I64, I64, I64, P, SZ, P], INT),
        "w8a8_gemm_ex": ([P, P, P, P, P, P, I64, I64, I64, P, SZ, INT, P], INT),
        "w8a8_gemm_workspace_bytes": ([I64, I64, I64], SZ),
        "w8a8_gemm_workspace_bytes_ex": ([I64, I64, I64, INT], SZ),
        "w8a8_linear": ([P, P, P, P, P, I64, I64, I64, P, SZ, P], INT),
        "w8a8_linear_workspace_bytes": ([I64, I64, I64], SZ),
        "w8a8_linear_one_launch": ([I64, I64, I64], INT),
        "w8a8_gemm_acc_i32": ([P, P, P, I64, I64, I64, P], INT),
        "w8a8_gemm_acc_i32_ex": ([P, P, P, I64, I64, I64, INT, P], INT),
        "w8a8_tile_count": ([], INT),
        "w8a8_tile_name": ([INT], ctypes.c_char_p),
        "w8a8_select_tile": ([I64, I64, I64], INT),
        "w8a8_default_tile": ([I64, I64, I64], INT),
        "w8a8_status_string": ([INT], ctypes.c_char_p),
        "w8a8_version": ([], ctypes.c_char_p),
        "w8a8_mfma_ceiling_ops": ([I64], I64),
        "w8a8_mfma_ceiling": ([P, P, I64, I64, I64, I64, P, P], INT),
        "w8a8_read_ceiling": ([P, I64, P, P], INT),
    }
    for name, (args, res) in sigs.items():
        f = getattr(lib, name)
        f.argtypes = args
        f.restype = res
    _lib = lib
    return lib


def _call(name: str, *args) -> None:
    lib = load_library()
    st = getattr(lib, name)(*args)
    if st != 0:
        raise W8A8Error(name, st, lib.w8a8_status_string(st).decode())


def _ptr(t: torch.Tensor | None):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _stream(device: torch.device):
    return ctypes.c_void_p(torch.cuda.current_stream(device).cuda_stream)


def _check(t: torch.Tensor, dtype: torch.dtype, ndim: int, name: str):
    if not isinstance(t, torch.Tensor):
        raise TypeError(f"{name} must be a torch.Tensor")
    if t.dtype != dtype:
        raise TypeError(f"{name} must be {dtype}, got {t.dtype}")
    if t.dim() != ndim:
        raise ValueError(f"{name} must be {ndim}-D, got shape {tuple(t.shape)}")
    if t.device.type != "cuda":
        raise ValueError(f"{name} must be on a HIP device, got {t.device}")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")


def _check_out(t, dtype: torch.dtype, shape: tuple, device, name: str = "out"):
    """A caller-provided output: the dtype, shape and device the kernels will write,
    contiguous (they write shape[0] * shape[1] elements from its first element)."""
    _check(t, dtype, len(shape), name)
    if tuple(t.shape) != tuple(shape):
        raise ValueError(f"{name} must have shape {tuple(shape)}, got {tuple(t.shape)}")
    if t.device != torch.device(device):
        raise ValueError(f"{name} is on {t.device}, expected {device}")


def _same_device(*ts):
    devs = {t.device for t in ts if t is not None}
    if len(devs) > 1:
        raise ValueError(f"tensors on different devices: {devs}")


def version() -> str:
    return load_library().w8a8_version().decode()


def tile_count() -> int:
    return int(load_library().w8a8_tile_count())


def tile_name(tile_id: int) -> str:
    r = load_library().w8a8_tile_name(tile_id)
    if r is None:
        raise ValueError(f"no tile {tile_id}")
    return r.decode()


def select_tile(M: int, N: int, K: int) -> int:
    return int(load_library().w8a8_select_tile(M, N, K))


def default_tile(M: int, N: int, K: int) -> int:
    """The fallback rule's tile for a shape, ignoring the offline table."""
    return int(load_library().w8a8_default_tile(M, N, K))


def gemm_workspace_bytes(M: int, N: int, K: int, tile: int = -1) -> int:
    return int(load_library().w8a8_gemm_workspace_bytes_ex(M, N, K, int(tile)))


def linear_workspace_bytes(M: int, N: int, K: int) -> int:
    return int(load_library().w8a8_linear_workspace_bytes(M, N, K))


def linear_one_launch(M: int, N: int, K: int) -> bool:
    """Whether linear() runs quantizer and GEMM as one launch for this shape (16-byte
    aligned x and wq): a host query, no device needed."""
    return bool(load_library().w8a8_linear_one_launch(M, N, K))


ACTS = {"none": 0, "gelu": 1}


def _act(act: str) -> int:
    if act not in ACTS:
        raise ValueError(f"act must be one of {sorted(ACTS)}, got {act!r}")
    return ACTS[act]


def _col_mul(col_mul, K: int, device):
    if col_mul is None:
        return None
    _check(col_mul, torch.float32, 1, "col_mul")
    if col_mul.shape[0] != K:
        raise ValueError(f"col_mul must have K={K} entries, got {col_mul.shape[0]}")
    if col_mul.device != torch.device(device):
        raise ValueError(f"col_mul is on {col_mul.device}, expected {device}")
    return col_mul


def quantize_weight(w: torch.Tensor, *, col_mul=None):
    """Per-output-channel int8 weights: w bf16 [N,K] -> (wq int8 [N,K], sw fp32 [N]).
    col_mul: optional fp32 [K] multiplier (the SmoothQuant factors s)."""
    _check(w, torch.bfloat16, 2, "w")
    N, K = w.shape
    cm = _col_mul(col_mul, K, w.device)
    q = torch.empty((N, K), dtype=torch.int8, device=w.device)
    s = torch.empty((N,), dtype=torch.float32, device=w.device)
    with torch.cuda.device(w.device):
        _call("w8a8_quantize_weight_ex", _ptr(w), N, K, _ptr(cm), _ptr(q), _ptr(s),
              _stream(w.device))
    return q, s


def quantize_act(x: torch.Tensor, *, act: str = "none", col_mul=None):
    """Per-token int8 activations: x bf16 [M,K] -> (xq int8 [M,K], sx fp32 [M]) of
    T(x) * col_mul (T = identity or GELU)."""
    a = _act(act)
    _check(x, torch.bfloat16, 2, "x")
    M, K = x.shape
    cm = _col_mul(col_mul, K, x.device)
    q = torch.empty((M, K), dtype=torch.int8, device=x.device)
    s = torch.empty((M,), dtype=torch.float32, device=x.device)
    with torch.cuda.device(x.device):
        _call("w8a8_quantize_act_ex", _ptr(x), M, K, a, _ptr(cm), _ptr(q), _ptr(s),
              _stream(x.device))
    return q, s


def col_absmax(v: torch.Tensor, *, act: str = "none", out=None, accumulate: bool = False):
    """Per-column max |T(v)| of a bf16 [R,K] matrix -> fp32 [K]. With accumulate=True the
    maxima are merged into `out` (several calibration batches)."""
    a = _act(act)
    if out is None and accumulate:
        raise ValueError("accumulate needs out")
    _check(v, torch.bfloat16, 2, "v")
    R, K = v.shape
    if out is None:
        out = torch.empty((K,), dtype=torch.float32, device=v.device)
    _check(out, torch.float32, 1, "out")
    if out.shape[0] != K:
        raise ValueError("out must be [K]")
    with torch.cuda.device(v.device):
        _call("w8a8_col_absmax", _ptr(v), R, K, a, _ptr(out), int(bool(accumulate)),
              _stream(v.device))
    return out


def smooth_factors(x_amax: torch.Tensor, w_amax: torch.Tensor, alpha: float = 0.5):
    """SmoothQuant factors (s, s_inv), fp32 [K]: s = x_amax^alpha / w_amax^(1-alpha)."""
    _check(x_amax, torch.float32, 1, "x_amax")
    _check(w_amax, torch.float32, 1, "w_amax")
    _same_device(x_amax, w_amax)
    if x_amax.shape != w_amax.shape:
        raise ValueError("x_amax and w_amax must both be [K]")
    K = x_amax.shape[0]
    s = torch.empty_like(x_amax)
    si = torch.empty_like(x_amax)
    with torch.cuda.device(x_amax.device):
        _call("w8a8_smooth_factors", _ptr(x_amax), _ptr(w_amax), K, float(alpha), _ptr(s),
              _ptr(si), _stream(x_amax.device))
    return s, si


def _workspace(nbytes: int, device, workspace):
    if nbytes == 0:
        return None
    if workspace is not None:
        if not isinstance(workspace, torch.Tensor) or not workspace.is_contiguous():
            raise ValueError("workspace must be a contiguous torch.Tensor")
        if workspace.device != torch.device(device):
            raise ValueError(f"workspace is on {workspace.device}, expected {device}")
        if workspace.numel() * workspace.element_size() < nbytes:
            raise ValueError(f"workspace needs {nbytes} bytes")
        return workspace
    return torch.empty(nbytes, dtype=torch.uint8, device=device)


def gemm(xq, x_scale, wq, w_scale, bias=None, *, tile: int = -1, out=None,
         workspace=None):
    """Fused int8 GEMM + epilogue: bf16(fmaf(float(xq @ wq^T), sx[m]*sw[n], b[n]))."""
    _check(xq, torch.int8, 2, "xq")
    _check(wq, torch.int8, 2, "wq")
    _check(x_scale, torch.float32, 1, "x_scale")
    _check(w_scale, torch.float32, 1, "w_scale")
    if bias is not None:
        _check(bias, torch.bfloat16, 1, "bias")
    _same_device(xq, wq, x_scale, w_scale, bias)
    M, K = xq.shape
    N = wq.shape[0]
    if wq.shape[1] != K or x_scale.shape[0] != M or w_scale.shape[0] != N or (
            bias is not None and bias.shape[0] != N):
        raise ValueError("shape mismatch")
    if out is not None:
        _check_out(out, torch.bfloat16, (M, N), xq.device)
    y = out if out is not None else torch.empty((M, N), dtype=torch.bfloat16,
                                                device=xq.device)
    ws = _workspace(gemm_workspace_bytes(M, N, K, tile), xq.device, workspace)
    nws = 0 if ws is None else ws.numel() * ws.element_size()
    with torch.cuda.device(xq.device):
        _call("w8a8_gemm_ex", _ptr(xq), _ptr(x_scale), _ptr(wq), _ptr(w_scale), _ptr(bias),
              _ptr(y), M, N, K, _ptr(ws), nws, int(tile), _stream(xq.device))
    return y


def linear(x, wq, w_scale, bias=None, *, act: str = "none", col_mul=None, out=None,
           workspace=None):
    """The whole W8A8 linear: x bf16 [..., K] -> y bf16 [..., N] (per-token
    quantization of T(x) * col_mul, int8 GEMM, fused dequantization + bias)."""
    a = _act(act)
    if not isinstance(x, torch.Tensor) or x.dtype != torch.bfloat16:
        raise TypeError("x must be a bf16 torch.Tensor")
    lead = x.shape[:-1]
    K = x.shape[-1]
    x2 = x.reshape(lead.numel(), K)
    _check(x2, torch.bfloat16, 2, "x")
    _check(wq, torch.int8, 2, "wq")
    _check(w_scale, torch.float32, 1, "w_scale")
    if bias is not None:
        _check(bias, torch.bfloat16, 1, "bias")
    _same_device(x2, wq, w_scale, bias)
    M = x2.shape[0]
    N = wq.shape[0]
    if wq.shape[1] != K or w_scale.shape[0] != N or (bias is not None and bias.shape[0] != N):
        raise ValueError("shape mismatch")
    cm = _col_mul(col_mul, K, x.device)
    if out is not None:
        _check_out(out, torch.bfloat16, (M, N), x.device)
    y = out if out is not None else torch.empty((M, N), dtype=torch.bfloat16,
                                                device=x.device)
    if M == 0 or N == 0:
        return y.reshape(*lead, N)
    ws = _workspace(linear_workspace_bytes(M, N, K), x.device, workspace)
    with torch.cuda.device(x.device):
        _call("w8a8_linear_ex", _ptr(x2), a, _ptr(cm), _ptr(wq), _ptr(w_scale), _ptr(bias),
              _ptr(y), M, N, K, _ptr(ws), ws.numel() * ws.element_size(), _stream(x.device))
    return y.reshape(*lead, N)


def gemm_acc_i32(xq, wq, *, tile: int = -1, out=None):
    """Debug: the raw int32 accumulator xq @ wq^T (no epilogue)."""
    _check(xq, torch.int8, 2, "xq")
    _check(wq, torch.int8, 2, "wq")
    _same_device(xq, wq)
    M, K = xq.shape
    N = wq.shape[0]
    if wq.shape[1] != K:
        raise ValueError("shape mismatch")
    if out is not None:
        _check_out(out, torch.int32, (M, N), xq.device)
    acc = out if out is not None else torch.empty((M, N), dtype=torch.int32,
                                                  device=xq.device)
    with torch.cuda.device(xq.device):
        _call("w8a8_gemm_acc_i32_ex", _ptr(xq), _ptr(wq), _ptr(acc), M, N, K, int(tile),
              _stream(xq.device))
    return acc


def mfma_ceiling_ops(iters: int) -> int:
    """Int8 ops (2 per multiply-accumulate) of one mfma_ceiling launch."""
    n = int(load_library().w8a8_mfma_ceiling_ops(int(iters)))
    if n < 0:
        raise ValueError(f"iters out of range: {iters}")
    return n


def mfma_ceiling(xq, wq, iters: int, *, out=None):
    """Measurement aid: the GEMM's MFMA sequence replayed from registers on fragments
    of xq [M,K] / wq [N,K] (K % 32 == 0), `iters` sweeps. Returns the per-wavefront
    checksums (int32 [1024], the uint32 sums of the accumulators); its launch time
    against mfma_ceiling_ops(iters) is the matrix-core ceiling on these codes."""
    _check(xq, torch.int8, 2, "xq")
    _check(wq, torch.int8, 2, "wq")
    _same_device(xq, wq)
    M, K = xq.shape
    N = wq.shape[0]
    if wq.shape[1] != K:
        raise ValueError("shape mismatch")
    sums = out if out is not None else torch.empty(1024, dtype=torch.int32, device=xq.device)
    _check(sums, torch.int32, 1, "out")
    if sums.numel() < 1024:
        raise ValueError("out needs 1024 entries")
    with torch.cuda.device(xq.device):
        _call("w8a8_mfma_ceiling", _ptr(xq), _ptr(wq), M, N, K, int(iters), _ptr(sums),
              _stream(xq.device))
    return sums


READ_BLOCKS = 2048


def read_ceiling(buf: torch.Tensor, *, out=None):
    """Measurement aid: a plain streaming read of buf's bytes (contiguous, 16-byte
    aligned, nbytes a multiple of 16 * READ_BLOCKS). Returns the per-workgroup XOR
    checksums (int32 [READ_BLOCKS]); its launch time is the HBM read floor for that
    many bytes."""
    if not buf.is_cuda or not buf.is_contiguous():
        raise ValueError("buf must be a contiguous device tensor")
    nbytes = buf.numel() * buf.element_size()
    sums = out if out is not None else torch.empty(READ_BLOCKS, dtype=torch.int32,
                                                   device=buf.device)
    _check(sums, torch.int32, 1, "out")
    if sums.numel() < READ_BLOCKS or sums.device != buf.device:
        raise ValueError(f"out needs {READ_BLOCKS} entries on buf's device")
    with torch.cuda.device(buf.device):
        _call("w8a8_read_ceiling", _ptr(buf), nbytes, _ptr(sums), _stream(buf.device))
    return sums
