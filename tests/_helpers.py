"""Comparison helpers shared by the tests (no method arithmetic)."""
import numpy as np


def ordered_bf16(u):
    """Map bf16 bit patterns to integers whose order is the float order (+0 == -0)."""
    u = np.asarray(u).astype(np.uint16).astype(np.int32)
    return np.where(u & 0x8000, -(u & 0x7FFF), u)


def ulp_distance(a_bits, b_bits):
    return np.abs(ordered_bf16(a_bits) - ordered_bf16(b_bits))


def bf16_bits_to_f64(bits):
    return (np.asarray(bits, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32).astype(np.float64)


def cosine(a_bits, b_bits):
    a = bf16_bits_to_f64(a_bits).ravel()
    b = bf16_bits_to_f64(b_bits).ravel()
    na, nb = np.linalg.norm(a), np.linalg.norm(b)
    if na == 0 and nb == 0:
        return 1.0
    return float(a @ b / (na * nb))


def assert_bf16_parity(got_bits, want_bits, what=""):
    """The bf16 gate: every element within 1 ulp, all finite, cosine >= 0.99999."""
    got_bits = np.asarray(got_bits)
    want_bits = np.asarray(want_bits)
    assert got_bits.shape == want_bits.shape, (what, got_bits.shape, want_bits.shape)
    if got_bits.size == 0:
        return {"max_ulp": 0, "mismatches": 0, "cosine": 1.0}
    d = ulp_distance(got_bits, want_bits)
    finite = np.isfinite(bf16_bits_to_f64(got_bits))
    assert finite.all(), f"{what}: non-finite outputs"
    cos = cosine(got_bits, want_bits)
    stats = {"max_ulp": int(d.max()), "mismatches": int((d != 0).sum()), "cosine": cos}
    assert d.max() <= 1, f"{what}: max ulp {d.max()} at {np.unravel_index(d.argmax(), d.shape)}"
    assert cos >= 0.99999, f"{what}: cosine {cos}"
    return stats


# Device round trips for the GPU tests (torch is imported lazily: the CPU suite does
# not need it here).
def dev_bf16(bits):
    import torch
    return torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).view(torch.bfloat16).cuda()


def dev_f32(a):
    import torch
    return torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).cuda()


def host_bits(t):
    import torch
    return t.contiguous().view(torch.int16).cpu().numpy().view(np.uint16)


def host(t):
    return t.cpu().numpy()


def say(*a):
    print(*a, flush=True)
