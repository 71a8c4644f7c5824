"""Small helpers shared by the tests (no method arithmetic)."""
import numpy as np
import torch


def u16(t: torch.Tensor) -> np.ndarray:
    """bf16 tensor -> numpy uint16 bit patterns (host copy)."""
    return t.detach().cpu().contiguous().view(torch.int16).numpy().view(np.uint16)


def host(t: torch.Tensor) -> np.ndarray:
    """Any tensor -> numpy (bf16 as uint16)."""
    if t.dtype == torch.bfloat16:
        return u16(t)
    return t.detach().cpu().numpy()


def bf16_bits_to_f32(a: np.ndarray) -> np.ndarray:
    return (np.asarray(a, np.uint16).astype(np.uint32) << 16).view(np.float32)


def within_tol(gpu_u16, ref_u16, atol=2e-2, rtol=1e-2):
    """Elementwise |gpu - ref| <= atol + rtol*|ref| on bf16 bit patterns; returns
    (ok, max_abs, worst_index)."""
    g = bf16_bits_to_f32(gpu_u16).astype(np.float64)
    r = bf16_bits_to_f32(ref_u16).astype(np.float64)
    err = np.abs(g - r)
    bound = atol + rtol * np.abs(r)
    bad = err > bound
    worst = int(np.argmax(err - bound)) if err.size else -1
    return (not bad.any()), (float(err.max()) if err.size else 0.0), worst


def ulp_diff_bf16(a_u16, b_u16) -> np.ndarray:
    """Distance in bf16 units in the last place between two bf16 arrays
    (same-sign ordering on the integer encoding)."""
    def key(v):
        v = np.asarray(v, np.uint16).astype(np.int32)
        return np.where(v & 0x8000, -(v & 0x7FFF), v)
    return np.abs(key(a_u16) - key(b_u16))
