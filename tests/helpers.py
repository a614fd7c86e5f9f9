"""Shared test helpers: host <-> device transfers of bit patterns and the
output tolerance of the linear layer."""
import numpy as np


def to_dev_bf16(bits: np.ndarray, device="cuda"):
    import torch
    t = torch.from_numpy(np.ascontiguousarray(bits, np.uint16).view(np.int16))
    return t.to(device).view(torch.bfloat16)


def to_host_u16(t) -> np.ndarray:
    import torch
    if t.dtype in (torch.bfloat16, torch.float16):
        t = t.view(torch.int16)
    return t.cpu().numpy().view(np.uint16)


def bf16_bits_to_f64(bits) -> np.ndarray:
    return (np.asarray(bits, np.uint16).astype(np.uint32) << 16).view(np.float32).astype(np.float64)


def y_tolerance(y64: np.ndarray, S: np.ndarray, K: int, gelu: bool = False) -> np.ndarray:
    """|y_gpu - y64| bound: 1e-2 relative plus an fp32-accumulation floor of
    4 (K/64 + 1) 2^-24 S, with S = sum_g |s_a s_w P_g| + |bias|; the floor is
    widened by 1.2 under GELU (its slope stays below 1.13)."""
    floor = 4.0 * (K / 64 + 1) * 2.0 ** -24 * S
    if gelu:
        floor = 1.2 * floor
    return 1e-2 * np.abs(y64) + floor


def bf16_ulp_distance(a_bits: np.ndarray, b_bits: np.ndarray) -> np.ndarray:
    """Distance in bf16 ulps between two bf16 bit patterns (sign-magnitude ordering)."""
    def ordered(b):
        b = np.asarray(b, np.uint16).astype(np.int32)
        return np.where(b & 0x8000, -(b & 0x7FFF), b)
    return np.abs(ordered(a_bits) - ordered(b_bits))
