"""Helpers of the GPU tests: move seeded host inputs to the device and back.
No arithmetic of the method lives here."""
import numpy as np
import torch


def dev_u16(a: np.ndarray) -> torch.Tensor:
    """uint16 bit patterns -> device int16 tensor (same bits)."""
    return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).cuda()


def dev(a: np.ndarray) -> torch.Tensor:
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def host_u16(t: torch.Tensor) -> np.ndarray:
    """device 16-bit tensor -> uint16 bit patterns on the host."""
    return t.detach().view(torch.int16).cpu().numpy().view(np.uint16)


def bf16_as_f64(bits: np.ndarray) -> np.ndarray:
    return ((bits.astype(np.uint32) << 16).view(np.float32)).astype(np.float64)


def say(msg: str):
    print(msg, flush=True)
