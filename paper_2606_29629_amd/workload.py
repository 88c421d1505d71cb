"""Device-side setup helpers: bf16 bit arrays (NumPy uint16) -> torch tensors
in HBM, and a layer bundle for the ctypes binding.  No arithmetic of the
layer happens here."""
from __future__ import annotations

from typing import Dict

import numpy as np

from ._lib import DeviceBatch, make_config


def to_device_bf16(bits: np.ndarray, device="cuda"):
    """uint16 bfloat16 bit patterns -> torch.bfloat16 tensor on `device` (exact)."""
    import torch
    t = torch.from_numpy(np.ascontiguousarray(bits).view(np.int16))
    return t.to(device).view(torch.bfloat16)


def to_host_f64(t) -> np.ndarray:
    """torch bfloat16/float tensor -> float64 NumPy array (exact widening)."""
    import torch
    return t.detach().to(torch.float32).cpu().numpy().astype(np.float64)


class DeviceLayer:
    """Weights of one layer resident in HBM plus its C config struct."""

    def __init__(self, cfg, weights_bits: Dict[str, np.ndarray], device="cuda"):
        self.cfg_py = cfg
        self.cfg = make_config(cfg)
        self.w = {k: to_device_bf16(v, device) for k, v in weights_bits.items()}


def device_cache(k_bits: np.ndarray, v_bits: np.ndarray, device="cuda"):
    return to_device_bf16(k_bits, device), to_device_bf16(v_bits, device)


def device_batch(batch, device="cuda") -> DeviceBatch:
    """DeviceBatch from any object with slot / ctx_len / q_len arrays."""
    return DeviceBatch(batch.slot, batch.ctx_len, batch.q_len, device=device)
