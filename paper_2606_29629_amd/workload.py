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


def to_device_f32(bits: np.ndarray, device="cuda"):
    """uint16 bfloat16 bit patterns -> torch.float32 tensor on `device` holding
    the same values (exact widening; the fp32 storage mode's inputs)."""
    import torch
    f = (np.ascontiguousarray(bits).astype(np.uint32) << 16).view(np.float32)
    return torch.from_numpy(f).to(device)


def to_host_f64(t) -> np.ndarray:
    """torch bfloat16/float tensor -> float64 NumPy array (exact widening)."""
    import torch
    return t.detach().to(torch.float32).cpu().numpy().astype(np.float64)


class DeviceLayer:
    """Weights of one layer resident in HBM plus its C config struct (bf16
    storage, or fp32 storage holding the same values with f32)."""

    def __init__(self, cfg, weights_bits: Dict[str, np.ndarray], device="cuda", f32=False):
        self.cfg_py = cfg
        self.cfg = make_config(cfg, f32=f32)
        to_dev = to_device_f32 if f32 else to_device_bf16
        self.w = {k: to_dev(v, device) for k, v in weights_bits.items()}


def device_cache(k_bits: np.ndarray, v_bits: np.ndarray, device="cuda", f32=False):
    to_dev = to_device_f32 if f32 else to_device_bf16
    return to_dev(k_bits, device), to_dev(v_bits, device)


def device_batch(batch, device="cuda") -> DeviceBatch:
    """DeviceBatch from any object with slot / ctx_len / q_len arrays."""
    pos3 = getattr(batch, "pos3", None)
    return DeviceBatch(batch.slot, batch.ctx_len, batch.q_len, device=device,
                       pos=None if pos3 is None else pos3)


def paged_from_contiguous(k, v, block_size: int, seed: int = 0, spare_blocks: int = 3,
                          fill=float("nan")):
    """A PagedCache holding the same rows as the contiguous cache (k, v)
    [n_slots, Hkv, max_seq, D]: every (slot, block) gets a distinct pool
    block in a seeded random order; `spare_blocks` extra pool blocks that no
    slot maps to are filled with `fill` (NaN by default, so any read of them
    would show in the results)."""
    import torch
    from ._lib import PagedCache
    n_slots, hkv, max_seq, d = k.shape
    assert max_seq % block_size == 0
    bps = max_seq // block_size
    n_blocks = n_slots * bps + spare_blocks
    rng = np.random.default_rng(seed)
    ids = rng.permutation(n_blocks)[:n_slots * bps].astype(np.int32).reshape(n_slots, bps)
    kp = torch.full((n_blocks, hkv, block_size, d), fill, dtype=k.dtype, device=k.device)
    vp = torch.full_like(kp, fill)
    src_k = k.reshape(n_slots, hkv, bps, block_size, d).permute(0, 2, 1, 3, 4)
    src_v = v.reshape(n_slots, hkv, bps, block_size, d).permute(0, 2, 1, 3, 4)
    idx = torch.from_numpy(ids.reshape(-1).astype(np.int64)).to(k.device)
    kp[idx] = src_k.reshape(-1, hkv, block_size, d)
    vp[idx] = src_v.reshape(-1, hkv, block_size, d)
    table = torch.from_numpy(ids).to(k.device)
    return PagedCache(kp, vp, table, max_seq)


def contiguous_from_paged(pc):
    """The contiguous (k, v) [n_slots, Hkv, max_seq, D] view of a PagedCache
    (gathered through its block table)."""
    ids = pc.block_table.long()
    n_slots, bps = ids.shape
    _, hkv, bs, d = pc.k.shape

    def gather(pool):
        g = pool[ids.reshape(-1)].reshape(n_slots, bps, hkv, bs, d).permute(0, 2, 1, 3, 4)
        return g.reshape(n_slots, hkv, bps * bs, d)

    return gather(pc.k), gather(pc.v)
