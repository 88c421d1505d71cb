"""Seeded synthetic inputs for the Thinker decoder layer.

This module only draws random numbers and lays them out; it holds none of the
layer's arithmetic.  Both the CPU oracle (through the tests and the bench) and
the HIP path receive exactly the arrays produced here, so the two sides see
bit-identical inputs.

Every tensor is drawn with NumPy ``Generator(PCG64(SeedSequence([seed, id])))``
in float32, scaled, and rounded to bfloat16 (round-to-nearest-even).  The
bfloat16 values are returned as ``uint16`` bit patterns; ``bf16_to_f32`` widens
them exactly.

The paper (Section II-A) describes the Thinker as a multimodal LLM that
consumes a token stream in a compute-bound prefill and then decodes
autoregressively over a KV cache; it gives no layer shapes.  The shapes below
are the 7B-class dense Thinker layer, a 30B-A3B-style MoE layer and a tiny
dense layer used for quick parity, with the value distributions stated in the
workload descriptions.
"""
from __future__ import annotations

import dataclasses
from typing import Dict, List, Optional, Tuple

import numpy as np

# Fixed tensor-id enumeration (second word of the seed sequence).
TID_ATTN_NORM = 0
TID_W_QKV = 1
TID_B_QKV = 2
TID_W_O = 3
TID_MLP_NORM = 4
TID_W_GATE_UP = 5
TID_W_DOWN = 6
TID_W_ROUTER = 7
TID_X_PREFILL = 8
TID_X_DECODE0 = 9          # step s uses TID_X_DECODE0 + s
TID_CACHE_K = 100
TID_CACHE_V = 101
TID_KV_LENGTHS = 102
TID_Q_NORM = 103
TID_K_NORM = 104


@dataclasses.dataclass(frozen=True)
class LayerConfig:
    hidden: int
    n_q_heads: int
    n_kv_heads: int
    head_dim: int
    ffn_dim: int = 0              # dense SwiGLU width F
    n_experts: int = 0            # MoE: E (0 = dense layer)
    top_k: int = 0
    expert_ffn_dim: int = 0       # MoE: per-expert SwiGLU width
    rms_eps: float = 1e-6
    rope_base: float = 1e6
    qkv_bias: bool = False
    moe_renorm: bool = True
    qk_norm: bool = False         # per-head RMSNorm of q and k before the rotation
    # multi-section rotary positions: (s_t, s_h, s_w) frequencies per section, sum D/2
    mrope_section: Optional[Tuple[int, int, int]] = None

    @property
    def moe(self) -> bool:
        return self.n_experts > 0

    @property
    def qkv_rows(self) -> int:
        return (self.n_q_heads + 2 * self.n_kv_heads) * self.head_dim


# ---------------------------------------------------------------- bfloat16 --

def to_bf16_bits(a: np.ndarray) -> np.ndarray:
    """float32 -> bfloat16 bit patterns, round to nearest even (finite input)."""
    u = np.ascontiguousarray(a, dtype=np.float32).view(np.uint32)
    lsb = (u >> np.uint32(16)) & np.uint32(1)
    return ((u + np.uint32(0x7FFF) + lsb) >> np.uint32(16)).astype(np.uint16)


def bf16_to_f32(bits: np.ndarray) -> np.ndarray:
    """bfloat16 bit patterns -> float32 (exact)."""
    return (np.asarray(bits, dtype=np.uint16).astype(np.uint32) << np.uint32(16)).view(np.float32)


def rng_for(seed: int, tensor_id: int) -> np.random.Generator:
    return np.random.Generator(np.random.PCG64(np.random.SeedSequence([seed, tensor_id])))


def normal_bf16(seed: int, tensor_id: int, shape, std: float = 1.0, mean: float = 0.0) -> np.ndarray:
    g = rng_for(seed, tensor_id)
    a = g.standard_normal(size=shape, dtype=np.float32)
    if std != 1.0:
        a *= np.float32(std)
    if mean != 0.0:
        a += np.float32(mean)
    return to_bf16_bits(a)


# ------------------------------------------------------------------ weights --

def make_weights(cfg: LayerConfig, seed: int = 0, w_std: float = 0.02,
                 gain_std: float = 0.1) -> Dict[str, np.ndarray]:
    """Random layer weights as bf16 bit patterns, row-major ``[out, in]``.

    Projection, expert and router matrices ~ N(0, w_std).  RMSNorm gains are
    1 + N(0, gain_std) so that the normalised activations keep unit scale.
    """
    H, D = cfg.hidden, cfg.head_dim
    w: Dict[str, np.ndarray] = {}
    w["attn_norm"] = normal_bf16(seed, TID_ATTN_NORM, (H,), gain_std, 1.0)
    w["w_qkv"] = normal_bf16(seed, TID_W_QKV, (cfg.qkv_rows, H), w_std)
    if cfg.qkv_bias:
        w["b_qkv"] = normal_bf16(seed, TID_B_QKV, (cfg.qkv_rows,), w_std * 10)
    w["w_o"] = normal_bf16(seed, TID_W_O, (H, cfg.n_q_heads * D), w_std)
    w["mlp_norm"] = normal_bf16(seed, TID_MLP_NORM, (H,), gain_std, 1.0)
    if cfg.qk_norm:
        w["q_norm"] = normal_bf16(seed, TID_Q_NORM, (D,), gain_std, 1.0)
        w["k_norm"] = normal_bf16(seed, TID_K_NORM, (D,), gain_std, 1.0)
    if cfg.moe:
        E, Fe = cfg.n_experts, cfg.expert_ffn_dim
        w["w_gate_up"] = normal_bf16(seed, TID_W_GATE_UP, (E, 2 * Fe, H), w_std)
        w["w_down"] = normal_bf16(seed, TID_W_DOWN, (E, H, Fe), w_std)
        w["w_router"] = normal_bf16(seed, TID_W_ROUTER, (E, H), w_std)
    else:
        F = cfg.ffn_dim
        w["w_gate_up"] = normal_bf16(seed, TID_W_GATE_UP, (2 * F, H), w_std)
        w["w_down"] = normal_bf16(seed, TID_W_DOWN, (H, F), w_std)
    return w


# ---------------------------------------------------------------- workloads --

@dataclasses.dataclass
class Batch:
    """A ragged batch: per sequence its cache slot, tokens already cached
    (``ctx_len``) and new tokens this call (``q_len``).  RoPE positions of the
    new tokens are ``ctx_len + i``, or, for multi-section rotary positions,
    the columns of ``pos3`` [3, T] (temporal, height, width ids)."""
    slot: np.ndarray      # int32 [n_seqs]
    ctx_len: np.ndarray   # int32 [n_seqs]
    q_len: np.ndarray     # int32 [n_seqs]
    pos3: Optional[np.ndarray] = None   # int32 [3, T] or None

    @property
    def n_seqs(self) -> int:
        return int(self.slot.shape[0])

    @property
    def cu_q(self) -> np.ndarray:
        return np.concatenate([[0], np.cumsum(self.q_len)]).astype(np.int32)

    @property
    def n_tokens(self) -> int:
        return int(self.q_len.sum())

    @property
    def pos(self) -> np.ndarray:
        return np.concatenate([np.arange(c, c + q, dtype=np.int32)
                               for c, q in zip(self.ctx_len, self.q_len)]).astype(np.int32)

    @property
    def rope_pos(self) -> np.ndarray:
        """The position array the layer reads: pos [T], or pos3 flattened [3 T]."""
        return self.pos if self.pos3 is None else np.ascontiguousarray(self.pos3, np.int32).ravel()

    def advanced(self) -> "Batch":
        """The batch after this call's tokens were appended (next decode step).
        With pos3, the next token of a sequence is text at one past the
        largest id its tokens of this call used."""
        nxt = None
        if self.pos3 is not None:
            cu = self.cu_q
            nxt = np.stack([np.full(3, self.pos3[:, cu[i]:cu[i + 1]].max() + 1, np.int32)
                            for i in range(self.n_seqs)], axis=1)
        return Batch(self.slot.copy(), (self.ctx_len + self.q_len).astype(np.int32),
                     np.ones_like(self.q_len), nxt)


def mrope_positions(segments, start: int = 0):
    """Multi-section position ids [3, n] (temporal, height, width) of a token
    stream and the id after it.  segments: ("text", n) -- ids start .. start+n-1
    on all three; ("image", gh, gw) -- gh x gw patches in row-major order,
    temporal id start, height start + row, width start + col; ("video", gt,
    gh, gw) -- gt frames of such patches, temporal id start + frame.  After an
    image or video the next id is start + its largest extent."""
    cols = []
    for seg in segments:
        kind = seg[0]
        if kind == "text":
            ids = np.arange(start, start + seg[1], dtype=np.int32)
            cols.append(np.stack([ids, ids, ids]))
            start += seg[1]
        else:
            gt, gh, gw = (1, seg[1], seg[2]) if kind == "image" else seg[1:4]
            f, r, c = np.meshgrid(np.arange(gt), np.arange(gh), np.arange(gw), indexing="ij")
            cols.append(np.stack([start + f.ravel(), start + r.ravel(), start + c.ravel()])
                        .astype(np.int32))
            start += max(gt, gh, gw)
    out = np.concatenate(cols, axis=1) if cols else np.zeros((3, 0), np.int32)
    return out.astype(np.int32), start


def mrope_batch(slot, ctx_len, segments_per_seq) -> Batch:
    """A Batch whose sequence s continues after ctx_len[s] cached text tokens
    (ids 0 .. ctx_len[s]-1) with the given segments."""
    pos, q = [], []
    for c, segs in zip(ctx_len, segments_per_seq):
        p3, _ = mrope_positions(segs, int(c))
        pos.append(p3)
        q.append(p3.shape[1])
    return Batch(np.asarray(slot, np.int32), np.asarray(ctx_len, np.int32),
                 np.asarray(q, np.int32), np.concatenate(pos, axis=1))


@dataclasses.dataclass
class Workload:
    name: str
    description: str
    cfg: LayerConfig
    n_slots: int
    max_seq: int
    batch: Batch              # first call
    decode_steps: int = 0     # further one-token steps after the first call
    cache_prefilled: bool = False  # caches hold N(0,1) rows below ctx_len
    seed: int = 0


def layer_c1() -> LayerConfig:
    return LayerConfig(hidden=256, n_q_heads=4, n_kv_heads=2, head_dim=64, ffn_dim=1024)


def layer_7b() -> LayerConfig:
    return LayerConfig(hidden=3584, n_q_heads=28, n_kv_heads=4, head_dim=128, ffn_dim=18944)


def layer_moe() -> LayerConfig:
    return LayerConfig(hidden=2048, n_q_heads=32, n_kv_heads=4, head_dim=128,
                       n_experts=128, top_k=8, expert_ffn_dim=768)


def layer_talker() -> LayerConfig:
    """A Talker-shaped layer: the paper's Talker (Section II-A) is an
    autoregressive transformer decoder whose shapes it does not give; the
    reading here is a 0.5B-class dense decoder of the same model family
    (hidden 896, 14 query / 2 KV heads of 64, SwiGLU 4864)."""
    return LayerConfig(hidden=896, n_q_heads=14, n_kv_heads=2, head_dim=64, ffn_dim=4864)


def _ints(*v) -> np.ndarray:
    return np.asarray(v, dtype=np.int32)


def workload(name: str, seed: int = 0) -> Workload:
    """The named workloads (tiny dense, 7B prefill/decode, MoE prefill/decode,
    mixed chunked-prefill + decode)."""
    if name == "tiny":
        return Workload(name, "tiny dense layer H256, 4q/2kv heads, D64, F1024; 32-token prefill "
                        "then 16 decode steps", layer_c1(), 1, 64,
                        Batch(_ints(0), _ints(0), _ints(32)), decode_steps=16, seed=seed)
    if name == "dense_prefill":
        return Workload(name, "7B dense layer prefill, 8 x 2048 tokens, causal", layer_7b(), 8, 2048,
                        Batch(np.arange(8, dtype=np.int32), np.zeros(8, np.int32),
                              np.full(8, 2048, np.int32)), seed=seed)
    if name == "dense_decode":
        return Workload(name, "7B dense layer decode, batch 64, KV 4096, 32 steps", layer_7b(), 64,
                        4096 + 32, Batch(np.arange(64, dtype=np.int32), np.full(64, 4096, np.int32),
                                         np.ones(64, np.int32)),
                        decode_steps=31, cache_prefilled=True, seed=seed)
    if name == "moe_prefill":
        return Workload(name, "MoE layer (128 experts, top-8) prefill, 4 x 1024 tokens", layer_moe(),
                        4, 1024, Batch(np.arange(4, dtype=np.int32), np.zeros(4, np.int32),
                                       np.full(4, 1024, np.int32)), seed=seed)
    if name == "moe_decode":
        return Workload(name, "MoE layer decode, batch 128, KV 2048, 32 steps", layer_moe(), 128,
                        2048 + 32, Batch(np.arange(128, dtype=np.int32), np.full(128, 2048, np.int32),
                                         np.ones(128, np.int32)),
                        decode_steps=31, cache_prefilled=True, seed=seed)
    if name == "mixed":
        lens = rng_for(seed, TID_KV_LENGTHS).integers(1024, 8193, size=32).astype(np.int32)
        return Workload(name, "7B dense layer mixed step: 512-token chunk at ctx 6144 plus 32 "
                        "decode sequences with KV lengths U[1024, 8192]", layer_7b(), 33, 8704,
                        Batch(np.arange(33, dtype=np.int32), np.concatenate([_ints(6144), lens]),
                              np.concatenate([_ints(512), np.ones(32, np.int32)])),
                        cache_prefilled=True, seed=seed)
    if name == "talker_prefill":
        return Workload(name, "Talker-shaped layer (H896, 14q/2kv heads, D64, F4864) prefill, "
                        "8 x 512 tokens", layer_talker(), 8, 512,
                        Batch(np.arange(8, dtype=np.int32), np.zeros(8, np.int32),
                              np.full(8, 512, np.int32)), seed=seed)
    if name == "talker_decode":
        return Workload(name, "Talker-shaped layer decode, batch 64 streams, KV 1024, 32 steps",
                        layer_talker(), 64, 1024 + 32,
                        Batch(np.arange(64, dtype=np.int32), np.full(64, 1024, np.int32),
                              np.ones(64, np.int32)),
                        decode_steps=31, cache_prefilled=True, seed=seed)
    if name in ("dense_prefill_bias", "dense_decode_bias"):
        # the 7B workloads with the q/k/v bias of the Qwen2 family (seeded, N(0, 0.2))
        base = workload(name[:-5], seed)
        return dataclasses.replace(
            base, name=name, cfg=dataclasses.replace(base.cfg, qkv_bias=True),
            description=base.description + ", q/k/v bias")
    if name in ("dense_prefill_qkn", "moe_prefill_qkn"):
        # the same prefills with the per-head q/k RMSNorm of the Qwen3-family
        # attention block (the MoE one then has the Qwen3-30B-A3B layer shape)
        base = workload(name[:-4], seed)
        return dataclasses.replace(
            base, name=name, cfg=dataclasses.replace(base.cfg, qk_norm=True),
            description=base.description + ", per-head q/k RMSNorm")
    raise KeyError(name)


WORKLOADS = ("tiny", "dense_prefill", "dense_decode", "moe_prefill", "moe_decode", "mixed",
             "dense_prefill_qkn", "moe_prefill_qkn", "dense_prefill_bias", "dense_decode_bias",
             "talker_prefill", "talker_decode")


def make_x(cfg: LayerConfig, n_tokens: int, seed: int = 0, step: Optional[int] = None) -> np.ndarray:
    """Token activations ~ N(0, 1) as bf16 bits ``[n_tokens, hidden]``; ``step``
    selects the fresh input of a decode step."""
    tid = TID_X_PREFILL if step is None else TID_X_DECODE0 + step
    return normal_bf16(seed, tid, (n_tokens, cfg.hidden))


def make_cache(cfg: LayerConfig, n_slots: int, max_seq: int, seed: int = 0):
    """K and V caches ``[n_slots, n_kv_heads, max_seq, head_dim]`` filled with
    N(0, 1) bf16 values (rows at or beyond a sequence's length are overwritten
    before they are read)."""
    shape = (n_slots, cfg.n_kv_heads, max_seq, cfg.head_dim)
    return normal_bf16(seed, TID_CACHE_K, shape), normal_bf16(seed, TID_CACHE_V, shape)


def random_batch(rng: np.random.Generator, n_seqs: int, max_q: int, max_ctx: int,
                 n_slots: Optional[int] = None) -> Batch:
    """A random ragged batch for edge-case tests (q_len >= 1)."""
    n_slots = n_slots or n_seqs
    slot = rng.permutation(n_slots)[:n_seqs].astype(np.int32)
    q = rng.integers(1, max_q + 1, size=n_seqs).astype(np.int32)
    c = rng.integers(0, max_ctx + 1, size=n_seqs).astype(np.int32)
    return Batch(slot, c, q)


__all__: List[str] = [n for n in dir() if not n.startswith("_")]
