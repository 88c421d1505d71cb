"""The fp32 storage mode (TRI_F32) on the GPU, through the C ABI.

Weights, activations and the KV cache are fp32 (the weights and inputs hold
the same bf16-representable seeded values as the bf16 tests); the layer runs
the same kernels on fp32 storage.  Every output element must lie within
max(1e-4, 1e-4 |r|) of the exact float64 oracle (no bf16 rounding anywhere),
and the rows written to the cache likewise.  Routing follows rule R2: the
GPU's experts are the oracle's top-k of its exact logits, except adjacent
ranks whose fp64 logit gap is <= 1e-4, and the output is checked against the
oracle run with the GPU's routes.
"""
import dataclasses

import numpy as np
import pytest

import oracle
from paper_2606_29629_amd import _lib as T
from paper_2606_29629_amd.workload import (DeviceLayer, device_batch, device_cache,
                                           paged_from_contiguous, to_device_f32, to_host_f64)
from parity import F32_TOL, check_e2e
from synth import (Batch, bf16_to_f32, layer_7b, layer_c1, make_cache, make_weights, make_x,
                   mrope_batch, workload)
from test_gpu_moe import TINY_MOE, routes_agree

pytestmark = pytest.mark.gpu

TAU_R2 = 1e-4


def f64(bits):
    return bf16_to_f32(bits).astype(np.float64)


def B(slot, ctx, q):
    return Batch(np.asarray(slot, np.int32), np.asarray(ctx, np.int32), np.asarray(q, np.int32))


def strict(got, exact, what):
    check_e2e(got, exact, what, strict=True, tol=F32_TOL)


class F32Case:
    """Seeded inputs of one fp32-storage layer call (host bits, device fp32)."""

    def __init__(self, cfg, batch, n_slots, max_seq, seed=0, x_step=None, paged_block=0):
        import torch
        self.cfg, self.batch = cfg, batch
        self.wb = make_weights(cfg, seed)
        self.kb, self.vb = make_cache(cfg, n_slots, max_seq, seed)
        self.xb = make_x(cfg, batch.n_tokens, seed, step=x_step)
        self.dl = DeviceLayer(cfg, self.wb, f32=True)
        k, v = device_cache(self.kb, self.vb, f32=True)
        self.cache = paged_from_contiguous(k, v, paged_block, seed=seed + 3) if paged_block else (k, v)
        self.db = device_batch(batch)
        self.route = None
        if getattr(cfg, "n_experts", 0):
            self.route = torch.full((batch.n_tokens, cfg.top_k), -1, dtype=torch.int32,
                                    device="cuda")
        torch.cuda.synchronize()

    def run(self, decode=False, x_bits=None):
        import torch
        fn = T.layer_decode if decode else T.layer_prefill
        x = to_device_f32(self.xb if x_bits is None else x_bits)
        out, ws = fn(self.dl.cfg, self.dl.w, self.cache, self.db, x, route_idx=self.route)
        torch.cuda.synchronize()
        assert out.dtype == torch.float32
        return out

    def cache_view(self):
        from paper_2606_29629_amd.workload import contiguous_from_paged
        return self.cache if isinstance(self.cache, tuple) else contiguous_from_paged(self.cache)

    def cache_rows(self, batch=None):
        b = self.batch if batch is None else batch
        k, v = self.cache_view()
        ks, vs = [], []
        for s, c, q in zip(b.slot, b.ctx_len, b.q_len):
            ks.append(to_host_f64(k[s, :, c:c + q]).transpose(1, 0, 2))
            vs.append(to_host_f64(v[s, :, c:c + q]).transpose(1, 0, 2))
        return np.concatenate(ks), np.concatenate(vs)

    def oracle(self, rows=None, x_bits=None, kc=None, vc=None, batch=None, forced=None):
        if not hasattr(self, "w64"):
            self.w64 = {k: f64(v) for k, v in self.wb.items()}
        return oracle.layer_forward(self.cfg, self.w64, f64(self.kb) if kc is None else kc,
                                    f64(self.vb) if vc is None else vc,
                                    self.batch if batch is None else batch,
                                    f64(self.xb if x_bits is None else x_bits), rows=rows,
                                    forced_routes=forced)


def test_f32_tiny_prefill_then_16_decode_steps():
    wl = workload("tiny")
    cs = F32Case(wl.cfg, wl.batch, wl.n_slots, wl.max_seq)
    out = cs.run()
    ex = cs.oracle()
    strict(to_host_f64(out), ex["out"], "f32 tiny prefill out")
    kr, vr = cs.cache_rows()
    strict(kr, ex["k_new"], "f32 tiny prefill K rows")
    strict(vr, ex["v_new"], "f32 tiny prefill V rows")
    batch = wl.batch
    for step in range(wl.decode_steps):
        batch = batch.advanced()
        k, v = cs.cache_view()
        kc, vc = to_host_f64(k), to_host_f64(v)        # the cache the GPU wrote so far
        cs.batch, cs.db = batch, device_batch(batch)
        xb = make_x(wl.cfg, batch.n_tokens, wl.seed, step=step)
        out = cs.run(decode=True, x_bits=xb)
        ex = cs.oracle(x_bits=xb, kc=kc, vc=vc)
        strict(to_host_f64(out), ex["out"], f"f32 tiny decode step {step}")
        kr, vr = cs.cache_rows()
        strict(kr, ex["k_new"], f"f32 tiny decode K row {step}")


@pytest.mark.parametrize("variant", ["bias", "qk_norm", "mrope", "paged"])
def test_f32_tiny_ragged_variants(variant):
    """A fresh prefill, a chunk after a cached prefix, decodes; with the q/k/v
    bias, the per-head q/k RMSNorm, multi-section positions, or a paged cache."""
    cfg = layer_c1()
    batch = B([3, 0, 2, 1, 4], [0, 40, 7, 0, 150], [200, 9, 1, 1, 1])
    block = 0
    if variant == "bias":
        cfg = dataclasses.replace(cfg, qkv_bias=True)
    elif variant == "qk_norm":
        cfg = dataclasses.replace(cfg, qk_norm=True, qkv_bias=True)
    elif variant == "mrope":
        cfg = dataclasses.replace(cfg, mrope_section=(8, 12, 12))
        batch = mrope_batch([3, 0, 2, 1, 4], [0, 40, 7, 0, 150], [
            [("text", 20), ("image", 8, 10), ("text", 40)], [("video", 2, 3, 3)],
            [("text", 1)], [("text", 1)], [("text", 1)]])
    else:
        block = 64
    cs = F32Case(cfg, batch, 5, 256, seed=3, paged_block=block)
    out = cs.run()
    ex = cs.oracle()
    strict(to_host_f64(out), ex["out"], f"f32 tiny {variant} out")
    kr, vr = cs.cache_rows()
    strict(kr, ex["k_new"], f"f32 tiny {variant} K rows")
    strict(vr, ex["v_new"], f"f32 tiny {variant} V rows")


def test_f32_7b_ragged_prefill_sampled_rows():
    batch = B([0, 1, 2, 3], [0, 37, 500, 0], [300, 129, 1, 64])
    cs = F32Case(layer_7b(), batch, 4, 640, seed=1)
    out = cs.run()
    rows = np.array([0, 1, 127, 128, 255, 256, 299, 300, 301, 365, 428, 429, 430, 460, 493])
    ex = cs.oracle(rows=rows)
    strict(to_host_f64(out)[rows], ex["out"], "f32 7B ragged prefill rows")
    kr, vr = cs.cache_rows()
    strict(kr, ex["k_new"], "f32 7B K rows")
    strict(vr, ex["v_new"], "f32 7B V rows")


def test_f32_7b_decode_step():
    ctx = [1, 63, 64, 127, 128, 129, 1000, 4095]
    batch = B(list(range(8)), ctx, [1] * 8)
    cs = F32Case(layer_7b(), batch, 8, 4100, seed=2, x_step=0)
    out = cs.run(decode=True)
    ex = cs.oracle()
    strict(to_host_f64(out), ex["out"], "f32 7B decode out")
    kr, vr = cs.cache_rows()
    strict(kr, ex["k_new"], "f32 7B decode K rows")


def moe_check(cs, out, rows, label):
    """Rule R2 on the GPU's routes, then the output with those routes."""
    gi = cs.route.cpu().numpy()
    ex = cs.oracle()
    n_tie = routes_agree(gi, ex["logits"], cs.cfg.top_k, TAU_R2)
    forced = cs.oracle(rows=rows, forced=gi)
    strict(to_host_f64(out)[rows], forced["out"], f"{label} out")
    return n_tie


@pytest.mark.parametrize("decode", [False, True])
def test_f32_tiny_moe(decode):
    if decode:
        batch = B([0, 1, 2, 3, 4], [5, 0, 17, 33, 2], [1] * 5)
    else:
        batch = B([0, 1, 2], [0, 7, 0], [40, 9, 1])
    cs = F32Case(TINY_MOE, batch, 5, 64, seed=4, x_step=0 if decode else None)
    out = cs.run(decode=decode)
    moe_check(cs, out, np.arange(batch.n_tokens), f"f32 tiny MoE (decode {decode})")


def test_f32_moe_layer_shape():
    """The 128-expert top-8 layer (H 2048, 32/4 heads, Fe 768) on 2 x 48 tokens."""
    wl = workload("moe_prefill")
    batch = B([0, 1], [0, 100], [48, 48])
    cs = F32Case(wl.cfg, batch, 2, 256, seed=5)
    out = cs.run()
    n_tie = moe_check(cs, out, np.array([0, 1, 47, 48, 70, 95]), "f32 MoE layer shape")
    assert n_tie <= 2, n_tie


def test_f32_kvcache_append():
    import torch
    cfg = layer_c1()
    batch = B([2, 0], [5, 0], [3, 4])
    k = torch.full((3, cfg.n_kv_heads, 16, cfg.head_dim), 7.0, dtype=torch.float32, device="cuda")
    v = k.clone()
    kn = torch.randn(7, cfg.n_kv_heads, cfg.head_dim, device="cuda")
    vn = torch.randn_like(kn)
    T.kvcache_append(T.make_config(cfg, f32=True), (k, v), device_batch(batch), kn, vn)
    torch.cuda.synchronize()
    ck, cv = oracle.kvcache_append(np.full(k.shape, 7.0), np.full(v.shape, 7.0), batch,
                                   kn.double().cpu().numpy(), vn.double().cpu().numpy())
    assert np.array_equal(k.double().cpu().numpy(), ck)
    assert np.array_equal(v.double().cpu().numpy(), cv)
