"""Multi-section rotary positions (the multimodal rotary embedding of the
Qwen2-VL / Qwen2.5-Omni family) on the GPU, through the C ABI.

Every token carries three position ids (temporal, height, width) and each
rotary frequency takes the id of its section; only the rotary table of the
layer prologue depends on them.  Batches mix text, image (a patch grid at one
temporal id) and video (several frames) segments after cached text prefixes,
at head_dim 64 and 128, then run decode steps whose text tokens continue one
past the largest id used.  Gates as in test_gpu_layer.py: per-kernel parity on
identical inputs plus the end-to-end tolerance against the oracle.
"""
import dataclasses

import numpy as np
import pytest

import oracle
from paper_2606_29629_amd.workload import device_batch, to_device_bf16, to_host_f64
from synth import layer_7b, layer_c1, make_x, mrope_batch
from parity import strict_shape
from test_gpu_layer import Case, assert_e2e, check_down, f64, stage_parity

pytestmark = pytest.mark.gpu


def run_and_check(cfg, batch, n_slots, max_seq, label, seed=0, decode_steps=0):
    cs = Case(cfg, batch, n_slots, max_seq, seed=seed)
    out, ws = cs.run()
    rows = np.arange(batch.n_tokens)
    x1, act, w = stage_parity(cs, ws, rows, label=label)
    check_down(cs, out, x1, act, w, rows, label)
    ref = cs.oracle()
    ex = cs.oracle(storage=None)
    strict = strict_shape(cfg)
    assert_e2e(to_host_f64(out), ex["out"], f"{label} out", emul=ref["out"], strict=strict)
    kr, vr = cs.cache_rows()
    assert_e2e(kr, ex["k_new"], f"{label} K rows", emul=ref["k_new"], strict=strict)
    assert_e2e(vr, ex["v_new"], f"{label} V rows", emul=ref["v_new"], strict=strict)
    b = batch
    for step in range(decode_steps):
        b = b.advanced()
        cs.batch, cs.db = b, device_batch(b)
        cs.xb = make_x(cfg, b.n_tokens, seed, step=step)
        out, ws = cs.run(decode=True, x=to_device_bf16(cs.xb))
        x1, act, w = stage_parity(cs, ws, np.arange(b.n_tokens), label=f"{label} decode {step}")
        k, v = cs.cache
        w64 = {kk: f64(vv) for kk, vv in cs.wb.items()}
        args = (cfg, w64, to_host_f64(k), to_host_f64(v), b, f64(cs.xb))
        ref = oracle.layer_forward(*args, storage="bf16")
        assert_e2e(to_host_f64(out), oracle.layer_forward(*args)["out"],
                   f"{label} decode {step} out", emul=ref["out"], strict=strict)


def test_mrope_tiny_mixed_segments_then_decode():
    cfg = dataclasses.replace(layer_c1(), mrope_section=(8, 12, 12))
    batch = mrope_batch([2, 0, 1], [0, 37, 5], [
        [("text", 11), ("image", 6, 9), ("text", 20)],
        [("video", 3, 4, 4), ("text", 4)],
        [("text", 1)]])
    run_and_check(cfg, batch, 3, 256, "tiny mrope", seed=4, decode_steps=3)


def test_mrope_7b_shape_prefill_and_decode():
    cfg = dataclasses.replace(layer_7b(), mrope_section=(16, 24, 24))
    batch = mrope_batch([1, 0, 3, 2], [0, 64, 300, 7], [
        [("text", 30), ("image", 12, 16), ("text", 50)],
        [("image", 8, 8), ("video", 2, 6, 6)],
        [("text", 1)],
        [("text", 3), ("video", 4, 3, 5)]])
    run_and_check(cfg, batch, 4, 640, "7B mrope", seed=5, decode_steps=2)


def test_moe_layer_with_qk_norm_and_sections():
    """The Qwen3-Omni Thinker's kind of layer: MoE FFN, per-head q/k RMSNorm
    and multi-section positions together.  q and the written cache rows
    against the reference from the GPU's own normalised input, the MoE stages
    on identical inputs, then the end-to-end tolerance with the GPU's routes."""
    from oracle import layer as OL
    from paper_2606_29629_amd import _lib as T
    from test_gpu_layer import assert_rounded, ws_view
    from test_gpu_moe import TINY_MOE, MoECase, moe_stage_parity, routes_agree
    cfg = dataclasses.replace(TINY_MOE, qk_norm=True, mrope_section=(10, 11, 11))
    batch = mrope_batch([1, 0, 2], [0, 9, 30], [
        [("text", 5), ("image", 4, 6), ("text", 7)],
        [("video", 2, 3, 3)],
        [("text", 1)]])
    c = MoECase(cfg, batch, 3, 64, seed=8)
    Tn, H, D, Hq, Hkv = batch.n_tokens, cfg.hidden, cfg.head_dim, cfg.n_q_heads, cfg.n_kv_heads
    m = T.workspace_layout(c.dl.cfg, c.db)
    w = {k: f64(v) for k, v in c.wb.items()}
    h = to_host_f64(ws_view(c.ws, m.h, (Tn, H)))
    q = to_host_f64(ws_view(c.ws, m.q, (Tn, Hq, D)))
    hq = h @ w["w_qkv"].T
    ang = OL.rope_angles_sections(batch.pos3, D, cfg.rope_base, cfg.mrope_section)
    q_ref = OL.rope(OL.rmsnorm(hq[:, :Hq * D].reshape(Tn, Hq, D), w["q_norm"], cfg.rms_eps), ang)
    k_ref = OL.rope(OL.rmsnorm(hq[:, Hq * D:(Hq + Hkv) * D].reshape(Tn, Hkv, D), w["k_norm"],
                               cfg.rms_eps), ang)
    assert_rounded(q, q_ref, "moe q")
    k_cache = c.cache[0]
    kr = np.concatenate([to_host_f64(k_cache[s, :, ct:ct + ql]).transpose(1, 0, 2)
                         for s, ct, ql in zip(batch.slot, batch.ctx_len, batch.q_len)])
    assert_rounded(kr, k_ref, "moe k cache rows")
    moe_stage_parity(c, np.arange(Tn))
    args = (cfg, w, f64(c.kb), f64(c.vb), batch, f64(c.xb))
    ref = oracle.layer_forward(*args, storage="bf16")
    gi = c.idx.cpu().numpy()
    routes_agree(gi, ref["logits"], cfg.top_k, 2e-2)
    forced = oracle.layer_forward(*args, storage="bf16", forced_routes=gi)
    exact = oracle.layer_forward(*args, forced_routes=gi)
    assert_e2e(to_host_f64(c.out), exact["out"], "tiny moe qk-norm sections out",
               emul=forced["out"], strict=True)
