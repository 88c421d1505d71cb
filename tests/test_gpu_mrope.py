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
from test_gpu_layer import Case, assert_close, check_down, f64, stage_parity

pytestmark = pytest.mark.gpu


def run_and_check(cfg, batch, n_slots, max_seq, label, seed=0, decode_steps=0):
    cs = Case(cfg, batch, n_slots, max_seq, seed=seed)
    out, ws = cs.run()
    rows = np.arange(batch.n_tokens)
    x1, act, w = stage_parity(cs, ws, rows, label=label)
    check_down(cs, out, x1, act, w, rows, label)
    ref = cs.oracle()
    assert_close(to_host_f64(out), ref["out"], f"{label} out", exact=cs.oracle(storage=None)["out"])
    kr, vr = cs.cache_rows()
    assert_close(kr, ref["k_new"], f"{label} K rows")
    assert_close(vr, ref["v_new"], f"{label} V rows")
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
        assert_close(to_host_f64(out), ref["out"], f"{label} decode {step} out",
                     exact=oracle.layer_forward(*args)["out"])


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
