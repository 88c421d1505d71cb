"""The Talker-shaped layer on the GPU, through the C ABI.

The paper's Talker (Section II-A) is an autoregressive transformer decoder
that turns the Thinker's output into speech-codec tokens; the paper gives no
shapes, and the reading here is a 0.5B-class dense decoder of the same family
(hidden 896, 14 query / 2 KV heads of 64, SwiGLU 4864): a second workload for
the same kernels at a narrow width.  Gates as in test_gpu_layer.py:
per-kernel parity on identical inputs and the end-to-end bar against the
exact oracle, at the bench's prefill launch (8 x 512) and its decode launch
(64 streams at KV 1024) over several steps.
"""
import numpy as np
import pytest

import oracle
from paper_2606_29629_amd.workload import device_batch, to_device_bf16, to_host_f64
from synth import Batch, make_x, workload
from test_gpu_layer import Case, assert_e2e, check_down, f64, stage_parity

pytestmark = pytest.mark.gpu


def B(slot, ctx, q):
    return Batch(np.asarray(slot, np.int32), np.asarray(ctx, np.int32), np.asarray(q, np.int32))


def test_talker_prefill_sampled():
    wl = workload("talker_prefill")
    cs = Case(wl.cfg, wl.batch, wl.n_slots, wl.max_seq)
    out, ws = cs.run()
    rows = np.array([0, 1, 63, 64, 511, 512, 3 * 512 + 200, 4095])
    x1, act, w = stage_parity(cs, ws, rows, label="talker prefill")
    check_down(cs, out, x1, act, w, rows, "talker prefill")
    s = 3
    sub = B([s], [0], [512])
    local = np.array([0, 1, 127, 128, 200, 511])
    args = (wl.cfg, w, f64(cs.kb), f64(cs.vb), sub, f64(cs.xb[s * 512:(s + 1) * 512]))
    ex = oracle.layer_forward(*args, rows=local)
    emul = oracle.layer_forward(*args, rows=local, storage="bf16")
    assert_e2e(to_host_f64(out)[s * 512 + local], ex["out"], "talker prefill rows",
               emul=emul["out"])


def test_talker_decode_steps():
    """Three decode steps of the 64-stream launch, each checked against the
    oracle over the cache the previous steps wrote."""
    wl = workload("talker_decode")
    cs = Case(wl.cfg, wl.batch, wl.n_slots, wl.max_seq, x_step=0)
    b = wl.batch
    pick = np.array([0, 9, 33, 63])
    for step in range(3):
        if step:
            b = b.advanced()
            cs.batch, cs.db = b, device_batch(b)
            cs.xb = make_x(wl.cfg, b.n_tokens, wl.seed, step=step)
        k, v = cs.cache
        kb, vb = to_host_f64(k[pick]), to_host_f64(v[pick])   # cache before this step
        out, ws = cs.run(decode=True, x=to_device_bf16(cs.xb))
        label = f"talker decode {step}"
        x1, act, w = stage_parity(cs, ws, pick, label=label)
        check_down(cs, out, x1, act, w, pick, label)
        sub = B(np.arange(len(pick)), b.ctx_len[pick], b.q_len[pick])
        args = (wl.cfg, w, kb, vb, sub, f64(cs.xb[pick]))
        ex = oracle.layer_forward(*args)
        emul = oracle.layer_forward(*args, storage="bf16")
        assert_e2e(to_host_f64(out)[pick], ex["out"], f"{label} rows", emul=emul["out"])
