"""The layer at the limits of its configuration space (GPU, through the C ABI):
the largest query group (Hq / Hkv = 32) at both head sizes, the largest
hidden size (8192) on the short-batch (skinny, fused-norm) and the large-batch
GEMM paths, and the largest MoE routing (256 experts, top 16).  Same gates as
test_gpu_layer.py / test_gpu_moe.py: per-kernel parity on identical inputs
plus the end-to-end tolerance against the oracle."""
import numpy as np
import pytest

import oracle
from paper_2606_29629_amd.workload import to_host_f64
from synth import LayerConfig
from parity import strict_shape
from test_gpu_layer import B, Case, assert_e2e, check_down, f64, stage_parity
from test_gpu_moe import MoECase, moe_stage_parity, routes_agree

pytestmark = pytest.mark.gpu

WIDE = LayerConfig(hidden=8192, n_q_heads=64, n_kv_heads=2, head_dim=128, ffn_dim=128)
NARROW_HEADS = LayerConfig(hidden=512, n_q_heads=32, n_kv_heads=1, head_dim=64, ffn_dim=256)
MAX_MOE = LayerConfig(hidden=256, n_q_heads=4, n_kv_heads=2, head_dim=64, n_experts=256,
                      top_k=16, expert_ffn_dim=64)


def dense_case(cfg, batch, n_slots, max_seq, decode=False, seed=2):
    cs = Case(cfg, batch, n_slots, max_seq, seed=seed, x_step=0 if decode else None)
    out, ws = cs.run(decode=decode)
    rows = np.arange(batch.n_tokens)
    x1, act, w = stage_parity(cs, ws, rows, label=f"{cfg.hidden}/{cfg.n_q_heads}")
    check_down(cs, out, x1, act, w, rows, f"{cfg.hidden}/{cfg.n_q_heads}")
    ref = cs.oracle()
    assert_e2e(to_host_f64(out), cs.oracle(storage=None)["out"],
               f"H{cfg.hidden} G{cfg.n_q_heads // cfg.n_kv_heads} out", emul=ref["out"],
               strict=strict_shape(cfg))


@pytest.mark.parametrize("cfg", [WIDE, NARROW_HEADS], ids=["H8192_D128_G32", "H512_D64_G32"])
def test_group32_short_batch(cfg):
    # 104 tokens: skinny projections, the O projection's fused residual + norm
    dense_case(cfg, B([0, 1, 2], [0, 70, 5], [33, 1, 70]), 3, 256)


@pytest.mark.parametrize("cfg", [WIDE, NARROW_HEADS], ids=["H8192_D128_G32", "H512_D64_G32"])
def test_group32_decode(cfg):
    dense_case(cfg, B([0, 1, 2, 3], [0, 64, 130, 255], [1, 1, 1, 1]), 4, 320, decode=True)


def test_hidden8192_large_batch():
    # 200 tokens: 256 x 256 GEMM tiles with a ragged M tail at the largest width
    dense_case(WIDE, B([0, 1], [0, 40], [130, 70]), 2, 256)


@pytest.mark.parametrize("decode", [False, True])
def test_moe_256_experts_top16(decode):
    if decode:
        batch = B([0, 1, 2, 3, 4, 5], [5, 0, 17, 33, 2, 60], [1] * 6)
    else:
        batch = B([0, 1, 2], [0, 7, 0], [40, 9, 1])
    c = MoECase(MAX_MOE, batch, 6, 64, seed=6, decode=decode)
    moe_stage_parity(c, np.arange(batch.n_tokens))
    w64 = {k: f64(v) for k, v in c.wb.items()}
    args = (c.cfg, w64, f64(c.kb), f64(c.vb), batch, f64(c.xb))
    ref = oracle.layer_forward(*args, storage="bf16")
    gi = c.idx.cpu().numpy()
    routes_agree(gi, ref["logits"], c.cfg.top_k, 2e-2)
    forced = oracle.layer_forward(*args, storage="bf16", forced_routes=gi)
    exact = oracle.layer_forward(*args, forced_routes=gi)
    assert_e2e(to_host_f64(c.out), exact["out"], "max MoE out", emul=forced["out"],
               strict=strict_shape(c.cfg))
