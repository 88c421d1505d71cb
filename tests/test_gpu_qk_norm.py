"""The per-head q/k RMSNorm layer variant (the Qwen3-family attention block:
every head of q and of k normalised over head_dim with its own gains before
the rotation) on the GPU, through the C ABI.

The variant changes the q/k/v projection's epilogue only, which has three
implementations: the short-batch split-K reduction (<= 128 tokens), the
reduction of the split tail tiles of a large GEMM, and the large GEMM's own
tile epilogue (whole tiles: over one round of 256 tiles).  Each is covered,
at head_dim 64 and 128, with and without the q/k/v bias: per-kernel parity
on identical inputs (the q rows and every written cache row against the
reference computed from the GPU's own normalised input), then the
end-to-end tolerance against the oracle.
"""
import dataclasses

import numpy as np
import pytest

import oracle
from oracle import layer as OL
from paper_2606_29629_amd import _lib as T
from paper_2606_29629_amd.workload import to_host_f64
from synth import LayerConfig, layer_7b, layer_c1
from parity import strict_shape
from test_gpu_layer import (B, Case, assert_e2e, assert_rounded, check_down, f64,
                            stage_parity, ws_view)

pytestmark = pytest.mark.gpu


def qkn(cfg, bias=False):
    return dataclasses.replace(cfg, qk_norm=True, qkv_bias=bias)


# two layers whose q/k/v projection has more than one round of 256 x 256
# tiles at these batch sizes (whole tiles plus a split tail)
MID_D128 = LayerConfig(hidden=1024, n_q_heads=8, n_kv_heads=2, head_dim=128, ffn_dim=512)
MID_D64 = LayerConfig(hidden=512, n_q_heads=8, n_kv_heads=4, head_dim=64, ffn_dim=256)


def qkv_all_rows(cs, ws, label):
    """q (workspace) and the cache rows written, for every token, against
    h W^T (+ b) -> per-head RMSNorm -> rotation, h being the GPU's own."""
    cfg, b = cs.cfg, cs.batch
    m = T.workspace_layout(cs.dl.cfg, cs.db)
    Tn, H, D, Hq, Hkv = b.n_tokens, cfg.hidden, cfg.head_dim, cfg.n_q_heads, cfg.n_kv_heads
    h = to_host_f64(ws_view(ws, m.h, (Tn, H)))
    q = to_host_f64(ws_view(ws, m.q, (Tn, Hq, D)))
    w = {k: f64(v) for k, v in cs.wb.items()}
    hq = h @ w["w_qkv"].T
    if cfg.qkv_bias:
        hq = hq + w["b_qkv"]
    ang = OL.rope_angles(b.pos, D, cfg.rope_base)
    q_ref = OL.rope(OL.rmsnorm(hq[:, :Hq * D].reshape(Tn, Hq, D), w["q_norm"], cfg.rms_eps), ang)
    k_ref = OL.rope(OL.rmsnorm(hq[:, Hq * D:(Hq + Hkv) * D].reshape(Tn, Hkv, D), w["k_norm"],
                               cfg.rms_eps), ang)
    v_ref = hq[:, (Hq + Hkv) * D:].reshape(Tn, Hkv, D)
    assert_rounded(q, q_ref, f"{label} q (all rows)")
    kr, vr = cs.cache_rows()
    assert_rounded(kr, k_ref, f"{label} k cache rows (all)")
    assert_rounded(vr, v_ref, f"{label} v cache rows (all)")


def end_to_end(cs, out, s, local, label):
    """Oracle on sequence s alone (its cached prefix from the seeded cache),
    rows `local` of it, against the GPU output rows of that sequence."""
    b = cs.batch
    sl, c0, ql = int(b.slot[s]), int(b.ctx_len[s]), int(b.q_len[s])
    t0 = int(b.cu_q[s])
    sub = B([0], [c0], [ql])
    w = {k: f64(v) for k, v in cs.wb.items()}
    args = (cs.cfg, w, f64(cs.kb[[sl]]), f64(cs.vb[[sl]]), sub, f64(cs.xb[t0:t0 + ql]))
    ref = oracle.layer_forward(*args, rows=local, storage="bf16")
    ex = oracle.layer_forward(*args, rows=local)
    assert_e2e(to_host_f64(out)[t0 + np.asarray(local)], ex["out"], label, emul=ref["out"],
               strict=strict_shape(cs.cfg))


@pytest.mark.parametrize("bias", [False, True])
def test_tiny_ragged_mixed(bias):
    # 212 tokens: one GEMM tile column pair, all split tail tiles
    cfg = qkn(layer_c1(), bias)
    batch = B([3, 0, 2, 1, 4], [0, 40, 7, 0, 150], [200, 9, 1, 1, 1])
    cs = Case(cfg, batch, 5, 256, seed=3)
    out, ws = cs.run()
    qkv_all_rows(cs, ws, "tiny")
    rows = np.arange(batch.n_tokens)
    x1, act, w = stage_parity(cs, ws, rows, label="tiny qk-norm")
    check_down(cs, out, x1, act, w, rows, "tiny qk-norm")
    ex = cs.oracle(storage=None)
    assert_e2e(to_host_f64(out), ex["out"], f"tiny qk-norm out (bias {bias})", strict=True)
    kr, vr = cs.cache_rows()
    assert_e2e(kr, ex["k_new"], "tiny qk-norm K", strict=True)
    assert_e2e(vr, ex["v_new"], "tiny qk-norm V", strict=True)


@pytest.mark.parametrize("cfg", [qkn(layer_c1()), qkn(layer_7b(), True)], ids=["D64", "D128_bias"])
def test_short_batch_and_decode(cfg):
    # <= 128 tokens: split-K projections reduced by the split-K epilogue
    cs = Case(cfg, B([0, 1, 2], [0, 70, 5], [33, 1, 70]), 3, 256, seed=4)
    out, ws = cs.run()
    qkv_all_rows(cs, ws, "short")
    rows = np.arange(cs.batch.n_tokens)
    x1, act, w = stage_parity(cs, ws, rows, label="short qk-norm")
    check_down(cs, out, x1, act, w, rows, "short qk-norm")
    ref = cs.oracle()
    assert_e2e(to_host_f64(out), cs.oracle(storage=None)["out"], f"H{cfg.hidden} short qk-norm out",
               emul=ref["out"], strict=strict_shape(cfg))

    cs = Case(cfg, B([0, 1, 2, 3], [1, 64, 129, 250], [1, 1, 1, 1]), 4, 256, seed=5, x_step=0)
    out, ws = cs.run(decode=True)
    qkv_all_rows(cs, ws, "decode")
    rows = np.arange(4)
    x1, act, w = stage_parity(cs, ws, rows, label="decode qk-norm")
    check_down(cs, out, x1, act, w, rows, "decode qk-norm")
    ref = cs.oracle()
    assert_e2e(to_host_f64(out), cs.oracle(storage=None)["out"],
               f"H{cfg.hidden} decode qk-norm out", emul=ref["out"], strict=strict_shape(cfg))


def test_7b_ragged_prefill():
    # 494 tokens at the 7B shape: every tile is a split tail tile
    cfg = qkn(layer_7b())
    batch = B([0, 1, 2, 3], [0, 37, 500, 0], [300, 129, 1, 64])
    cs = Case(cfg, batch, 4, 640, seed=1)
    out, ws = cs.run()
    qkv_all_rows(cs, ws, "7B")
    rows = np.array([0, 1, 127, 128, 255, 256, 299, 300, 301, 365, 428, 429, 430, 460, 493])
    x1, act, w = stage_parity(cs, ws, rows, label="7B qk-norm")
    check_down(cs, out, x1, act, w, rows, "7B qk-norm")
    end_to_end(cs, out, 1, [0, 1, 64, 127, 128], "7B qk-norm rows")


@pytest.mark.parametrize("cfg,q_lens,ctx,max_seq", [
    # 48 row tiles x 6 column tiles = 288: 256 whole tiles + 32 split tail tiles
    (qkn(MID_D128), [2048] * 5 + [1900, 48], [0, 0, 0, 0, 0, 100, 7], 2112),
    # 65 row tiles x 4 column tiles = 260: 256 whole + 4 tail, with the bias
    (qkn(MID_D64, True), [4096] * 4 + [200], [0, 0, 0, 0, 37], 4160),
    # 64 row tiles x 6 column tiles = 384: 256 whole + 128 tail tiles run as
    # 128-row halves
    (qkn(MID_D128), [2048] * 8, [0] * 8, 2048),
    # 53 row tiles x 6 = 318: 62 tail tiles (four-way split at K = 1024) as halves
    (qkn(MID_D128), [2048] * 6 + [1280], [0] * 7, 2048),
], ids=["D128", "D64_bias", "D128_half_tail", "D128_half_tail4"])
def test_whole_tiles_and_tail(cfg, q_lens, ctx, max_seq):
    n = len(q_lens)
    batch = B(np.arange(n), ctx, q_lens)
    cs = Case(cfg, batch, n, max_seq, seed=7)
    out, ws = cs.run()
    qkv_all_rows(cs, ws, f"D{cfg.head_dim} tiles")
    Tn = batch.n_tokens
    rows = np.unique([r for r in (0, 31, 32, 255, 256, 4000, 8191, 8192, Tn // 2 + 17, 12300, 14000,
                                  Tn - 257, Tn - 2, Tn - 1) if r < Tn])
    x1, act, w = stage_parity(cs, ws, rows, label=f"D{cfg.head_dim} tiles")
    check_down(cs, out, x1, act, w, rows, f"D{cfg.head_dim} tiles")
    s = n - 1
    last = int(batch.q_len[s])
    end_to_end(cs, out, s, sorted({0, 1, last // 2, last - 1}), f"D{cfg.head_dim} tiles rows")
