"""GPU parity of the HIP decoder layer against the CPU oracle, through the C ABI.

The HIP path stores activations in bfloat16 between kernels and accumulates
in fp32 inside them.  Two gates, on the same seeded bf16 inputs:

1. Per-kernel parity on identical inputs (the tight gate).  Every stage's GPU
   output is compared with the oracle's definition of that stage evaluated in
   float64 on the GPU's own inputs to the stage (read back from the
   workspace) and rounded to bf16: each element must be that value or an
   adjacent bf16 value (<= 1 ulp; a flip is possible when the exact value lies
   within fp32 error of a rounding boundary), and at most 1% of elements may
   be the adjacent one.
2. End to end against the exact float64 oracle (tests/parity.py): at the tiny
   shapes every element within max(2e-2, 1e-2 |r|); at the 7B shapes the
   count of elements outside that bound and the largest error are held to
   those of the CPU bf16-storage emulation on the same rows (plus a stated
   margin); the normwise error of every row is also <= 1e-2.

Index results are bit-exact.  Sizes span several GEMM / attention tiles with
ragged tails; the full-size workloads are checked on sampled rows in the
launch configuration the bench times.
"""
import numpy as np
import pytest

import oracle
from oracle import layer as OL
from paper_2606_29629_amd import _lib as T
from paper_2606_29629_amd.workload import (DeviceLayer, device_batch, device_cache,
                                           to_device_bf16, to_host_f64)
from synth import (Batch, LayerConfig, bf16_to_f32, layer_7b, layer_c1, make_cache,
                   make_weights, make_x, to_bf16_bits, workload)
from parity import check_e2e

pytestmark = pytest.mark.gpu


def assert_e2e(got, exact, what, emul=None, strict=False, norm_rtol=1e-2):
    """End-to-end check against the exact oracle (tests/parity.py), plus the
    normwise error of every row."""
    got = np.asarray(got, np.float64)
    ex = np.asarray(exact, np.float64)
    if got.ndim >= 2:
        g2, e2 = got.reshape(got.shape[0], -1), ex.reshape(ex.shape[0], -1)
        nrm = np.linalg.norm(g2 - e2, axis=1) / np.maximum(np.linalg.norm(e2, axis=1), 1e-30)
        assert nrm.max() <= norm_rtol, f"{what}: row normwise error vs exact oracle {nrm.max():.3g}"
    check_e2e(got, ex, what, emul=emul, strict=strict)


def bf16_ordinal(a):
    """Monotone integer index of bf16 values (adjacent bf16 values differ by 1)."""
    b = to_bf16_bits(np.asarray(a, np.float32)).astype(np.int64)
    return np.where(b & 0x8000, -(b & 0x7FFF), b)


def assert_rounded(got, exact, what, max_flip_frac=0.01, abs_scale=None):
    """got (bf16 values) is the bf16 rounding of `exact` or an adjacent bf16 value.

    Elements within 1e-5 of the rms of `exact`, or within 2^-14 abs_scale
    (per element) of it, are exempt: a result that is small through
    cancellation carries the absolute error of its largest terms, and
    abs_scale states that scale (for attention, the attention of |V|: fp32
    sums and a 16-bit P bound the error by a few 2^-16 of it)."""
    got = np.asarray(got, np.float64)
    exact = np.asarray(exact, np.float64)
    assert got.shape == exact.shape, (what, got.shape, exact.shape)
    assert np.all(np.isfinite(got)), f"{what}: non-finite"
    d = np.abs(bf16_ordinal(got) - bf16_ordinal(OL.round_bf16(exact)))
    tiny = np.abs(got - exact) <= 1e-5 * np.sqrt(np.mean(exact ** 2))  # values near 0
    if abs_scale is not None:
        tiny |= np.abs(got - exact) <= 2.0 ** -14 * np.asarray(abs_scale, np.float64)
    bad = (d > 1) & ~tiny
    if bad.any():
        i = np.unravel_index(np.argmax(np.where(tiny, 0, d)), d.shape)
        raise AssertionError(f"{what}: {int(bad.sum())}/{d.size} elements > 1 ulp from the "
                             f"rounded exact value (worst {d[i]} ulps at {i}: gpu {got[i]:.6g} "
                             f"exact {exact[i]:.6g})")
    frac = np.mean((d == 1) & ~tiny)
    assert frac <= max_flip_frac, f"{what}: {frac:.3%} of elements one ulp off"


def f64(bits):
    return bf16_to_f32(bits).astype(np.float64)


class Case:
    """Seeded inputs of one layer call, resident on host (bits) and device."""

    def __init__(self, cfg, batch, n_slots, max_seq, seed=0, x_step=None):
        import torch
        self.cfg, self.batch = cfg, batch
        self.wb = make_weights(cfg, seed)
        self.kb, self.vb = make_cache(cfg, n_slots, max_seq, seed)
        self.xb = make_x(cfg, batch.n_tokens, seed, step=x_step)
        self.dl = DeviceLayer(cfg, self.wb)
        self.cache = device_cache(self.kb, self.vb)
        self.x = to_device_bf16(self.xb)
        self.db = device_batch(batch)
        torch.cuda.synchronize()

    def run(self, decode=False, x=None):
        import torch
        fn = T.layer_decode if decode else T.layer_prefill
        out, ws = fn(self.dl.cfg, self.dl.w, self.cache, self.db, self.x if x is None else x)
        torch.cuda.synchronize()
        return out, ws

    def oracle(self, rows=None, x_bits=None, storage="bf16"):
        w = {k: f64(v) for k, v in self.wb.items()}
        return oracle.layer_forward(self.cfg, w, f64(self.kb), f64(self.vb), self.batch,
                                    f64(self.xb if x_bits is None else x_bits), rows=rows,
                                    storage=storage)

    def cache_view(self):
        """The cache as contiguous (K, V) [n_slots, Hkv, max_seq, D] device tensors."""
        return self.cache

    def cache_rows(self):
        """GPU cache rows written by this call, as [T, Hkv, D] (K and V)."""
        k, v = self.cache_view()
        ks, vs = [], []
        for s, c, q in zip(self.batch.slot, self.batch.ctx_len, self.batch.q_len):
            ks.append(to_host_f64(k[s, :, c:c + q]).transpose(1, 0, 2))
            vs.append(to_host_f64(v[s, :, c:c + q]).transpose(1, 0, 2))
        return np.concatenate(ks), np.concatenate(vs)


def B(slot, ctx, q):
    return Batch(np.asarray(slot, np.int32), np.asarray(ctx, np.int32), np.asarray(q, np.int32))


def ws_view(ws, off, shape):
    import torch
    n = int(np.prod(shape))
    return ws[off:off + 2 * n].view(torch.bfloat16).view(*shape)


def stage_parity(cs, ws, rows, x_bits=None, label=""):
    """Per-kernel parity on identical inputs for the given token rows."""
    import torch
    cfg, b = cs.cfg, cs.batch
    m = T.workspace_layout(cs.dl.cfg, cs.db)
    Tn, H, D, Hq, Hkv = b.n_tokens, cfg.hidden, cfg.head_dim, cfg.n_q_heads, cfg.n_kv_heads
    F = cfg.ffn_dim
    rows = np.asarray(rows)
    ridx = torch.as_tensor(rows, device=ws.device)

    def rd(off, n, shape):
        return to_host_f64(ws_view(ws, off, (Tn, n))[ridx]).reshape(len(rows), *shape)

    h, q = rd(m.h, H, (H,)), rd(m.q, Hq * D, (Hq, D))
    attn, x1, h2 = rd(m.attn, Hq * D, (Hq * D,)), rd(m.x1, H, (H,)), rd(m.h2, H, (H,))
    act = rd(m.act, F, (F,))
    w = {k: f64(v) for k, v in cs.wb.items()}
    x = f64((cs.xb if x_bits is None else x_bits)[rows])
    # token -> (sequence, cache slot, cache row); only the slots involved are read back
    seq = np.searchsorted(b.cu_q, rows, side="right") - 1
    crow = b.ctx_len[seq] + rows - b.cu_q[seq]
    slots, sidx = np.unique(b.slot[seq], return_inverse=True)
    st = torch.as_tensor(slots, device=ws.device)
    kview, vview = cs.cache_view()
    kc, vc = to_host_f64(kview[st]), to_host_f64(vview[st])
    # RMSNorm
    assert_rounded(h, OL.rmsnorm(x, w["attn_norm"], cfg.rms_eps), f"{label} rmsnorm_attn")
    # q/k/v projection + rotary + cache write
    hq = h @ w["w_qkv"].T
    if "b_qkv" in w:
        hq = hq + w["b_qkv"]
    if getattr(cfg, "mrope_section", None):
        ang = OL.rope_angles_sections(b.pos3[:, rows], D, cfg.rope_base, cfg.mrope_section)
    else:
        ang = OL.rope_angles(b.pos[rows], D, cfg.rope_base)
    q_pre = hq[:, :Hq * D].reshape(-1, Hq, D)
    k_pre = hq[:, Hq * D:(Hq + Hkv) * D].reshape(-1, Hkv, D)
    if getattr(cfg, "qk_norm", False):
        q_pre = OL.rmsnorm(q_pre, w["q_norm"], cfg.rms_eps)
        k_pre = OL.rmsnorm(k_pre, w["k_norm"], cfg.rms_eps)
    assert_rounded(q, OL.rope(q_pre, ang), f"{label} q")
    k_ref = OL.rope(k_pre, ang)
    v_ref = hq[:, (Hq + Hkv) * D:].reshape(-1, Hkv, D)
    assert_rounded(kc[sidx, :, crow], k_ref, f"{label} k cache rows")
    assert_rounded(vc[sidx, :, crow], v_ref, f"{label} v cache rows")
    # attention over the GPU-written cache
    att_ref = np.stack([OL.attention(q[i:i + 1], kc[sidx[i], :, :crow[i] + 1],
                                     vc[sidx[i], :, :crow[i] + 1], np.array([crow[i]]))[0]
                        for i in range(len(rows))]).reshape(len(rows), Hq * D)
    att_abs = np.stack([OL.attention(q[i:i + 1], kc[sidx[i], :, :crow[i] + 1],
                                     np.abs(vc[sidx[i], :, :crow[i] + 1]), np.array([crow[i]]))[0]
                        for i in range(len(rows))]).reshape(len(rows), Hq * D)
    assert_rounded(attn, att_ref, f"{label} attention", abs_scale=att_abs)
    assert_rounded(x1, x + attn @ w["w_o"].T, f"{label} o_proj + residual")
    assert_rounded(h2, OL.rmsnorm(x1, w["mlp_norm"], cfg.rms_eps), f"{label} rmsnorm_mlp")
    g = h2 @ w["w_gate_up"][:F].T
    u = h2 @ w["w_gate_up"][F:].T
    assert_rounded(act, OL.silu(g) * u, f"{label} gate_up + SwiGLU")
    return x1, act, w


def check_down(cs, out, x1, act, w, rows, label=""):
    assert_rounded(to_host_f64(out)[np.asarray(rows)], x1 + act @ w["w_down"].T,
                   f"{label} down + residual")


# ------------------------------------------------------------- tiny layer --

def test_tiny_prefill_then_16_decode_steps():
    wl = workload("tiny")
    cs = Case(wl.cfg, wl.batch, wl.n_slots, wl.max_seq)
    out, _ = cs.run()
    ex = cs.oracle(storage=None)
    assert_e2e(to_host_f64(out), ex["out"], "tiny prefill out", strict=True)
    kr, vr = cs.cache_rows()
    assert_e2e(kr, ex["k_new"], "tiny prefill K rows", strict=True)
    assert_e2e(vr, ex["v_new"], "tiny prefill V rows", strict=True)
    # decode: fresh N(0,1) input each step, oracle fed the GPU-written cache
    batch = wl.batch
    for step in range(wl.decode_steps):
        batch = batch.advanced()
        cs.batch, cs.db = batch, device_batch(batch)
        xb = make_x(wl.cfg, batch.n_tokens, wl.seed, step=step)
        k, v = cs.cache
        w64 = {kk: f64(vv) for kk, vv in cs.wb.items()}
        ex = oracle.layer_forward(wl.cfg, w64, to_host_f64(k), to_host_f64(v), batch, f64(xb))
        out, _ = cs.run(decode=True, x=to_device_bf16(xb))
        assert_e2e(to_host_f64(out), ex["out"], f"tiny decode step {step}", strict=True)
        kr, vr = cs.cache_rows()
        assert_e2e(kr, ex["k_new"], f"tiny decode K row {step}", strict=True)
        assert_e2e(vr, ex["v_new"], f"tiny decode V row {step}", strict=True)


def test_tiny_intermediates():
    cfg = layer_c1()
    batch = B([0, 1], [0, 5], [37, 20])
    cs = Case(cfg, batch, 2, 64)
    out, ws = cs.run()
    ex = cs.oracle(storage=None)
    m = T.workspace_layout(cs.dl.cfg, cs.db)
    Tn, H, D, Hq = batch.n_tokens, cfg.hidden, cfg.head_dim, cfg.n_q_heads
    assert_e2e(to_host_f64(ws_view(ws, m.h, (Tn, H))), ex["h"], "tiny h", strict=True)
    assert_e2e(to_host_f64(ws_view(ws, m.q, (Tn, Hq, D))), ex["q"], "tiny q", strict=True)
    assert_e2e(to_host_f64(ws_view(ws, m.attn, (Tn, Hq * D))), ex["attn"], "tiny attn",
               strict=True)
    assert_e2e(to_host_f64(ws_view(ws, m.x1, (Tn, H))), ex["x1"], "tiny x1", strict=True)
    assert_e2e(to_host_f64(ws_view(ws, m.h2, (Tn, H))), ex["h2"], "tiny h2", strict=True)
    assert_e2e(to_host_f64(out), ex["out"], "tiny out", strict=True)
    rows = np.arange(batch.n_tokens)
    x1, act, w = stage_parity(cs, ws, rows, label="tiny")
    check_down(cs, out, x1, act, w, rows, "tiny")


@pytest.mark.parametrize("bias", [False, True])
def test_tiny_ragged_mixed_batch(bias):
    import dataclasses
    cfg = dataclasses.replace(layer_c1(), qkv_bias=bias)
    # a long prefill over two flash tiles, a chunk with cached prefix, decodes
    batch = B([3, 0, 2, 1, 4], [0, 40, 7, 0, 150], [200, 9, 1, 1, 1])
    cs = Case(cfg, batch, 5, 256, seed=3)
    out, ws = cs.run()
    rows = np.arange(batch.n_tokens)
    x1, act, w = stage_parity(cs, ws, rows, label="ragged")
    check_down(cs, out, x1, act, w, rows, "ragged")
    ex = cs.oracle(storage=None)
    assert_e2e(to_host_f64(out), ex["out"], f"tiny ragged out (bias {bias})", strict=True)
    kr, vr = cs.cache_rows()
    assert_e2e(kr, ex["k_new"], "tiny ragged K", strict=True)
    assert_e2e(vr, ex["v_new"], "tiny ragged V", strict=True)


@pytest.mark.parametrize("q_lens", [[150, 0, 1, 0, 70, 0], [40, 0, 1, 0, 30, 0]],
                         ids=["large", "short"])
def test_empty_sequences_in_a_ragged_batch(q_lens):
    # sequences with no new token inside and at the end of the batch (large:
    # the 256 x 256 GEMM path; short: the split-K path of <= 128 tokens)
    cfg = layer_c1()
    batch = B([3, 0, 2, 1, 4, 5], [0, 40, 7, 0, 150, 10], q_lens)
    cs = Case(cfg, batch, 6, 256, seed=9)
    out, ws = cs.run()
    ex = cs.oracle(storage=None)
    assert_e2e(to_host_f64(out), ex["out"], "tiny empty-seq out", strict=True)
    kr, vr = cs.cache_rows()
    assert_e2e(kr, ex["k_new"], "tiny empty-seq K", strict=True)
    assert_e2e(vr, ex["v_new"], "tiny empty-seq V", strict=True)
    # the empty sequences' slots are untouched, bit for bit
    k, v = cs.cache
    for s, q in zip(batch.slot, batch.q_len):
        if q == 0:
            assert np.array_equal(to_host_f64(k[s]), f64(cs.kb[s])), f"slot {s} K changed"
            assert np.array_equal(to_host_f64(v[s]), f64(cs.vb[s])), f"slot {s} V changed"


# --------------------------------------------------------- 7B layer shapes --

def test_7b_ragged_prefill_sampled_rows():
    cfg = layer_7b()
    # M = 494 (> the skinny threshold): big GEMM tiles with a ragged M tail,
    # flash tiles with ragged tails, a cached-prefix chunk and a decode sequence
    batch = B([0, 1, 2, 3], [0, 37, 500, 0], [300, 129, 1, 64])
    cs = Case(cfg, batch, 4, 640, seed=1)
    out, ws = cs.run()
    rows = np.array([0, 1, 127, 128, 255, 256, 299, 300, 301, 365, 428, 429, 430, 460, 493])
    x1, act, w = stage_parity(cs, ws, rows, label="7B ragged")
    check_down(cs, out, x1, act, w, rows, "7B ragged")
    ref = cs.oracle(rows=rows)
    ex = cs.oracle(rows=rows, storage=None)
    assert_e2e(to_host_f64(out)[rows], ex["out"], "7B ragged prefill rows", emul=ref["out"])
    kr, vr = cs.cache_rows()
    assert_e2e(kr, ex["k_new"], "7B K rows", emul=ref["k_new"])
    assert_e2e(vr, ex["v_new"], "7B V rows", emul=ref["v_new"])


@pytest.mark.parametrize("n_tok", [129, 257, 640, 641, 1025])
def test_7b_mid_size_prefill_gemm_paths(n_tok):
    """Batches of a few hundred tokens take the mid-size GEMM tiles (128 x 128
    with three stages for q/k/v and O, 128 x 256 for gate/up up to 640 rows),
    skip the row blocks past the last valid row, and split the down
    projection's K unevenly (1025 rows: three splits of 99, 99, 98 k-tiles).
    Sampled rows on both sides of every tile boundary and the last rows."""
    cfg = layer_7b()
    batch = B([0, 1], [0, 100], [n_tok - 7, 7])
    cs = Case(cfg, batch, 2, n_tok + 8, seed=7)
    out, ws = cs.run()
    rows = np.unique([r for r in (0, 1, 127, 128, 255, 256, 511, 512, 639, 640, 1023, 1024,
                                  n_tok - 8, n_tok - 7, n_tok - 2, n_tok - 1)
                     if 0 <= r < n_tok])
    x1, act, w = stage_parity(cs, ws, rows, label=f"7B T={n_tok}")
    check_down(cs, out, x1, act, w, rows, f"7B T={n_tok}")
    ref = cs.oracle(rows=rows)
    ex = cs.oracle(rows=rows, storage=None)
    assert_e2e(to_host_f64(out)[rows], ex["out"], f"7B T={n_tok} rows", emul=ref["out"])


def test_7b_decode_step_all_rows():
    cfg = layer_7b()
    ctx = [1, 63, 64, 127, 128, 129, 1000, 4095]
    batch = B(list(range(8)), ctx, [1] * 8)
    cs = Case(cfg, batch, 8, 4100, seed=2)
    out, ws = cs.run(decode=True)
    rows = np.arange(8)
    x1, act, w = stage_parity(cs, ws, rows, label="7B decode")
    check_down(cs, out, x1, act, w, rows, "7B decode")
    ref = cs.oracle()
    ex = cs.oracle(storage=None)
    assert_e2e(to_host_f64(out), ex["out"], "7B decode out", emul=ref["out"])
    kr, vr = cs.cache_rows()
    assert_e2e(kr, ex["k_new"], "7B decode K", emul=ref["k_new"])
    assert_e2e(vr, ex["v_new"], "7B decode V", emul=ref["v_new"])


def test_full_size_dense_prefill_sampled():
    """8 x 2048 tokens (the bench's prefill launch), rows sampled from one sequence."""
    wl = workload("dense_prefill")
    cs = Case(wl.cfg, wl.batch, wl.n_slots, wl.max_seq)
    out, ws = cs.run()
    # (rows 12300 and up lie in the projections' last-round tiles, which run
    # as 128-row halves)
    rows = np.array([0, 63, 64, 2047, 2048, 5 * 2048 + 1000, 12300, 14337, 15000, 16383])
    x1, act, w = stage_parity(cs, ws, rows, label="full prefill")
    check_down(cs, out, x1, act, w, rows, "full prefill")
    s = 5
    sub = B([s], [0], [2048])
    local = np.array([0, 1, 255, 256, 1023, 1024, 2046, 2047])
    w = {k: f64(v) for k, v in cs.wb.items()}
    args = (wl.cfg, w, f64(cs.kb), f64(cs.vb), sub, f64(cs.xb[s * 2048:(s + 1) * 2048]))
    ref = oracle.layer_forward(*args, rows=local, storage="bf16")
    ex = oracle.layer_forward(*args, rows=local)
    assert_e2e(to_host_f64(out)[s * 2048 + local], ex["out"], "full prefill sampled rows",
               emul=ref["out"])


def test_full_size_dense_decode_sampled():
    """64 sequences at KV 4096 (the decode launch), 6 sequences checked."""
    wl = workload("dense_decode")
    cs = Case(wl.cfg, wl.batch, wl.n_slots, wl.max_seq)
    out, ws = cs.run(decode=True)
    pick = np.array([0, 1, 17, 31, 62, 63])
    x1, act, w = stage_parity(cs, ws, pick, label="full decode")
    check_down(cs, out, x1, act, w, pick, "full decode")
    # the oracle sees only the picked slots' caches, renumbered 0..5
    sub = B(np.arange(len(pick)), wl.batch.ctx_len[pick], wl.batch.q_len[pick])
    w = {k: f64(v) for k, v in cs.wb.items()}
    args = (wl.cfg, w, f64(cs.kb[wl.batch.slot[pick]]), f64(cs.vb[wl.batch.slot[pick]]), sub,
            f64(cs.xb[pick]))
    ref = oracle.layer_forward(*args, storage="bf16")
    assert_e2e(to_host_f64(out)[pick], oracle.layer_forward(*args)["out"],
               "full decode sampled rows", emul=ref["out"])


# ------------------------------------------------------------- invariants --

def test_zero_projections_give_exact_identity():
    import torch
    cfg = layer_c1()
    batch = B([0, 1], [0, 3], [50, 1])
    cs = Case(cfg, batch, 2, 64)
    cs.dl.w["w_o"].zero_()
    cs.dl.w["w_down"].zero_()
    out, _ = cs.run()
    assert torch.equal(out, cs.x)


def test_first_query_returns_its_value_exactly():
    cfg = layer_7b()
    batch = B([0, 1], [0, 0], [130, 1])   # a flash-path prefill and a decode-path single token
    cs = Case(cfg, batch, 2, 256)
    out, ws = cs.run()
    m = T.workspace_layout(cs.dl.cfg, cs.db)
    attn = ws_view(ws, m.attn, (131, cfg.n_q_heads, cfg.head_dim))
    v = cs.cache[1]
    g = cfg.n_q_heads // cfg.n_kv_heads
    import torch
    for t, sl in ((0, 0), (130, 1)):
        for j in range(cfg.n_q_heads):
            assert torch.equal(attn[t, j], v[sl, j // g, 0]), (t, j)


def test_causal_invariance_bit_exact():
    import torch
    cfg = layer_c1()
    batch = B([0], [0], [150])
    cs = Case(cfg, batch, 1, 256)
    out0, _ = cs.run()
    out0 = out0.clone()
    x2 = cs.x.clone()
    x2[100:] = torch.randn_like(x2[100:].float()).to(torch.bfloat16) * 3
    out1, _ = cs.run(x=x2)
    assert torch.equal(out0[:100], out1[:100])
    assert not torch.equal(out0[100:], out1[100:])


def test_run_twice_bit_identical():
    import torch
    cfg = layer_7b()
    batch = B([0, 1, 2], [0, 100, 2000], [200, 1, 1])
    cs = Case(cfg, batch, 3, 2304)
    a, _ = cs.run()
    a = a.clone()
    b, _ = cs.run()
    assert torch.equal(a, b)


def test_decode_equals_recompute():
    cfg = layer_c1()
    n = 70
    full = Case(cfg, B([0], [0], [n + 1]), 1, 128, seed=5)
    ref_out, _ = full.run()
    ref_row = to_host_f64(ref_out)[n]
    # prefill n tokens, then decode token n from the cache the prefill wrote
    part = Case(cfg, B([0], [0], [n]), 1, 128, seed=5)
    part.x = full.x[:n].contiguous()
    part.run()
    part.batch = B([0], [n], [1])
    part.db = device_batch(part.batch)
    out, _ = part.run(decode=True, x=full.x[n:n + 1].contiguous())
    # both sides are the GPU: the strict bar against the recomputed row
    check_e2e(to_host_f64(out)[0], ref_row, "tiny decode vs recompute", strict=True)


def test_kvcache_append_and_canaries():
    import torch
    cfg = layer_c1()
    batch = B([2, 0], [5, 0], [3, 4])
    k = torch.full((3, cfg.n_kv_heads, 16, cfg.head_dim), 7.0, dtype=torch.bfloat16, device="cuda")
    v = k.clone()
    kn = torch.randn(7, cfg.n_kv_heads, cfg.head_dim, device="cuda").to(torch.bfloat16)
    vn = torch.randn_like(kn.float()).to(torch.bfloat16)
    T.kvcache_append(T.make_config(cfg), (k, v), device_batch(batch), kn, vn)
    torch.cuda.synchronize()
    ck, cv = oracle.kvcache_append(to_host_f64(k) * 0 + 7, to_host_f64(v) * 0 + 7, batch,
                                   to_host_f64(kn), to_host_f64(vn))
    assert np.array_equal(to_host_f64(k), ck)
    assert np.array_equal(to_host_f64(v), cv)


def test_output_buffer_canary():
    import torch
    cfg = layer_c1()
    batch = B([0], [0], [33])
    cs = Case(cfg, batch, 1, 64)
    big = torch.full((40, cfg.hidden), -3.0, dtype=torch.bfloat16, device="cuda")
    T.layer_prefill(cs.dl.cfg, cs.dl.w, cs.cache, cs.db, cs.x, out=big[:33])
    torch.cuda.synchronize()
    assert torch.all(big[33:] == -3.0)


def test_full_size_mixed_step_sampled():
    """One call: a 512-token chunk at ctx 6144 plus 32 decode sequences with KV
    lengths U[1024, 8192] (flash and split-KV paths in one launch sequence)."""
    wl = workload("mixed")
    cs = Case(wl.cfg, wl.batch, wl.n_slots, wl.max_seq)
    out, ws = cs.run()
    rows = np.array([0, 1, 255, 256, 511, 512, 513, 530, 543])
    x1, act, w = stage_parity(cs, ws, rows, label="mixed")
    check_down(cs, out, x1, act, w, rows, "mixed")
    # end to end for two decode sequences and the chunk's last rows
    pick = np.array([1, 7, 32])                      # sequences (0 = the chunk)
    sub = B(np.arange(3), wl.batch.ctx_len[pick], wl.batch.q_len[pick])
    w64 = {k: f64(v) for k, v in cs.wb.items()}
    tok = wl.batch.cu_q[pick]
    args = (wl.cfg, w64, f64(cs.kb[wl.batch.slot[pick]]), f64(cs.vb[wl.batch.slot[pick]]), sub,
            f64(cs.xb[tok]))
    ref = oracle.layer_forward(*args, storage="bf16")
    assert_e2e(to_host_f64(out)[tok], oracle.layer_forward(*args)["out"], "mixed decode rows",
               emul=ref["out"])
    chunk = B([0], [wl.batch.ctx_len[0]], [512])
    args = (wl.cfg, w64, f64(cs.kb[:1]), f64(cs.vb[:1]), chunk, f64(cs.xb[:512]))
    local = np.array([0, 300, 511])
    ref = oracle.layer_forward(*args, rows=local, storage="bf16")
    assert_e2e(to_host_f64(out)[local], oracle.layer_forward(*args, rows=local)["out"],
               "mixed chunk rows", emul=ref["out"])
