"""Pins of the CPU oracle against mathematics it must satisfy (no GPU).

Each test fixes the oracle to something other than itself: closed forms,
invariants, special cases that reduce to a textbook formula, and a naive
scalar brute force written separately.  The paper prints no worked example of
the layer, so there are no stored golden values (see tests/golden/README.md).
"""
import math

import numpy as np
import pytest

import oracle
from oracle import layer as L
from synth import Batch, LayerConfig, bf16_to_f32, make_cache, make_weights, make_x

TINY = LayerConfig(hidden=16, n_q_heads=4, n_kv_heads=2, head_dim=8, ffn_dim=24)
TINY_MOE = LayerConfig(hidden=16, n_q_heads=4, n_kv_heads=2, head_dim=8, n_experts=6, top_k=2,
                       expert_ffn_dim=12)


def widen(wb):
    return {k: bf16_to_f32(v).astype(np.float64) for k, v in wb.items()}


def setup(cfg, batch, n_slots, max_seq, seed=0, w_std=0.3):
    w = widen(make_weights(cfg, seed, w_std=w_std))
    ck, cv = (bf16_to_f32(a).astype(np.float64) for a in make_cache(cfg, n_slots, max_seq, seed))
    x = bf16_to_f32(make_x(cfg, batch.n_tokens, seed)).astype(np.float64)
    return w, ck, cv, x


def B(slot, ctx, q):
    return Batch(np.asarray(slot, np.int32), np.asarray(ctx, np.int32), np.asarray(q, np.int32))


# --------------------------------------------------------------- P1 RMSNorm --

def test_project_matches_scalar_sums():
    """y[i, j] = sum_k a[i, k] w[j, k], written out as scalar loops on a tiny
    integer case (exact in float64), and the identity weight."""
    rng = np.random.default_rng(5)
    a = rng.integers(-9, 10, (3, 5)).astype(np.float64)
    w = rng.integers(-9, 10, (4, 5)).astype(np.float64)
    y = L.project(a, w)
    assert y.shape == (3, 4)
    for i in range(3):
        for j in range(4):
            acc = 0.0
            for k in range(5):
                acc += a[i, k] * w[j, k]
            assert y[i, j] == acc
    assert np.array_equal(L.project(a, np.eye(5)), a)


def test_rmsnorm_constant_vector():
    H, c, eps = 64, 3.0, 1e-6
    g = np.linspace(0.5, 1.5, H)
    y = L.rmsnorm(np.full((1, H), c), g, eps)
    assert np.allclose(y[0], g * c / math.sqrt(c * c + eps), rtol=1e-15, atol=0)


def test_rmsnorm_one_hot():
    H, a, eps, j = 32, -2.5, 1e-6, 7
    g = np.linspace(0.9, 1.1, H)
    x = np.zeros((1, H))
    x[0, j] = a
    y = L.rmsnorm(x, g, eps)
    assert y[0, j] == pytest.approx(g[j] * a / math.sqrt(a * a / H + eps), rel=1e-15)
    assert np.count_nonzero(y) == 1


def test_rmsnorm_scale_invariant_without_eps():
    rng = np.random.default_rng(1)
    x = rng.standard_normal((5, 40))
    g = rng.standard_normal(40)
    assert np.allclose(L.rmsnorm(7.25 * x, g, 0.0), L.rmsnorm(x, g, 0.0), rtol=1e-14, atol=1e-15)


# -------------------------------------------------------------- P2 softmax --

def test_attention_weights_sum_to_one():
    """V with a constant-one column: that output column is the row sum of P."""
    rng = np.random.default_rng(2)
    n, hq, hkv, d, Lk = 6, 4, 2, 8, 9
    q = rng.standard_normal((n, hq, d))
    k = rng.standard_normal((hkv, Lk, d)) * 3
    v = rng.standard_normal((hkv, Lk, d))
    v[:, :, 0] = 1.0
    o = L.attention(q, k, v, np.arange(Lk - n, Lk))
    assert np.allclose(o[:, :, 0], 1.0, atol=1e-12)


def test_router_softmax_sums_to_one():
    rng = np.random.default_rng(3)
    p = L.softmax(rng.standard_normal((10, 128)) * 4)
    assert np.allclose(p.sum(-1), 1.0, atol=1e-12)
    assert np.all(p > 0)


# ------------------------------------------------------- P3 single key / equal keys --

def test_single_key_returns_value_exactly():
    cfg = TINY
    b = B([0], [0], [1])
    w, ck, cv, x = setup(cfg, b, 1, 4)
    r = L.layer_forward(cfg, w, ck, cv, b, x)
    group = cfg.n_q_heads // cfg.n_kv_heads
    for j in range(cfg.n_q_heads):
        got = r["attn"][0, j * cfg.head_dim:(j + 1) * cfg.head_dim]
        assert np.array_equal(got, r["v_new"][0, j // group])


def test_equal_keys_return_mean_value():
    rng = np.random.default_rng(4)
    Lk, d = 11, 8
    k = np.tile(rng.standard_normal((1, 1, d)), (1, Lk, 1))
    v = rng.standard_normal((1, Lk, d))
    q = rng.standard_normal((1, 1, d))
    o = L.attention(q, k, v, np.array([Lk - 1]))
    assert np.allclose(o[0, 0], v[0].mean(0), atol=1e-14)


# ---------------------------------------------------------- P4 causal mask --

def test_causal_invariance_bit_exact():
    cfg = TINY
    b = B([0, 1], [0, 3], [7, 5])
    w, ck, cv, x = setup(cfg, b, 2, 12)
    r0 = L.layer_forward(cfg, w, ck, cv, b, x)
    x2 = x.copy()
    x2[4:7] = np.random.default_rng(5).standard_normal((3, cfg.hidden)) * 5   # seq 0, tokens 4..6
    x2[10:12] = 9.0                                                          # seq 1, tokens 3..4
    r1 = L.layer_forward(cfg, w, ck, cv, b, x2)
    assert np.array_equal(r0["out"][:4], r1["out"][:4])
    assert np.array_equal(r0["out"][7:10], r1["out"][7:10])
    assert not np.allclose(r0["out"][4:7], r1["out"][4:7])


# ---------------------------------------------- P5 decode / chunk = recompute --

@pytest.mark.parametrize("cfg", [TINY, TINY_MOE])
def test_decode_with_cache_equals_recompute(cfg):
    n = 6
    full = B([0], [0], [n + 1])
    w, ck, cv, x = setup(cfg, full, 1, 8)
    ref = L.layer_forward(cfg, w, ck, cv, full, x)
    pre = L.layer_forward(cfg, w, ck, cv, B([0], [0], [n]), x[:n])
    ck2, cv2 = L.kvcache_append(ck, cv, B([0], [0], [n]), pre["k_new"], pre["v_new"])
    dec = L.layer_forward(cfg, w, ck2, cv2, B([0], [n], [1]), x[n:n + 1])
    assert np.allclose(dec["out"][0], ref["out"][n], rtol=1e-12, atol=1e-12)
    assert np.allclose(pre["out"], ref["out"][:n], rtol=1e-12, atol=1e-12)


def test_chunked_prefill_equals_recompute():
    cfg = TINY
    a, bb = 4, 9
    w, ck, cv, x = setup(cfg, B([0], [0], [bb]), 1, 12)
    ref = L.layer_forward(cfg, w, ck, cv, B([0], [0], [bb]), x)
    first = L.layer_forward(cfg, w, ck, cv, B([0], [0], [a]), x[:a])
    ck2, cv2 = L.kvcache_append(ck, cv, B([0], [0], [a]), first["k_new"], first["v_new"])
    second = L.layer_forward(cfg, w, ck2, cv2, B([0], [a], [bb - a]), x[a:])
    assert np.allclose(second["out"], ref["out"][a:], rtol=1e-12, atol=1e-12)


# ------------------------------------------------------------ P6 brute force --

def _lists(a):
    return np.asarray(a, dtype=np.float64).tolist()


@pytest.mark.parametrize("cfg,bias,qkn", [(TINY, False, False), (TINY, True, False),
                                          (TINY_MOE, False, False), (TINY, True, True),
                                          (TINY_MOE, False, True)])
def test_oracle_matches_brute_force(cfg, bias, qkn):
    import dataclasses
    cfg = dataclasses.replace(cfg, qkv_bias=bias, qk_norm=qkn)
    b = B([2, 0, 1], [3, 0, 5], [4, 3, 1])       # ragged: a chunk with prefix, a prefill, a decode
    w, ck, cv, x = setup(cfg, b, 3, 8)
    r = L.layer_forward(cfg, w, ck, cv, b, x)
    wl = {k: _lists(v) for k, v in w.items()}
    out, kr, vr, ridx, rw = oracle.layer_brute(cfg, wl, _lists(ck), _lists(cv), b.slot.tolist(),
                                               b.ctx_len.tolist(), b.q_len.tolist(), _lists(x))
    assert np.allclose(r["out"], np.array(out), rtol=1e-12, atol=1e-12)
    assert np.allclose(r["k_new"], np.array(kr), rtol=1e-12, atol=1e-12)
    assert np.allclose(r["v_new"], np.array(vr), rtol=1e-12, atol=1e-12)
    if cfg.n_experts:
        assert np.array_equal(r["route_idx"], np.array(ridx))
        assert np.allclose(r["route_w"], np.array(rw), rtol=1e-12)


def test_fp32_oracle_close_to_fp64():
    cfg = TINY_MOE
    b = B([0, 1], [2, 0], [5, 3])
    w, ck, cv, x = setup(cfg, b, 2, 8, w_std=0.1)
    r64 = L.layer_forward(cfg, w, ck, cv, b, x)
    r32 = L.layer_forward(cfg, w, ck, cv, b, x, dtype=np.float32)
    assert r32["out"].dtype == np.float32
    assert np.allclose(r32["out"], r64["out"], rtol=1e-5, atol=1e-5)


def test_row_subset_matches_full():
    cfg = TINY
    b = B([0, 1], [1, 0], [6, 4])
    w, ck, cv, x = setup(cfg, b, 2, 8)
    full = L.layer_forward(cfg, w, ck, cv, b, x)
    rows = np.array([0, 5, 7, 9])
    part = L.layer_forward(cfg, w, ck, cv, b, x, rows=rows)
    assert np.allclose(part["out"], full["out"][rows], rtol=1e-13, atol=1e-13)


# ------------------------------------------------------------------ P7 RoPE --

def test_rope_position_zero_is_identity():
    x = np.random.default_rng(6).standard_normal((1, 3, 16))
    assert np.array_equal(L.rope(x, L.rope_angles(np.array([0]), 16, 1e6)), x)


def test_rope_preserves_pair_norms_and_relative_phase():
    rng = np.random.default_rng(7)
    D = 16
    q = rng.standard_normal((1, 1, D))
    k = rng.standard_normal((1, 1, D))
    rq = L.rope(q, L.rope_angles(np.array([37]), D, 1e4))
    n0 = q[0, 0, :D // 2] ** 2 + q[0, 0, D // 2:] ** 2
    n1 = rq[0, 0, :D // 2] ** 2 + rq[0, 0, D // 2:] ** 2
    assert np.allclose(n0, n1, rtol=1e-13)
    dots = []
    for shift in (0, 100, 5000):
        a = L.rope(q, L.rope_angles(np.array([50 + shift]), D, 1e4))
        bq = L.rope(k, L.rope_angles(np.array([20 + shift]), D, 1e4))
        dots.append(float(np.sum(a * bq)))
    assert np.allclose(dots, dots[0], rtol=1e-10)


def test_rope_d2_is_plane_rotation():
    x = np.array([[[0.6, -1.3]]])
    p = 3
    y = L.rope(x, L.rope_angles(np.array([p]), 2, 1e6))
    c, s = math.cos(p), math.sin(p)
    assert np.allclose(y[0, 0], [0.6 * c + 1.3 * s, -1.3 * c + 0.6 * s], rtol=1e-15)


# ------------------------------------------------------------------- P8 GQA --

def test_gqa_equals_mha_with_duplicated_heads():
    import dataclasses
    gqa = TINY
    mha = dataclasses.replace(TINY, n_kv_heads=TINY.n_q_heads)
    b = B([0, 1], [3, 0], [4, 2])
    w, ck, cv, x = setup(gqa, b, 2, 8)
    D, Hq, Hkv = gqa.head_dim, gqa.n_q_heads, gqa.n_kv_heads
    grp = Hq // Hkv
    qkv = w["w_qkv"]
    wq, wk, wv = qkv[:Hq * D], qkv[Hq * D:(Hq + Hkv) * D], qkv[(Hq + Hkv) * D:]
    dup = lambda m: np.concatenate([m[(j // grp) * D:(j // grp + 1) * D] for j in range(Hq)])
    w2 = dict(w, w_qkv=np.concatenate([wq, dup(wk), dup(wv)]))
    ck2 = np.repeat(ck, grp, axis=1)
    cv2 = np.repeat(cv, grp, axis=1)
    r1 = L.layer_forward(gqa, w, ck, cv, b, x)
    r2 = L.layer_forward(mha, w2, ck2, cv2, b, x)
    assert np.array_equal(r1["attn"], r2["attn"])
    assert np.array_equal(r1["out"], r2["out"])


# -------------------------------------------------------- P9/P10 residual, SwiGLU --

def test_zero_projections_give_identity():
    cfg = TINY
    b = B([0], [2], [5])
    w, ck, cv, x = setup(cfg, b, 1, 8)
    w = dict(w, w_o=np.zeros_like(w["w_o"]), w_down=np.zeros_like(w["w_down"]))
    assert np.array_equal(L.layer_forward(cfg, w, ck, cv, b, x)["out"], x)


def test_silu_and_zero_up():
    assert L.silu(np.array([0.0]))[0] == 0.0
    assert L.silu(np.array([1.0]))[0] == pytest.approx(1.0 / (1.0 + math.exp(-1.0)), rel=1e-15)
    assert L.silu(np.array([-40.0]))[0] == pytest.approx(-40.0 * math.exp(-40.0), rel=1e-12)
    rng = np.random.default_rng(8)
    wgu = rng.standard_normal((20, 8))
    wgu[10:] = 0.0
    assert np.array_equal(L.swiglu(rng.standard_normal((3, 8)), wgu, rng.standard_normal((8, 10))),
                          np.zeros((3, 8)))


# ------------------------------------------------------------------ P11 MoE --

def test_moe_identical_experts_equal_dense():
    import dataclasses
    b = B([0], [0], [5])
    w, ck, cv, x = setup(TINY_MOE, b, 1, 8)
    E = TINY_MOE.n_experts
    w_moe = dict(w, w_gate_up=np.repeat(w["w_gate_up"][:1], E, 0), w_down=np.repeat(w["w_down"][:1], E, 0))
    dense = dataclasses.replace(TINY_MOE, n_experts=0, top_k=0, ffn_dim=TINY_MOE.expert_ffn_dim)
    w_dense = dict(w, w_gate_up=w["w_gate_up"][0], w_down=w["w_down"][0])
    w_dense.pop("w_router")
    r1 = L.layer_forward(TINY_MOE, w_moe, ck, cv, b, x)
    r2 = L.layer_forward(dense, w_dense, ck, cv, b, x)
    assert np.allclose(r1["out"], r2["out"], rtol=1e-12, atol=1e-12)


def test_moe_all_experts_is_full_softmax_mixture():
    import dataclasses
    cfg = dataclasses.replace(TINY_MOE, top_k=TINY_MOE.n_experts)
    b = B([0], [0], [3])
    w, ck, cv, x = setup(cfg, b, 1, 4)
    r = L.layer_forward(cfg, w, ck, cv, b, x)
    h2 = r["h2"]
    p = L.softmax(h2 @ w["w_router"].T)
    mix = sum(p[:, e:e + 1] * L.swiglu(h2, w["w_gate_up"][e], w["w_down"][e]) for e in range(cfg.n_experts))
    assert np.allclose(r["out"], r["x1"] + mix, rtol=1e-12, atol=1e-12)
    assert np.allclose(r["route_w"].sum(-1), 1.0)


# ------------------------------------------------------------------ P12 top-k --

def test_topk_matches_sorted_order_and_ties_go_low():
    rng = np.random.default_rng(9)
    logits = rng.standard_normal((50, 16))
    idx = L.topk_lower_index(logits, 5)
    for r in range(50):
        ref = sorted(range(16), key=lambda e: (-logits[r, e], e))[:5]
        assert idx[r].tolist() == ref
    tied = np.array([[0.5, 2.0, 2.0, -1.0, 2.0, 0.0]])
    assert L.topk_lower_index(tied, 3).tolist() == [[1, 2, 4]]


def test_duplicated_router_rows_pick_lower_expert():
    b = B([0], [0], [16])
    w, ck, cv, x = setup(TINY_MOE, b, 1, 16)
    wr = w["w_router"].copy()
    wr[4] = wr[1]                      # experts 1 and 4 tie on every token
    r = L.layer_forward(TINY_MOE, dict(w, w_router=wr), ck, cv, b, x)
    seen_pair = seen_single = 0
    for row in r["route_idx"].tolist():
        if 4 in row:                   # 4 may only be chosen after 1
            assert 1 in row and row.index(1) == row.index(4) - 1
            seen_pair += 1
        elif 1 in row:
            seen_single += 1
    assert seen_pair > 0


# ------------------------------------------------------- P13 token permutation --

@pytest.mark.parametrize("cfg", [TINY, TINY_MOE])
def test_token_permutation_permutes_outputs(cfg):
    n = 5
    b = B(list(range(n)), [2, 0, 4, 1, 3], [1] * n)
    w, ck, cv, x = setup(cfg, b, n, 8)
    r = L.layer_forward(cfg, w, ck, cv, b, x)
    perm = np.array([3, 0, 4, 2, 1])
    bp = B(b.slot[perm], b.ctx_len[perm], b.q_len[perm])
    rp = L.layer_forward(cfg, w, ck, cv, bp, x[perm])
    assert np.allclose(rp["out"], r["out"][perm], rtol=1e-13, atol=1e-13)
    if cfg.n_experts:
        assert np.array_equal(rp["route_idx"], r["route_idx"][perm])


def test_kvcache_append_rows():
    cfg = TINY
    b = B([1, 0], [2, 5], [3, 1])
    ck = np.zeros((2, 2, 8, 8))
    kn = np.arange(4 * 2 * 8, dtype=np.float64).reshape(4, 2, 8) + 1
    ck2, _ = L.kvcache_append(ck, ck, b, kn, kn)
    assert np.array_equal(ck2[1, :, 2:5], kn[:3].transpose(1, 0, 2))
    assert np.array_equal(ck2[0, :, 5], kn[3])
    assert np.count_nonzero(ck2) == kn.size


# ------------------------------------------------------- bf16 storage reading --

def test_round_bf16_ties_to_even_and_matches_bit_rounding():
    assert L.round_bf16(np.array([1.0 + 2.0 ** -8]))[0] == 1.0                     # tie -> even
    assert L.round_bf16(np.array([1.0 + 3 * 2.0 ** -8]))[0] == 1.0 + 2.0 ** -6      # tie -> even
    assert L.round_bf16(np.array([1.0 + 2.0 ** -8 + 2.0 ** -20]))[0] == 1.0 + 2.0 ** -7
    assert L.round_bf16(np.array([-0.0, 0.0, 2.0 ** -130])).tolist() == [-0.0, 0.0, 2.0 ** -130]
    from synth import to_bf16_bits
    v = (np.random.default_rng(11).standard_normal(100000) *
         np.exp(np.random.default_rng(12).uniform(-20, 20, 100000))).astype(np.float32)
    assert np.array_equal(L.round_bf16(v.astype(np.float64)), bf16_to_f32(to_bf16_bits(v)).astype(np.float64))


def test_bf16_storage_rounds_exactly_the_declared_points():
    cfg = TINY
    b = B([0, 1], [2, 0], [5, 3])
    w, ck, cv, x = setup(cfg, b, 2, 8)
    r = L.layer_forward(cfg, w, ck, cv, b, x, storage="bf16")
    for k in ("h", "q", "k_new", "v_new", "attn", "x1", "h2", "out"):
        assert np.array_equal(L.round_bf16(r[k]), r[k]), k
    exact = L.layer_forward(cfg, w, ck, cv, b, x)
    assert np.allclose(r["out"], exact["out"], rtol=3e-2, atol=3e-2)
    assert not np.array_equal(r["out"], exact["out"])


@pytest.mark.parametrize("cfg", [TINY, TINY_MOE])
def test_bf16_storage_matches_brute_force_with_bit_rounding(cfg):
    """The storage points of the vectorised oracle agree with the brute force
    given an independent (bit-pattern) bf16 rounding."""
    import struct
    from synth import to_bf16_bits

    def bit_round(v):
        f32 = np.float32(struct.unpack("f", struct.pack("f", v))[0])  # nearest fp32 first
        return float(bf16_to_f32(to_bf16_bits(np.array([f32])))[0])

    b = B([1, 0], [3, 0], [3, 4])
    w, ck, cv, x = setup(cfg, b, 2, 8)
    r = L.layer_forward(cfg, w, ck, cv, b, x, storage="bf16")
    wl = {k: _lists(v) for k, v in w.items()}
    out, kr, vr, ridx, rw = oracle.layer_brute(cfg, wl, _lists(ck), _lists(cv), b.slot.tolist(),
                                               b.ctx_len.tolist(), b.q_len.tolist(), _lists(x),
                                               store=bit_round)
    assert np.allclose(r["k_new"], np.array(kr), rtol=1e-12, atol=1e-12)
    assert np.allclose(r["out"], np.array(out), rtol=1e-12, atol=1e-12)


# ------------------------------------------------------------ q/k norm variant --

def test_qk_norm_unit_gains_give_unit_rms_heads():
    """With unit gains and eps = 0 every head of q and k has RMS exactly 1
    before the rotation, hence after it (the rotation preserves pair norms)."""
    import dataclasses
    cfg = dataclasses.replace(TINY, qk_norm=True, rms_eps=0.0)
    b = B([0, 1], [2, 0], [3, 4])
    w, ck, cv, x = setup(cfg, b, 2, 8)
    w["q_norm"] = np.ones(cfg.head_dim)
    w["k_norm"] = np.ones(cfg.head_dim)
    r = L.layer_forward(cfg, w, ck, cv, b, x)
    assert np.allclose(np.mean(r["q"] ** 2, axis=-1), 1.0, rtol=1e-13)
    assert np.allclose(np.mean(r["k_new"] ** 2, axis=-1), 1.0, rtol=1e-13)


def test_qk_norm_makes_the_layer_invariant_to_query_and_key_scale():
    """Scaling the q (or k) rows of W_qkv by a positive factor per head leaves
    the layer unchanged with eps = 0; without the norm it does not."""
    import dataclasses
    b = B([0, 1], [0, 0], [5, 3])
    for qkn in (True, False):
        cfg = dataclasses.replace(TINY, qk_norm=qkn, rms_eps=0.0)
        w, ck, cv, x = setup(cfg, b, 2, 8)
        ck[:] = 0.0
        cv[:] = 0.0   # no cached prefix: every key comes from the scaled projection
        r0 = L.layer_forward(cfg, w, ck, cv, b, x)
        w2 = dict(w)
        w2["w_qkv"] = w["w_qkv"].copy()
        D, Hq, Hkv = cfg.head_dim, cfg.n_q_heads, cfg.n_kv_heads
        for j, a in enumerate([0.5, 3.0, 1.7, 0.9]):           # q heads
            w2["w_qkv"][j * D:(j + 1) * D] *= a
        for j, a in enumerate([2.5, 0.4]):                     # k heads
            w2["w_qkv"][(Hq + j) * D:(Hq + j + 1) * D] *= a
        r1 = L.layer_forward(cfg, w2, ck, cv, b, x)
        same = np.allclose(r1["out"], r0["out"], rtol=1e-12, atol=1e-12)
        assert same == qkn


# ----------------------------------------------- multi-section rotary positions --

def test_mrope_angles_hand_computed():
    """D = 8 (four frequencies), base 100, sections (1, 2, 1), ids (t, h, w) =
    (2, 5, 7): inverse frequencies 100^(-i/4) = 1, 10^-0.5, 0.1, 10^-1.5, so
    the angles are 2 * 1, 5 * 10^-0.5, 5 * 0.1 and 7 * 10^-1.5."""
    ang = L.rope_angles_sections(np.array([[2], [5], [7]]), 8, 100.0, (1, 2, 1))
    want = [2.0, 1.5811388300841898, 0.5, 0.22135943621178655]
    assert np.allclose(ang[0], want, rtol=1e-15, atol=0)


def test_mrope_equal_ids_is_the_one_dimensional_layer():
    """Three equal ids per token reduce the embedding to the 1-D one: the
    layer output is bit-identical for any sections."""
    import dataclasses
    from synth import mrope_positions
    b = B([1, 0], [3, 0], [4, 5])
    pos = b.pos
    b3 = Batch(b.slot, b.ctx_len, b.q_len, np.stack([pos, pos, pos]))
    for sec in [(1, 2, 1), (4, 0, 0), (0, 0, 4), (2, 1, 1)]:
        cfg = dataclasses.replace(TINY, mrope_section=sec)
        w, ck, cv, x = setup(cfg, b, 2, 12)
        r0 = L.layer_forward(TINY, w, ck, cv, b, x)
        r1 = L.layer_forward(cfg, w, ck, cv, b3, x)
        assert np.array_equal(r0["out"], r1["out"]) and np.array_equal(r0["k_new"], r1["k_new"])
    # text segments of the position generator are equal ids
    p3, nxt = mrope_positions([("text", 5)], 7)
    assert np.array_equal(p3, np.tile(np.arange(7, 12), (3, 1))) and nxt == 12


def test_mrope_single_section_ignores_the_other_ids():
    """Sections (D/2, 0, 0): only the temporal id matters."""
    import dataclasses
    rng = np.random.default_rng(3)
    b = B([0], [0], [6])
    t = np.array([0, 0, 1, 1, 4, 9], np.int32)
    b3 = Batch(b.slot, b.ctx_len, b.q_len, np.stack([t, rng.integers(0, 50, 6),
                                                     rng.integers(0, 50, 6)]).astype(np.int32))
    bt = Batch(b.slot, b.ctx_len, b.q_len, np.stack([t, t, t]))
    cfg = dataclasses.replace(TINY, mrope_section=(4, 0, 0))
    w, ck, cv, x = setup(cfg, b, 1, 8)
    r0 = L.layer_forward(cfg, w, ck, cv, bt, x)
    r1 = L.layer_forward(cfg, w, ck, cv, b3, x)
    assert np.array_equal(r0["out"], r1["out"])


def test_mrope_scores_depend_on_per_section_differences_only():
    """Shifting every token's temporal, height and width ids by three
    different constants leaves a fresh prefill unchanged: q.k after the
    rotation depends only on the ids' differences, section by section."""
    import dataclasses
    from synth import mrope_batch
    b = mrope_batch([0, 1], [0, 0], [[("text", 3), ("image", 2, 3), ("text", 2)],
                                     [("video", 2, 2, 2), ("text", 1)]])
    cfg = dataclasses.replace(TINY, mrope_section=(1, 2, 1))
    w, ck, cv, x = setup(cfg, b, 2, 16)
    r0 = L.layer_forward(cfg, w, ck, cv, b, x)
    shifted = Batch(b.slot, b.ctx_len, b.q_len, b.pos3 + np.array([[5], [11], [2]], np.int32))
    r1 = L.layer_forward(cfg, w, ck, cv, shifted, x)
    assert np.allclose(r0["out"], r1["out"], rtol=1e-10, atol=1e-10)
    assert not np.allclose(r0["k_new"], r1["k_new"])       # the keys themselves moved
    # a shift of one section only, by different amounts per token, changes it
    moved = Batch(b.slot, b.ctx_len, b.q_len,
                  b.pos3 + np.array([[0], [1], [0]], np.int32) * np.arange(b.n_tokens)[None, :])
    r2 = L.layer_forward(cfg, w, ck, cv, moved, x)
    assert not np.allclose(r0["out"], r2["out"], rtol=1e-6, atol=1e-6)


@pytest.mark.parametrize("sec", [(1, 2, 1), (0, 3, 1), (2, 0, 2)])
def test_mrope_oracle_matches_brute_force(sec):
    import dataclasses
    from synth import mrope_batch
    b = mrope_batch([1, 0], [2, 0], [[("image", 2, 2), ("text", 1)], [("video", 2, 1, 2)]])
    cfg = dataclasses.replace(TINY, mrope_section=sec)
    w, ck, cv, x = setup(cfg, b, 2, 10)
    r = L.layer_forward(cfg, w, ck, cv, b, x)
    wl = {k: _lists(v) for k, v in w.items()}
    out, kr, vr, _, _ = oracle.layer_brute(cfg, wl, _lists(ck), _lists(cv), b.slot.tolist(),
                                           b.ctx_len.tolist(), b.q_len.tolist(), _lists(x),
                                           pos3=b.pos3.T.tolist())
    assert np.allclose(r["k_new"], np.array(kr), rtol=1e-12, atol=1e-12)
    assert np.allclose(r["out"], np.array(out), rtol=1e-12, atol=1e-12)
