"""GPU parity of the mixture-of-experts layer (router, permutation, grouped
expert GEMMs, combine) against the CPU oracle, through the C ABI.

Routing protocol (top-k is decided by floating-point comparisons):
* on identical fp32 router inputs (tri_moe_route), the expert indices are
  bit-exact except where two experts at adjacent ranks have fp64 logits within
  1e-5 of each other (fp32 accumulation order may swap such near-ties);
* inside the layer the router reads the GPU's bf16 h2; each token's experts are
  compared with the oracle's routing of that same h2 under the same rule, and
  the layer output is compared with the oracle run with the GPU's routes
  (forced_routes), so near-tie swaps cannot hide an arithmetic error.
"""
import dataclasses

import numpy as np
import pytest

import oracle
from oracle import layer as OL
from paper_2606_29629_amd import _lib as T
from paper_2606_29629_amd.workload import (DeviceLayer, device_batch, device_cache,
                                           to_device_bf16, to_host_f64)
from synth import Batch, LayerConfig, bf16_to_f32, make_cache, make_weights, make_x, workload
from parity import strict_shape
from test_gpu_layer import B, assert_e2e, assert_rounded, f64, ws_view

pytestmark = pytest.mark.gpu

TINY_MOE = LayerConfig(hidden=256, n_q_heads=4, n_kv_heads=2, head_dim=64, n_experts=8, top_k=2,
                       expert_ffn_dim=128)


def routes_agree(gpu_idx, logits64, k, tau):
    """gpu_idx [T, k] must be the top-k of logits64 (desc, ties low) except for
    swaps among experts whose logits lie within tau of the k-th boundary or of
    each other.  Returns the number of tokens that needed the tie allowance."""
    ref = OL.topk_lower_index(logits64, k)
    n_tie = 0
    for t in range(gpu_idx.shape[0]):
        if np.array_equal(gpu_idx[t], ref[t]):
            continue
        n_tie += 1
        g, r = gpu_idx[t], ref[t]
        assert len(set(g.tolist())) == k, (t, g)
        # every chosen expert must be within tau of the reference value at its rank
        lg = logits64[t]
        assert np.all(np.abs(lg[g] - lg[r]) <= tau), (t, g, r, lg[g], lg[r])
    return n_tie


def test_router_bit_exact_on_identical_fp32_input():
    import torch
    cfg = dataclasses.replace(workload("moe_prefill").cfg)
    Tn = 1024
    rng = np.random.default_rng(21)
    h = rng.standard_normal((Tn, cfg.hidden)).astype(np.float32)
    wr = make_weights(cfg, 0)["w_router"]
    idx = torch.empty(Tn, cfg.top_k, dtype=torch.int32, device="cuda")
    w = torch.empty(Tn, cfg.top_k, dtype=torch.float32, device="cuda")
    T.moe_route(T.make_config(cfg), torch.from_numpy(h).cuda(), to_device_bf16(wr), idx, w)
    torch.cuda.synchronize()
    logits = h.astype(np.float64) @ f64(wr).T
    n_tie = routes_agree(idx.cpu().numpy(), logits, cfg.top_k, 1e-5)
    assert n_tie <= 3, n_tie
    p = OL.softmax(logits)
    gi = idx.cpu().numpy().astype(np.int64)
    ref_w = np.take_along_axis(p, gi, 1)
    ref_w = ref_w / ref_w.sum(1, keepdims=True)
    assert np.allclose(w.cpu().numpy(), ref_w, rtol=1e-5, atol=1e-7)


def test_router_exact_ties_pick_lower_index():
    import torch
    cfg = dataclasses.replace(TINY_MOE, top_k=3)
    wr = make_weights(cfg, 0)["w_router"].copy()
    wr[5] = wr[2]                       # experts 2 and 5 always tie exactly
    h = np.random.default_rng(3).standard_normal((64, cfg.hidden)).astype(np.float32)
    idx = torch.empty(64, 3, dtype=torch.int32, device="cuda")
    w = torch.empty(64, 3, dtype=torch.float32, device="cuda")
    T.moe_route(T.make_config(cfg), torch.from_numpy(h).cuda(), to_device_bf16(wr), idx, w)
    torch.cuda.synchronize()
    for row in idx.cpu().numpy().tolist():
        if 5 in row:
            assert 2 in row and row.index(2) == row.index(5) - 1, row


class MoECase:
    def __init__(self, cfg, batch, n_slots, max_seq, seed=0, decode=False):
        import torch
        self.cfg, self.batch, self.decode = cfg, batch, decode
        self.wb = make_weights(cfg, seed)
        self.kb, self.vb = make_cache(cfg, n_slots, max_seq, seed)
        self.xb = make_x(cfg, batch.n_tokens, seed)
        self.dl = DeviceLayer(cfg, self.wb)
        self.cache = device_cache(self.kb, self.vb)
        self.db = device_batch(batch)
        k = cfg.top_k
        self.idx = torch.empty(batch.n_tokens, k, dtype=torch.int32, device="cuda")
        self.w = torch.empty(batch.n_tokens, k, dtype=torch.float32, device="cuda")
        fn = T.layer_decode if decode else T.layer_prefill
        self.out, self.ws = fn(self.dl.cfg, self.dl.w, self.cache, self.db, to_device_bf16(self.xb),
                               route_idx=self.idx, route_w=self.w)
        torch.cuda.synchronize()


def moe_stage_parity(c, rows):
    """Router, expert gate/up, expert down and combine on identical inputs."""
    import torch
    cfg, b = c.cfg, c.batch
    m = T.workspace_layout(c.dl.cfg, c.db)
    Tn, H, k, Fe = b.n_tokens, cfg.hidden, cfg.top_k, cfg.expert_ffn_dim
    P = Tn * k
    w = {kk: f64(v) for kk, v in c.wb.items()}
    h2 = to_host_f64(ws_view(c.ws, m.h2, (Tn, H)))
    x1 = to_host_f64(ws_view(c.ws, m.x1, (Tn, H)))
    idx = c.idx.cpu().numpy().astype(np.int64)
    gw = c.w.cpu().numpy().astype(np.float64)
    # router on the GPU's own h2
    logits = h2 @ w["w_router"].T
    routes_agree(idx, logits, k, 1e-5)
    p = OL.softmax(logits)
    ref_w = np.take_along_axis(p, idx, 1)
    ref_w = ref_w / ref_w.sum(1, keepdims=True)
    assert np.allclose(gw, ref_w, rtol=1e-5, atol=1e-7), "routing weights"
    # permutation: grouped by expert, ascending pair id within an expert
    perm = c.ws[m.perm:m.perm + 4 * P].view(torch.int32).cpu().numpy().astype(np.int64)
    flat = idx.reshape(-1)
    assert np.array_equal(np.sort(perm), np.arange(P)), "perm is not a permutation"
    assert np.array_equal(perm, np.lexsort((np.arange(P), flat))), "routed order"
    # expert FFN rows for the sampled tokens
    pos_of = np.empty(P, np.int64)
    pos_of[perm] = np.arange(P)
    act = ws_view(c.ws, m.act, (P, Fe))
    y = c.ws[m.y:m.y + 4 * P * H].view(torch.float32).view(P, H)
    sel = np.array([pos_of[t * k + j] for t in rows for j in range(k)])
    st = torch.as_tensor(sel, device="cuda")
    act_g = to_host_f64(act[st])
    y_g = y[st].double().cpu().numpy()
    ex = flat[perm[sel]]
    tok = perm[sel] // k
    g_ref = np.stack([h2[t] @ w["w_gate_up"][e, :Fe].T for t, e in zip(tok, ex)])
    u_ref = np.stack([h2[t] @ w["w_gate_up"][e, Fe:].T for t, e in zip(tok, ex)])
    assert_rounded(act_g, OL.silu(g_ref) * u_ref, "expert gate/up + SwiGLU")
    y_ref = np.stack([act_g[i] @ w["w_down"][e].T for i, e in enumerate(ex)])
    scale = np.sqrt(np.mean(y_ref ** 2))
    assert np.max(np.abs(y_g - y_ref)) <= 2e-5 * scale, "expert down (fp32 output)"
    # combine
    out_ref = np.stack([x1[t] + sum(gw[t, j] * y[pos_of[t * k + j]].double().cpu().numpy()
                                    for j in range(k)) for t in rows])
    assert_rounded(to_host_f64(c.out)[rows], out_ref, "combine + residual")


@pytest.mark.parametrize("decode", [False, True])
def test_tiny_moe_layer(decode):
    if decode:
        batch = B([0, 1, 2, 3, 4], [5, 0, 17, 33, 2], [1] * 5)
    else:
        batch = B([0, 1, 2], [0, 7, 0], [40, 9, 1])
    c = MoECase(TINY_MOE, batch, 5, 64, seed=4, decode=decode)
    rows = np.arange(batch.n_tokens)
    moe_stage_parity(c, rows)
    w64 = {k: f64(v) for k, v in c.wb.items()}
    args = (c.cfg, w64, f64(c.kb), f64(c.vb), batch, f64(c.xb))
    ref = oracle.layer_forward(*args, storage="bf16")
    gi = c.idx.cpu().numpy()
    routes_agree(gi, ref["logits"], c.cfg.top_k, 2e-2)
    forced = oracle.layer_forward(*args, storage="bf16", forced_routes=gi)
    exact = oracle.layer_forward(*args, forced_routes=gi)
    assert_e2e(to_host_f64(c.out), exact["out"], f"tiny MoE out (decode {decode})",
               emul=forced["out"], strict=True)


def test_moe_prefill_full_size_sampled():
    """4 x 1024 tokens, 128 experts top-8 (the MoE prefill launch), sampled rows."""
    wl = workload("moe_prefill")
    c = MoECase(wl.cfg, wl.batch, wl.n_slots, wl.max_seq)
    rows = np.array([0, 1, 511, 1023, 1024, 2047, 3000, 4095])
    moe_stage_parity(c, rows)
    counts = np.bincount(c.idx.cpu().numpy().reshape(-1), minlength=wl.cfg.n_experts)
    assert counts.sum() == wl.batch.n_tokens * wl.cfg.top_k
    # end to end on one sequence with the GPU's routes
    s = 2
    sub = B([s], [0], [1024])
    w64 = {k: f64(v) for k, v in c.wb.items()}
    local = np.array([0, 100, 1023])
    gi = c.idx.cpu().numpy()[s * 1024:(s + 1) * 1024]
    args = (wl.cfg, w64, f64(c.kb), f64(c.vb), sub, f64(c.xb[s * 1024:(s + 1) * 1024]))
    forced = oracle.layer_forward(*args, rows=local, storage="bf16", forced_routes=gi)
    exact = oracle.layer_forward(*args, rows=local, forced_routes=gi)
    assert_e2e(to_host_f64(c.out)[s * 1024 + local], exact["out"], "MoE prefill rows",
               emul=forced["out"])


def test_moe_decode_full_size_sampled():
    """Batch 128 at KV 2048 (the MoE decode launch), sampled sequences."""
    wl = workload("moe_decode")
    c = MoECase(wl.cfg, wl.batch, wl.n_slots, wl.max_seq, decode=True)
    pick = np.array([0, 5, 64, 127])
    moe_stage_parity(c, pick)
    sub = B(np.arange(len(pick)), wl.batch.ctx_len[pick], wl.batch.q_len[pick])
    w64 = {k: f64(v) for k, v in c.wb.items()}
    gi = c.idx.cpu().numpy()[pick]
    args = (wl.cfg, w64, f64(c.kb[wl.batch.slot[pick]]), f64(c.vb[wl.batch.slot[pick]]), sub,
            f64(c.xb[pick]))
    forced = oracle.layer_forward(*args, storage="bf16", forced_routes=gi)
    exact = oracle.layer_forward(*args, forced_routes=gi)
    assert_e2e(to_host_f64(c.out)[pick], exact["out"], "MoE decode rows", emul=forced["out"])


def test_moe_decode_twice_bit_identical():
    """The MoE decode launch twice on the same inputs: output, routes and
    weights bit-identical (each expert workgroup's k-order and each decode
    attention wave's tile order are fixed functions of the tile and wave)."""
    import torch
    wl = workload("moe_decode")
    c = MoECase(wl.cfg, wl.batch, wl.n_slots, wl.max_seq, decode=True)
    out0, idx0, w0 = c.out.clone(), c.idx.clone(), c.w.clone()
    out1, _ = T.layer_decode(c.dl.cfg, c.dl.w, c.cache, c.db, to_device_bf16(c.xb),
                             route_idx=c.idx, route_w=c.w)
    torch.cuda.synchronize()
    assert torch.equal(idx0, c.idx) and torch.equal(w0, c.w)
    assert torch.equal(out0, out1)


@pytest.mark.parametrize("n_tok", [600, 1000], ids=["128-row tiles", "256-row tiles"])
def test_moe_grouped_tile_sizes(n_tok):
    """The grouped expert GEMMs pick their tile rows from the mean rows per
    expert: 1200 routed rows over 8 experts take 128-row tiles, 2000 take
    256-row tiles (ragged: most experts end in a partial tile)."""
    batch = B([0, 1], [0, 5], [n_tok - 100, 100])
    c = MoECase(TINY_MOE, batch, 2, 1024, seed=9)
    rows = np.array([0, 1, 255, 256, 257, n_tok - 101, n_tok - 100, n_tok - 1])
    moe_stage_parity(c, rows)
    w64 = {k: f64(v) for k, v in c.wb.items()}
    args = (c.cfg, w64, f64(c.kb), f64(c.vb), batch, f64(c.xb))
    gi = c.idx.cpu().numpy()
    forced = oracle.layer_forward(*args, rows=rows, storage="bf16", forced_routes=gi)
    exact = oracle.layer_forward(*args, rows=rows, forced_routes=gi)
    assert_e2e(to_host_f64(c.out)[rows], exact["out"], f"tiny MoE {n_tok} tokens rows",
               emul=forced["out"], strict=True)
