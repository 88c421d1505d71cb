"""Work model of the layer stages (tri_layer_work) and the time-weighted phase
intensity of Section III-C, Eq. 5 (tri_phase_intensity).  Host code only:
nothing here touches a GPU.

The totals are pinned to the algorithmic flop and byte counts derived for the
benchmark workloads by hand (7B-class dense layer: 233.05 M linear parameters;
30B-A3B-style MoE layer: 128 experts of 4.72 M parameters), not recomputed
from the library's own formulas.
"""
import math
import os

import numpy as np
import pytest

from paper_2606_29629_amd import _lib as T
from synth import workload


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(T.LIB_PATH):
        pytest.skip("libtri.so not built (run python -m paper_2606_29629_amd.build)")
    return T.lib()


def work(name, decode=None, batch=None, expert_rows=None):
    wl = workload(name)
    b = wl.batch if batch is None else batch
    if decode is None:
        decode = int(b.q_len.max()) == 1
    return T.layer_work(T.make_config(wl.cfg), decode, b.q_len, b.ctx_len, expert_rows)


def stages(w):
    return T.work_dict(w)


def total(w, key):
    return sum(v[key] for v in stages(w).values())


LINEAR = ("qkv_rope", "o_proj", "gate_up", "down")


def test_dense_prefill_flops(lib):
    s = stages(work("dense_prefill"))
    # 2 x 233.05 M parameters x 16384 tokens; 8 causal 2048-token sequences
    assert sum(s[k]["flops"] for k in LINEAR) == pytest.approx(7.636e12, rel=2e-4)
    assert s["attn_prefill"]["flops"] == pytest.approx(0.2406e12, rel=2e-4)
    assert total(work("dense_prefill"), "flops") == pytest.approx(7.877e12, rel=5e-4)
    # every sequence has 2048 new tokens: the split-KV stages are not launched
    assert "attn_decode" not in s and "attn_combine" not in s
    # ragged prefill lengths (no single-token sequence either): launched, no work
    from synth import Batch
    rag = Batch(np.arange(2, dtype=np.int32), np.zeros(2, np.int32),
                np.array([2048, 1000], np.int32))
    sr = stages(work("dense_prefill", batch=rag))
    assert sr["attn_decode"]["flops"] == 0 and sr["attn_combine"]["bytes"] == 0
    assert not any(k.startswith("moe_") for k in s)


def test_qk_norm_adds_its_elementwise_work(lib):
    """The per-head q/k RMSNorm: two multiply-adds per q and k element and
    the two D-long gain vectors; nothing else changes."""
    import dataclasses
    wl = workload("dense_prefill")
    b = wl.batch
    plain = stages(T.layer_work(T.make_config(wl.cfg), False, b.q_len, b.ctx_len))
    cfg = dataclasses.replace(wl.cfg, qk_norm=True)
    normed = stages(T.layer_work(T.make_config(cfg), False, b.q_len, b.ctx_len))
    n_tok = int(b.q_len.sum())
    # 16384 tokens x (28 + 4) heads x 128 x 4
    assert normed["qkv_rope"]["flops"] - plain["qkv_rope"]["flops"] == 16384 * 32 * 128 * 4
    assert n_tok == 16384
    assert normed["qkv_rope"]["bytes"] - plain["qkv_rope"]["bytes"] == 2 * 128 * 2
    for k in plain:
        if k != "qkv_rope":
            assert normed[k] == plain[k]


def test_dense_decode_bytes(lib):
    w = work("dense_decode")
    s = stages(w)
    assert "attn_prefill" not in s
    weights = sum(s[k]["bytes"] for k in LINEAR)
    # 466.1 MB of projection weights; the activations the four stages read and
    # write (64 rows, the 18944-wide SwiGLU activation twice) add under 10 MB
    assert 466.1e6 <= weights <= 476.1e6
    # K and V of 64 sequences x 4 KV heads x 4097 keys x 128 x bf16
    kv = 64 * 4097 * 2048
    assert kv == pytest.approx(537.0e6, rel=1e-3)
    assert kv <= s["attn_decode"]["bytes"] <= kv * 1.02
    assert 1.004e9 <= total(w, "bytes") <= 1.04e9
    assert total(w, "flops") == pytest.approx(33.6e9, rel=5e-3)


def test_decode_attention_intensity_is_the_group_size(lib):
    # Every K/V byte serves Hq / Hkv query heads with 2 flops per multiply-add
    # over two products: flops / bytes -> Hq / Hkv as the KV dominates.
    s = stages(work("dense_decode"))
    ai = s["attn_decode"]["flops"] / s["attn_decode"]["bytes"]
    assert 6.8 < ai < 7.0
    # Projections at batch 64: 2 * 64 flops per 2-byte weight -> 64 flop/B.
    ai_gu = s["gate_up"]["flops"] / s["gate_up"]["bytes"]
    assert 63.0 < ai_gu < 64.0


def test_moe_prefill_flops(lib):
    s = stages(work("moe_prefill"))
    # projections 154.6 + router 2.1 + experts 309.2 + attention 34.4 GFLOP
    assert s["qkv_rope"]["flops"] + s["o_proj"]["flops"] == pytest.approx(154.6e9, rel=5e-4)
    assert s["moe_router"]["flops"] == pytest.approx(2.15e9, rel=5e-3)
    assert s["moe_gate_up"]["flops"] + s["moe_down"]["flops"] == pytest.approx(309.2e9, rel=5e-4)
    assert s["attn_prefill"]["flops"] == pytest.approx(34.4e9, rel=5e-4)
    assert total(work("moe_prefill"), "flops") == pytest.approx(500.4e9, rel=1e-3)
    assert "gate_up" not in s and "down" not in s


def test_moe_decode_bytes_and_touched_experts(lib):
    w = work("moe_decode")
    s = stages(w)
    experts = s["moe_gate_up"]["bytes"] + s["moe_down"]["bytes"]
    assert experts >= 1.208e9                   # all 128 experts streamed
    # experts 1.208 GB + attention weights 37.7 MB + router 0.5 MB + KV 537 MB;
    # fp32 expert rows and split-KV partials (each written, then read) add ~40 MB
    assert 1.783e9 <= total(w, "bytes") <= 1.85e9
    # only 3 of 128 experts routed to: their weights alone
    wl = workload("moe_decode")
    rows = np.zeros(128, np.int64)
    rows[[0, 5, 77]] = [400, 400, wl.batch.n_tokens * wl.cfg.top_k - 800]
    s3 = stages(work("moe_decode", expert_rows=rows))
    per_expert = 3 * 768 * 2048 * 2
    assert s["moe_gate_up"]["bytes"] - s3["moe_gate_up"]["bytes"] == pytest.approx(
        125 * 2 / 3 * per_expert, rel=1e-12)
    assert s3["moe_gate_up"]["flops"] == s["moe_gate_up"]["flops"]


def test_mixed_step(lib):
    s = stages(work("mixed", decode=False))
    # 544 tokens through 233.05 M parameters; the 512-token chunk at ctx 6144
    assert sum(s[k]["flops"] for k in LINEAR) == pytest.approx(253.6e9, rel=5e-4)
    assert s["attn_prefill"]["flops"] == pytest.approx(47.0e9, rel=5e-4)
    # 32 single-token sequences with KV ~ U[1024, 8192]: about 2.1 GFLOP
    assert s["attn_decode"]["flops"] == pytest.approx(2.1e9, rel=0.15)


def test_phase_intensity_eq5(lib):
    w = work("dense_decode")
    s = stages(w)
    names = list(s)
    idx = {w.name[i].decode(): i for i in range(w.n_stages)}

    def prof(times):
        p = T.Profile()
        p.n_stages = w.n_stages
        for k, t in times.items():
            p.total_ms[idx[k]] = t
        return p

    ai = {k: v["flops"] / v["bytes"] for k, v in s.items()}
    # durations proportional to bytes: the duration-weighted mean of flops/bytes
    # is total flops / total bytes
    got = T.phase_intensity(w, prof({k: s[k]["bytes"] * 1e-9 for k in names}))
    assert got == pytest.approx(total(w, "flops") / total(w, "bytes"), rel=1e-12)
    # equal durations: the plain mean
    got = T.phase_intensity(w, prof({k: 0.5 for k in names}))
    assert got == pytest.approx(sum(ai.values()) / len(ai), rel=1e-12)
    # a single timed stage: its own intensity
    got = T.phase_intensity(w, prof({"gate_up": 3.0}))
    assert got == pytest.approx(ai["gate_up"], rel=1e-12)
    # time on a stage the call does not launch is ignored
    got = T.phase_intensity(w, prof({"gate_up": 3.0, "attn_prefill": 5.0}))
    assert got == pytest.approx(ai["gate_up"], rel=1e-12)
    # a launched stage with no work (split-KV stages of a ragged all-prefill
    # batch) drops out whatever its time
    from synth import Batch
    rag = Batch(np.arange(2, dtype=np.int32), np.zeros(2, np.int32),
                np.array([2048, 1000], np.int32))
    wp = work("dense_prefill", batch=rag)
    sp = stages(wp)
    assert sp["attn_decode"]["bytes"] == 0
    p = T.Profile()
    p.n_stages = wp.n_stages
    for k in sp:
        p.total_ms[idx[k]] = 1.0
    p_noop = T.phase_intensity(wp, p)
    p.total_ms[idx["attn_decode"]] = 0.0
    p.total_ms[idx["attn_combine"]] = 0.0
    assert T.phase_intensity(wp, p) == p_noop
    # random durations: a convex combination
    rng = np.random.default_rng(3)
    for _ in range(20):
        got = T.phase_intensity(w, prof({k: float(rng.uniform(0, 2)) for k in names}))
        assert min(ai.values()) - 1e-9 <= got <= max(ai.values()) + 1e-9
    with pytest.raises(T.TriError) as e:
        T.phase_intensity(w, prof({}))
    assert e.value.status == T.TRI_ERR_SHAPE
    with pytest.raises(T.TriError) as e:
        T.phase_intensity(w, prof({"gate_up": -1.0}))
    assert e.value.status == T.TRI_ERR_RANGE


def test_work_sum_over_decode_steps(lib):
    wl = workload("dense_decode")
    b = wl.batch
    ws = []
    for _ in range(3):
        ws.append(T.layer_work(T.make_config(wl.cfg), True, b.q_len, b.ctx_len))
        b = b.advanced()
    tot = T.work_sum(ws)
    s = stages(tot)
    # one more key per sequence and step: 3 steps add 0 + 1 + 2 keys per sequence
    kv0 = stages(ws[0])["attn_decode"]["flops"]
    assert s["attn_decode"]["flops"] == pytest.approx(kv0 * 3 * (1 + 1 / 4097), rel=1e-12)
    assert s["gate_up"]["bytes"] == 3 * stages(ws[0])["gate_up"]["bytes"]


def test_work_validation(lib):
    wl = workload("dense_decode")
    c = T.make_config(wl.cfg)
    with pytest.raises(T.TriError) as e:
        T.layer_work(c, True, [2, 1], [5, 5])
    assert e.value.status == T.TRI_ERR_SHAPE
    with pytest.raises(T.TriError) as e:
        T.layer_work(c, False, [-1], [5])
    assert e.value.status == T.TRI_ERR_SHAPE
    wm = workload("moe_decode")
    with pytest.raises(T.TriError) as e:
        T.layer_work(T.make_config(wm.cfg), True, [1] * 4, [10] * 4, expert_rows=[1] * 128)
    assert e.value.status == T.TRI_ERR_SHAPE
    # an empty batch is no work
    w = T.layer_work(c, False, [], [])
    assert not any(w.runs[i] for i in range(w.n_stages))
    # a prefill-entry batch of single-token sequences has no flash stage
    s = stages(T.layer_work(c, False, [1, 1, 1], [100, 7, 0]))
    assert "attn_prefill" not in s
    assert s["attn_decode"]["flops"] == 4 * 128 * 28 * (101 + 8 + 1)
    assert math.isfinite(s["attn_combine"]["bytes"])
