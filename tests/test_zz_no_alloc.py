"""The allocation-free decode entry (tri_layer_decode_noalloc) against the
workspace entry (tri_layer_decode), through the C ABI.

Both run the same kernels, so on identical inputs (weights, cache contents,
batch, activations) the outputs, the cache rows written and the MoE routes
must be bit-identical.  Two calls in a row on the fixed scratch, the second
with a smaller batch, so a stale first call's scratch could show; then the
end-to-end bar against the exact oracle on sampled rows.
"""
import numpy as np
import pytest

import oracle
from paper_2606_29629_amd import _lib as T
from paper_2606_29629_amd.workload import (DeviceLayer, device_batch, device_cache,
                                           to_device_bf16, to_host_f64)
from parity import check_e2e
from synth import Batch, make_cache, make_weights, make_x, workload

pytestmark = pytest.mark.gpu


def f64(bits):
    from synth import bf16_to_f32
    return bf16_to_f32(bits).astype(np.float64)


def both(dl, kb, vb, batch, xb, moe_k=0):
    """The same decode step through both entries, each on its own copy of the
    cache; returns (out_ws, out_noalloc, caches, routes)."""
    import torch
    db = device_batch(batch)
    x = to_device_bf16(xb)
    c1, c2 = device_cache(kb, vb), device_cache(kb, vb)
    r1 = r2 = None
    if moe_k:
        r1 = torch.full((batch.n_tokens, moe_k), -1, dtype=torch.int32, device="cuda")
        r2 = torch.full_like(r1, -1)
    o1, _ = T.layer_decode(dl.cfg, dl.w, c1, db, x, route_idx=r1)
    o2 = torch.full_like(o1, float("nan"))
    T.layer_decode_noalloc(dl.cfg, dl.w, c2, db, x, out=o2, route_idx=r2)
    torch.cuda.synchronize()
    return o1, o2, c1, c2, r1, r2


def assert_identical(o1, o2, c1, c2, r1, r2, what):
    import torch
    assert torch.equal(o1.view(torch.int16), o2.view(torch.int16)), f"{what}: outputs differ"
    assert torch.equal(c1[0].view(torch.int16), c2[0].view(torch.int16)), f"{what}: K differs"
    assert torch.equal(c1[1].view(torch.int16), c2[1].view(torch.int16)), f"{what}: V differs"
    if r1 is not None:
        assert torch.equal(r1, r2), f"{what}: routes differ"


def B(slot, ctx, q):
    return Batch(np.asarray(slot, np.int32), np.asarray(ctx, np.int32), np.asarray(q, np.int32))


def test_noalloc_dense_decode_two_calls():
    wl = workload("dense_decode")
    wb = make_weights(wl.cfg, 0)
    kb, vb = make_cache(wl.cfg, wl.n_slots, wl.max_seq, 0)
    dl = DeviceLayer(wl.cfg, wb)
    # call 1: the full decode launch, 64 sequences at KV 4096
    xb = make_x(wl.cfg, wl.batch.n_tokens, 0, step=0)
    res = both(dl, kb, vb, wl.batch, xb)
    assert_identical(*res, "64 x KV 4096")
    # call 2: a smaller batch, 8 sequences of mixed lengths in other slots
    small = B([5, 0, 63, 17, 30, 2, 41, 9], [1, 4095, 127, 2000, 64, 0, 129, 3000], [1] * 8)
    xs = make_x(wl.cfg, small.n_tokens, 3, step=1)
    o1, o2, c1, c2, r1, r2 = both(dl, kb, vb, small, xs)
    assert_identical(o1, o2, c1, c2, r1, r2, "8 mixed")
    # and the end-to-end bar against the exact oracle for the smaller call
    w64 = {k: f64(v) for k, v in wb.items()}
    sub = B(np.arange(8), small.ctx_len, small.q_len)
    args = (wl.cfg, w64, f64(kb[small.slot]), f64(vb[small.slot]), sub, f64(xs))
    ex = oracle.layer_forward(*args)
    emul = oracle.layer_forward(*args, storage="bf16")
    check_e2e(to_host_f64(o2), ex["out"], "noalloc 8 mixed out", emul=emul["out"])


def test_noalloc_moe_decode_two_calls():
    wl = workload("moe_decode")
    wb = make_weights(wl.cfg, 0)
    kb, vb = make_cache(wl.cfg, wl.n_slots, wl.max_seq, 0)
    dl = DeviceLayer(wl.cfg, wb)
    k = wl.cfg.top_k
    xb = make_x(wl.cfg, wl.batch.n_tokens, 0, step=0)
    assert_identical(*both(dl, kb, vb, wl.batch, xb, moe_k=k), "MoE 128 x KV 2048")
    small = B([7, 100, 3], [10, 2047, 500], [1, 1, 1])
    xs = make_x(wl.cfg, small.n_tokens, 4, step=2)
    assert_identical(*both(dl, kb, vb, small, xs, moe_k=k), "MoE 3 mixed")


def test_noalloc_rejects_a_batch_beyond_its_scratch():
    import torch
    wl = workload("dense_decode")
    dl = DeviceLayer(wl.cfg, make_weights(wl.cfg, 0))
    n = 512
    big = B(np.arange(n), np.full(n, 8000), np.ones(n))
    kc = torch.zeros(1, dtype=torch.bfloat16, device="cuda")
    with pytest.raises(T.TriError) as e:
        T.layer_decode_noalloc(dl.cfg, dl.w, (kc.expand(n, wl.cfg.n_kv_heads, 8192, 128),
                                              kc.expand(n, wl.cfg.n_kv_heads, 8192, 128)),
                               device_batch(big), torch.zeros(n, wl.cfg.hidden,
                                                              dtype=torch.bfloat16, device="cuda"))
    assert e.value.status == T.TRI_ERR_SCRATCH
