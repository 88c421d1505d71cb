"""Paged KV cache (the PagedAttention block layout of the serving framework in
Section II-A) on the GPU, through the C ABI.

The paged layout changes where cache rows live, not what is computed: every
launch reads and writes the same rows through a block table, so a layer call
on a paged cache must give bit-identical outputs to the same call on the
contiguous cache holding the same rows, and the rows it writes must land in
the blocks the table names.  The pools hold spare blocks that no slot maps
to, filled with NaN: a read of any of them would show in the outputs.

The paged path is also checked against the oracle on its own (no contiguous
cache in the process): per-kernel parity on identical inputs and the
end-to-end bar, at the full decode launch (64 sequences at KV 4096) and at a
7B ragged prefill whose chunk continues a cached prefix that ends mid-block,
with 64- and 128-row blocks in a shuffled pool.
"""
import numpy as np
import pytest

import oracle
from paper_2606_29629_amd import _lib as T
from paper_2606_29629_amd.workload import (DeviceLayer, contiguous_from_paged, device_batch,
                                           device_cache, paged_from_contiguous, to_device_bf16,
                                           to_host_f64)
from synth import Batch, layer_7b, layer_c1, make_cache, make_weights, make_x, workload
from test_gpu_layer import Case, assert_e2e, check_down, f64, stage_parity

pytestmark = pytest.mark.gpu


def B(slot, ctx, q):
    return Batch(np.asarray(slot, np.int32), np.asarray(ctx, np.int32), np.asarray(q, np.int32))


def run_both(cfg, batch, n_slots, max_seq, block_size, decode=False, seed=0, table_edit=None):
    """The same call on a contiguous cache and on its paged copy; returns the
    two outputs and the two caches (the paged one gathered back)."""
    import torch
    wb = make_weights(cfg, seed)
    kb, vb = make_cache(cfg, n_slots, max_seq, seed)
    dl = DeviceLayer(cfg, wb)
    cont = device_cache(kb, vb)
    paged = paged_from_contiguous(cont[0], cont[1], block_size, seed=seed + 11)
    if table_edit is not None:
        table_edit(paged)
    x = to_device_bf16(make_x(cfg, batch.n_tokens, seed, step=0 if decode else None))
    db = device_batch(batch)
    fn = T.layer_decode if decode else T.layer_prefill
    out_c, _ = fn(dl.cfg, dl.w, cont, db, x)
    out_p, _ = fn(dl.cfg, dl.w, paged, db, x)
    torch.cuda.synchronize()
    return out_c, out_p, cont, paged


def assert_same(out_c, out_p, cont, paged, what):
    import torch
    assert torch.equal(out_c.view(torch.int16), out_p.view(torch.int16)), f"{what}: outputs differ"
    kg, vg = contiguous_from_paged(paged)
    assert torch.equal(kg.view(torch.int16), cont[0].view(torch.int16)), f"{what}: K cache differs"
    assert torch.equal(vg.view(torch.int16), cont[1].view(torch.int16)), f"{what}: V cache differs"
    assert not torch.isnan(out_p.float()).any(), f"{what}: a spare block was read"


def test_paged_7b_ragged_prefill_chunk_and_decode_sequence():
    cfg = layer_7b()
    # fresh prefill, a chunk over a cached prefix that ends mid-block, a
    # single-token sequence (split-KV path) and a chunk crossing blocks
    batch = B([0, 2, 3, 1], [0, 130, 513, 64], [300, 200, 1, 65])
    out_c, out_p, cont, paged = run_both(cfg, batch, 4, 1024, 64)
    assert_same(out_c, out_p, cont, paged, "7B ragged prefill")


def test_paged_7b_decode_step_block_size_128():
    cfg = layer_7b()
    batch = B(np.arange(16), np.array([5, 63, 64, 65, 127, 128, 129, 300, 511, 512, 700, 1000,
                                       1023, 1, 0, 255]), np.ones(16, np.int64))
    out_c, out_p, cont, paged = run_both(cfg, batch, 16, 1152, 128, decode=True)
    assert_same(out_c, out_p, cont, paged, "7B decode bs128")


def test_paged_full_size_decode():
    # the decode workload's shape: 64 sequences at KV 4096, 64-row blocks
    cfg = layer_7b()
    batch = B(np.arange(64), np.full(64, 4096), np.ones(64, np.int64))
    out_c, out_p, cont, paged = run_both(cfg, batch, 64, 4160, 64, decode=True)
    assert_same(out_c, out_p, cont, paged, "full decode")


def test_paged_tiny_head_dim_64():
    cfg = layer_c1()
    batch = B([1, 0, 2], [0, 70, 129], [90, 40, 1])
    out_c, out_p, cont, paged = run_both(cfg, batch, 3, 256, 64)
    assert_same(out_c, out_p, cont, paged, "tiny prefill")
    batch = B([0, 1, 2], [130, 64, 191], [1, 1, 1])
    out_c, out_p, cont, paged = run_both(cfg, batch, 3, 256, 64, decode=True)
    assert_same(out_c, out_p, cont, paged, "tiny decode")


def test_paged_invalid_table_entries_are_contained():
    """Entries outside the pool are never dereferenced: the call completes,
    and sequences whose blocks are all valid are unaffected."""
    import torch
    cfg = layer_c1()
    batch = B([0, 1, 2], [100, 100, 100], [20, 20, 20])

    def corrupt(paged):
        t = paged.block_table
        t[1, 0] = -1                       # a prefix block of slot 1
        t[2, 1] = paged.n_blocks + 5       # the block slot 2 writes to
    out_c, out_p, cont, paged = run_both(cfg, batch, 3, 256, 64, table_edit=corrupt)
    assert torch.equal(out_c[:20].view(torch.int16), out_p[:20].view(torch.int16))
    # slot 0's cache rows (its own blocks) match the contiguous cache
    ids = paged.block_table.long()
    k0 = paged.k[ids[0]].permute(1, 0, 2, 3).reshape(cfg.n_kv_heads, -1, cfg.head_dim)
    assert torch.equal(k0.view(torch.int16), cont[0][0].view(torch.int16))


def test_paged_kvcache_append():
    import torch
    cfg = layer_c1()
    batch = B([2, 0, 1], [63, 0, 130], [3, 70, 1])
    kb, vb = make_cache(cfg, 3, 256, 4)
    cont = device_cache(kb, vb)
    paged = paged_from_contiguous(cont[0], cont[1], 64, seed=5)
    kn = torch.randn(74, cfg.n_kv_heads, cfg.head_dim, device="cuda").to(torch.bfloat16)
    vn = torch.randn_like(kn.float()).to(torch.bfloat16)
    T.kvcache_append(T.make_config(cfg), cont, device_batch(batch), kn, vn)
    T.kvcache_append(T.make_config(cfg), paged, device_batch(batch), kn, vn)
    torch.cuda.synchronize()
    kg, vg = contiguous_from_paged(paged)
    assert torch.equal(kg.view(torch.int16), cont[0].view(torch.int16))
    assert torch.equal(vg.view(torch.int16), cont[1].view(torch.int16))


class PagedCase(Case):
    """A Case whose layer calls see only a paged copy of the seeded cache
    (blocks of `block_size` rows dealt to a shuffled pool with NaN spare
    blocks); the contiguous device copy is dropped before any call."""

    def __init__(self, cfg, batch, n_slots, max_seq, block_size, seed=0, x_step=None):
        import torch
        super().__init__(cfg, batch, n_slots, max_seq, seed=seed, x_step=x_step)
        k, v = self.cache
        self.cache = paged_from_contiguous(k, v, block_size, seed=seed + 23)
        del k, v
        torch.cuda.synchronize()

    def cache_view(self):
        return contiguous_from_paged(self.cache)


@pytest.mark.parametrize("block_size", [64, 128])
def test_paged_full_size_decode_against_oracle(block_size):
    """The decode launch (64 sequences at KV 4096) on a paged cache only."""
    wl = workload("dense_decode")
    max_seq = -(-wl.max_seq // block_size) * block_size
    cs = PagedCase(wl.cfg, wl.batch, wl.n_slots, max_seq, block_size)
    out, ws = cs.run(decode=True)
    pick = np.array([0, 3, 31, 40, 63])
    label = f"paged bs{block_size} decode"
    x1, act, w = stage_parity(cs, ws, pick, label=label)
    check_down(cs, out, x1, act, w, pick, label)
    sub = B(np.arange(len(pick)), wl.batch.ctx_len[pick], wl.batch.q_len[pick])
    w64 = {k: f64(v) for k, v in cs.wb.items()}
    args = (wl.cfg, w64, f64(cs.kb[wl.batch.slot[pick]]), f64(cs.vb[wl.batch.slot[pick]]), sub,
            f64(cs.xb[pick]))
    ref = oracle.layer_forward(*args, storage="bf16")
    ex = oracle.layer_forward(*args)
    assert_e2e(to_host_f64(out)[pick], ex["out"], f"{label} rows", emul=ref["out"])
    # the rows written went to the blocks the table names
    kr, vr = cs.cache_rows()
    assert_e2e(kr[pick], ex["k_new"], f"{label} K rows", emul=ref["k_new"])
    assert_e2e(vr[pick], ex["v_new"], f"{label} V rows", emul=ref["v_new"])


@pytest.mark.parametrize("block_size", [64, 128])
def test_paged_7b_ragged_prefill_against_oracle(block_size):
    """A fresh prefill, a chunk whose cached prefix ends mid-block (130 rows),
    a single-token sequence and a chunk crossing blocks, on a paged cache only."""
    cfg = layer_7b()
    batch = B([0, 2, 3, 1], [0, 130, 513, 64], [300, 200, 1, 65])
    cs = PagedCase(cfg, batch, 4, 1024, block_size, seed=7)
    out, ws = cs.run()
    rows = np.array([0, 1, 127, 128, 299, 300, 301, 363, 364, 499, 500, 501, 564])
    label = f"paged bs{block_size} ragged"
    x1, act, w = stage_parity(cs, ws, rows, label=label)
    check_down(cs, out, x1, act, w, rows, label)
    ref = cs.oracle(rows=rows)
    ex = cs.oracle(rows=rows, storage=None)
    assert_e2e(to_host_f64(out)[rows], ex["out"], f"{label} rows", emul=ref["out"])
    kr, vr = cs.cache_rows()
    assert_e2e(kr, ex["k_new"], f"{label} K rows", emul=ref["k_new"])
    assert_e2e(vr, ex["v_new"], f"{label} V rows", emul=ref["v_new"])
