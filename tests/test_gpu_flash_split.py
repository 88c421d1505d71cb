"""Chunked prefill over a long cached prefix: when a batch has too few query
tiles to fill the GPU, the flash kernel deals each query tile's key tiles to
several workgroups and a second kernel merges their partial (max, sum,
output) in split order.  The attention output is checked on identical inputs
against the reference over the GPU-written cache, then the layer end to end
against the oracle; the paged layout gives bit-identical results.
"""
import numpy as np
import pytest

import oracle
from paper_2606_29629_amd.workload import (DeviceLayer, contiguous_from_paged, device_batch,
                                           paged_from_contiguous, to_device_bf16, to_host_f64)
from paper_2606_29629_amd import _lib as T
from synth import layer_7b, layer_c1, make_cache, make_weights, make_x
from parity import strict_shape
from test_gpu_layer import B, Case, assert_e2e, check_down, f64, stage_parity

pytestmark = pytest.mark.gpu


def run_case(cfg, batch, n_slots, max_seq, label, seed=0, e2e_rows=None):
    cs = Case(cfg, batch, n_slots, max_seq, seed=seed)
    out, ws = cs.run()
    rows = np.arange(batch.n_tokens) if e2e_rows is None else np.asarray(e2e_rows)
    x1, act, w = stage_parity(cs, ws, rows, label=label)
    check_down(cs, out, x1, act, w, rows, label)
    ref = cs.oracle(rows=rows)
    assert_e2e(to_host_f64(out)[rows], cs.oracle(rows=rows, storage=None)["out"], f"{label} out",
               emul=ref["out"], strict=strict_shape(cfg))
    return cs, out


def test_tiny_chunk_over_long_prefix():
    # 130 new tokens after 2000 cached: 8 query tiles x heads, 34 key tiles -> 4 splits
    run_case(layer_c1(), B([0], [2000], [130]), 1, 2176, "tiny split chunk", seed=3)


def test_tiny_chunks_and_decodes_mixed():
    # chunks of different lengths and prefixes next to single-token sequences
    batch = B([2, 0, 3, 1], [1500, 0, 700, 900], [70, 40, 1, 1])
    run_case(layer_c1(), batch, 4, 1600, "tiny split mixed", seed=4)


def test_7b_chunk_with_decodes():
    # a 300-token chunk at ctx 3000 beside three decode sequences (the mixed step's shape)
    batch = B([0, 1, 2, 3], [3000, 100, 2500, 4000], [300, 1, 1, 1])
    rows = np.array([0, 1, 63, 64, 127, 128, 255, 256, 299, 300, 301, 302])
    run_case(layer_7b(), batch, 4, 4160, "7B split chunk", seed=5, e2e_rows=rows)


def test_paged_split_chunk_is_bit_identical():
    import torch
    cfg = layer_7b()
    batch = B([1, 0], [2600, 900], [200, 1])
    wb = make_weights(cfg, 6)
    kb, vb = make_cache(cfg, 2, 2880, 6)
    dl = DeviceLayer(cfg, wb)
    from paper_2606_29629_amd.workload import device_cache
    cont = device_cache(kb, vb)
    paged = paged_from_contiguous(cont[0], cont[1], 64, seed=17)
    x = to_device_bf16(make_x(cfg, batch.n_tokens, 6))
    db = device_batch(batch)
    out_c, _ = T.layer_prefill(dl.cfg, dl.w, cont, db, x)
    out_p, _ = T.layer_prefill(dl.cfg, dl.w, paged, db, x)
    torch.cuda.synchronize()
    assert torch.equal(out_c.view(torch.int16), out_p.view(torch.int16))
    kg, vg = contiguous_from_paged(paged)
    assert torch.equal(kg.view(torch.int16), cont[0].view(torch.int16))
    assert not torch.isnan(out_p.float()).any()
