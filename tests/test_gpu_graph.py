"""Layer calls captured into HIP graphs (torch.cuda.graph) and replayed.

Each graph is replayed three times with eager work and synchronisations
between the replays, and every replay must give the eager call's output bit
for bit (kernels that re-run on the same inputs are deterministic; the call
rewrites this step's cache rows with the same values).  Cases: a mixed batch
through tri_layer_prefill (a chunk beside single-token sequences, so the
split-KV attention runs on the library's side stream, forked and joined
inside the capture) and a decode step through tri_layer_decode_noalloc (the
entry for callers that cannot allocate, on the library's fixed scratch).
"""
import numpy as np
import pytest

from paper_2606_29629_amd import _lib as T
from paper_2606_29629_amd.workload import to_device_bf16
from synth import Batch, layer_c1, make_x
from test_gpu_layer import Case

pytestmark = pytest.mark.gpu


def B(slot, ctx, q):
    return Batch(np.asarray(slot, np.int32), np.asarray(ctx, np.int32), np.asarray(q, np.int32))


def replay_matches(graph, out, ref):
    import torch
    for i in range(3):
        graph.replay()
        torch.cuda.synchronize()
        assert torch.equal(out, ref), f"replay {i}"
        junk = torch.randn(1 << 20, device="cuda") * 3.0   # eager work between replays
        del junk
        torch.cuda.synchronize()


def test_graph_mixed_batch_with_side_stream():
    import torch
    cfg = layer_c1()
    batch = B([0, 1, 2, 3], [50, 7, 120, 0], [40, 1, 1, 1])
    cs = Case(cfg, batch, 4, 256, seed=9)
    x = to_device_bf16(cs.xb)
    out = torch.empty_like(x)
    ws = torch.empty(T.workspace_size(cs.dl.cfg, cs.db), dtype=torch.uint8, device="cuda")
    stream = torch.cuda.Stream()
    call = lambda: T.layer_prefill(cs.dl.cfg, cs.dl.w, cs.cache, cs.db, x, out=out, workspace=ws,
                                   stream=stream)
    with torch.cuda.stream(stream):
        call()                          # eager: creates the side stream, sets kernel attributes
    torch.cuda.synchronize()
    ref = out.clone()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g, stream=stream):
        call()
    torch.cuda.synchronize()
    replay_matches(g, out, ref)


def test_graph_noalloc_decode():
    import torch
    cfg = layer_c1()
    batch = B([0, 1, 2, 3, 4], [5, 60, 17, 33, 200], [1] * 5)
    cs = Case(cfg, batch, 5, 256, seed=10, x_step=0)
    x = to_device_bf16(make_x(cfg, batch.n_tokens, 10, step=0))
    out = torch.empty_like(x)
    stream = torch.cuda.Stream()
    call = lambda: T.layer_decode_noalloc(cs.dl.cfg, cs.dl.w, cs.cache, cs.db, x, out=out,
                                          stream=stream)
    with torch.cuda.stream(stream):
        call()
    torch.cuda.synchronize()
    ref = out.clone()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g, stream=stream):
        call()
    torch.cuda.synchronize()
    replay_matches(g, out, ref)
