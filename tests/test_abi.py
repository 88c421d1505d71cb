"""C-ABI checks that need no GPU: the library loads, exports every function
declared in include/tri.h, its structs match the ctypes mirrors, and host-side
validation rejects bad arguments before any launch.

Every call below fails validation, so no kernel is ever launched (the fake
device addresses are never dereferenced).
"""
import ctypes
import os
import re
import subprocess
import tempfile

import pytest

from paper_2606_29629_amd import _lib as T

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "tri.h")


@pytest.fixture(scope="module")
def lib():
    import torch
    if torch.cuda.is_available():
        pytest.skip("fake-address validation tests run only where no GPU is visible")
    if not os.path.exists(T.LIB_PATH):
        pytest.skip("libtri.so not built (run python -m paper_2606_29629_amd.build)")
    return T.lib()


def declared_functions():
    src = open(HEADER).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(tri_[a-z_]+)\s*\(", src)))


def test_exports_every_declared_function(lib):
    names = declared_functions()
    assert "tri_layer_prefill" in names and "tri_kvcache_append" in names
    for n in names:
        assert hasattr(lib, n), n
    out = subprocess.run(["nm", "-D", "--defined-only", T.LIB_PATH], capture_output=True,
                         text=True).stdout
    exported = set(re.findall(r" T (tri_\w+)", out))
    assert set(names) <= exported
    assert lib.tri_version() >= 100


STRUCTS = {
    "tri_layer_config": (T.LayerConfig, [f for f, _ in T.LayerConfig._fields_]),
    "tri_layer_weights": (T.LayerWeights, [f for f, _ in T.LayerWeights._fields_]),
    "tri_kv_cache": (T.KVCache, [f for f, _ in T.KVCache._fields_]),
    "tri_batch": (T.BatchStruct, [f for f, _ in T.BatchStruct._fields_]),
    "tri_workspace_map": (T.WorkspaceMap, [f for f, _ in T.WorkspaceMap._fields_]),
    "tri_profile": (T.Profile, [f for f, _ in T.Profile._fields_]),
    "tri_work": (T.Work, [f for f, _ in T.Work._fields_]),
}


def test_struct_layout_matches_header():
    lines = ['#include <stdio.h>', '#include <stddef.h>', '#include "tri.h"', "int main(void){"]
    for cname, (_, fields) in STRUCTS.items():
        lines.append(f'printf("{cname} size %zu\\n", sizeof({cname}));')
        for f in fields:
            lines.append(f'printf("{cname} {f} %zu\\n", offsetof({cname}, {f}));')
    lines.append("return 0;}")
    with tempfile.TemporaryDirectory() as d:
        c = os.path.join(d, "probe.c")
        open(c, "w").write("\n".join(lines))
        exe = os.path.join(d, "probe")
        subprocess.run(["gcc", "-std=c99", "-I", os.path.dirname(HEADER), c, "-o", exe], check=True)
        out = subprocess.run([exe], capture_output=True, text=True, check=True).stdout
    got = {}
    for line in out.splitlines():
        a, b, v = line.split()
        got[(a, b)] = int(v)
    for cname, (cls, fields) in STRUCTS.items():
        assert got[(cname, "size")] == ctypes.sizeof(cls), cname
        for f in fields:
            assert got[(cname, f)] == getattr(cls, f).offset, (cname, f)


# ------------------------------------------------------------ validation --

FAKE = 0x7F0000000000  # 256-byte aligned fake device address, never dereferenced


def cfg(**kw):
    base = dict(hidden=256, n_q_heads=4, n_kv_heads=2, head_dim=64, ffn_dim=1024,
                n_experts=0, top_k=0, expert_ffn_dim=0, rms_eps=1e-6, rope_base=1e6,
                dtype=T.TRI_BF16, flags=0)
    base.update(kw)
    return T.LayerConfig(**base)


def batch(n_seqs=1, n_tokens=4, max_q=4, max_ctx=0, ptr=FAKE):
    return T.BatchStruct(n_seqs, n_tokens, max_q, max_ctx, ptr, ptr + 256, ptr + 512, ptr + 768)


def weights(ptr=FAKE):
    w = T.LayerWeights(*[ptr + 4096 * i for i in range(10)])
    w.b_qkv = None
    w.w_router = None
    return w


def call(lib, fn="tri_layer_prefill", c=None, w=None, kv=None, b=None, x=FAKE + (1 << 20),
         out=FAKE + (2 << 20), ws=FAKE + (3 << 20), ws_bytes=1 << 30):
    c = cfg() if c is None else c
    w = weights() if w is None else w
    kv = T.KVCache(FAKE + (4 << 20), FAKE + (5 << 20), 1, 64, None, 0, 0) if kv is None else kv
    b = batch() if b is None else b
    return getattr(lib, fn)(ctypes.byref(c), ctypes.byref(w), ctypes.byref(kv), ctypes.byref(b),
                            x, out, None, None, ws, ws_bytes, None)


def test_null_and_unsupported(lib):
    assert lib.tri_layer_prefill(None, None, None, None, None, None, None, None, None, 0,
                                 None) == T.TRI_ERR_NULL
    assert call(lib, c=cfg(head_dim=96)) == T.TRI_ERR_UNSUPPORTED
    assert call(lib, c=cfg(dtype=2)) == T.TRI_ERR_UNSUPPORTED        # no such storage type
    assert call(lib, c=cfg(flags=64)) == T.TRI_ERR_UNSUPPORTED
    assert call(lib, c=cfg(hidden=200)) == T.TRI_ERR_UNSUPPORTED
    assert call(lib, c=cfg(ffn_dim=100)) == T.TRI_ERR_UNSUPPORTED
    assert call(lib, c=cfg(n_q_heads=5)) == T.TRI_ERR_SHAPE
    assert call(lib, c=cfg(n_q_heads=66, n_kv_heads=2)) == T.TRI_ERR_UNSUPPORTED  # group > 32
    assert call(lib, c=cfg(rope_base=0.0)) == T.TRI_ERR_RANGE
    assert call(lib, w=T.LayerWeights()) == T.TRI_ERR_NULL
    assert call(lib, x=None) == T.TRI_ERR_NULL
    assert call(lib, c=cfg(flags=T.TRI_F_QKV_BIAS)) == T.TRI_ERR_NULL    # bias flag, no bias
    for name in ("q_norm", "k_norm"):                                      # q/k norm gains
        w = weights()
        setattr(w, name, None)
        assert call(lib, c=cfg(flags=T.TRI_F_QK_NORM), w=w) == T.TRI_ERR_NULL
        setattr(w, name, FAKE + 2)
        assert call(lib, c=cfg(flags=T.TRI_F_QK_NORM), w=w) == T.TRI_ERR_ALIGN
        w = weights()
        setattr(w, name, None)                                             # ignored without the flag
        assert call(lib, w=w, ws_bytes=1024) == T.TRI_ERR_WORKSPACE
    bb = batch()
    bb.cu_q = None
    assert call(lib, b=bb) == T.TRI_ERR_NULL


def test_mrope_config_checks(lib):
    def mc(sec):
        c = cfg(flags=T.TRI_F_MROPE)
        c.mrope_section[:] = sec
        return c
    assert call(lib, c=mc((8, 12, 12)), ws_bytes=1024) == T.TRI_ERR_WORKSPACE   # valid: D/2 = 32
    assert call(lib, c=mc((32, 0, 0)), ws_bytes=1024) == T.TRI_ERR_WORKSPACE
    assert call(lib, c=mc((8, 12, 11))) == T.TRI_ERR_SHAPE                     # sums to 31
    assert call(lib, c=mc((-1, 21, 12))) == T.TRI_ERR_SHAPE
    assert call(lib, c=mc((0, 0, 0))) == T.TRI_ERR_SHAPE
    c = cfg()
    c.mrope_section[:] = (1, 1, 1)                                              # ignored without the flag
    assert call(lib, c=c, ws_bytes=1024) == T.TRI_ERR_WORKSPACE


def test_moe_config_checks(lib):
    moe = dict(flags=T.TRI_F_MOE, n_experts=8, top_k=2, expert_ffn_dim=128, ffn_dim=0)
    assert call(lib, c=cfg(**dict(moe, top_k=9))) == T.TRI_ERR_SHAPE
    assert call(lib, c=cfg(**dict(moe, top_k=0))) == T.TRI_ERR_SHAPE
    assert call(lib, c=cfg(**dict(moe, n_experts=300))) == T.TRI_ERR_UNSUPPORTED
    assert call(lib, c=cfg(**dict(moe, expert_ffn_dim=100))) == T.TRI_ERR_UNSUPPORTED
    assert call(lib, c=cfg(**moe)) == T.TRI_ERR_NULL          # MoE needs w_router


def test_batch_checks(lib):
    assert call(lib, b=batch(n_seqs=0, n_tokens=4)) == T.TRI_ERR_SHAPE
    assert call(lib, b=batch(n_seqs=1, n_tokens=4, max_q=2)) == T.TRI_ERR_SHAPE
    assert call(lib, b=batch(n_seqs=-1)) == T.TRI_ERR_SHAPE
    assert call(lib, b=batch(max_ctx=64)) == T.TRI_ERR_RANGE               # no row left
    assert call(lib, b=batch(n_seqs=2, n_tokens=65, max_q=65)) == T.TRI_ERR_RANGE
    assert call(lib, fn="tri_layer_decode", b=batch(n_seqs=1, n_tokens=1, max_q=1, max_ctx=64)) == T.TRI_ERR_RANGE
    assert call(lib, kv=T.KVCache(FAKE, FAKE + 256, 0, 64, None, 0, 0)) == T.TRI_ERR_SHAPE
    # decode needs one token per sequence
    assert call(lib, fn="tri_layer_decode", b=batch(n_seqs=2, n_tokens=4, max_q=2)) == T.TRI_ERR_SHAPE


def test_alignment_workspace_alias(lib):
    assert call(lib, x=FAKE + (1 << 20) + 8) == T.TRI_ERR_ALIGN
    assert call(lib, ws=FAKE + (3 << 20) + 16) == T.TRI_ERR_ALIGN   # workspace needs 256 B
    w = weights()
    w.w_o = FAKE + 2
    assert call(lib, w=w) == T.TRI_ERR_ALIGN
    assert call(lib, ws_bytes=1024) == T.TRI_ERR_WORKSPACE
    assert call(lib, out=FAKE + (1 << 20) + 256) == T.TRI_ERR_ALIAS          # overlaps x_in
    assert call(lib, ws=FAKE + (1 << 20)) == T.TRI_ERR_ALIAS


def test_empty_batch_is_a_noop(lib):
    # n_tokens == 0: nothing to do, nothing launched, null data pointers allowed
    assert call(lib, b=batch(n_seqs=0, n_tokens=0, max_q=0), x=None, out=None, ws=None) == T.TRI_OK


def test_workspace_size_and_layout(lib):
    c = cfg()
    sizes = []
    for n in (1, 32, 200, 4096):
        b = batch(n_seqs=1, n_tokens=n, max_q=n, max_ctx=0)
        s = ctypes.c_size_t()
        assert lib.tri_workspace_size(ctypes.byref(c), ctypes.byref(b), ctypes.byref(s)) == 0
        m = T.WorkspaceMap()
        assert lib.tri_workspace_layout(ctypes.byref(c), ctypes.byref(b), ctypes.byref(m)) == 0
        assert m.total == s.value
        offs = [m.h, m.q, m.attn, m.x1, m.h2, m.act]
        assert offs == sorted(offs) and all(o % 256 == 0 for o in offs)
        assert m.act + n * 1024 * 2 <= m.total
        sizes.append(s.value)
    assert sizes == sorted(sizes)
    assert lib.tri_workspace_size(ctypes.byref(c), None, None) == T.TRI_ERR_NULL


def test_workspace_of_f32_storage(lib):
    """fp32 storage: fp32 activations and the bf16 operand planes (three per
    value) of every weight matrix and of the widest activation operand."""
    H, Hq, Hkv, D, F = 256, 4, 2, 64, 1024
    c = cfg(dtype=T.TRI_F32)
    T_ = 40
    b = batch(n_seqs=1, n_tokens=T_, max_q=T_, max_ctx=0)
    s = ctypes.c_size_t()
    assert lib.tri_workspace_size(ctypes.byref(c), ctypes.byref(b), ctypes.byref(s)) == 0
    params = (Hq + 2 * Hkv) * D * H + H * Hq * D + 3 * F * H
    acts = T_ * (3 * H + 2 * Hq * D + F) * 4
    assert s.value >= params * 6 + acts + T_ * F * 6
    m = T.WorkspaceMap()
    assert lib.tri_workspace_layout(ctypes.byref(c), ctypes.byref(b), ctypes.byref(m)) == 0
    assert m.x1 - m.attn == -(-T_ * Hq * D * 4 // 256) * 256      # attention output in fp32
    sb = ctypes.c_size_t()
    cb = cfg()
    assert lib.tri_workspace_size(ctypes.byref(cb), ctypes.byref(b), ctypes.byref(sb)) == 0
    assert s.value > sb.value


def test_workspace_of_long_chunked_prefill(lib):
    """Chunked prefill over a long cached prefix: the workspace holds the
    layer's activations plus scratch that grows with the number of sequences,
    not with tokens x prefix (the split-KV partials serve single-token
    sequences and are indexed by sequence)."""
    H, Hq, Hkv, D, F = 3584, 28, 4, 128, 18944
    c = cfg(hidden=H, n_q_heads=Hq, n_kv_heads=Hkv, head_dim=D, ffn_dim=F)

    def size(n_seqs, q, ctx, n_tokens=None):
        n_tokens = n_seqs * q if n_tokens is None else n_tokens
        b = batch(n_seqs=n_seqs, n_tokens=n_tokens, max_q=q, max_ctx=ctx)
        s = ctypes.c_size_t()
        assert lib.tri_workspace_size(ctypes.byref(c), ctypes.byref(b), ctypes.byref(s)) == 0
        return s.value

    def activations(t):
        return t * (4 + 4 + (D // 2) * 8 + 3 * H * 2 + 2 * Hq * D * 2 + F * 2)

    # scratch beyond the activations: the large GEMMs' tail-tile partials (one
    # 256 x 256 fp32 tile per compute unit, 256 CUs without a device), which the
    # split-KV partials share, plus 256-byte alignment of the regions
    scratch = 256 * 256 * 256 * 4 + 20 * 256
    for ctx in (8192, 30000):
        t = 8 * 2048
        assert size(8, 2048, ctx) <= activations(t) + scratch + 8 * Hq * 235 * (D + 2) * 4, ctx
    assert size(8, 2048, 8192) <= activations(8 * 2048) + scratch
    # the prefix adds only per-sequence partials: 8 x Hq x ceil(dctx / 128) x (D + 2) floats
    grow = size(8, 2048, 30000) - size(8, 2048, 8192)
    assert 0 <= grow <= 8 * Hq * -(-(30000 - 8192) // 128 + 1) * (D + 2) * 4 + 4096
    # the mixed step's shape: a 512-token chunk at 6144 plus 32 decodes up to 8192
    assert size(33, 512, 8192, n_tokens=544) <= activations(544) + scratch


def test_kvcache_append_and_route_validation(lib):
    c = cfg()
    kv = T.KVCache(FAKE, FAKE + 4096, 1, 64, None, 0, 0)
    b = batch(max_ctx=64)
    assert lib.tri_kvcache_append(ctypes.byref(c), ctypes.byref(kv), ctypes.byref(b), FAKE,
                                  FAKE, None) == T.TRI_ERR_RANGE
    b = batch()
    assert lib.tri_kvcache_append(ctypes.byref(c), ctypes.byref(kv), ctypes.byref(b), FAKE + 8,
                                  FAKE, None) == T.TRI_ERR_ALIGN
    assert lib.tri_kvcache_append(ctypes.byref(c), ctypes.byref(kv), ctypes.byref(b), None,
                                  FAKE, None) == T.TRI_ERR_NULL
    assert lib.tri_moe_route(ctypes.byref(c), FAKE, FAKE, 4, FAKE, FAKE, None) == T.TRI_ERR_SHAPE
    m = cfg(flags=T.TRI_F_MOE, n_experts=8, top_k=2, expert_ffn_dim=128, ffn_dim=0)
    assert lib.tri_moe_route(ctypes.byref(m), None, FAKE, 4, FAKE, FAKE, None) == T.TRI_ERR_NULL
    assert lib.tri_moe_route(ctypes.byref(m), FAKE + 4, FAKE, 4, FAKE, FAKE, None) == T.TRI_ERR_ALIGN
    assert lib.tri_moe_route(ctypes.byref(m), FAKE, FAKE, -1, FAKE, FAKE, None) == T.TRI_ERR_SHAPE


def test_noalloc_rejects_batches_beyond_its_scratch(lib):
    """The no-allocation decode entry refuses, before touching any device, a
    batch whose workspace would exceed its fixed scratch."""
    c = cfg(hidden=3584, n_q_heads=28, n_kv_heads=4, head_dim=128, ffn_dim=18944)
    b = batch(n_seqs=512, n_tokens=512, max_q=1, max_ctx=30000)
    need = ctypes.c_size_t()
    assert lib.tri_workspace_size(ctypes.byref(c), ctypes.byref(b), ctypes.byref(need)) == 0
    assert need.value > T.NOALLOC_SCRATCH_BYTES
    kv = T.KVCache(FAKE, FAKE + (1 << 30), 512, 30080, None, 0, 0)
    w = weights()
    st = lib.tri_layer_decode_noalloc(ctypes.byref(c), ctypes.byref(w), ctypes.byref(kv),
                                      ctypes.byref(b), FAKE + (2 << 30), FAKE + (3 << 30), None,
                                      None, None)
    assert st == T.TRI_ERR_SCRATCH
    # validation errors come first, as in tri_layer_decode
    st = lib.tri_layer_decode_noalloc(None, ctypes.byref(w), ctypes.byref(kv), ctypes.byref(b),
                                      FAKE, FAKE, None, None, None)
    assert st == T.TRI_ERR_NULL


def test_decode_batches_fit_the_noalloc_scratch(lib):
    """The decode workloads fit the no-allocation entry's scratch: a batch
    with no multi-token sequence reserves no flash-attention partials (they
    sit beside the split-KV partials only when both kernels run)."""
    dense = cfg(hidden=3584, n_q_heads=28, n_kv_heads=4, head_dim=128, ffn_dim=18944)
    moe = cfg(hidden=2048, n_q_heads=32, n_kv_heads=4, head_dim=128, ffn_dim=768,
              flags=T.TRI_F_MOE, n_experts=128, top_k=8, expert_ffn_dim=768)
    for c, n, ctx in ((dense, 64, 4096), (moe, 128, 2048)):
        need = ctypes.c_size_t()
        b = batch(n_seqs=n, n_tokens=n, max_q=1, max_ctx=ctx)
        assert lib.tri_workspace_size(ctypes.byref(c), ctypes.byref(b), ctypes.byref(need)) == 0
        assert need.value <= T.NOALLOC_SCRATCH_BYTES, (n, ctx, need.value)
    # a chunk beside decodes reserves both kinds of attention partials
    b1 = batch(n_seqs=33, n_tokens=544, max_q=512, max_ctx=8192)
    b2 = batch(n_seqs=1, n_tokens=512, max_q=512, max_ctx=8192)
    s1, s2 = ctypes.c_size_t(), ctypes.c_size_t()
    assert lib.tri_workspace_size(ctypes.byref(dense), ctypes.byref(b1), ctypes.byref(s1)) == 0
    assert lib.tri_workspace_size(ctypes.byref(dense), ctypes.byref(b2), ctypes.byref(s2)) == 0
    assert s1.value >= s2.value


def test_linear_validation(lib):
    """tri_linear checks shapes, pointers, alignment, ranges, workspace and
    aliasing before any launch (fake device addresses: nothing runs)."""
    ws = ctypes.c_size_t()
    assert lib.tri_linear_workspace_size(64, 4096, 4096, ctypes.byref(ws)) == 0
    assert ws.value > 0                       # short batch: split-K partials
    big = ctypes.c_size_t()
    assert lib.tri_linear_workspace_size(1024, 4096, 4096, ctypes.byref(big)) == 0
    assert big.value == 256 * 256 * 256 * 4   # the large GEMMs' tail tiles
    assert lib.tri_linear_workspace_size(8, 64, 100, ctypes.byref(ws)) == T.TRI_ERR_SHAPE
    assert lib.tri_linear_workspace_size(8, 6, 64, ctypes.byref(ws)) == T.TRI_ERR_SHAPE
    assert lib.tri_linear_workspace_size(0, 64, 64, ctypes.byref(ws)) == T.TRI_ERR_SHAPE
    assert lib.tri_linear_workspace_size(8, 64, 64, None) == T.TRI_ERR_NULL
    # Every call below must fail validation (the pointers are fake): the
    # shape needs split-K partials, so a missing workspace is an error too.
    A, B, C, W = FAKE, FAKE + (1 << 30), FAKE + (2 << 30), FAKE + (3 << 30)
    M, N, K = 64, 4096, 4096
    need = ctypes.c_size_t()
    assert lib.tri_linear_workspace_size(M, N, K, ctypes.byref(need)) == 0 and need.value > 0
    f = lib.tri_linear
    ok_ws = need.value
    assert f(None, B, C, M, N, K, W, ok_ws, None) == T.TRI_ERR_NULL
    assert f(A + 8, B, C, M, N, K, W, ok_ws, None) == T.TRI_ERR_ALIGN
    assert f(A, B, C, M, N, K, None, 0, None) == T.TRI_ERR_WORKSPACE
    assert f(A, B, C, M, N, K, W, ok_ws - 1, None) == T.TRI_ERR_WORKSPACE
    assert f(A, B, C, M, N, K, W + 16, ok_ws, None) == T.TRI_ERR_ALIGN
    assert f(A, B, A, M, N, K, W, ok_ws, None) == T.TRI_ERR_ALIAS
    assert f(A, B, C, 8, 1 << 20, 1024, W, 1 << 30, None) == T.TRI_ERR_RANGE
    assert f(A, B, C, M, N, 96, W, ok_ws, None) == T.TRI_ERR_SHAPE


def test_status_strings(lib):
    for s in range(-9, 1):
        assert T.status_string(s) and T.status_string(s) != "unknown status"
    assert T.status_string(-99) == "unknown status"


def test_paged_cache_validation(lib):
    tab = FAKE + (6 << 20)
    ok = T.KVCache(FAKE + (4 << 20), FAKE + (5 << 20), 1, 128, tab, 64, 4)
    assert call(lib, kv=ok, ws_bytes=0) == T.TRI_ERR_WORKSPACE  # passes the cache checks
    assert call(lib, kv=T.KVCache(FAKE, FAKE + 256, 1, 128, tab, 32, 4)) == T.TRI_ERR_UNSUPPORTED
    assert call(lib, kv=T.KVCache(FAKE, FAKE + 256, 1, 96, tab, 64, 4)) == T.TRI_ERR_SHAPE
    assert call(lib, kv=T.KVCache(FAKE, FAKE + 256, 1, 128, tab, 64, 0)) == T.TRI_ERR_SHAPE
    assert call(lib, kv=T.KVCache(FAKE, FAKE + 256, 1, 128, tab + 2, 64, 4)) == T.TRI_ERR_ALIGN
    b = batch()
    kn = FAKE + (7 << 20)
    assert lib.tri_kvcache_append(ctypes.byref(cfg()), ctypes.byref(
        T.KVCache(FAKE, FAKE + 256, 1, 128, tab, 48, 4)), ctypes.byref(b), kn, kn + 4096,
        None) == T.TRI_ERR_UNSUPPORTED


def test_workspace_size_never_shrinks_as_tokens_grow(lib):
    """tri_workspace_size is non-decreasing in n_tokens for a fixed config (the
    header's promise): a workspace sized for the largest batch serves every
    smaller one.  Checked token by token across the short-batch paths, whose
    64-row and 128-row tiles split K differently, and past them."""
    dense = cfg(hidden=3584, n_q_heads=28, n_kv_heads=4, head_dim=128, ffn_dim=18944)
    moe = cfg(hidden=2048, n_q_heads=32, n_kv_heads=4, head_dim=128, ffn_dim=0,
              n_experts=128, top_k=8, expert_ffn_dim=768, flags=T.TRI_F_MOE)
    shapes = (lambda n: batch(n_seqs=n, n_tokens=n, max_q=1, max_ctx=4096),  # decode steps
              lambda n: batch(n_seqs=1, n_tokens=n, max_q=n, max_ctx=0))     # one prompt
    for c in (dense, moe):
        for shape in shapes:
            prev = 0
            for n in list(range(1, 300)) + [512, 1024, 4096]:
                b = shape(n)
                s = ctypes.c_size_t()
                assert lib.tri_workspace_size(ctypes.byref(c), ctypes.byref(b),
                                              ctypes.byref(s)) == 0
                assert s.value >= prev, (c.hidden, n, s.value, prev)
                prev = s.value
