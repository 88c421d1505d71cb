"""ctypes binding of libtri (include/tri.h).

Argument marshalling only: every step of the layer runs in the HIP kernels of
libtri.so.  torch supplies device memory (``tensor.data_ptr()``) and the
current HIP stream.  Loading fails loudly if the library has not been built.
"""
from __future__ import annotations

import ctypes
import os
from typing import Dict, Optional, Sequence

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libtri.so")

TRI_OK, TRI_ERR_NULL, TRI_ERR_SHAPE, TRI_ERR_UNSUPPORTED = 0, -1, -2, -3
TRI_ERR_RANGE, TRI_ERR_ALIGN, TRI_ERR_WORKSPACE, TRI_ERR_HIP, TRI_ERR_ALIAS = -4, -5, -6, -7, -8
TRI_ERR_SCRATCH = -9
NOALLOC_SCRATCH_BYTES = 64 << 20
TRI_BF16, TRI_F32 = 0, 1
TRI_F_QKV_BIAS, TRI_F_MOE, TRI_F_MOE_RENORM, TRI_F_QK_NORM, TRI_F_MROPE = 1, 2, 4, 8, 16


class LayerConfig(ctypes.Structure):
    _fields_ = [("hidden", ctypes.c_int32), ("n_q_heads", ctypes.c_int32),
                ("n_kv_heads", ctypes.c_int32), ("head_dim", ctypes.c_int32),
                ("ffn_dim", ctypes.c_int32), ("n_experts", ctypes.c_int32),
                ("top_k", ctypes.c_int32), ("expert_ffn_dim", ctypes.c_int32),
                ("rms_eps", ctypes.c_float), ("rope_base", ctypes.c_float),
                ("dtype", ctypes.c_int32), ("flags", ctypes.c_int32),
                ("mrope_section", ctypes.c_int32 * 3)]


class LayerWeights(ctypes.Structure):
    _fields_ = [(n, ctypes.c_void_p) for n in
                ("attn_norm", "w_qkv", "b_qkv", "w_o", "mlp_norm", "w_gate_up", "w_down",
                 "w_router", "q_norm", "k_norm")]


class KVCache(ctypes.Structure):
    _fields_ = [("k", ctypes.c_void_p), ("v", ctypes.c_void_p), ("n_slots", ctypes.c_int32),
                ("max_seq", ctypes.c_int32), ("block_table", ctypes.c_void_p),
                ("block_size", ctypes.c_int32), ("n_blocks", ctypes.c_int32)]


class BatchStruct(ctypes.Structure):
    _fields_ = [("n_seqs", ctypes.c_int32), ("n_tokens", ctypes.c_int32),
                ("max_q_len", ctypes.c_int32), ("max_ctx_len", ctypes.c_int32),
                ("cu_q", ctypes.c_void_p), ("ctx_len", ctypes.c_void_p),
                ("slot", ctypes.c_void_p), ("pos", ctypes.c_void_p)]


class WorkspaceMap(ctypes.Structure):
    _fields_ = [(n, ctypes.c_size_t) for n in ("h", "q", "attn", "x1", "h2", "act", "perm", "y",
                                                "total")]


class Profile(ctypes.Structure):
    _fields_ = [("n_stages", ctypes.c_int32), ("name", ctypes.c_char_p * 16),
                ("launches", ctypes.c_int32 * 16), ("total_ms", ctypes.c_double * 16)]


class Work(ctypes.Structure):
    _fields_ = [("n_stages", ctypes.c_int32), ("name", ctypes.c_char_p * 16),
                ("runs", ctypes.c_int32 * 16), ("flops", ctypes.c_double * 16),
                ("bytes", ctypes.c_double * 16)]


class TriError(RuntimeError):
    def __init__(self, status: int, what: str):
        self.status = status
        super().__init__(f"{what}: tri status {status} ({status_string(status)})")


_lib: Optional[ctypes.CDLL] = None

_FUNCS = {
    "tri_workspace_size": (ctypes.c_int, [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p]),
    "tri_workspace_layout": (ctypes.c_int, [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p]),
    "tri_layer_prefill": (ctypes.c_int, [ctypes.c_void_p] * 4 + [ctypes.c_void_p] * 4
                          + [ctypes.c_void_p, ctypes.c_size_t, ctypes.c_void_p]),
    "tri_layer_decode": (ctypes.c_int, [ctypes.c_void_p] * 4 + [ctypes.c_void_p] * 4
                         + [ctypes.c_void_p, ctypes.c_size_t, ctypes.c_void_p]),
    "tri_layer_decode_noalloc": (ctypes.c_int, [ctypes.c_void_p] * 4 + [ctypes.c_void_p] * 4
                                 + [ctypes.c_void_p]),
    "tri_kvcache_append": (ctypes.c_int, [ctypes.c_void_p] * 6),
    "tri_moe_route": (ctypes.c_int, [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p,
                                     ctypes.c_int32, ctypes.c_void_p, ctypes.c_void_p,
                                     ctypes.c_void_p]),
    "tri_status_string": (ctypes.c_char_p, [ctypes.c_int]),
    "tri_profile_enable": (ctypes.c_int, [ctypes.c_int32]),
    "tri_profile_read": (ctypes.c_int, [ctypes.c_void_p]),
    "tri_layer_work": (ctypes.c_int, [ctypes.c_void_p, ctypes.c_int32, ctypes.c_int32,
                                      ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p,
                                      ctypes.c_void_p]),
    "tri_phase_intensity": (ctypes.c_int, [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p]),
    "tri_version": (ctypes.c_int32, []),
    "tri_linear_workspace_size": (ctypes.c_int, [ctypes.c_int32] * 3 + [ctypes.c_void_p]),
    "tri_linear": (ctypes.c_int, [ctypes.c_void_p] * 3 + [ctypes.c_int32] * 3
                   + [ctypes.c_void_p, ctypes.c_size_t, ctypes.c_void_p]),
}


def lib() -> ctypes.CDLL:
    """The loaded libtri.so (raises if it has not been built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"libtri.so not built at {LIB_PATH}; run "
                               "`python -m paper_2606_29629_amd.build` first")
        l = ctypes.CDLL(LIB_PATH)
        for name, (res, args) in _FUNCS.items():
            f = getattr(l, name)
            f.restype = res
            f.argtypes = args
        _lib = l
    return _lib


def status_string(s: int) -> str:
    return lib().tri_status_string(s).decode()


def _check(status: int, what: str) -> None:
    if status != TRI_OK:
        raise TriError(status, what)


def make_config(cfg, f32: bool = False) -> LayerConfig:
    """LayerConfig from any object with the layer's attribute names; f32
    selects the fp32 storage mode (TRI_F32: fp32 weights, activations and
    cache)."""
    flags = 0
    if getattr(cfg, "qkv_bias", False):
        flags |= TRI_F_QKV_BIAS
    if getattr(cfg, "qk_norm", False):
        flags |= TRI_F_QK_NORM
    sec = getattr(cfg, "mrope_section", None)
    if sec:
        flags |= TRI_F_MROPE
    n_exp = int(getattr(cfg, "n_experts", 0) or 0)
    if n_exp > 0:
        flags |= TRI_F_MOE
        if getattr(cfg, "moe_renorm", True):
            flags |= TRI_F_MOE_RENORM
    return LayerConfig(int(cfg.hidden), int(cfg.n_q_heads), int(cfg.n_kv_heads),
                       int(cfg.head_dim), int(getattr(cfg, "ffn_dim", 0) or 0), n_exp,
                       int(getattr(cfg, "top_k", 0) or 0),
                       int(getattr(cfg, "expert_ffn_dim", 0) or 0), float(cfg.rms_eps),
                       float(cfg.rope_base), TRI_F32 if f32 else TRI_BF16, flags,
                       (ctypes.c_int32 * 3)(*(sec or (0, 0, 0))))


def _ptr(t) -> Optional[int]:
    return None if t is None else t.data_ptr()


def _stream(stream) -> Optional[int]:
    if stream is None:
        import torch
        return torch.cuda.current_stream().cuda_stream
    return getattr(stream, "cuda_stream", stream)


class DeviceBatch:
    """A ragged batch: device int32 arrays plus the host scalars that size launches."""

    def __init__(self, slot: Sequence[int], ctx_len: Sequence[int], q_len: Sequence[int],
                 device="cuda", pos=None):
        """pos: the rotary positions (default ctx_len + i per token), or the
        three planes [3, n_tokens] of a TRI_F_MROPE layer."""
        import numpy as np
        import torch
        slot = np.asarray(slot, dtype=np.int32)
        ctx = np.asarray(ctx_len, dtype=np.int32)
        q = np.asarray(q_len, dtype=np.int32)
        cu = np.concatenate([[0], np.cumsum(q)]).astype(np.int32)
        if pos is not None:
            pos = np.ascontiguousarray(pos, dtype=np.int32).ravel()
        elif len(q):
            pos = np.concatenate([np.arange(c, c + n) for c, n in zip(ctx, q)]).astype(np.int32)
        else:
            pos = np.zeros(0, np.int32)
        self.n_seqs, self.n_tokens = int(len(q)), int(cu[-1])
        self.max_q_len = int(q.max()) if len(q) else 0
        self.max_ctx_len = int(ctx.max()) if len(ctx) else 0
        dev = lambda a: torch.from_numpy(np.ascontiguousarray(a)).to(device)
        self.cu_q, self.ctx_len, self.slot, self.pos = dev(cu), dev(ctx), dev(slot), dev(pos)
        self.host = dict(slot=slot, ctx_len=ctx, q_len=q)

    def struct(self) -> BatchStruct:
        return BatchStruct(self.n_seqs, self.n_tokens, self.max_q_len, self.max_ctx_len,
                           _ptr(self.cu_q), _ptr(self.ctx_len), _ptr(self.slot), _ptr(self.pos))

    def advance(self) -> None:
        """In place: every sequence has appended its new tokens; next step is one token each."""
        import numpy as np
        h = self.host
        ctx = (h["ctx_len"] + h["q_len"]).astype(np.int32)
        self.__init__(h["slot"], ctx, np.ones_like(h["q_len"]), device=self.cu_q.device)


def weights_struct(w: Dict[str, object]) -> LayerWeights:
    return LayerWeights(*[_ptr(w.get(n)) for n in
                          ("attn_norm", "w_qkv", "b_qkv", "w_o", "mlp_norm", "w_gate_up",
                           "w_down", "w_router", "q_norm", "k_norm")])


def workspace_size(cfg: LayerConfig, batch: DeviceBatch) -> int:
    n = ctypes.c_size_t(0)
    b = batch.struct()
    _check(lib().tri_workspace_size(ctypes.byref(cfg), ctypes.byref(b), ctypes.byref(n)),
           "tri_workspace_size")
    return n.value


def workspace_layout(cfg: LayerConfig, batch: DeviceBatch) -> WorkspaceMap:
    m = WorkspaceMap()
    b = batch.struct()
    _check(lib().tri_workspace_layout(ctypes.byref(cfg), ctypes.byref(b), ctypes.byref(m)),
           "tri_workspace_layout")
    return m


class PagedCache:
    """A paged KV cache: K and V pools [n_blocks, Hkv, block_size, D] (bf16) and
    a device int32 block table [n_slots, max_seq / block_size]."""

    def __init__(self, k_pool, v_pool, block_table, max_seq: int):
        self.k, self.v, self.block_table = k_pool, v_pool, block_table
        self.n_slots = int(block_table.shape[0])
        self.max_seq = int(max_seq)
        self.block_size = int(k_pool.shape[2])
        self.n_blocks = int(k_pool.shape[0])

    def __getitem__(self, i):
        return (self.k, self.v)[i]


def kv_struct(cache) -> KVCache:
    """KVCache for a contiguous (k, v) pair [n_slots, Hkv, max_seq, D] or a PagedCache."""
    if isinstance(cache, PagedCache):
        return KVCache(_ptr(cache.k), _ptr(cache.v), cache.n_slots, cache.max_seq,
                       _ptr(cache.block_table), cache.block_size, cache.n_blocks)
    return KVCache(_ptr(cache[0]), _ptr(cache[1]), int(cache[0].shape[0]),
                   int(cache[0].shape[2]), None, 0, 0)


def _layer(fn_name, cfg, w, cache, batch, x, out, workspace, route_idx, route_w, stream):
    import torch
    if out is None:
        out = torch.empty_like(x)
    need = workspace_size(cfg, batch)
    if workspace is None:
        workspace = torch.empty(max(need, 1), dtype=torch.uint8, device=x.device)
    ws = weights_struct(w)
    kc = kv_struct(cache)
    b = batch.struct()
    st = getattr(lib(), fn_name)(ctypes.byref(cfg), ctypes.byref(ws), ctypes.byref(kc),
                                 ctypes.byref(b), _ptr(x), _ptr(out), _ptr(route_idx),
                                 _ptr(route_w), _ptr(workspace), workspace.numel(),
                                 _stream(stream))
    _check(st, fn_name)
    return out, workspace


def layer_prefill(cfg, w, cache, batch, x, out=None, workspace=None, route_idx=None,
                  route_w=None, stream=None):
    """One decoder layer over a ragged batch; returns (out, workspace)."""
    return _layer("tri_layer_prefill", cfg, w, cache, batch, x, out, workspace, route_idx,
                  route_w, stream)


def layer_decode(cfg, w, cache, batch, x, out=None, workspace=None, route_idx=None,
                 route_w=None, stream=None):
    """One decode step (one new token per sequence); returns (out, workspace)."""
    return _layer("tri_layer_decode", cfg, w, cache, batch, x, out, workspace, route_idx,
                  route_w, stream)


def layer_decode_noalloc(cfg, w, cache, batch, x, out=None, route_idx=None, route_w=None,
                         stream=None):
    """One decode step on the library's fixed device scratch (no workspace;
    tri_layer_decode_noalloc); returns out."""
    import torch
    if out is None:
        out = torch.empty_like(x)
    ws = weights_struct(w)
    kc = kv_struct(cache)
    b = batch.struct()
    _check(lib().tri_layer_decode_noalloc(ctypes.byref(cfg), ctypes.byref(ws), ctypes.byref(kc),
                                          ctypes.byref(b), _ptr(x), _ptr(out), _ptr(route_idx),
                                          _ptr(route_w), _stream(stream)),
           "tri_layer_decode_noalloc")
    return out


def kvcache_append(cfg, cache, batch, k_new, v_new, stream=None) -> None:
    kc = kv_struct(cache)
    b = batch.struct()
    _check(lib().tri_kvcache_append(ctypes.byref(cfg), ctypes.byref(kc), ctypes.byref(b),
                                    _ptr(k_new), _ptr(v_new), _stream(stream)),
           "tri_kvcache_append")


def linear_workspace_size(M: int, N: int, K: int) -> int:
    n = ctypes.c_size_t()
    _check(lib().tri_linear_workspace_size(int(M), int(N), int(K), ctypes.byref(n)),
           "tri_linear_workspace_size")
    return n.value


def linear(a, b, out=None, workspace=None, stream=None):
    """out = a @ b^T (bf16 [M, K] x bf16 [N, K] -> bf16 [M, N]) through tri_linear."""
    import torch
    M, K = a.shape
    N = b.shape[0]
    if out is None:
        out = torch.empty((M, N), dtype=torch.bfloat16, device=a.device)
    need = linear_workspace_size(M, N, K)
    if workspace is None and need:
        workspace = torch.empty(need, dtype=torch.uint8, device=a.device)
    wb = workspace.numel() * workspace.element_size() if workspace is not None else 0
    _check(lib().tri_linear(_ptr(a), _ptr(b), _ptr(out), M, N, K, _ptr(workspace), wb,
                            _stream(stream)), "tri_linear")
    return out


def moe_route(cfg, h2_f32, w_router, idx, w, stream=None) -> None:
    _check(lib().tri_moe_route(ctypes.byref(cfg), _ptr(h2_f32), _ptr(w_router),
                               int(h2_f32.shape[0]), _ptr(idx), _ptr(w), _stream(stream)),
           "tri_moe_route")


def profile_enable(on: bool = True) -> None:
    """Start (and reset) or stop per-stage HIP-event timing inside the library."""
    _check(lib().tri_profile_enable(1 if on else 0), "tri_profile_enable")


def profile_read(raw: bool = False):
    """Per-stage launches and total milliseconds recorded since profile_enable(True)
    (the Profile struct itself if raw)."""
    p = Profile()
    _check(lib().tri_profile_read(ctypes.byref(p)), "tri_profile_read")
    if raw:
        return p
    return {p.name[i].decode(): {"launches": p.launches[i], "total_ms": p.total_ms[i]}
            for i in range(p.n_stages)}


def _i32_array(v) -> ctypes.Array:
    v = [int(a) for a in v]
    return (ctypes.c_int32 * max(len(v), 1))(*v)


def layer_work(cfg: LayerConfig, decode: bool, q_len: Sequence[int], ctx_len: Sequence[int],
               expert_rows: Optional[Sequence[int]] = None) -> Work:
    """Algorithmic flops and HBM bytes per stage of one layer call (tri_layer_work)."""
    if len(q_len) != len(ctx_len):
        raise ValueError("q_len and ctx_len differ in length")
    w = Work()
    er = None if expert_rows is None else _i32_array(expert_rows)
    _check(lib().tri_layer_work(ctypes.byref(cfg), 1 if decode else 0, len(q_len),
                                _i32_array(q_len), _i32_array(ctx_len), er, ctypes.byref(w)),
           "tri_layer_work")
    return w


def work_sum(works: Sequence[Work]) -> Work:
    """Stage-by-stage sum of the work of several calls."""
    out = Work()
    out.n_stages = works[0].n_stages
    for i in range(16):
        out.name[i] = works[0].name[i]
        out.runs[i] = int(any(w.runs[i] for w in works))
        out.flops[i] = sum(w.flops[i] for w in works)
        out.bytes[i] = sum(w.bytes[i] for w in works)
    return out


def work_dict(w: Work) -> Dict[str, Dict[str, float]]:
    return {w.name[i].decode(): {"flops": w.flops[i], "bytes": w.bytes[i]}
            for i in range(w.n_stages) if w.runs[i]}


def phase_intensity(work: Work, prof: Profile) -> float:
    """Time-weighted arithmetic intensity of a phase (tri_phase_intensity, Eq. 5)."""
    ai = ctypes.c_double()
    _check(lib().tri_phase_intensity(ctypes.byref(work), ctypes.byref(prof), ctypes.byref(ai)),
           "tri_phase_intensity")
    return ai.value
