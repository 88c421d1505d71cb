"""CPU oracle for the Thinker decoder-layer forward (prefill, decode, mixed).

TEST INFRASTRUCTURE ONLY.  Only the test-suite, the smoke check and the
bench's CPU-baseline leg may import this module; the product path never does.

The paper's Thinker stage (Section II-A) is a multimodal LLM that consumes its
token stream in a compute-bound prefill phase and then emits tokens in an
autoregressive decode loop over a KV cache kept under PagedAttention memory
management; Section II-C (Observation 2) characterises prefill as dense GEMM
kernels and decode as GEMV-like operators, and Section III-A1 labels scheduler
steps prefill, decode or mixed.  The paper gives no equations for the layer
itself: it names the model (Qwen2.5-Omni-7B, Section IV-A), whose Thinker is a
Qwen2-family pre-norm decoder.  Every convention below that the paper does not
fix is a declared reading:

  * pre-norm residual order  x1 = x + Attn(RMSNorm(x)),  out = x1 + FFN(RMSNorm(x1));
  * RMSNorm  y = x / sqrt(mean(x^2) + eps) * g;
  * rotary embedding, rotate-half pairing (i, i + D/2), inverse frequency
    base^(-2i/D), angle pos * inv_freq formed in float64;
  * grouped-query attention with consecutive grouping (query head j reads KV
    head floor(j * Hkv / Hq)), scale 1/sqrt(D), causal over cache rows
    0 .. ctx_len + i, keys stored after rotation;
  * optional per-head query/key normalisation (the Qwen3-family variant of
    the layer, ``cfg.qk_norm``): before the rotation every head of q and of k
    is RMS-normalised over its D values with gains q_norm / k_norm [D] and
    the layer's eps;
  * optional multi-section rotary positions (the multimodal rotary embedding
    of the Qwen2-VL / Qwen2.5-Omni family, ``cfg.mrope_section`` = (s_t, s_h,
    s_w), s_t + s_h + s_w = D/2): every token carries three position ids
    (temporal, height, width; ``batch.pos3`` [3, T]) and rotary frequency i
    takes its position from the section it falls in, frequencies
    [0, s_t) the temporal id, [s_t, s_t + s_h) the height id, the rest the
    width id.  With equal ids it is the one-dimensional embedding;
  * SwiGLU  a = silu(h W_g^T) * (h W_u^T),  silu(z) = z / (1 + exp(-z));
  * MoE: softmax over all expert logits, top-k by logit (descending, ties to
    the lower expert index), weights renormalised over the chosen k, no shared
    expert, no capacity limit.

This is the plain definition: full softmax attention (flash or split-KV
attention are exact re-orderings of it), no blocking, no fusion.  Arithmetic is
float64 by default; ``dtype=np.float32`` gives the plain fp32 layer.

Storage precision (a declared reading; the paper states none).  With
``storage="bf16"`` the layer's activations are held in bfloat16 between
operations, as a bf16 deployment of the model stores them: the value at each
storage point is rounded to the nearest bfloat16 (ties to even) and the
arithmetic between storage points stays exact.  The storage points are the
normalised input h, the rotated q and k and the value v (the KV cache is
bf16), the attention output, the residual x1, the normalised h2, the SwiGLU
activation, and the layer output.  ``storage=None`` rounds nothing.
"""
from __future__ import annotations

from typing import Dict, Optional

import numpy as np


def round_bf16(x: np.ndarray) -> np.ndarray:
    """Nearest bfloat16 value (8 significant bits, ties to even), same dtype back."""
    x = np.asarray(x)
    m, e = np.frexp(x.astype(np.float64))          # x = m 2^e, 0.5 <= |m| < 1
    return np.ldexp(np.rint(np.ldexp(m, 8)), e - 8).astype(x.dtype)


def project(a: np.ndarray, w: np.ndarray) -> np.ndarray:
    """A projection y = a W^T with an nn.Linear weight W [out, in]: the
    matrix multiply of the layer's q/k/v, O and MLP projections (Section
    II-A) and of the roofline benchmark kernel (Section II-C)."""
    return a @ w.T


def rmsnorm(x: np.ndarray, g: np.ndarray, eps: float) -> np.ndarray:
    """RMSNorm over the last axis: x / sqrt(mean(x^2) + eps) * g."""
    ms = np.mean(x * x, axis=-1, keepdims=True)
    return x / np.sqrt(ms + x.dtype.type(eps)) * g


def rope_angles(pos: np.ndarray, head_dim: int, base: float) -> np.ndarray:
    """Rotary angles [n, D/2] in float64: pos * base^(-2i/D)."""
    i = np.arange(head_dim // 2, dtype=np.float64)
    inv_freq = np.float64(base) ** (-2.0 * i / head_dim)
    return np.asarray(pos, dtype=np.float64)[:, None] * inv_freq[None, :]


def rope_angles_sections(pos3: np.ndarray, head_dim: int, base: float, sections) -> np.ndarray:
    """Multi-section rotary angles [n, D/2] in float64: frequency i of a token
    uses position id pos3[k, token] of the section k that i falls in
    (sections = (s_t, s_h, s_w) consecutive frequency counts)."""
    i = np.arange(head_dim // 2, dtype=np.float64)
    inv_freq = np.float64(base) ** (-2.0 * i / head_dim)
    sec = np.repeat(np.arange(3), np.asarray(sections, dtype=np.int64))
    assert sec.shape[0] == head_dim // 2, "sections must sum to D/2"
    p = np.asarray(pos3, dtype=np.float64)[sec, :]          # [D/2, n]
    return p.T * inv_freq[None, :]


def rope(x: np.ndarray, angles: np.ndarray) -> np.ndarray:
    """Rotate-half rotary embedding. x [n, heads, D]; angles [n, D/2]."""
    half = x.shape[-1] // 2
    c = np.cos(angles).astype(x.dtype)[:, None, :]
    s = np.sin(angles).astype(x.dtype)[:, None, :]
    x1, x2 = x[..., :half], x[..., half:]
    return np.concatenate([x1 * c - x2 * s, x2 * c + x1 * s], axis=-1)


def softmax(s: np.ndarray, axis: int = -1) -> np.ndarray:
    m = np.max(s, axis=axis, keepdims=True)
    e = np.exp(s - m)
    return e / np.sum(e, axis=axis, keepdims=True)


def attention(q: np.ndarray, k: np.ndarray, v: np.ndarray, q_index: np.ndarray) -> np.ndarray:
    """Causal grouped-query softmax attention for one sequence.

    q [n, Hq, D]; k, v [Hkv, L, D] (cache rows 0..L-1, already rotated);
    q_index[i] = cache row of query i; query i sees rows 0..q_index[i].
    Returns o [n, Hq, D].
    """
    n, hq, d = q.shape
    hkv, L, _ = k.shape
    scale = q.dtype.type(1.0 / np.sqrt(d))
    keys = np.arange(L)
    masked = keys[None, :] > np.asarray(q_index)[:, None]          # [n, L]
    o = np.empty_like(q)
    for j in range(hq):
        g = (j * hkv) // hq
        s = (q[:, j, :] @ k[g].T) * scale
        s = np.where(masked, -np.inf, s)
        o[:, j, :] = softmax(s) @ v[g]
    return o


def silu(z: np.ndarray) -> np.ndarray:
    return z / (z.dtype.type(1) + np.exp(-z))


def swiglu(h: np.ndarray, w_gate_up: np.ndarray, w_down: np.ndarray,
           store=lambda a: a) -> np.ndarray:
    """SwiGLU FFN: gate rows [0, F), up rows [F, 2F) of w_gate_up [2F, H]; w_down [H, F].
    ``store`` is applied to the activation silu(g) * u (its storage precision)."""
    f = w_gate_up.shape[0] // 2
    g = h @ w_gate_up[:f].T
    u = h @ w_gate_up[f:].T
    return store(silu(g) * u) @ w_down.T


def topk_lower_index(logits: np.ndarray, k: int) -> np.ndarray:
    """Indices of the k largest logits per row, descending, ties to the lower index."""
    order = np.argsort(-logits, axis=-1, kind="stable")
    return order[:, :k].astype(np.int32)


def moe_route(h: np.ndarray, w_router: np.ndarray, k: int, renorm: bool = True):
    """Router: logits = h W_r^T, p = softmax(logits), top-k by logit, weights p[idx]
    (divided by their sum when ``renorm``).  Returns (idx int32 [T,k], w [T,k], logits)."""
    logits = h @ w_router.T
    p = softmax(logits)
    idx = topk_lower_index(logits, k)
    wts = np.take_along_axis(p, idx, axis=-1)
    if renorm:
        wts = wts / np.sum(wts, axis=-1, keepdims=True)
    return idx, wts, logits


def moe_ffn(h: np.ndarray, idx: np.ndarray, wts: np.ndarray,
            w_gate_up: np.ndarray, w_down: np.ndarray, store=lambda a: a) -> np.ndarray:
    """Weighted sum of the chosen experts' SwiGLU outputs.
    w_gate_up [E, 2Fe, H]; w_down [E, H, Fe]."""
    y = np.zeros_like(h)
    for e in np.unique(idx):
        t, j = np.nonzero(idx == e)
        y_e = swiglu(h[t], w_gate_up[e], w_down[e], store)
        np.add.at(y, t, wts[t, j][:, None] * y_e)
    return y


def _as(a, dtype):
    return None if a is None else np.asarray(a, dtype=dtype)


def layer_forward(cfg, w: Dict[str, np.ndarray], cache_k: np.ndarray, cache_v: np.ndarray,
                  batch, x: np.ndarray, *, dtype=np.float64,
                  forced_routes: Optional[np.ndarray] = None,
                  rows: Optional[np.ndarray] = None,
                  storage: Optional[str] = None) -> Dict[str, np.ndarray]:
    """One decoder-layer forward over a ragged batch.

    cfg      object with hidden, n_q_heads, n_kv_heads, head_dim, ffn_dim,
             n_experts, top_k, rms_eps, rope_base, moe_renorm (and optionally
             qk_norm, with weights q_norm / k_norm).
    w        weights as float arrays, row-major [out, in] (see module docstring).
    cache_k, cache_v   [n_slots, Hkv, max_seq, D]; rows below a sequence's
             ctx_len are its cached (rotated) keys / values.  Not modified.
    batch    object with slot, ctx_len, q_len (int arrays); new token i of a
             sequence sits at cache row and RoPE position ctx_len + i.
    x        [T, H] token activations, sequences concatenated in batch order.
    forced_routes  optional [T, k] expert indices used instead of the router's.
    rows     optional token indices: outputs are produced only for these rows
             (keys and values are still computed for every token).
    storage  None (exact) or "bf16" (activations rounded to bfloat16 at the
             storage points listed in the module docstring).

    Returns a dict with ``out`` [len(rows) or T, H], ``k_new``/``v_new``
    [T, Hkv, D] (the rows written to the cache), and the intermediates
    ``h``, ``q``, ``attn``, ``x1``, ``h2`` (for the selected rows) plus
    ``route_idx``/``route_w``/``logits`` for an MoE layer.
    """
    H, Hq, Hkv, D = cfg.hidden, cfg.n_q_heads, cfg.n_kv_heads, cfg.head_dim
    if storage not in (None, "bf16"):
        raise ValueError(storage)
    st = round_bf16 if storage == "bf16" else (lambda a: a)
    x = _as(x, dtype)
    T = x.shape[0]
    rows = np.arange(T) if rows is None else np.asarray(rows)
    slot = np.asarray(batch.slot)
    ctx = np.asarray(batch.ctx_len)
    qlen = np.asarray(batch.q_len)
    cu = np.concatenate([[0], np.cumsum(qlen)])
    pos = np.concatenate([np.arange(c, c + q) for c, q in zip(ctx, qlen)])

    # Attention block: RMSNorm, fused q/k/v projection, rotary embedding.
    h = st(rmsnorm(x, _as(w["attn_norm"], dtype), cfg.rms_eps))
    w_qkv = _as(w["w_qkv"], dtype)
    qkv = h @ w_qkv.T
    if w.get("b_qkv") is not None:
        qkv = qkv + _as(w["b_qkv"], dtype)
    if getattr(cfg, "mrope_section", None):
        ang = rope_angles_sections(batch.pos3, D, cfg.rope_base, cfg.mrope_section)
    else:
        ang = rope_angles(pos, D, cfg.rope_base)
    q_pre = qkv[:, :Hq * D].reshape(T, Hq, D)
    k_pre = qkv[:, Hq * D:(Hq + Hkv) * D].reshape(T, Hkv, D)
    if getattr(cfg, "qk_norm", False):
        q_pre = rmsnorm(q_pre, _as(w["q_norm"], dtype), cfg.rms_eps)
        k_pre = rmsnorm(k_pre, _as(w["k_norm"], dtype), cfg.rms_eps)
    q = st(rope(q_pre, ang))
    k_new = st(rope(k_pre, ang))
    v_new = st(qkv[:, (Hq + Hkv) * D:].reshape(T, Hkv, D))

    # Causal attention per sequence over its cached prefix plus its new rows.
    attn = np.zeros((T, Hq, D), dtype=dtype)
    want = np.zeros(T, dtype=bool)
    want[rows] = True
    for s in range(len(slot)):
        a, b = int(cu[s]), int(cu[s + 1])
        sel = np.nonzero(want[a:b])[0]
        if sel.size == 0:
            continue
        c = int(ctx[s])
        kk = np.concatenate([_as(cache_k[slot[s], :, :c], dtype),
                             k_new[a:b].transpose(1, 0, 2)], axis=1)
        vv = np.concatenate([_as(cache_v[slot[s], :, :c], dtype),
                             v_new[a:b].transpose(1, 0, 2)], axis=1)
        attn[a + sel] = st(attention(q[a + sel], kk, vv, c + sel))

    xr = x[rows]
    x1 = st(xr + attn[rows].reshape(len(rows), Hq * D) @ _as(w["w_o"], dtype).T)
    h2 = st(rmsnorm(x1, _as(w["mlp_norm"], dtype), cfg.rms_eps))
    res = {"h": h[rows], "q": q[rows], "k_new": k_new, "v_new": v_new,
           "attn": attn[rows].reshape(len(rows), Hq * D), "x1": x1, "h2": h2}
    if cfg.n_experts > 0:
        idx, wts, logits = moe_route(h2, _as(w["w_router"], dtype), cfg.top_k, cfg.moe_renorm)
        if forced_routes is not None:
            idx = np.asarray(forced_routes, dtype=np.int32)[rows]
            p = softmax(logits)
            wts = np.take_along_axis(p, idx, axis=-1)
            if cfg.moe_renorm:
                wts = wts / np.sum(wts, axis=-1, keepdims=True)
        y = moe_ffn(h2, idx, wts, _as(w["w_gate_up"], dtype), _as(w["w_down"], dtype), st)
        res.update(route_idx=idx, route_w=wts, logits=logits)
    else:
        y = swiglu(h2, _as(w["w_gate_up"], dtype), _as(w["w_down"], dtype), st)
    res["out"] = st(x1 + y)
    return res


def kvcache_append(cache_k: np.ndarray, cache_v: np.ndarray, batch, k_new: np.ndarray,
                   v_new: np.ndarray):
    """Reference for the cache append: returns copies of the caches with
    cache[slot][h][ctx_len + i] = new[token][h] for every new token."""
    ck, cv = cache_k.copy(), cache_v.copy()
    t = 0
    for s, c, q in zip(batch.slot, batch.ctx_len, batch.q_len):
        for i in range(int(q)):
            ck[s, :, c + i, :] = k_new[t]
            cv[s, :, c + i, :] = v_new[t]
            t += 1
    return ck, cv
