"""Naive float64 brute force of the decoder layer, for tiny shapes only.

TEST INFRASTRUCTURE ONLY (see ``oracle/__init__.py``).

Written independently of ``oracle/layer.py``: scalar Python loops over the
literal formulas, Python ``math`` in double precision, no NumPy arithmetic.
It exists to pin the vectorised oracle (a dropped term, a wrong sign, a
transposed operand or a wrong head mapping there disagrees with this).

Readings are the same as in ``oracle/layer.py`` (pre-norm Qwen2-family layer,
optional per-head q/k RMSNorm before the rotation, rotate-half rotary
embedding, consecutive GQA grouping, SwiGLU, top-k softmax routing with ties
to the lower index).
"""
from __future__ import annotations

import math
from typing import Dict, List, Optional


def _matvec(wmat, vec):
    """wmat given as list of rows [out][in]; returns [out]."""
    return [sum(wr[i] * vec[i] for i in range(len(vec))) for wr in wmat]


def layer_brute(cfg, w: Dict[str, list], cache_k, cache_v, slots: List[int],
                ctx_lens: List[int], q_lens: List[int], x: List[List[float]],
                forced_routes: Optional[List[List[int]]] = None, store=None,
                pos3: Optional[List[List[int]]] = None):
    """Arguments are nested Python lists of floats (cache_k[slot][h][row][d]).
    ``store`` (scalar -> scalar), if given, is applied to every activation value
    at the storage points: h, q, k, v, attention output, x1, h2, the SwiGLU
    activation and the output.  ``pos3`` ([token][3] temporal, height, width
    ids) replaces the one-dimensional positions when ``cfg.mrope_section``
    is set.
    Returns (out rows, k_new, v_new, route_idx, route_w)."""
    S = (lambda v: v) if store is None else store
    H, Hq, Hkv, D = cfg.hidden, cfg.n_q_heads, cfg.n_kv_heads, cfg.head_dim
    eps = cfg.rms_eps
    T = len(x)
    out, k_rows, v_rows, ridx, rw = [], [], [], [], []

    def norm(vec, gain):
        ms = sum(t * t for t in vec) / len(vec)
        r = 1.0 / math.sqrt(ms + eps)
        return [vec[i] * r * gain[i] for i in range(len(vec))]

    sections = getattr(cfg, "mrope_section", None)

    def rotate(vec, p):
        # p: the position, or the token's (temporal, height, width) ids
        half = D // 2
        res = [0.0] * D
        for i in range(half):
            if sections:
                k = 0 if i < sections[0] else (1 if i < sections[0] + sections[1] else 2)
                pi = p[k]
            else:
                pi = p
            theta = pi * math.pow(cfg.rope_base, -2.0 * i / D)
            c, s = math.cos(theta), math.sin(theta)
            res[i] = vec[i] * c - vec[i + half] * s
            res[i + half] = vec[i + half] * c + vec[i] * s
        return res

    # Per token: q, k, v for every token first (keys of earlier tokens are needed).
    toks = []   # (seq, position, q heads, k heads, v heads)
    t = 0
    for s in range(len(slots)):
        for i in range(q_lens[s]):
            p = ctx_lens[s] + i
            rp = pos3[t] if sections else p     # rotary position(s) of the token
            h = [S(v) for v in norm(x[t], w["attn_norm"])]
            qkv = _matvec(w["w_qkv"], h)
            if w.get("b_qkv") is not None:
                qkv = [qkv[j] + w["b_qkv"][j] for j in range(len(qkv))]
            qpre = [qkv[j * D:(j + 1) * D] for j in range(Hq)]
            kpre = [qkv[(Hq + j) * D:(Hq + j + 1) * D] for j in range(Hkv)]
            if getattr(cfg, "qk_norm", False):   # per-head RMSNorm before the rotation
                qpre = [norm(vec, w["q_norm"]) for vec in qpre]
                kpre = [norm(vec, w["k_norm"]) for vec in kpre]
            qh = [[S(v) for v in rotate(qpre[j], rp)] for j in range(Hq)]
            kh = [[S(v) for v in rotate(kpre[j], rp)] for j in range(Hkv)]
            vh = [[S(v) for v in qkv[(Hq + Hkv + j) * D:(Hq + Hkv + j + 1) * D]] for j in range(Hkv)]
            toks.append((s, p, qh, kh, vh))
            k_rows.append(kh)
            v_rows.append(vh)
            t += 1

    for t in range(T):
        s, p, qh, _, _ = toks[t]
        # keys of sequence s at cache rows 0..p: cached prefix, then new tokens
        keys, vals = [], []
        for m in range(p + 1):
            if m < ctx_lens[s]:
                keys.append([cache_k[slots[s]][g][m] for g in range(Hkv)])
                vals.append([cache_v[slots[s]][g][m] for g in range(Hkv)])
            else:
                u = [tt for tt in range(T) if toks[tt][0] == s and toks[tt][1] == m][0]
                keys.append(toks[u][3])
                vals.append(toks[u][4])
        o = []
        for j in range(Hq):
            g = (j * Hkv) // Hq
            sc = [sum(qh[j][d] * keys[m][g][d] for d in range(D)) / math.sqrt(D)
                  for m in range(p + 1)]
            mx = max(sc)
            e = [math.exp(z - mx) for z in sc]
            den = sum(e)
            o.extend(S(sum(e[m] / den * vals[m][g][d] for m in range(p + 1))) for d in range(D))
        x1 = [S(x[t][i] + v) for i, v in enumerate(_matvec(w["w_o"], o))]
        h2 = [S(v) for v in norm(x1, w["mlp_norm"])]

        def expert_ffn(wgu, wd):
            f = len(wgu) // 2
            gate = _matvec(wgu[:f], h2)
            up = _matvec(wgu[f:], h2)
            a = [S(gate[i] / (1.0 + math.exp(-gate[i])) * up[i]) for i in range(f)]
            return _matvec(wd, a)

        if cfg.n_experts > 0:
            logits = _matvec(w["w_router"], h2)
            mx = max(logits)
            ex = [math.exp(z - mx) for z in logits]
            den = sum(ex)
            prob = [e_ / den for e_ in ex]
            if forced_routes is not None:
                chosen = list(forced_routes[t])
            else:
                # selection sort: largest logit first, ties to the lower index
                remaining = list(range(cfg.n_experts))
                chosen = []
                for _ in range(cfg.top_k):
                    best = remaining[0]
                    for e_ in remaining[1:]:
                        if logits[e_] > logits[best]:
                            best = e_
                    chosen.append(best)
                    remaining.remove(best)
            ws = [prob[e_] for e_ in chosen]
            if cfg.moe_renorm:
                tot = sum(ws)
                ws = [v / tot for v in ws]
            y = [0.0] * H
            for e_, wt in zip(chosen, ws):
                ye = expert_ffn(w["w_gate_up"][e_], w["w_down"][e_])
                y = [y[i] + wt * ye[i] for i in range(H)]
            ridx.append(chosen)
            rw.append(ws)
        else:
            y = expert_ffn(w["w_gate_up"], w["w_down"])
        out.append([S(x1[i] + y[i]) for i in range(H)])
    return out, k_rows, v_rows, ridx, rw
