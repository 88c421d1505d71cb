// Algorithmic work (flops, compulsory HBM bytes) of each stage of one layer
// call, and the time-weighted phase intensity of Section III-C (Eq. 5) formed
// from it and the measured stage times.  Host code only.
#include <stdint.h>

#include <algorithm>

#include "../../include/tri.h"
#include "host.hpp"
#include "kernels.hpp"

using namespace tri;

namespace {

struct Acc {
  tri_work* w;
  void add(int st, double flops, double bytes) {
    w->runs[st] = 1;
    w->flops[st] += flops;
    w->bytes[st] += bytes;
  }
};

}  // namespace

extern "C" {

tri_status tri_layer_work(const tri_layer_config* cfg, int32_t decode, int32_t n_seqs,
                          const int32_t* q_len, const int32_t* ctx_len,
                          const int32_t* expert_rows, tri_work* out) {
  if (!out) return TRI_ERR_NULL;
  tri_status st = check_config(cfg);
  if (st != TRI_OK) return st;
  if (n_seqs < 0) return TRI_ERR_SHAPE;
  if (n_seqs > 0 && (!q_len || !ctx_len)) return TRI_ERR_NULL;
  const bool moe = (cfg->flags & TRI_F_MOE) != 0;

  double T = 0.0;
  int max_q = 0, max_ctx = 0;
  for (int s = 0; s < n_seqs; ++s) {
    if (q_len[s] < 0 || ctx_len[s] < 0) return TRI_ERR_SHAPE;
    if (decode && q_len[s] != 1) return TRI_ERR_SHAPE;
    T += q_len[s];
    max_q = std::max(max_q, q_len[s]);
    max_ctx = std::max(max_ctx, ctx_len[s]);
  }

  out->n_stages = ST_COUNT;
  for (int i = 0; i < TRI_MAX_STAGES; ++i) {
    out->name[i] = i < ST_COUNT ? kStageName[i] : nullptr;
    out->runs[i] = 0;
    out->flops[i] = 0.0;
    out->bytes[i] = 0.0;
  }
  if (T == 0.0) return TRI_OK;

  Acc a{out};
  const double H = cfg->hidden, D = cfg->head_dim, Hq = cfg->n_q_heads, Hkv = cfg->n_kv_heads;
  const double Nqkv = (Hq + 2.0 * Hkv) * D;
  // bytes of one stored element (bf16, or fp32 in the fp32 storage mode)
  const double bf = cfg->dtype == TRI_F32 ? 4.0 : 2.0, f32 = 4.0, i32 = 4.0;
  const double rope_table = T * (D / 2) * 8.0;  // (cos, sin) fp32 per token and pair
  const double token_map = T * 2 * i32;         // (slot, cache row) per token

  // Token map + rotary table + RMSNorm(x; attn_norm): sum of squares and the
  // scaled product, two multiply-adds per element.
  a.add(ST_PROLOGUE, 4.0 * T * H, T * H * bf + H * bf + T * H * bf + rope_table + token_map);

  // q/k/v projection, optional per-head q/k RMSNorm (sum of squares and the
  // scaled product, two multiply-adds per q and k element), rotary
  // embedding, cache write.
  {
    double bytes = Nqkv * H * bf + T * H * bf + rope_table + token_map + T * Hq * D * bf +
                   T * 2.0 * Hkv * D * bf;
    double flops = 2.0 * T * Nqkv * H;
    if (cfg->flags & TRI_F_QKV_BIAS) bytes += Nqkv * bf;
    if (cfg->flags & TRI_F_QK_NORM) {
      bytes += 2.0 * D * bf;
      flops += 4.0 * T * (Hq + Hkv) * D;
    }
    a.add(ST_QKV, flops, bytes);
  }

  // Attention: sequences with several new tokens take the causal flash path
  // (prefill entry point only), single-token sequences the split-KV path.
  const int split = attn_decode_split_keys(n_seqs, cfg->n_kv_heads, max_ctx + 1, cfg->head_dim,
                                           cfg->n_q_heads / cfg->n_kv_heads, 0);
  bool flash = !decode && max_q > 1;
  double fl_pairs = 0, fl_tok = 0, fl_rows = 0;
  double dec_keys = 0, dec_tok = 0, dec_parts = 0;
  for (int s = 0; s < n_seqs; ++s) {
    const double c = ctx_len[s], q = q_len[s];
    if (q == 0) continue;
    if (q == 1) {
      dec_keys += c + 1;
      dec_tok += 1;
      dec_parts += (ctx_len[s] + 1 + split - 1) / split;
    } else {
      // query i sees keys 0 .. c + i: q c + q (q + 1) / 2 pairs
      fl_pairs += q * c + q * (q + 1) / 2;
      fl_tok += q;
      fl_rows += c + q;
    }
  }
  if (flash)
    a.add(ST_ATTN_PREFILL, 4.0 * D * Hq * fl_pairs,
          fl_tok * Hq * D * bf * 2 + fl_rows * Hkv * D * bf * 2);
  // The split-KV and merge stages are launched unless every sequence has
  // max_q > 1 new tokens (then none is theirs); sequences that are not theirs
  // exit at once.
  if (decode || max_q == 1 || (double)n_seqs * max_q != T) {
    const double part_elems = dec_parts * Hq * (D + 2);  // (m, l, acc[D]) per split
    a.add(ST_ATTN_DECODE, 4.0 * D * Hq * dec_keys,
          dec_tok * Hq * D * bf + dec_keys * Hkv * D * bf * 2 + part_elems * f32);
    a.add(ST_ATTN_COMBINE, 2.0 * dec_parts * Hq * D, part_elems * f32 + dec_tok * Hq * D * bf);
  }

  // O projection + residual, then RMSNorm(x1; mlp_norm) -- one stage for a
  // short batch, whose split-K reduction applies the norm (x1 then never
  // re-read).
  const double o_flops = 2.0 * T * H * Hq * D, o_bytes = H * Hq * D * bf + T * Hq * D * bf +
                                                         2.0 * T * H * bf;
  if (skinny_resid_norm_fused((int)T, cfg->hidden, cfg->n_q_heads * cfg->head_dim)) {
    a.add(ST_OPROJ, o_flops + 4.0 * T * H, o_bytes + T * H * bf + H * bf);
  } else {
    a.add(ST_OPROJ, o_flops, o_bytes);
    a.add(ST_NORM2, 4.0 * T * H, 2.0 * T * H * bf + H * bf);
  }

  if (!moe) {
    const double F = cfg->ffn_dim;
    a.add(ST_GATEUP, 2.0 * T * 2.0 * F * H, 2.0 * F * H * bf + T * H * bf + T * F * bf);
    a.add(ST_DOWN, 2.0 * T * H * F, H * F * bf + T * F * bf + 2.0 * T * H * bf);
    return TRI_OK;
  }

  const double E = cfg->n_experts, k = cfg->top_k, Fe = cfg->expert_ffn_dim, P = T * k;
  double touched = std::min(E, P);
  if (expert_rows) {
    double rows = 0;
    touched = 0;
    for (int e = 0; e < cfg->n_experts; ++e) {
      if (expert_rows[e] < 0) return TRI_ERR_SHAPE;
      rows += expert_rows[e];
      touched += expert_rows[e] > 0;
    }
    if (rows != P) return TRI_ERR_SHAPE;
  }
  // Router logits, softmax, top-k: reads h2 and W_r, writes (idx, w).
  a.add(ST_ROUTER, 2.0 * T * E * H, T * H * bf + E * H * bf + P * (i32 + f32));
  // Counting sort of the (token, expert) pairs: idx in; perm, inv, segment
  // and tile offsets out.
  a.add(ST_MOE_PERMUTE, 0.0, P * i32 + 2.0 * P * i32 + 2.0 * (E + 1) * i32);
  // Expert gate/up + SwiGLU over gathered rows (h2 counted once).
  a.add(ST_MOE_GATEUP, 2.0 * P * 2.0 * Fe * H,
        touched * 2.0 * Fe * H * bf + T * H * bf + P * i32 + P * Fe * bf);
  // Expert down projections, fp32 rows out.
  a.add(ST_MOE_DOWN, 2.0 * P * H * Fe, touched * H * Fe * bf + P * Fe * bf + P * H * f32);
  // Weighted sum of each token's k expert rows + residual.
  a.add(ST_MOE_COMBINE, 2.0 * P * H,
        P * H * f32 + 2.0 * T * H * bf + P * (f32 + i32));
  return TRI_OK;
}

tri_status tri_phase_intensity(const tri_work* work, const tri_profile* prof, double* ai) {
  if (!work || !prof || !ai) return TRI_ERR_NULL;
  if (work->n_stages != prof->n_stages || work->n_stages > TRI_MAX_STAGES) return TRI_ERR_SHAPE;
  double num = 0.0, den = 0.0;
  for (int i = 0; i < work->n_stages; ++i) {
    if (!work->runs[i]) continue;
    const double d = prof->total_ms[i];
    if (!(d >= 0.0)) return TRI_ERR_RANGE;
    const double b = work->bytes[i];
    // a launch with nothing to do (e.g. the split-KV stages of a batch with
    // no single-token sequence) has no intensity and drops out like d = 0
    if (d == 0.0 || (b == 0.0 && work->flops[i] == 0.0)) continue;
    if (!(b > 0.0)) return TRI_ERR_RANGE;
    num += d * (work->flops[i] / b);
    den += d;
  }
  if (den == 0.0) return TRI_ERR_SHAPE;
  *ai = num / den;
  return TRI_OK;
}

}  // extern "C"
