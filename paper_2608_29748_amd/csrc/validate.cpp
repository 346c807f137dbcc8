// Configuration checks and workspace layout (host only).
#include <math.h>
#include <stdarg.h>
#include <stdio.h>

#include "host.h"

namespace rt {

static thread_local std::string g_err;

void set_error(const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  g_err = buf;
}

int fail(int code, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  g_err = buf;
  return code;
}

const char* last_error() { return g_err.c_str(); }

int validate_config(const rt_config* c) {
  if (!c) return fail(RT_ERR_INVALID, "config is null");
  if (c->dtype != RT_F32 && c->dtype != RT_BF16) return fail(RT_ERR_INVALID, "dtype must be RT_F32 or RT_BF16");
  if (c->vocab < 16 || c->vocab % 16) return fail(RT_ERR_INVALID, "vocab must be a positive multiple of 16");
  if (c->hidden < 32 || c->hidden % 32 || c->hidden > 8192)
    return fail(RT_ERR_INVALID, "hidden must be a multiple of 32 in [32, 8192]");
  if (c->n_layers < 1 || c->n_layers > 99) return fail(RT_ERR_INVALID, "n_layers must be in [1, 99]");
  if (c->head_dim != 64 && c->head_dim != 128) return fail(RT_ERR_INVALID, "head_dim must be 64 or 128");
  if (c->n_kv_heads < 1 || c->n_q_heads < c->n_kv_heads || c->n_q_heads % c->n_kv_heads)
    return fail(RT_ERR_INVALID, "n_q_heads must be a positive multiple of n_kv_heads");
  if ((c->n_q_heads * c->head_dim) % 128 || (c->n_kv_heads * c->head_dim) % 128)
    return fail(RT_ERR_INVALID, "q and kv projection widths must be multiples of 128");
  if (c->ffn < 16 || c->ffn % 16) return fail(RT_ERR_INVALID, "ffn must be a positive multiple of 16");
  if (c->draft_layers < 1 || c->draft_layers > 99) return fail(RT_ERR_INVALID, "draft_layers must be in [1, 99]");
  if (c->n_cond_layers < 1 || c->n_cond_layers > RT_MAX_COND_LAYERS)
    return fail(RT_ERR_INVALID, "n_cond_layers must be in [1, %d]", RT_MAX_COND_LAYERS);
  for (int i = 0; i < c->n_cond_layers; ++i) {
    const int id = c->cond_layer_ids[i];
    if (id < 0 || id >= c->n_layers) return fail(RT_ERR_INVALID, "cond_layer_ids[%d] = %d out of range", i, id);
    if (i && id <= c->cond_layer_ids[i - 1]) return fail(RT_ERR_INVALID, "cond_layer_ids must increase");
  }
  if (c->block_size < 2 || c->block_size > 64) return fail(RT_ERR_INVALID, "block_size must be in [2, 64]");
  if (c->mask_token_id < 0 || c->mask_token_id >= c->vocab) return fail(RT_ERR_TOKEN, "mask_token_id out of range");
  if (!isfinite(c->beta)) return fail(RT_ERR_INVALID, "beta must be finite");
  if (!(c->rope_theta > 0.f) || !(c->rms_eps >= 0.f)) return fail(RT_ERR_INVALID, "rope_theta / rms_eps invalid");
  if (c->cond_mode < RT_COND_OFF || c->cond_mode > RT_COND_LOWRANK)
    return fail(RT_ERR_INVALID, "cond_mode must be RT_COND_OFF, _RETRACE, _RAW_GATED, _OVERWRITE or _LOWRANK");
  if (c->max_batch < 1 || c->max_batch > 1024) return fail(RT_ERR_INVALID, "max_batch must be in [1, 1024]");
  if (c->max_seq_len < c->block_size + 1 || c->max_seq_len > (1 << 20))
    return fail(RT_ERR_INVALID, "max_seq_len must be in [block_size + 1, 2^20]");
  if (c->dtype == RT_F32 && c->max_seq_len > 16384)   // fp32 attention keeps a split's page ids in LDS
    return fail(RT_ERR_INVALID, "fp32 storage supports max_seq_len up to 16384");
  if (c->page_size != 16) return fail(RT_ERR_INVALID, "page_size must be 16");
  if (!(c->temperature >= 0.f) || !isfinite(c->temperature)) return fail(RT_ERR_INVALID, "temperature must be >= 0");
  if (c->temperature > 0.f) {
    if (c->top_k < 1 || c->top_k > RT_MAX_TOP_K || c->top_k > c->vocab)
      return fail(RT_ERR_INVALID, "top_k must be in [1, %d] and at most vocab", RT_MAX_TOP_K);
    if (!(c->top_p > 0.f && c->top_p <= 1.f)) return fail(RT_ERR_INVALID, "top_p must be in (0, 1]");
  }
  return RT_OK;
}

int weight_count(const rt_config* c) {
  return 1 + 11 * c->n_layers + 4 + 11 * c->draft_layers + 1 + 3 + (c->cond_mode == RT_COND_LOWRANK ? 5 : 0);
}

// Elements of weight tensor i in the canonical order of rt_init_models (0 if out of range).
size_t weight_elems(const rt_config* c, int i) {
  const size_t d = c->hidden, q = (size_t)c->n_q_heads * c->head_dim, kv = (size_t)c->n_kv_heads * c->head_dim;
  const size_t hd = c->head_dim, F = c->ffn, V = c->vocab, nc = c->n_cond_layers;
  // the eleven tensors of a decoder layer: input_norm, q, k, v, q_norm, k_norm, o, post_norm, gate, up, down
  const size_t layer[11] = {d, q * d, kv * d, kv * d, hd, hd, d * q, d, F * d, F * d, d * F};
  if (i < 0 || i >= weight_count(c)) return 0;
  if (i == 0) return V * d;                                  // embed
  i -= 1;
  if (i < 11 * c->n_layers) return layer[i % 11];
  i -= 11 * c->n_layers;
  if (i < 4) {
    const size_t head[4] = {d, V * d, d * nc * d, d};        // final_norm, lm_head, fc, hidden_norm
    return head[i];
  }
  i -= 4;
  if (i < 11 * c->draft_layers) return layer[i % 11];
  i -= 11 * c->draft_layers;
  const size_t tail[9] = {d, d * 2 * d, d * d, d * 2 * d,      // draft final_norm, W_c, W_v, W_g
                          64 * d, 32 * 2 * d, 64 * 32, d * 64, d * 64};   // low-rank A, C_down, C_up, V, G
  return tail[i];
}

int make_plan(const rt_config* c, Plan* p) {
  int st = validate_config(c);
  if (st) return st;
  Plan& q = *p;
  q.V = c->vocab; q.d = c->hidden; q.L = c->n_layers; q.Hq = c->n_q_heads; q.Hkv = c->n_kv_heads;
  q.hd = c->head_dim; q.F = c->ffn; q.LD = c->draft_layers; q.nc = c->n_cond_layers;
  q.bk = c->block_size; q.B = q.bk - 1; q.bmax = c->max_batch; q.T = c->max_seq_len;
  q.G = q.Hq / q.Hkv;
  q.qN = q.Hq * q.hd; q.kvN = q.Hkv * q.hd; q.qkvN = q.qN + 2 * q.kvN;
  q.Kp_d = (int)rup(q.d, 32); q.Kp_q = (int)rup(q.qN, 32); q.Kp_F = (int)rup(q.F, 32);
  q.Kp_nc = (int)rup((size_t)q.nc * q.d, 32); q.Kp_2d = (int)rup(2 * (size_t)q.d, 32);
  q.esz = c->dtype == RT_BF16 ? 2 : 4;
  q.ksz = c->dtype == RT_BF16 ? 2 : 4;
  q.pages_per_seq = (q.T + 15) / 16;
  q.n_pages = q.bmax * q.pages_per_seq;
  q.R = q.bmax * q.bk;
  q.PF = kPrefillChunk;
  q.Mrows = (int)rup((size_t)(q.R > q.PF ? q.R : q.PF), 128);
  // one row block per sequence and KV head when the block has at most 96 (token, head)
  // rows (bf16), so each KV head's keys are read once
  q.attn_rows = (c->dtype == RT_BF16 && q.bk * q.G > 64 && q.bk * q.G <= 96) ? 96 : 64;
  q.attn_rb = (q.bk * q.G + q.attn_rows - 1) / q.attn_rows;
  // key splits: about one workgroup per compute unit, at most 64 (one per lane of the
  // merge), and at least two 64-key chunks per split at the longest sequence
  auto key_splits = [&](int row_blocks) {
    const int base = q.bmax * q.Hkv * row_blocks;
    int sp = (256 + base - 1) / base;
    const int maxsp = ((q.T + 63) / 64) / 2;
    if (sp > maxsp) sp = maxsp;
    if (sp > 64) sp = 64;
    if (sp < 1) sp = 1;
    return sp;
  };
  q.attn_splits = key_splits(q.attn_rb);
  q.ar_rb = (q.G + kAttnRowsAr - 1) / kAttnRowsAr;   // one query token: G rows per KV head
  q.ar_splits = key_splits(q.ar_rb);
  q.pf_rb = (q.PF * q.G + 63) / 64;
  q.cache_layer_elems = (size_t)q.n_pages * q.Hkv * 16 * q.hd;

  size_t off = 0;
  auto take = [&](size_t bytes) { size_t o = off; off = rup(off + bytes, 256); return o; };
  const size_t e = q.esz;
  auto packed = [&](size_t N, size_t Kp) { return N * Kp * e; };
  q.embed = take((size_t)q.V * q.d * e);
  q.lm_head = take(packed(q.V, q.Kp_d));
  q.t_final_norm = take(q.d * e);
  q.d_final_norm = take(q.d * e);
  q.fc = take(packed(q.d, q.Kp_nc));
  q.hidden_norm = take(q.d * e);
  q.ctxkv = take(packed((size_t)q.LD * 2 * q.kvN, q.Kp_d));
  q.ctx_knorm = take((size_t)q.LD * q.hd * e);
  q.wc = take(packed(q.d, q.Kp_2d));
  q.wg = take(packed(q.d, q.Kp_2d));
  q.wv = take(packed(q.d, q.Kp_d));
  if (c->cond_mode == RT_COND_LOWRANK) {
    q.lr_down = take(packed(kLowRankRows, q.Kp_2d));        // [A | 0 ; C_down], packed
    q.lr_cup = take((size_t)64 * 32 * e);
    q.lr_v = take((size_t)q.d * 64 * e);
    q.lr_g = take((size_t)q.d * 64 * e);
    q.lr_ge = take((size_t)q.d * 4);
  }
  // per-layer block
  size_t lo = 0;
  auto ltake = [&](size_t bytes) { size_t o = lo; lo = rup(lo + bytes, 256); return o; };
  q.lo_qkv = ltake(packed(q.qkvN, q.Kp_d));
  q.lo_o = ltake(packed(q.d, q.Kp_q));
  q.lo_gu = ltake(packed(2 * (size_t)q.F, q.Kp_d));
  q.lo_down = ltake(packed(q.d, q.Kp_F));
  q.lo_in = ltake(q.d * e);
  q.lo_post = ltake(q.d * e);
  q.lo_qn = ltake(q.hd * e);
  q.lo_kn = ltake(q.hd * e);
  q.layer_bytes = lo;
  q.t_layers = take(q.layer_bytes * q.L);
  q.d_layers = take(q.layer_bytes * q.LD);
  q.zero_from = off;
  q.kc = take(q.cache_layer_elems * e * q.L);
  q.vc = take(q.cache_layer_elems * e * q.L);
  q.dkc = take(q.cache_layer_elems * e * q.LD);
  q.dvc = take(q.cache_layer_elems * e * q.LD);
  q.page_table = take((size_t)q.n_pages * 4);
  q.rope = take((size_t)q.T * (q.hd / 2) * 2 * 4);
  q.state = take((size_t)q.bmax * kStateSlots * 4);
  q.pf_ints = take(16 * 4);
  q.first_tok = take((size_t)q.bmax * 4);
  q.counters = take((size_t)kMaxTiles * 4);
  q.partial = take(kPartialFloats * 4);
  q.rpart_rows = q.R > 32 ? q.R : 32;
  q.rpart = take((size_t)kResidSplitsMax * q.rpart_rows * q.d * 4);
  {
    size_t rb = q.attn_rb > q.pf_rb ? q.attn_rb : q.pf_rb;
    (void)rb;
    // per KV head one partial block per slot, plus one per unit boundary (a slot of the
    // spanning plan writes one block per unit it meets)
    size_t rows = (size_t)q.Hkv * ((size_t)q.bmax * q.attn_rb * (q.attn_splits + 1) - 1) * q.attn_rows;
    const size_t ar_rows = (size_t)q.Hkv * ((size_t)q.bmax * q.ar_rb * (q.ar_splits + 1) - 1) * kAttnRowsAr;
    if (ar_rows > rows) rows = ar_rows;
    q.opart = take(rows * q.hd * 4);
    q.mlpart = take(rows * 2 * 4);
    q.attn_plan = take(2 * 64 * 4);
  }
  const size_t M = q.Mrows;
  q.x = take(M * q.d * 4);
  q.xa = take(M * q.Kp_d * e);
  q.qbuf = take(M * q.qN * e);
  q.attn = take(M * q.Kp_q * e);
  q.mlp = take(M * q.Kp_F * e);
  q.g = take(M * q.Kp_nc * e);
  q.fcout = take(M * q.d * 4);
  q.fa = take(M * q.Kp_d * e);
  const size_t Rp = rup(q.R, 32);
  q.etilde = take((size_t)q.R * q.d * 4);
  q.mu = take(Rp * q.Kp_2d * 4);
  q.er = take(Rp * q.Kp_2d * 4);
  q.gate = take(Rp * q.d * 4);
  q.lr_lat = take(Rp * kLowRankRows * 4);
  q.hd_keep = take((size_t)q.R * q.d * q.ksz);
  q.ht_keep = take((size_t)q.R * q.d * q.ksz);
  q.dlogits = take((size_t)q.R * q.V * 4);
  q.vlogits = take((size_t)q.R * q.V * 4);
  q.dkeys = take(M * 8);
  q.tkeys = take(M * 8);
  {
    const size_t qc = (size_t)q.qkvN > (size_t)q.LD * 2 * q.kvN ? (size_t)q.qkvN : (size_t)q.LD * 2 * q.kvN;
    q.qkvf = take(M * qc * 4);
    q.lm_parts = (q.V + 31) / 32 / 8 + 1;                 // skinny LM head workgroups
    if (2 * ((q.V + 63) / 64) > q.lm_parts) q.lm_parts = 2 * ((q.V + 63) / 64);   // mid-size: 2 per workgroup
    if (q.lm_parts < kLmPartsMin) q.lm_parts = kLmPartsMin;   // LDS-staged skinny LM head
    q.part_keys = take((size_t)q.lm_parts * M * 8);
  }
  q.dtok = take((size_t)q.R * 4);
  q.ttok = take((size_t)q.R * 4);
  q.out_tok = take((size_t)q.R * 4);
  q.out_n = take((size_t)q.bmax * 4);
  q.out_a = take((size_t)q.bmax * 4);
  q.tokbuf = take((size_t)q.T * 4);
  q.ar_tok = take((size_t)q.bmax * kArMaxSteps * 4);
  q.dist_ids_d = take((size_t)q.R * RT_MAX_TOP_K * 4);
  q.dist_p_d = take((size_t)q.R * RT_MAX_TOP_K * 4);
  q.dist_ids_v = take((size_t)q.R * RT_MAX_TOP_K * 4);
  q.dist_p_v = take((size_t)q.R * RT_MAX_TOP_K * 4);
  q.stok = take((size_t)q.bmax * 4);
  q.topk_cand = take((size_t)q.R * ((q.V + kTopkChunk - 1) / kTopkChunk) * RT_MAX_TOP_K * 8);
  q.total = off;
  // the same partial-result buffers, from offset 0 (static scratch)
  {
    size_t so = 0;
    auto stake = [&](size_t bytes) { size_t o = so; so = rup(so + bytes, 256); return o; };
    q.s_partial = stake(kPartialFloats * 4);
    q.s_counters = stake((size_t)kMaxTiles * 4);
    q.s_rpart = stake((size_t)kResidSplitsMax * q.rpart_rows * q.d * 4);
    q.s_opart = stake(q.mlpart - q.opart);
    q.s_mlpart = stake(q.attn_plan - q.mlpart);
    q.s_attn_plan = stake(2 * 64 * 4);
    q.s_total = so;
  }
  return RT_OK;
}

}  // namespace rt
