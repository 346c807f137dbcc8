// Host-side planning shared by the C ABI: configuration checks, derived sizes and the
// workspace layout.  Nothing here touches the GPU, so the checks can be exercised
// without one.
#pragma once
#include <stddef.h>
#include <stdint.h>

#include <string>

#include "../../include/retrace.h"

namespace rt {

void set_error(const char* fmt, ...);
int fail(int code, const char* fmt, ...);   // sets the message, returns code

int validate_config(const rt_config* c);
int weight_count(const rt_config* c);
size_t weight_elems(const rt_config* c, int i);

inline size_t rup(size_t x, size_t a) { return (x + a - 1) / a * a; }

constexpr int kPrefillChunk = 512;     // prompt rows per prefill pass
constexpr int kMaxTiles = 1 << 16;     // split-K arrival counters
constexpr size_t kPartialFloats = (size_t)8 << 20;   // split-K partial capacity (32 MiB)
constexpr int kResidSplits = 4;   // k slabs of the round's o / down projections (skinny kernel)
constexpr int kResidSplitsMax = 8;  // at most, on the mid-size kernel (the norm folds up to 8)
constexpr int kArMaxSteps = RT_AR_MAX_STEPS;   // target-only greedy steps per rt_ar_steps call
constexpr int kAttnRowsAr = 64;   // attention rows per block in target-only steps (the 64-row kernel)
constexpr int kStateSlots = 16;   // int32 slots of per-sequence round state (fields in misc.h)
constexpr int kTopkChunk = 8192;  // logits per first-stage top-k workgroup (sample.hip)
constexpr int kLmPartsMin = 512;  // LM-head key rows always reserved (LDS-staged LM head grid, gemm.hip)
constexpr int kLowRankRows = 96;  // low-rank conditioning: 64 latent + 32 correction rows

struct Plan {
  // dimensions
  int V, d, L, Hq, Hkv, hd, F, LD, nc, bk, B, bmax, T, G;
  int qN, kvN, qkvN;                     // q columns, k (= v) columns, fused q|k|v columns
  int Kp_d, Kp_q, Kp_F, Kp_nc, Kp_2d;    // padded reduction lengths
  int esz, ksz;                          // storage / retained element bytes
  int pages_per_seq, n_pages;
  int R, PF, Mrows;                      // round rows, prefill rows, allocated activation rows
  int attn_rb, attn_splits;              // round attention row blocks / key splits
  int attn_rows;                         // round attention rows per block (64, or 96)
  int ar_rb, ar_splits;                  // target-only steps: 64-row attention blocks / key splits
  int pf_rb;
  size_t cache_layer_elems;
  // byte offsets into the workspace
  size_t embed, lm_head, t_final_norm, d_final_norm, fc, hidden_norm, ctxkv, ctx_knorm, wc, wg, wv;
  size_t t_layers, d_layers, layer_bytes;               // per-layer blocks
  size_t lo_qkv, lo_o, lo_gu, lo_down, lo_in, lo_post, lo_qn, lo_kn;   // offsets within a layer block
  size_t kc, vc, dkc, dvc;
  size_t page_table, rope, state, pf_ints, first_tok, counters, partial, opart, mlpart, attn_plan;
  size_t x, xa, qbuf, attn, mlp, g, fcout, fa, etilde, mu, er, gate;
  size_t hd_keep, ht_keep, dlogits, vlogits, dkeys, tkeys, dtok, ttok, out_tok, out_n, out_a, tokbuf;
  size_t qkvf, part_keys;        // fp32 q|k|v projection output; LM-head partial argmax keys
  size_t rpart;                  // k-slab partials of the deferred residual GEMMs [kResidSplitsMax][rpart_rows][d]
  size_t ar_tok;                 // target-only step tokens [bmax][kArMaxSteps]
  size_t dist_ids_d, dist_p_d;   // sampling: drafter filtered distributions [R][RT_MAX_TOP_K]
  size_t dist_ids_v, dist_p_v;   // sampling: target filtered distributions [R][RT_MAX_TOP_K]
  size_t stok;                   // sampling: first / target-only step tokens [bmax]
  size_t topk_cand;              // sampling: per-chunk top-k keys [R][chunks][RT_MAX_TOP_K]
  size_t lr_down, lr_cup, lr_v, lr_g, lr_ge, lr_lat;   // low-rank conditioning (0 unless that mode)
  int rpart_rows;                // max(32, rows of a round)
  int lm_parts;                  // upper bound of LM-head workgroups
  size_t zero_from;                      // everything from here on is zero-filled at init
  size_t total;
  // the partial-result buffers (split partials, split-K arrival counters, residual k-slab
  // partials, attention key-split partials and plan) laid out from offset 0, for the
  // allocation-free round whose partial results live in the library's static scratch
  size_t s_partial, s_counters, s_rpart, s_opart, s_mlpart, s_attn_plan, s_total;
};

// Bytes of the library's static scratch array (one per GPU), which holds the partial
// results of rt_spec_round_static; configurations whose s_total exceeds it are refused.
constexpr size_t kStaticScratchBytes = (size_t)128 << 20;

int make_plan(const rt_config* c, Plan* p);

}  // namespace rt
