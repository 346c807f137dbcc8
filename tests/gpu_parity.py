"""Teacher-forced round-by-round comparison of the HIP path (through the C ABI) with
the oracle, shared by the GPU parity tests.

Per round: the conditioned drafter inputs, retained drafter / target final states
and both LM heads' logits must agree within `tol` (max abs error); every argmax
decision whose oracle top-2 gap exceeds `tol` must agree exactly; at near-ties the
GPU's choice is adopted by the oracle so both continue from the same tokens.  The
acceptance length, committed tokens and round state must then agree exactly.
"""
from __future__ import annotations

import sys
from dataclasses import dataclass, field
from typing import List

import numpy as np

from oracle import OracleModel, OracleRunner
from oracle.model import rms_norm
from paper_2608_29748_amd import binding as B
from paper_2608_29748_amd.engine import RoundEngine, config_from
from workloads import weight_specs


def log(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def engine_for(wl, W, max_batch=None, cond_mode=None):
    if cond_mode is None:
        cond_mode = B.COND_MODES[wl.cond_mode]
    cfg = config_from(wl.target, dtype=wl.dtype, draft_layers=wl.draft_layers,
                      cond_layers=wl.cond_layers, block_size=wl.block_size,
                      mask_token_id=wl.mask_token_id, max_batch=max_batch or wl.batch,
                      max_seq_len=wl.max_seq_len, rope_theta=wl.rope_theta, rms_eps=wl.rms_eps,
                      beta=wl.beta, cond_mode=cond_mode, temperature=wl.temperature, top_k=wl.top_k,
                      top_p=wl.top_p, sample_seed=wl.sample_seed)
    return RoundEngine(cfg, [W[name] for name, _, _ in weight_specs(wl)])


def keep_dtype(wl):
    return np.float16 if wl.dtype == "bf16" else np.float32


def store_to_f64(arr, wl):
    if wl.dtype == "bf16":
        return (arr.astype(np.uint16).astype(np.uint32) << 16).view(np.float32).astype(np.float64)
    return arr.astype(np.float64)


def top2_gap(logits):
    part = np.partition(logits, -2, axis=-1)
    return part[..., -1] - part[..., -2]


@dataclass
class Report:
    rounds: int = 0
    max_err: dict = field(default_factory=dict)
    near_ties: int = 0
    decisions: int = 0
    accept: List[int] = field(default_factory=list)
    conditioned: int = 0         # sequence rounds checked with conditioned rows (cond_len > 0)
    stage_decisions: int = 0     # argmax decisions checked per stage (from the GPU's LM-head operands)
    stage_near_ties: int = 0     # of those, top-2 gap within the tolerance (GPU's choice adopted)

    p999: dict = field(default_factory=dict)

    def err(self, name, a, b):
        d = np.abs(np.asarray(a, np.float64) - np.asarray(b, np.float64))
        e = float(np.max(d)) if np.size(a) else 0.0
        self.max_err[name] = max(self.max_err.get(name, 0.0), e)
        if np.size(a):
            self.p999[name] = max(self.p999.get(name, 0.0), float(np.quantile(d, 0.999)))
        return e

    def stored_err(self, name, a, b, tol, wl):
        """Error in excess of the allowance for values both sides store in the
        storage type: where the unrounded values straddle a rounding boundary the
        stored ones differ by one unit in the last place (2**-7 relative for bf16),
        so the bound is tol + ulp(|ref|).  Returns the largest excess (<= 0 passes)."""
        a = np.asarray(a, np.float64)
        b = np.asarray(b, np.float64)
        self.err(name, a, b)
        if not np.size(a):
            return 0.0
        ulp = np.ldexp(1.0, np.frexp(np.abs(b))[1] - 8) if wl.dtype == "bf16" else np.zeros_like(b)
        return float(np.max(np.abs(a - b) - tol - ulp))


def kept_excess(g, ref, bound, wl):
    """Retained final states are rounded to the keep type (fp16 for bf16 models) on
    both sides; where the unrounded values differ by up to `bound` and straddle a
    rounding boundary the kept values differ by one more fp16 unit in the last place,
    so the allowance is bound + ulp16(|ref|).  Returns the largest excess (<= 0 passes)."""
    g = np.asarray(g, np.float64)
    ref = np.asarray(ref, np.float64)
    if not np.size(ref):
        return 0.0
    ulp = np.ldexp(1.0, np.frexp(np.abs(ref))[1] - 11) if wl.dtype == "bf16" else np.zeros_like(ref)
    return float(np.max(np.abs(g - ref) - bound - ulp))


def check_decisions(rep, o_logits, gpu_tok, tol, what, stage=False):
    """Oracle argmax must equal the GPU token wherever the oracle's top-2 gap > tol."""
    o_tok = np.argmax(o_logits, axis=-1)
    gap = top2_gap(o_logits)
    for i in range(len(gpu_tok)):
        if stage:
            rep.stage_decisions += 1
        else:
            rep.decisions += 1
        if gap[i] > tol:
            assert o_tok[i] == gpu_tok[i], f"{what} row {i}: oracle {o_tok[i]} gpu {gpu_tok[i]} gap {gap[i]}"
        elif stage:
            rep.stage_near_ties += 1
        else:
            rep.near_ties += 1


def kv_check(rep, name, g, ref, tol, wl, what, exact=None):
    """Cached K/V are intermediate tensors of a deep bf16 network.  There, any sub-ulp
    difference (fp32 MFMA accumulation order, fp32 versus float64 softmax) is amplified
    within two or three layers into bf16-rounding-level noise: at the Qwen3-0.6B shape
    the oracle's own mixed-precision K differs from its pure-float64 K by ~7e-3
    (relative Frobenius) at every layer past the first, and perturbing only the
    residual's precision by 6e-8 already moves layer-3 K by 3e-3.  The bound is
    therefore relative and calibrated per tensor when the float64 oracle's value
    `exact` is given: the GPU may be at most twice as far from the mixed-precision
    oracle as that oracle is from exact arithmetic (floor 1e-3); without it, 1e-2.  No
    element may be off by more than 0.25 (wrong positions, pages, RoPE angles or heads
    give O(1) errors).  Final hidden states and logits keep the absolute tolerance."""
    g = np.asarray(g, np.float64)
    ref = np.asarray(ref, np.float64)
    e = rep.err(name, g, ref)
    nrm = lambda a: max(float(np.linalg.norm(a)), 1e-30)
    rel = float(np.linalg.norm(g - ref)) / nrm(ref)
    rep.max_err[name + "_rel"] = max(rep.max_err.get(name + "_rel", 0.0), rel)
    if wl.dtype != "bf16":
        rel_bound, abs_bound = 1e-5, 1e-4
    elif exact is not None:
        q = float(np.linalg.norm(ref - np.asarray(exact, np.float64))) / nrm(ref)
        rep.max_err[name + "_quant_rel"] = max(rep.max_err.get(name + "_quant_rel", 0.0), q)
        rel_bound, abs_bound = max(2.0 * q, 1e-3), 0.25
    else:
        rel_bound, abs_bound = 1e-2, 0.25
    assert rel <= rel_bound and e <= abs_bound, f"{what}: relative error {rel} (bound {rel_bound}), max abs {e}"


def compare_prefill(eng, R, wl, prompts, seq_states, tol, layers=None, exact_states=None, gpu_seqs=None):
    """Target and drafter-context KV of every prompt position (exact_states: the same
    prefill by the float64 oracle, which calibrates the bf16 bound).  gpu_seqs[i] is
    the GPU sequence that prompts[i] / seq_states[i] describe (default: i)."""
    s = wl.target
    et = np.uint16 if wl.dtype == "bf16" else np.float32
    rep = Report()
    for i, st in enumerate(seq_states):
        b = gpu_seqs[i] if gpu_seqs is not None else i
        n = len(prompts[i])
        for l in (layers if layers is not None else range(s.n_layers)):
            for tid, ref in ((B.RT_T_TARGET_K + l, st.tgt_k[l]), (B.RT_T_TARGET_V + l, st.tgt_v[l])):
                g = store_to_f64(eng.read(tid, b, (n, s.n_kv_heads, s.head_dim), et), wl)
                ex = None
                if exact_states is not None:
                    xs = exact_states[i]
                    ex = (xs.tgt_k if tid < B.RT_T_TARGET_V else xs.tgt_v)[l][:n]
                kv_check(rep, "target_kv", g, ref[:n], tol, wl, f"seq {b} layer {l} target kv", ex)
        for l in range(wl.draft_layers):
            for tid, ref in ((B.RT_T_DRAFT_K + l, st.ctx_k[l]), (B.RT_T_DRAFT_V + l, st.ctx_v[l])):
                g = store_to_f64(eng.read(tid, b, (n, s.n_kv_heads, s.head_dim), et), wl)
                ex = None
                if exact_states is not None:
                    xs = exact_states[i]
                    ex = (xs.ctx_k if tid < B.RT_T_DRAFT_V else xs.ctx_v)[l][:n]
                kv_check(rep, "draft_ctx_kv", g, ref[:n], tol, wl, f"seq {b} drafter layer {l} ctx kv", ex)
    return rep


def carried_state(eng, b, wl):
    s, bk = wl.target, wl.block_size
    kd = keep_dtype(wl)
    return (eng.read(B.RT_T_HD, b, (bk, s.hidden), kd).astype(np.float64),
            eng.read(B.RT_T_HT, b, (bk, s.hidden), kd).astype(np.float64))


def inject_state(eng, st, b, wl, carried, kv=False):
    """Starts the oracle's round from the GPU's carried state (read before the GPU
    round): the retained drafter / target final states, optionally both KV caches."""
    s = wl.target
    st.hD_prev, st.hT_prev = carried
    if kv:
        et = np.uint16 if wl.dtype == "bf16" else np.float32
        shp = (st.P, s.n_kv_heads, s.head_dim)
        for l in range(s.n_layers):
            st.tgt_k[l, :st.P] = store_to_f64(eng.read(B.RT_T_TARGET_K + l, b, shp, et), wl)
            st.tgt_v[l, :st.P] = store_to_f64(eng.read(B.RT_T_TARGET_V + l, b, shp, et), wl)
        for l in range(wl.draft_layers):
            st.ctx_k[l, :st.P] = store_to_f64(eng.read(B.RT_T_DRAFT_K + l, b, shp, et), wl)
            st.ctx_v[l, :st.P] = store_to_f64(eng.read(B.RT_T_DRAFT_V + l, b, shp, et), wl)


def sync_kv_rows(eng, st, b, wl, p0, n):
    """Copies the GPU's target and drafter-context KV rows p0..p0+n-1 of sequence b into
    the oracle state st."""
    s = wl.target
    et = np.uint16 if wl.dtype == "bf16" else np.float32
    shp = (n, s.n_kv_heads, s.head_dim)
    for l in range(s.n_layers):
        st.tgt_k[l, p0:p0 + n] = store_to_f64(eng.read_rows(B.RT_T_TARGET_K + l, b, p0, shp, et), wl)
        st.tgt_v[l, p0:p0 + n] = store_to_f64(eng.read_rows(B.RT_T_TARGET_V + l, b, p0, shp, et), wl)
    for l in range(wl.draft_layers):
        st.ctx_k[l, p0:p0 + n] = store_to_f64(eng.read_rows(B.RT_T_DRAFT_K + l, b, p0, shp, et), wl)
        st.ctx_v[l, p0:p0 + n] = store_to_f64(eng.read_rows(B.RT_T_DRAFT_V + l, b, p0, shp, et), wl)


def check_layer_steps(eng, R: OracleRunner, wl, st, b, l, draft, rep, tol, exact, what, block_kv=None):
    """One decoder layer of the last round, step by step from the GPU's own operands
    (layer trace): q (and the block K/V) from the GPU's residual input; the attention
    output from the GPU's q over the GPU's cached keys; the post-attention residual from
    the GPU's attention output; the norm from that residual; the SwiGLU product from the
    GPU's norm output; the layer output from the GPU's residual and SwiGLU product.  Each
    step spans one kernel (or one GEMM and its epilogue), so it is held to `tol` (stored
    values to tol plus one unit in the last place).  The whole layer recomputed from its
    input alone is held to `tol` too, or with `exact` (a float64 runner) to twice the
    mixed-precision oracle's own distance from float64 arithmetic for that layer: in a
    random model with small residuals (an early layer), the post-attention norm scales
    fp32 rounding differences up by the inverse residual norm.  Returns the GPU output."""
    m, W, P = R.m, R.m.W, R.m.prec
    s, bk, d = wl.target, wl.block_size, wl.target.hidden
    et = np.uint16 if wl.dtype == "bf16" else np.float32
    pre, xb, sb = (f"draft.{l}", B.RT_T_TRACE_DRAFT_X, 1100) if draft else (f"target.{l}", B.RT_T_TRACE_TARGET_X, 2100)
    tag = "draft" if draft else "target"
    qN, F = s.n_q_heads * s.head_dim, s.ffn

    def tr(tid, width, f32=False):
        if f32:
            return eng.read(tid, b, (bk, width), np.float32).astype(np.float64)
        return store_to_f64(eng.read(tid, b, (bk, width), et), wl)

    x_in = tr(xb + l, d, True)
    x_out = tr(xb + l + 1, d, True)
    pos = st.P + np.arange(bk)
    q, k, v = m._qkv(pre, x_in, pos)
    g_q = tr(sb + l, qN).reshape(q.shape)
    assert rep.stored_err(f"step_{tag}_q", g_q, q, tol, wl) <= 0, f"{what} {tag} layer {l}: q"
    if draft:
        keys = np.concatenate([st.ctx_k[l, :st.P], k])
        vals = np.concatenate([st.ctx_v[l, :st.P], v])
        k_pos, causal = np.concatenate([np.arange(st.P), pos]), False
    else:
        gk, gv = block_kv
        assert rep.stored_err("step_target_block_kv", gk, k, tol, wl) <= 0, f"{what} target layer {l}: block K"
        assert rep.stored_err("step_target_block_kv", gv, v, tol, wl) <= 0, f"{what} target layer {l}: block V"
        keys = np.concatenate([st.tgt_k[l, :st.P], gk])
        vals = np.concatenate([st.tgt_v[l, :st.P], gv])
        k_pos, causal = np.arange(st.P + bk), True
    o = m.attn_out(g_q, keys, vals, pos, k_pos, causal)
    g_o = tr(sb + 100 + l, qN)
    assert rep.stored_err(f"step_{tag}_attn", g_o, o, tol, wl) <= 0, f"{what} {tag} layer {l}: attention output"
    x_mid = m.o_residual(pre, x_in, g_o)
    g_xm = tr(sb + 200 + l, d, True)
    e = rep.err(f"step_{tag}_o_resid", g_xm, x_mid)
    assert e <= tol, f"{what} {tag} layer {l}: residual after attention, max abs error {e}"
    h2 = m.mlp_input(pre, g_xm)
    g_h2 = tr(sb + 300 + l, d)
    assert rep.stored_err(f"step_{tag}_norm", g_h2, h2, tol, wl) <= 0, f"{what} {tag} layer {l}: post-attention norm"
    a = m.swiglu(pre, g_h2)
    g_a = tr(sb + 400 + l, F)
    assert rep.stored_err(f"step_{tag}_swiglu", g_a, a, tol, wl) <= 0, f"{what} {tag} layer {l}: SwiGLU product"
    y = m.down_residual(pre, g_xm, g_a)
    e = rep.err(f"step_{tag}_down_resid", x_out, y)
    assert e <= tol, f"{what} {tag} layer {l}: layer output from the GPU's SwiGLU product, max abs error {e}"
    # the whole layer from its input alone
    if draft:
        ref = m.drafter_layer(st, l, x_in)
        ref_x = exact.m.drafter_layer(st, l, x_in) if exact is not None else None
    else:
        ref_x = exact.m.target_layer(st, l, x_in, st.P) if exact is not None else None
        ref = m.target_layer(st, l, x_in, st.P)
    e = rep.err(f"stage_{tag}_layer", x_out, ref)
    bound = tol
    if ref_x is not None:
        qd = float(np.max(np.abs(ref - ref_x)))
        rep.max_err[f"stage_{tag}_layer_quant"] = max(rep.max_err.get(f"stage_{tag}_layer_quant", 0.0), qd)
        bound = max(tol, 2.0 * qd)
    assert e <= bound, f"{what} {tag} layer {l}: output from the layer input, max abs error {e} (bound {bound})"
    return x_out


def check_stages(eng, R: OracleRunner, wl, st, b, y_hat, forced, rep, tol, target_layers, draft_layers, what,
                 exact=None):
    """Per-stage teacher-forced check of the last round of GPU sequence b (layer trace on,
    fp32 logits stored): every checked layer step by step from the GPU's own operands
    (check_layer_steps; the oracle's caches hold the GPU's rows 0..P-1), the final norms
    from the GPU's final residuals, each LM head from the GPU's own operand.  Logits,
    final states and every argmax decision whose top-2 gap exceeds `tol` must agree:
    no decision is left to a calibrated bound.  Each comparison spans one step, so the
    error amplification of a deep random network across layers does not enter."""
    m, W, P = R.m, R.m.W, R.m.prec
    s, bk, d = wl.target, wl.block_size, wl.target.hidden
    et = np.uint16 if wl.dtype == "bf16" else np.float32
    kd = keep_dtype(wl)

    def tr(base, l):
        return eng.read(base + l, b, (bk, d), np.float32).astype(np.float64)

    # drafter: B+1 rows at P..P+B over the context cache
    for l in draft_layers:
        check_layer_steps(eng, R, wl, st, b, l, True, rep, tol, exact, what)
    h = rms_norm(tr(B.RT_T_TRACE_DRAFT_X, wl.draft_layers), W["draft.final_norm"], m.eps)
    g_hd = eng.read(B.RT_T_HD, b, (bk, d), kd)
    rep.err("stage_h_draft", g_hd, P.k(h))
    assert kept_excess(g_hd, P.k(h), tol, wl) <= 0, f"{what}: h^D from the GPU's final residual"
    head = store_to_f64(eng.read(B.RT_T_TRACE_DRAFT_HEAD, b, (bk, d), et), wl)
    assert rep.stored_err("stage_draft_head_in", head, P.a(h), tol, wl) <= 0, f"{what}: drafter LM-head input"
    logits = m.lm_logits(head)
    g_dl = eng.read(B.RT_T_DRAFT_LOGITS, b, (bk, s.vocab), np.float32)
    e = rep.err("stage_draft_logits", g_dl[1:], logits[1:])
    assert e <= tol, f"{what}: drafter logits from the GPU's LM-head input, max abs error {e}"
    if not forced:
        g_dt = eng.read(B.RT_T_DRAFT_TOKENS, b, (bk,), np.int32)
        check_decisions(rep, logits[1:], g_dt[1:], tol, f"{what} draft (per stage)", stage=True)
    # verify: [anchor, drafts] at P..P+B, causal over the target cache
    toks = np.array([st.anchor] + [int(t) for t in y_hat])
    e = rep.err("stage_embed", tr(B.RT_T_TRACE_TARGET_X, 0), P.r(W.rows("embed", toks)))
    assert e == 0.0, f"{what}: verify embedding rows differ by {e}"
    shp = (bk, s.n_kv_heads, s.head_dim)
    for l in target_layers:
        gk = store_to_f64(eng.read_rows(B.RT_T_TARGET_K + l, b, st.P, shp, et), wl)
        gv = store_to_f64(eng.read_rows(B.RT_T_TARGET_V + l, b, st.P, shp, et), wl)
        check_layer_steps(eng, R, wl, st, b, l, False, rep, tol, exact, what, block_kv=(gk, gv))
    xT = tr(B.RT_T_TRACE_TARGET_X, s.n_layers)
    h = rms_norm(xT, W["target.final_norm"], m.eps)
    g_ht = eng.read(B.RT_T_HT, b, (bk, d), kd)
    rep.err("stage_h_target", g_ht, P.k(h))
    assert kept_excess(g_ht, P.k(h), tol, wl) <= 0, f"{what}: h^T from the GPU's final residual"
    head = store_to_f64(eng.read(B.RT_T_TRACE_VERIFY_HEAD, b, (bk, d), et), wl)
    assert rep.stored_err("stage_verify_head_in", head, P.a(h), tol, wl) <= 0, f"{what}: verify LM-head input"
    logits = m.lm_logits(head)
    g_vl = eng.read(B.RT_T_VERIFY_LOGITS, b, (bk, s.vocab), np.float32)
    e = rep.err("stage_verify_logits", g_vl, logits)
    assert e <= tol, f"{what}: verify logits from the GPU's LM-head input, max abs error {e}"
    g_tt = eng.read(B.RT_T_TARGET_TOKENS, b, (bk,), np.int32)
    check_decisions(rep, logits, g_tt, tol, f"{what} verify (per stage)", stage=True)
    # captured conditioning-layer states: the storage rounding of the traced residuals
    g = store_to_f64(eng.read(B.RT_T_G, b, (bk, len(wl.cond_layers) * d), et), wl)
    for i, l in enumerate(wl.cond_layers):
        e = rep.err("stage_capture", g[:, i * d:(i + 1) * d], P.a(tr(B.RT_T_TRACE_TARGET_X, l + 1)))
        assert e == 0.0, f"{what}: captured state of layer {l} differs by {e}"
    return g


def check_context_rows(eng, R: OracleRunner, wl, st, b, g, P0, n, rep, tol, what):
    """The drafter context rows P0..P0+n-1 the GPU appended, against the oracle's context
    pathway applied to the GPU's own captured states g[:n]; then st takes the GPU's rows."""
    s = wl.target
    et = np.uint16 if wl.dtype == "bf16" else np.float32
    R.m.context_append(st, g[:n], P0)
    shp = (n, s.n_kv_heads, s.head_dim)
    for l in range(wl.draft_layers):
        for tid, cache in ((B.RT_T_DRAFT_K + l, st.ctx_k), (B.RT_T_DRAFT_V + l, st.ctx_v)):
            gkv = store_to_f64(eng.read_rows(tid, b, P0, shp, et), wl)
            assert rep.stored_err("stage_context_kv", gkv, cache[l, P0:P0 + n], tol, wl) <= 0, \
                f"{what} drafter layer {l}: appended context K/V"


def run_teacher_forced(eng, R: OracleRunner, wl, seq_states, n_rounds, tol, forced=None, rep=None,
                       inject=True, inject_kv=False, exact: OracleRunner = None, stages=None):
    """Runs n_rounds GPU rounds (debug: logits stored, no graph) and checks each
    against the oracle continuing from the same decisions.  With inject, every
    round starts the oracle from the GPU's carried state, so each comparison
    measures one round.  forced: optional list (per round) of [n_seqs][B] drafts.
    seq_states[b] = None leaves GPU sequence b unchecked (sampled batches).

    exact: a float64 runner of the same model.  The absolute tolerance then widens,
    per tensor, to twice the mixed-precision oracle's own distance from float64
    arithmetic on the same inputs (deep random bf16 networks sit near 2e-2 there),
    never below `tol`; the widened bound and the distance are reported.  Argmax
    decisions are then fixed only where the oracle's top-2 gap exceeds twice the
    logit bound (otherwise where it exceeds `tol`).

    stages: per-stage checks (check_stages) with the layer trace on, a dict with the
    target and drafter layers to recompute ("target_layers", "draft_layers"; default
    all).  The oracle's caches then always hold the GPU's rows: all of them before the
    first round, and the rows each round commits after it, so every layer is checked
    on the GPU's own inputs at tolerance `tol`; the end-to-end comparison above stays
    as an additional check."""
    s, bk, B_ = wl.target, wl.block_size, wl.B
    rep = rep or Report()
    eng.set_debug(11 if stages is not None else 3)
    if stages is not None:
        inject, inject_kv = True, True
        t_layers = list(stages.get("target_layers", range(s.n_layers)))
        d_layers = list(stages.get("draft_layers", range(wl.draft_layers)))
    kd = keep_dtype(wl)
    ns = len(seq_states)
    for t in range(n_rounds):
        carried = [carried_state(eng, b, wl) if inject and seq_states[b] is not None else None for b in range(ns)]
        if forced is not None:
            tok, n_c, acc = eng.spec_round_forced(forced[t])
        else:
            tok, n_c, acc = eng.spec_round()
        for b, st in enumerate(seq_states):
            if st is None:        # sequence not sampled
                continue
            if st.done:
                assert n_c[b] == 0
                continue
            if inject:
                inject_state(eng, st, b, wl, carried[b], kv=inject_kv and t == 0)
            rep.conditioned += st.cond_len > 0 and wl.cond_mode != "off"
            d = R.draft(st)
            dx = exact.draft(st) if exact is not None else None

            def decision_tol(bd):
                # a calibrated logit bound bd lets each of the top two logits move by bd,
                # so only decisions whose oracle gap exceeds 2 * bd are fixed by it
                return tol if bd <= tol else 2.0 * bd

            def bound(name, mixed, ex):
                if ex is None:
                    return tol
                q = float(np.max(np.abs(np.asarray(mixed) - np.asarray(ex))))
                rep.max_err[name + "_quant"] = max(rep.max_err.get(name + "_quant", 0.0), q)
                return max(tol, 2.0 * q)

            g_et = eng.read(B.RT_T_ETILDE, b, (bk, s.hidden), np.float32)
            e = rep.err("e_tilde", g_et, d.e_tilde)
            assert e <= tol, f"round {t} seq {b}: e_tilde err {e}"
            g_hd = eng.read(B.RT_T_HD, b, (bk, s.hidden), kd)
            e = rep.err("h_draft", g_hd, R.m.prec.k(d.h))
            bd = bound("h_draft", d.h, dx.h if dx else None)
            assert kept_excess(g_hd, R.m.prec.k(d.h), bd, wl) <= 0, f"round {t} seq {b}: h^D err {e} (bound {bd} + ulp)"
            g_dl = eng.read(B.RT_T_DRAFT_LOGITS, b, (bk, s.vocab), np.float32)
            e = rep.err("draft_logits", g_dl[1:], d.logits[1:])
            bd = bound("draft_logits", d.logits[1:], dx.logits[1:] if dx else None)
            assert e <= bd, f"round {t} seq {b}: draft logits err {e} (bound {bd})"
            g_dt = eng.read(B.RT_T_DRAFT_TOKENS, b, (bk,), np.int32)
            if forced is None:
                check_decisions(rep, d.logits[1:], g_dt[1:], decision_tol(bd), f"round {t} seq {b} draft")
            else:
                assert list(g_dt[1:]) == list(forced[t][b])
            y_hat = g_dt[1:].astype(np.int64)
            g_cap = None
            if stages is not None:
                g_cap = check_stages(eng, R, wl, st, b, y_hat, forced is not None, rep, tol, t_layers, d_layers,
                                     f"round {t} seq {b}", exact=exact)
            vx = exact.verify(st, y_hat) if exact is not None else None   # before the mixed verify,
            v = R.verify(st, y_hat)                                        # which rewrites rows P..P+B
            g_ht = eng.read(B.RT_T_HT, b, (bk, s.hidden), kd)
            e = rep.err("h_target", g_ht, R.m.prec.k(v.h))
            bd = bound("h_target", v.h, vx.h if vx else None)
            assert kept_excess(g_ht, R.m.prec.k(v.h), bd, wl) <= 0, f"round {t} seq {b}: h^T err {e} (bound {bd} + ulp)"
            g_vl = eng.read(B.RT_T_VERIFY_LOGITS, b, (bk, s.vocab), np.float32)
            e = rep.err("verify_logits", g_vl, v.logits)
            bd = bound("verify_logits", v.logits, vx.logits if vx else None)
            assert e <= bd, f"round {t} seq {b}: verify logits err {e} (bound {bd})"
            g_tt = eng.read(B.RT_T_TARGET_TOKENS, b, (bk,), np.int32)
            check_decisions(rep, v.logits, g_tt, decision_tol(bd), f"round {t} seq {b} verify")
            P_before = st.P
            A, new = R.commit(st, y_hat, g_tt.astype(np.int64), d, v)
            assert A == acc[b], f"round {t} seq {b}: A oracle {A} gpu {acc[b]}"
            assert list(tok[b][: n_c[b]]) == new, f"round {t} seq {b}: committed {tok[b][:n_c[b]]} vs {new}"
            if stages is not None:
                check_context_rows(eng, R, wl, st, b, g_cap, P_before, A + 1, rep, tol, f"round {t} seq {b}")
                sync_kv_rows(eng, st, b, wl, P_before, A + 1)
            gst = eng.read(B.RT_T_STATE, b, (8,), np.int32)
            assert gst[0] == st.P and gst[1] == st.anchor, f"state {gst} vs P {st.P} anchor {st.anchor}"
            assert gst[3] == st.cond_len and (st.cond_len == 0 or gst[2] == st.r), f"carry {gst} vs {st.r},{st.cond_len}"
            assert gst[5] == P_before and gst[6] == A + 1
            rep.accept.append(A)
        rep.rounds += 1
    return rep


def planted_drafts(eng, wl, n_seqs, plan):
    """Forced drafts with a known acceptance length per sequence.  plan[b] = k plants a
    mismatch at block position k (A = k - 1); None gives the full greedy continuation
    (A = B); sequences absent from plan draft token 0.  The target's greedy
    continuation is found on the GPU: the next round is run with forced drafts and
    undone (retained states and round state written back; the caches only hold rows
    beyond the committed length, which the next round rewrites) until every planned
    prefix matches the target's own verify tokens, one block position or more per
    repeat.  Returns drafts [n_seqs][B]; the GPU is left in the state it had."""
    bk, B_, V = wl.block_size, wl.B, wl.target.vocab
    kd, d = keep_dtype(wl), wl.target.hidden
    saved = [(eng.read(B.RT_T_STATE, b, (9,), np.int32), eng.read(B.RT_T_HD, b, (bk, d), kd),
              eng.read(B.RT_T_HT, b, (bk, d), kd)) for b in range(n_seqs)]
    need = {b: (B_ if k is None else k - 1) for b, k in plan.items()}
    drafts = np.zeros((n_seqs, B_), np.int32)

    def restore():
        for b, (stv, hd, ht) in enumerate(saved):
            eng.write(B.RT_T_STATE, b, stv)
            eng.write(B.RT_T_HD, b, hd)
            eng.write(B.RT_T_HT, b, ht)

    for _ in range(B_ + 1):
        eng.spec_round_forced(drafts)
        done = True
        for b, n in need.items():
            y_t = eng.read(B.RT_T_TARGET_TOKENS, b, (bk,), np.int32)
            A = 0
            while A < B_ and drafts[b][A] == y_t[A]:
                A += 1
            if A < n:
                drafts[b][A] = y_t[A]      # verify row A saw the continuation's first A tokens
                done = False
        restore()
        if done:
            break
    else:
        raise AssertionError("greedy continuations not found within B + 1 repeats")
    for b, k in plan.items():
        if k is not None:
            drafts[b][k - 1] = (drafts[b][k - 1] + 1) % V
    return drafts
