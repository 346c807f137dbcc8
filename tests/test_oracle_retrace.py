"""Pins for the oracle's ReTrace round: the paper's worked index example, closed
forms of the conditioning under special weights, its stated reductions (W_v = 0,
beta = 0), losslessness against target-only greedy decoding, brute-force
recomputation, planted drafts with known acceptance lengths, the reset rule,
budget clipping, the component-ablation conditioning variants (Table 3), and the
drafter's internal consistency."""
import dataclasses
import json
import os

import numpy as np
import pytest

import oracle.retrace as ort
from oracle import OracleModel, OracleRunner, Precision
from oracle.model import rms_norm
from oracle.retrace import accept_length, align_rejected, condition_inputs
from workloads import get, make_prompts, make_weights

from hf_reference import qwen3_from_weights

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


# ------------------------------------------------------------ index arithmetic

def check_fig3(align=align_rejected, accept=accept_length):
    g = json.load(open(os.path.join(GOLDEN, "fig3_alignment.json")))
    B, exp = g["B"], g["expected"]
    A = accept(g["draft_tokens"], g["target_tokens"][:B])
    assert A == exp["A"]
    r = A + 1
    assert r == exp["first_rejected"]
    committed = g["draft_tokens"][:A] + [g["target_tokens"][A]]
    assert committed == exp["committed"]
    cond_len = B - r
    assert cond_len == exp["cond_len"]
    d = 3
    hD = np.array([[10.0 * j + c for c in range(d)] for j in range(B + 1)])   # row j labelled 10j
    hT = np.array([[-10.0 * j - c for c in range(d)] for j in range(B + 1)])
    m, u = align(hD, hT, r, B)
    for j, src in enumerate(exp["m_rows_from_draft_positions"], start=1):
        np.testing.assert_array_equal(m[j], hD[src])
    for j, src in enumerate(exp["u_rows_from_verify_rows"], start=1):
        np.testing.assert_array_equal(u[j], hT[src])
    for j in [0] + exp["zero_rows"]:
        assert not m[j].any() and not u[j].any()


def test_fig3_worked_example():
    check_fig3()


def test_alignment_all_rejection_points():
    B, d = 15, 2
    hD = np.arange((B + 1) * d, dtype=float).reshape(B + 1, d) + 1
    hT = -hD
    for A in range(B - 1):
        r = A + 1
        m, u = align_rejected(hD, hT, r, B)
        n = B - r
        assert (np.abs(m).sum(axis=1) > 0).sum() == n
        if n:
            np.testing.assert_array_equal(m[1:n + 1], hD[r + 1:B + 1])
            np.testing.assert_array_equal(u[1:n + 1], hT[r:B])


def test_accept_length_cases():
    assert accept_length([1, 2, 3], [1, 2, 4]) == 2
    assert accept_length([5, 2, 3], [1, 2, 3]) == 0
    assert accept_length([1, 2, 3], [1, 2, 3]) == 3


# ------------------------------------------------------------ conditioning closed forms

D = 3


def _rows(rng, n=5):
    return rng.standard_normal((n, D))


def check_concat_order(cond=condition_inputs):
    """W_c = [0 | I] selects u, W_v = I, W_g = 0 (gate 1/2), beta = 1/2:
    e~_j = e_j + (m_j + u_j / 2) / 2."""
    rng = np.random.default_rng(0)
    e, m, u = _rows(rng), _rows(rng), _rows(rng)
    I, Z = np.eye(D), np.zeros((D, D))
    out = cond(e, m, u, 3, np.hstack([Z, I]), I, np.hstack([Z, Z]), 0.5)
    np.testing.assert_allclose(out[1:4], e[1:4] + 0.5 * (m[1:4] + 0.5 * u[1:4]), rtol=1e-14)
    np.testing.assert_array_equal(out[0], e[0])
    np.testing.assert_array_equal(out[4:], e[4:])


def check_gate_inputs(cond=condition_inputs):
    """Hand-worked d=2 rows: W_c = 0, W_v = I.  W_g = [I | 0] gates by sigmoid(e);
    W_g = [0 | I] gates by sigmoid(r) with r = m."""
    e = np.array([[9.0, 9.0], [0.0, np.log(3.0)]])
    m = np.array([[0.0, 0.0], [2.0, 4.0]])
    u = np.array([[0.0, 0.0], [7.0, -7.0]])
    I, Z = np.eye(2), np.zeros((2, 2))
    out = cond(e, m, u, 1, np.hstack([Z, Z]), I, np.hstack([I, Z]), 1.0)
    np.testing.assert_allclose(out[1], [1.0, np.log(3.0) + 3.0], rtol=1e-14)
    out = cond(e, m, u, 1, np.hstack([Z, Z]), I, np.hstack([Z, I]), 1.0)
    s = lambda x: 1 / (1 + np.exp(-x))
    np.testing.assert_allclose(out[1], [2 * s(2.0), np.log(3.0) + 4 * s(4.0)], rtol=1e-14)


def check_beta_scales_correction(cond=condition_inputs):
    """W_c = [I | 0]: c = m, so r = (1 + beta) m; with W_v = I, W_g = 0: e~ = e + (1+beta) m / 2."""
    rng = np.random.default_rng(1)
    e, m, u = _rows(rng), _rows(rng), _rows(rng)
    I, Z = np.eye(D), np.zeros((D, D))
    for beta in (0.0, 0.5, 1.0):
        out = cond(e, m, u, 4, np.hstack([I, Z]), I, np.hstack([Z, Z]), beta)
        np.testing.assert_allclose(out[1:], e[1:] + 0.5 * (1 + beta) * m[1:], rtol=1e-14)


def test_conditioning_closed_forms():
    check_concat_order()
    check_gate_inputs()
    check_beta_scales_correction()


def test_wv_zero_keeps_inputs_exactly():
    """Zero-initialised W_v: the residual vanishes and the draft input is unchanged."""
    rng = np.random.default_rng(2)
    e, m, u = _rows(rng, 16), _rows(rng, 16), _rows(rng, 16)
    out = condition_inputs(e, m, u, 14, rng.standard_normal((D, 2 * D)), np.zeros((D, D)),
                           rng.standard_normal((D, 2 * D)), 1.0)
    np.testing.assert_array_equal(out, e)


def test_beta_zero_is_raw_gated():
    """beta = 0 leaves the aligned draft state uncorrected: r_j = m_j."""
    rng = np.random.default_rng(3)
    e, m, u = _rows(rng), _rows(rng), _rows(rng)
    wv, wg = rng.standard_normal((D, D)), rng.standard_normal((D, 2 * D))
    out = condition_inputs(e, m, u, 4, rng.standard_normal((D, 2 * D)), wv, wg, 0.0)
    s = lambda x: 1 / (1 + np.exp(-x))
    for j in range(1, 5):
        np.testing.assert_allclose(out[j], e[j] + (wv @ m[j]) * s(wg @ np.concatenate([e[j], m[j]])),
                                   rtol=1e-13)


def check_raw_gated_ignores_correction(cond=condition_inputs):
    """Raw gated fusion (Table 3): r_j = m_j, so W_c, u and beta drop out and the result
    equals the corrected form at beta = 0; hand-worked d = 2 row with W_v = I,
    W_g = [0 | I]: e~ = e + m * sigmoid(m)."""
    rng = np.random.default_rng(5)
    e, m, u = _rows(rng), _rows(rng), _rows(rng)
    wv, wg = rng.standard_normal((D, D)), rng.standard_normal((D, 2 * D))
    ref = condition_inputs(e, m, u, 4, np.zeros((D, 2 * D)), wv, wg, 1.0)   # W_c = 0: r = m
    for wc, uu, beta in ((rng.standard_normal((D, 2 * D)), u, 1.0), (np.eye(D, 2 * D), 3 * m, 0.5)):
        np.testing.assert_allclose(cond(e, m, uu, 4, wc, wv, wg, beta, "raw_gated"), ref, rtol=1e-13)
    e2 = np.array([[9.0, 9.0], [0.5, -1.0]])
    m2 = np.array([[0.0, 0.0], [2.0, -3.0]])
    u2 = np.array([[0.0, 0.0], [7.0, 5.0]])
    I, Z = np.eye(2), np.zeros((2, 2))
    s = lambda x: 1 / (1 + np.exp(-x))
    out = cond(e2, m2, u2, 1, np.hstack([I, I]), I, np.hstack([Z, I]), 1.0, "raw_gated")
    np.testing.assert_allclose(out[1], [0.5 + 2 * s(2.0), -1.0 - 3 * s(-3.0)], rtol=1e-14)
    np.testing.assert_array_equal(out[0], e2[0])


def check_overwrite_replaces_rows(cond=condition_inputs):
    """Overwrite (Table 3): conditioned rows 1..n become m_j exactly, whatever the
    weights; the anchor row and rows past n keep e."""
    rng = np.random.default_rng(6)
    e, m, u = _rows(rng, 8), _rows(rng, 8), _rows(rng, 8)
    w = lambda *s: rng.standard_normal(s)
    out = cond(e, m, u, 5, w(D, 2 * D), w(D, D), w(D, 2 * D), 1.0, "overwrite")
    np.testing.assert_array_equal(out[1:6], m[1:6])
    np.testing.assert_array_equal(out[0], e[0])
    np.testing.assert_array_equal(out[6:], e[6:])


def check_lowrank_reduces_to_full(cond=condition_inputs):
    """With d equal to the latent rank (64), A = I, V = W_v, G = W_g[:, d:] and a rank-32
    W_c = C_up C_down, the low-rank form is the full form of Eq.7-9 (parity of the
    low-rank reading itself is unpinned against the paper, which describes it in one
    sentence)."""
    rng = np.random.default_rng(11)
    d = 64
    e, m, u = (rng.standard_normal((6, d)) for _ in range(3))
    c_down, c_up = rng.standard_normal((32, 2 * d)) * 0.1, rng.standard_normal((d, 32)) * 0.1
    wv, wg = rng.standard_normal((d, d)) * 0.1, rng.standard_normal((d, 2 * d)) * 0.1
    for beta in (1.0, 0.5):
        full = condition_inputs(e, m, u, 4, c_up @ c_down, wv, wg, beta)
        low = cond(e, m, u, 4, None, None, wg, beta, "lowrank", (np.eye(d), c_down, c_up, wv, wg[:, d:]))
        np.testing.assert_allclose(low, full, rtol=1e-12, atol=1e-14)
    # beta = 0: rho = A m (no correction); V = 0: inputs unchanged
    A, V, G = rng.standard_normal((64, d)), rng.standard_normal((d, 64)), rng.standard_normal((d, 64))
    s = lambda x: 1 / (1 + np.exp(-x))
    low = cond(e, m, u, 3, None, None, wg, 0.0, "lowrank", (A, c_down, c_up, V, G))
    for j in range(1, 4):
        rho = A @ m[j]
        np.testing.assert_allclose(low[j], e[j] + (V @ rho) * s(wg[:, :d] @ e[j] + G @ rho), rtol=1e-12)
    np.testing.assert_array_equal(low[4:], e[4:])
    low = cond(e, m, u, 3, None, None, wg, 1.0, "lowrank", (A, c_down, c_up, np.zeros_like(V), G))
    np.testing.assert_array_equal(low, e)


def test_ablation_conditioning_closed_forms():
    check_raw_gated_ignores_correction()
    check_overwrite_replaces_rows()
    check_lowrank_reduces_to_full()
    for mode in ("retrace", "raw_gated", "overwrite"):   # nothing conditioned: inputs unchanged
        rng = np.random.default_rng(7)
        e, m, u = _rows(rng), _rows(rng), _rows(rng)
        out = condition_inputs(e, m, u, 0, w := rng.standard_normal((D, 2 * D)), rng.standard_normal((D, D)), w,
                               1.0, mode)
        np.testing.assert_array_equal(out, e)


# ------------------------------------------------------------ planted mistakes must be caught

def _align_off_by_one(hD, hT, r, B):
    m, u = align_rejected(hD, hT, r, B)
    u2 = np.zeros_like(u)
    for j in range(1, B - r + 1):
        u2[j] = hT[r + j] if r + j <= B else 0
    return m, u2


def _cond_swapped(e, m, u, n, wc, wv, wg, beta):
    return condition_inputs(e, u, m, n, wc, wv, wg, beta)


def _cond_gate_on_r_only(e, m, u, n, wc, wv, wg, beta):
    d = e.shape[1]
    return condition_inputs(np.zeros_like(e), m, u, n, wc, wv, wg, beta) + e


@pytest.mark.parametrize("check,kw", [
    (check_fig3, {"align": _align_off_by_one}),
    (check_fig3, {"accept": lambda a, b: accept_length(a, b) + 1}),
    (check_concat_order, {"cond": _cond_swapped}),
    (check_gate_inputs, {"cond": _cond_gate_on_r_only}),
    (check_beta_scales_correction, {"cond": lambda e, m, u, n, wc, wv, wg, b:
                                    condition_inputs(e, m, u, n, wc, wv, wg, 1.0)}),
    # raw gated fusion fed the target state instead of the drafter's, or still corrected
    (check_raw_gated_ignores_correction, {"cond": lambda e, m, u, n, wc, wv, wg, b, mode:
                                          condition_inputs(e, u, m, n, wc, wv, wg, 0.0)}),
    (check_raw_gated_ignores_correction, {"cond": lambda e, m, u, n, wc, wv, wg, b, mode:
                                          condition_inputs(e, m, u, n, wc, wv, wg, b)}),
    # overwrite that adds m to e, or shifts the aligned rows by one
    (check_overwrite_replaces_rows, {"cond": lambda e, m, u, n, wc, wv, wg, b, mode:
                                     np.concatenate([e[:1], e[1:n + 1] + m[1:n + 1], e[n + 1:]])}),
    (check_overwrite_replaces_rows, {"cond": lambda e, m, u, n, wc, wv, wg, b, mode:
                                     np.concatenate([e[:1], m[:n], e[n + 1:]])}),
    # low-rank form with the correction's factors swapped into the wrong order, or the
    # gate reading the latent through V instead of G
    (check_lowrank_reduces_to_full, {"cond": lambda e, m, u, n, wc, wv, wg, b, mode, lr:
                                     condition_inputs(e, m, u, n, wc, wv, wg, b, mode,
                                                      (lr[0], lr[1], lr[2], lr[3], lr[3]))}),
    (check_lowrank_reduces_to_full, {"cond": lambda e, m, u, n, wc, wv, wg, b, mode, lr:
                                     condition_inputs(e, u, m, n, wc, wv, wg, b, mode, lr)}),
])
def test_pins_catch_planted_mistakes(check, kw):
    with pytest.raises(AssertionError):
        check(**kw)


# ------------------------------------------------------------ whole-round pins

@pytest.fixture(scope="module")
def tiny():
    wl = get("tiny-f32", norm_init="perturbed")
    W = make_weights(wl)
    return wl, W, make_prompts(wl)[0]


@pytest.fixture(scope="module")
def mini():
    wl = get("mini-bf16", norm_init="perturbed")
    W = make_weights(wl)
    return wl, W, make_prompts(wl)[0]


@pytest.mark.parametrize("which,mode", [("tiny", "retrace"), ("mini", "retrace"), ("mini", "raw_gated"),
                                        ("mini", "overwrite"), ("mini", "lowrank"), ("mini", "off")])
def test_lossless_against_target_greedy(which, mode, tiny, mini):
    """Whatever the drafter's conditioning, greedy verification commits exactly the
    target's own greedy continuation (Section 3, lossless acceptance)."""
    wl, W, prompt = tiny if which == "tiny" else mini
    wl = dataclasses.replace(wl, cond_mode=mode)
    if mode == "lowrank":
        W = make_weights(wl)          # adds the low-rank factors; the other tensors are unchanged
    R = OracleRunner(OracleModel(wl, W))
    gen, recs, _ = R.spec_decode(prompt, wl.new_tokens)
    assert len(gen) == wl.new_tokens
    assert gen == R.ar_decode(prompt, wl.new_tokens)
    for rec in recs:   # rejected proposals are never committed
        assert list(rec.committed[: rec.A]) == list(rec.y_hat[: rec.A])
        if rec.A < wl.B:
            assert rec.y_hat[rec.A] != rec.y_t[rec.A]
            assert rec.committed[rec.A:] in ([], [rec.y_t[rec.A]])


def test_brute_force_recompute(tiny):
    wl, W, prompt = tiny
    R = OracleRunner(OracleModel(wl, W))
    gen, _, _ = R.spec_decode(prompt, 40)
    seq = np.concatenate([prompt, gen])
    logits = R.logits_nocache(seq[:-1])
    n = len(prompt)
    assert list(np.argmax(logits[n - 1:], axis=1)) == gen


def _planted_rounds(wl, W, prompt, plants, budget=80):
    """Rounds with drafts taken from the target's own greedy continuation, with a
    wrong token planted at block position k (None: no error)."""
    R = OracleRunner(OracleModel(wl, W))
    truth = R.ar_decode(prompt, budget + wl.B + 1)
    st = R.prefill(prompt, budget)
    out = []
    for k in plants:
        done = len(st.generated)
        draft = list(truth[done:done + wl.B])
        if k is not None:
            draft[k - 1] = (draft[k - 1] + 1) % wl.target.vocab
        rec = R.round(st, forced_draft=draft)
        out.append((k, rec, st.cond_len, st.r))
    return R, st, truth, out


def test_planted_drafts_fix_acceptance_and_reset(mini):
    wl, W, prompt = mini
    B = wl.B
    plants = [1, 3, B - 1, B, None, 2]
    R, st, truth, out = _planted_rounds(wl, W, prompt, plants)
    for k, rec, cond_len, r in out:
        A = B if k is None else k - 1
        assert rec.A == A
        if A < B - 1:
            assert (r, cond_len) == (A + 1, B - A - 1)
        else:
            assert cond_len == 0                      # full acceptance / last-position rejection
    assert st.generated == truth[: len(st.generated)]
    while not st.done:                                # continue unforced: still lossless
        R.round(st)
    assert st.generated == truth[:st.budget]


def test_budget_clips_last_round(mini):
    wl, W, prompt = mini
    R = OracleRunner(OracleModel(wl, W))
    truth = R.ar_decode(prompt, wl.B + 2)
    st = R.prefill(prompt, 10)
    rec = R.round(st, forced_draft=truth[1:1 + wl.B])   # would accept B+1 tokens
    assert rec.A == wl.B
    assert len(rec.committed) == 9
    assert st.generated == truth[:10] and st.done


def test_wv_zero_run_is_plain_dflash(mini):
    wl, _, prompt = mini
    W0 = make_weights(wl, wv_zero=True)
    R = OracleRunner(OracleModel(wl, W0))
    st = R.prefill(prompt, 20)
    for _ in range(4):
        d = R.draft(st)
        np.testing.assert_array_equal(d.e_tilde, d.e)
        R.round(st)


@pytest.mark.parametrize("mode", ["overwrite", "raw_gated", "lowrank", "off"])
def test_ablation_rounds_condition_the_drafter_input(mini, mode):
    """Within whole rounds: overwrite puts the previous round's aligned drafter states on
    the conditioned rows (Eq.5 alignment), raw gated and off leave the anchor and the
    unconditioned rows at their embeddings, and off leaves every row there."""
    wl, W, prompt = mini
    wl = dataclasses.replace(wl, cond_mode=mode)
    if mode == "lowrank":
        W = make_weights(wl)
    R = OracleRunner(OracleModel(wl, W))
    truth = R.ar_decode(prompt, 60)
    st = R.prefill(prompt, 50)
    seen = 0
    for k in (2, 5, None, 1, 3):
        r, n, hD = st.r, st.cond_len, None if st.hD_prev is None else st.hD_prev.copy()
        d = R.draft(st)
        if mode == "off" or n == 0:
            np.testing.assert_array_equal(d.e_tilde, d.e)
        else:
            seen += 1
            np.testing.assert_array_equal(d.e_tilde[0], d.e[0])
            np.testing.assert_array_equal(d.e_tilde[n + 1:], d.e[n + 1:])
            if mode == "overwrite":
                np.testing.assert_array_equal(d.e_tilde[1:n + 1], hD[r + 1:r + n + 1])
            else:
                assert not np.array_equal(d.e_tilde[1:n + 1], d.e[1:n + 1])
        done = len(st.generated)
        draft = list(truth[done:done + wl.B])
        if k is not None:
            draft[k - 1] = (draft[k - 1] + 1) % wl.target.vocab
        R.round(st, forced_draft=draft)
    assert mode == "off" or seen >= 3


def test_context_pathway_incremental_equals_recomputed(tiny):
    wl, W, prompt = tiny
    m = OracleModel(wl, W, prec=Precision.for_dtype("f64"))
    R = OracleRunner(m)
    truth = R.ar_decode(prompt, 60)
    st = R.prefill(prompt, 40)
    for k in (2, 5, None, 1):
        done = len(st.generated)
        draft = list(truth[done:done + wl.B])
        if k is not None:
            draft[k - 1] = (draft[k - 1] + 1) % wl.target.vocab
        R.round(st, forced_draft=draft)
    seq = np.concatenate([prompt, st.generated[:-1]])
    fresh = m.new_state(seq, 0)
    g = m.target_forward(fresh, seq, 0).g
    m.context_append(fresh, g, 0)
    np.testing.assert_allclose(fresh.ctx_k[:, :st.P], st.ctx_k[:, :st.P], atol=1e-11, rtol=0)
    np.testing.assert_allclose(fresh.ctx_v[:, :st.P], st.ctx_v[:, :st.P], atol=1e-11, rtol=0)
    np.testing.assert_allclose(fresh.tgt_k[:, :st.P], st.tgt_k[:, :st.P], atol=1e-11, rtol=0)


def test_drafter_without_context_is_noncausal_qwen3_stack(tiny):
    """With no context rows, the drafter block is a Qwen3 decoder stack over the
    conditioned inputs with an all-visible mask (transformers, CPU, float64)."""
    import torch
    from transformers import Qwen3Config, Qwen3Model
    wl, W, _ = tiny
    s = wl.target
    m = OracleModel(wl, W, prec=Precision.for_dtype("f64"))
    st = m.new_state(np.zeros(1, int), 0)
    st.P = 0
    e_t = np.random.default_rng(5).standard_normal((wl.block_size, s.hidden))
    h, _ = m.drafter_forward(st, e_t)
    cfg = Qwen3Config(vocab_size=s.vocab, hidden_size=s.hidden, intermediate_size=s.ffn,
                      num_hidden_layers=wl.draft_layers, num_attention_heads=s.n_q_heads,
                      num_key_value_heads=s.n_kv_heads, head_dim=s.head_dim,
                      rope_theta=wl.rope_theta, rms_norm_eps=wl.rms_eps,
                      attn_implementation="eager")
    hf = Qwen3Model(cfg).double().eval()
    from hf_reference import as_f32
    t = lambda n: torch.from_numpy(as_f32(W[n]).astype(np.float64))
    sd = {"embed_tokens.weight": t("embed"), "norm.weight": t("draft.final_norm")}
    for l in range(wl.draft_layers):
        for a, b in [("self_attn.q_proj", "q_proj"), ("self_attn.k_proj", "k_proj"),
                     ("self_attn.v_proj", "v_proj"), ("self_attn.o_proj", "o_proj"),
                     ("self_attn.q_norm", "q_norm"), ("self_attn.k_norm", "k_norm"),
                     ("input_layernorm", "input_norm"), ("post_attention_layernorm", "post_norm"),
                     ("mlp.gate_proj", "gate_proj"), ("mlp.up_proj", "up_proj"),
                     ("mlp.down_proj", "down_proj")]:
            sd[f"layers.{l}.{a}.weight"] = t(f"draft.{l}.{b}")
    hf.load_state_dict(sd, strict=True)
    n = wl.block_size
    with torch.no_grad():
        ref = hf(inputs_embeds=torch.from_numpy(e_t)[None],
                 attention_mask=torch.zeros(1, 1, n, n, dtype=torch.float64)).last_hidden_state[0]
    np.testing.assert_allclose(h, ref.numpy(), atol=2e-6, rtol=0)
