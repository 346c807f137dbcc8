"""GPU temperature sampling (temperature 1, top-k 20, top-p 0.95) through the C ABI.

Per round and sequence, with the oracle started from the GPU's carried state: both
LM heads' logits against the oracle's (tolerance); the GPU's filtered distributions
against the oracle's definition applied to the GPU's own logits; every draw (draft
tokens, acceptance tests, correction / bonus token) against the oracle's rule fed the
same counter-based uniforms and the GPU's distributions; then the committed tokens
and the round state.  Draws within 1e-5 of a decision boundary adopt the GPU's
outcome (fp32 against float64 sums).  Distribution tests: from identical states
across a batch, the first committed token of a round and the token of a target-only
step follow the target's filtered distribution (chi-square)."""
import numpy as np
import pytest

import oracle.sampling as smp
from oracle import OracleModel, OracleRunner
from paper_2608_29748_amd import binding as B
from workloads import get, make_prompts, make_weights

from gpu_parity import Report, carried_state, engine_for, inject_state, keep_dtype, log

pytestmark = pytest.mark.gpu

TOL = {"f32": 1e-4, "bf16": 2e-2}
EDGE = 1e-5          # draws this close to a boundary adopt the GPU's decision


def gpu_dist(ids, probs):
    keep = ids >= 0
    return smp.Dist(ids=ids[keep].astype(np.int64), probs=probs[keep].astype(np.float64))


def check_dist(g: smp.Dist, logits_row, wl, what):
    """The GPU's filtered distribution equals the definition applied to its own logits,
    up to fp32 sums: same ids in the same order and probabilities within 1e-5, unless the
    top-p cut or an order falls within EDGE (then the shorter of the two prefixes agrees)."""
    o = smp.filtered(logits_row, wl.temperature, wl.top_k, wl.top_p)
    n = min(len(o.ids), len(g.ids))
    if len(o.ids) != len(g.ids):
        # a cut at the top-p boundary: the cumulative probability there is within EDGE
        z = np.asarray(logits_row, np.float64)
        order = np.lexsort((np.arange(z.size), -z))[: wl.top_k]
        s = z[order] / wl.temperature
        pk = np.exp(s - s[0]) / np.exp(s - s[0]).sum()
        assert abs(np.cumsum(pk)[n - 1] - wl.top_p) < EDGE, f"{what}: kept {len(g.ids)} vs {len(o.ids)}"
    if list(g.ids[:n]) != list(o.ids[:n]):   # only an order among near-equal logits may differ
        gaps = np.abs(np.diff(np.sort(np.asarray(logits_row, np.float64)[o.ids])))
        assert gaps.size and gaps.min() < EDGE, f"{what}: ids {g.ids[:n]} vs {o.ids[:n]}"
    if len(o.ids) == len(g.ids):
        np.testing.assert_allclose(g.probs, o.probs, atol=1e-5, err_msg=what)


def near_cdf_edge(d: smp.Dist, u: float) -> bool:
    return bool(np.min(np.abs(np.cumsum(d.probs) - u)) < EDGE)


def run_sampled_rounds(eng, R, wl, states, n_rounds, forced=None):
    """forced: optional per-round [n_seqs][B] drafts (the drafter still runs; its
    distributions still enter the acceptance rule)."""
    s, bk, B_ = wl.target, wl.block_size, wl.B
    rep = Report()
    eng.set_debug(3)
    tol = TOL[wl.dtype]
    seed = wl.sample_seed
    adopted = 0
    for t in range(n_rounds):
        carried = [carried_state(eng, b, wl) for b in range(len(states))]
        if forced is not None:
            tok, n_c, acc = eng.spec_round_forced(np.asarray(forced[t], np.int32))
        else:
            tok, n_c, acc = eng.spec_round()
        for b, st in enumerate(states):
            if st.done:
                assert n_c[b] == 0
                continue
            inject_state(eng, st, b, wl, carried[b])
            rnd = st.rnd + 1
            d = R.draft(st)
            g_dl = eng.read(B.RT_T_DRAFT_LOGITS, b, (bk, s.vocab), np.float32).astype(np.float64)
            assert rep.err("draft_logits", g_dl[1:], d.logits[1:]) <= tol
            ids = eng.read(B.RT_T_DRAFT_DIST_IDS, b, (bk, B.RT_MAX_TOP_K), np.int32)
            prb = eng.read(B.RT_T_DRAFT_DIST_P, b, (bk, B.RT_MAX_TOP_K), np.float32)
            q = [gpu_dist(ids[i], prb[i]) for i in range(1, bk)]
            dtok = eng.read(B.RT_T_DRAFT_TOKENS, b, (bk,), np.int32)
            for i in range(1, bk):
                check_dist(q[i - 1], g_dl[i], wl, f"round {t} seq {b} draft row {i}")
                u = smp.uniform(seed, rnd, b, smp.U_DRAFT, i)
                rep.decisions += 1
                if forced is not None:
                    assert dtok[i] == forced[t][b][i - 1]
                elif near_cdf_edge(q[i - 1], u):
                    adopted += 1
                else:
                    assert smp.sample(q[i - 1], u) == dtok[i], f"round {t} seq {b}: draft {i}"
            y_hat = dtok[1:].astype(np.int64)
            v = R.verify(st, y_hat)
            g_vl = eng.read(B.RT_T_VERIFY_LOGITS, b, (bk, s.vocab), np.float32).astype(np.float64)
            assert rep.err("verify_logits", g_vl, v.logits) <= tol
            ids = eng.read(B.RT_T_VERIFY_DIST_IDS, b, (bk, B.RT_MAX_TOP_K), np.int32)
            prb = eng.read(B.RT_T_VERIFY_DIST_P, b, (bk, B.RT_MAX_TOP_K), np.float32)
            p = [gpu_dist(ids[i], prb[i]) for i in range(bk)]
            for i in range(bk):
                check_dist(p[i], g_vl[i], wl, f"round {t} seq {b} verify row {i}")
            u_acc = [smp.uniform(seed, rnd, b, smp.U_ACCEPT, i) for i in range(1, bk)]
            u_res = smp.uniform(seed, rnd, b, smp.U_RESAMPLE, 0)
            A, corr = smp.speculative_accept(y_hat, q, p, u_acc, u_res)
            g_A = int(acc[b])
            gst = eng.read(B.RT_T_STATE, b, (9,), np.int32)
            g_corr = int(gst[1])              # the new anchor is the correction / bonus token
            # decisions near a boundary: the acceptance ratio or the correction's draw
            edge = False
            for i in range(min(A, g_A) + 1):
                if i < B_:
                    pq, qq = p[i].prob(int(y_hat[i])), q[i].prob(int(y_hat[i]))
                    edge |= abs(u_acc[i] * qq - pq) < EDGE
            row = min(A, g_A)
            res = smp.residual(p[row], q[row]) if row < B_ else p[B_]
            edge |= near_cdf_edge(res, u_res)
            rep.decisions += 1
            if edge:
                adopted += 1
            else:
                assert A == g_A, f"round {t} seq {b}: A oracle {A} gpu {g_A}"
                assert corr == g_corr, f"round {t} seq {b}: correction {corr} vs {g_corr}"
            # continue from the GPU's decisions
            _, new = R.commit_tokens(st, y_hat, g_A, g_corr, d, v)
            assert list(tok[b][: n_c[b]]) == new
            assert gst[0] == st.P and gst[1] == st.anchor and gst[8] == st.rnd
            assert gst[3] == st.cond_len and (st.cond_len == 0 or gst[2] == st.r)
            rep.accept.append(g_A)
        rep.rounds += 1
    log(f"[{wl.name} sampled] rounds {rep.rounds} max err {rep.max_err} boundary draws adopted {adopted}/{rep.decisions} "
        f"A {rep.accept}")
    return rep


@pytest.mark.parametrize("name", ["tiny-f32", "mini-bf16", "mini-bf16-ragged"])
def test_sampled_rounds_match_oracle(name):
    wl = get(name, norm_init="perturbed", temperature=1.0, top_k=20, top_p=0.95)
    W = make_weights(wl)
    prompts = make_prompts(wl)
    eng = engine_for(wl, W)
    R = OracleRunner(OracleModel(wl, W))
    first = eng.prefill(prompts, wl.new_tokens)
    states = []
    for b, pr in enumerate(prompts):
        st = R.prefill(pr, wl.new_tokens, seq=b)
        if st.anchor != first[b]:     # the first draw may sit on a boundary: adopt the GPU's token
            st.anchor = int(first[b])
            st.generated = [int(first[b])]
        states.append(st)
    run_sampled_rounds(eng, R, wl, states, 6)
    eng.close()


def test_sampled_rounds_with_target_drafts():
    """Drafts taken from the target's own greedy continuation: most are kept (the drafter's
    q gives them little or no mass), so full blocks and the bonus draw are exercised."""
    wl = get("tiny-f32", norm_init="perturbed", temperature=1.0, top_k=20, top_p=0.95)
    W = make_weights(wl)
    prompt = make_prompts(wl)[0]
    eng = engine_for(wl, W)
    R = OracleRunner(OracleModel(wl, W))
    first = eng.prefill([prompt], wl.new_tokens)
    st = R.prefill(prompt, wl.new_tokens, seq=0)
    st.anchor, st.generated = int(first[0]), [int(first[0])]
    greedy = OracleRunner(OracleModel(get("tiny-f32", norm_init="perturbed"), W))
    accepted = []
    for t in range(4):
        ctx = np.concatenate([prompt, np.asarray(st.generated, np.int64)])
        truth = greedy.ar_decode(ctx, wl.B + 1)[: wl.B]
        accepted += run_sampled_rounds(eng, R, wl, [st], 1, forced=[[truth]]).accept
    log(f"[target drafts] accepted {accepted}")
    assert max(accepted) > 0
    eng.close()


def test_sampled_target_only_stream_matches_oracle():
    wl = get("tiny-f32", norm_init="perturbed", temperature=1.0, top_k=20, top_p=0.95)
    W = make_weights(wl)
    prompt = make_prompts(wl)[0]
    eng = engine_for(wl, W)
    first = eng.prefill([prompt], 30)
    t, n = eng.ar_steps(29)
    gpu = [int(first[0])] + [int(x) for x in t[0, : n[0]]]
    ref = OracleRunner(OracleModel(wl, W)).ar_decode(prompt, 30, seq=0)
    log(f"[sampled target-only] gpu {gpu[:12]} oracle {ref[:12]}")
    assert gpu == ref
    eng.close()


def _chi2_ok(counts: dict, d: smp.Dist, n: int):
    from scipy.stats import chi2 as chi2d
    assert set(counts) <= set(int(t) for t in d.ids), f"{set(counts) - set(int(t) for t in d.ids)}"
    obs = np.array([counts.get(int(t), 0) for t in d.ids], float)
    exp = d.probs * n
    big = exp >= 5
    o = np.append(obs[big], obs[~big].sum())
    e = np.append(exp[big], exp[~big].sum())
    if e[-1] == 0:
        o, e = o[:-1], e[:-1]
    stat = float(np.sum((o - e) ** 2 / e))
    assert stat < chi2d.ppf(0.999, max(len(e) - 1, 1)), f"chi2 {stat} over {len(e)} cells"
    return stat


def test_sampling_distributions_from_identical_states():
    """A batch of identical prompts; every sequence's state is set to the same anchor, so
    the first token committed by one round (whatever the drafts), and separately the
    token of one target-only step, must follow the target's filtered distribution."""
    n = 256
    wl = get("tiny-f32", norm_init="perturbed", temperature=1.0, top_k=20, top_p=0.95, batch=n)
    W = make_weights(wl)
    prompt = make_prompts(wl)[0]
    R = OracleRunner(OracleModel(wl, W))
    st0 = R.prefill(prompt, 40)
    p1 = R.dist(R.verify(st0, [0] * wl.B).logits[0])     # the anchor row sees only the context
    for what in ("round", "step"):
        eng = engine_for(wl, W, max_batch=n)
        eng.prefill([prompt] * n, 40)
        state = eng.read(B.RT_T_STATE, 0, (9,), np.int32)
        state[1] = st0.anchor
        state[2:4] = 0
        for b in range(n):
            eng.write(B.RT_T_STATE, b, state)
        counts = {}
        if what == "round":
            tok, n_c, acc = eng.spec_round()
            firsts = tok[:, 0]
            log(f"[distribution] round: rejected at the first draft in {int(np.sum(acc == 0))}/{n}")
        else:
            t, _ = eng.ar_steps(1)
            firsts = t[:, 0]
        for x in firsts:
            counts[int(x)] = counts.get(int(x), 0) + 1
        stat = _chi2_ok(counts, p1, n)
        log(f"[distribution] {what}: chi2 {stat:.1f} over {len(p1.ids)} tokens")
        eng.close()


def test_sampled_graph_replay_equals_eager():
    wl = get("mini-bf16", norm_init="perturbed", temperature=1.0)
    W = make_weights(wl)
    prompts = make_prompts(wl)
    outs = []
    for flags in (0, 2):
        eng = engine_for(wl, W)
        eng.set_debug(flags)
        eng.prefill(prompts, wl.new_tokens)
        outs.append([tuple(map(np.copy, eng.spec_round())) for _ in range(5)])
        eng.close()
    for (t0, n0, a0), (t1, n1, a1) in zip(*outs):
        np.testing.assert_array_equal(t0, t1)
        np.testing.assert_array_equal(n0, n1)
