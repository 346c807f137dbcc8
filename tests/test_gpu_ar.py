"""GPU target-only greedy decoding (the baseline that speculative decoding is measured
against) through the C ABI: per-step logits and decisions against the oracle with
teacher forcing, graph replay against eager launches, the lossless equality of the
speculative and target-only streams, budgets, and call-order errors."""
import numpy as np
import pytest

from oracle import OracleModel, OracleRunner
from paper_2608_29748_amd import binding as B
from workloads import get, make_prompts, make_weights

from gpu_parity import Report, check_decisions, engine_for, log, top2_gap

pytestmark = pytest.mark.gpu

TOL = {"f32": 1e-4, "bf16": 2e-2}


def _setup(name, **over):
    wl = get(name, norm_init="perturbed", **over)
    return wl, make_weights(wl), make_prompts(wl)


@pytest.mark.parametrize("name", ["tiny-f32", "mini-bf16-ragged", "mini-bf16-gqa5"])
def test_ar_steps_match_oracle_teacher_forced(name):
    wl, W, prompts = _setup(name)
    V, tol = wl.target.vocab, TOL[wl.dtype]
    eng = engine_for(wl, W)
    m = OracleModel(wl, W)
    first = eng.prefill(prompts, wl.new_tokens)
    eng.set_debug(3)   # keep logits, launch eagerly
    rep = Report()
    states, tok, pos = [], [], []
    for i, p in enumerate(prompts):
        st = m.new_state(p, wl.new_tokens)
        ol = m.target_forward(st, p, 0).logits[-1]
        check_decisions(rep, ol[None], [first[i]], tol, f"seq {i} first token")
        states.append(st)
        tok.append(int(first[i]))
        pos.append(len(p))
    n_steps = min(12, wl.new_tokens - 1)
    for step in range(n_steps):
        g_tok, n = eng.ar_steps(1)
        assert list(n) == [1] * len(prompts)
        for i, st in enumerate(states):
            gl = eng.read(B.RT_T_AR_LOGITS, i, (V,), np.float32)
            ol = m.target_forward(st, [tok[i]], pos[i]).logits[-1]
            e = rep.err("ar_logits", gl, ol)
            assert e <= tol, f"seq {i} step {step}: logit error {e}"
            check_decisions(rep, ol[None], [g_tok[i, 0]], tol, f"seq {i} step {step}")
            tok[i] = int(g_tok[i, 0])
            pos[i] += 1
    log(f"[{name}] target-only steps {n_steps} max err {rep.max_err} near-ties {rep.near_ties}/{rep.decisions}")
    eng.close()


def _ar_stream(eng, prompts, budget, chunks):
    first = eng.prefill(prompts, budget)
    out = [[int(f)] for f in first]
    for c in chunks:
        t, n = eng.ar_steps(c)
        for i in range(len(prompts)):
            assert np.all(t[i, :n[i]] >= 0) and np.all(t[i, n[i]:] == -1)
            out[i].extend(int(x) for x in t[i, :n[i]])
    return out


def _spec_stream(eng, prompts, budget):
    first = eng.prefill(prompts, budget)
    out = [[int(f)] for f in first]
    while True:
        t, n, _ = eng.spec_round()
        if not n.any():
            return out
        for i in range(len(prompts)):
            out[i].extend(int(x) for x in t[i, :n[i]])


@pytest.mark.parametrize("name", ["tiny-f32", "mini-bf16"])
def test_ar_stream_graph_eager_and_speculative_agree(name):
    """Target-only steps replayed from a graph equal eager launches bit for bit; the
    budget ends every stream; and the speculative stream equals the target-only one
    (lossless greedy verification) up to a near-tie of the target's own logits."""
    wl, W, prompts = _setup(name)
    budget = wl.new_tokens
    eng = engine_for(wl, W)
    g = _ar_stream(eng, prompts, budget, [5, 17, budget])          # the last call runs past the budget
    assert all(len(s) == budget for s in g)
    t, n = eng.ar_steps(3)
    assert not n.any() and np.all(t == -1)
    with pytest.raises(B.RetraceError) as ex:
        eng.spec_round()
    assert ex.value.code == B.RT_ERR_STATE
    eng.set_debug(2)
    e = _ar_stream(eng, prompts, budget, [budget - 1])
    assert e == g
    eng.set_debug(0)
    sp = _spec_stream(eng, prompts, budget)
    eng.close()
    m = OracleModel(wl, W)
    for i, p in enumerate(prompts):
        if sp[i] == g[i]:
            continue
        k = next(j for j in range(budget) if sp[i][j] != g[i][j])
        # the streams may part only where the target's top-2 logits nearly tie
        seq = np.concatenate([p, g[i][:k]]).astype(np.int64)
        ol = OracleRunner(m).logits_nocache(seq)[-1]
        gap = float(top2_gap(ol))
        log(f"[{name}] seq {i}: streams part at token {k}, oracle top-2 gap {gap:.3g}")
        assert wl.dtype == "bf16" and gap <= 2 * TOL[wl.dtype], f"seq {i} token {k}: gap {gap}"
    log(f"[{name}] target-only == speculative for {sum(a == b for a, b in zip(sp, g))}/{len(prompts)} sequences")


def test_ar_call_errors():
    wl, W, prompts = _setup("tiny-f32")
    eng = engine_for(wl, W)
    with pytest.raises(B.RetraceError) as ex:
        eng.ar_steps(1)
    assert ex.value.code == B.RT_ERR_STATE
    eng.prefill(prompts, 8)
    for bad in (0, B.RT_AR_MAX_STEPS + 1):
        with pytest.raises(B.RetraceError) as ex:
            eng.ar_steps(bad)
        assert ex.value.code == B.RT_ERR_INVALID
    eng.ar_steps(B.RT_AR_MAX_STEPS)     # runs past the budget: every later entry is -1
    eng.prefill(prompts, 8)             # a new prefill allows rounds again
    eng.spec_round()
    eng.close()
