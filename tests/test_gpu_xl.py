"""GPU parity at the batched, long-context shapes: the Qwen3-8B shape with 8 ragged
sequences (prompts of 1024..8192 tokens) and the Qwen3-14B shape with 16 (8192..16384).

The whole batch runs on the GPU in the launch configuration the benchmark times; the
oracle checks sampled outputs one sequence at a time.  First the GPU prefill of a
sampled sequence on a causal prefix of its prompt (KV rows of the first tokens depend on
nothing later).  Then four rounds of two sampled sequences, started from the GPU's KV
caches and carried state: two unforced rounds (the second conditions its drafts on the
first round's rejected suffix at batch shape), a round with planted drafts (one
sequence accepts a prefix and keeps a shorter rejected suffix, the other accepts the
whole block and resets), and at the 8B shape an unforced round after it.  Every round
is checked end to end (calibrated bound) and stage by stage at 2e-2: every drafter
layer and sampled target layers step by step from the GPU's own operands, both LM heads
from the GPU's own operands, every argmax decision with a top-2 gap above 2e-2.  The oracle keeps float32 copies of
the weights (exact for bf16)."""
import time

import numpy as np
import pytest

from oracle import OracleModel, OracleRunner, Precision
from paper_2608_29748_amd import binding as B
from workloads import get, make_prompts, make_weights

from gpu_parity import Report, compare_prefill, engine_for, log, planted_drafts, run_teacher_forced

pytestmark = pytest.mark.gpu
TOL = 2e-2


def sampled_layers(wl):
    """First two, conditioning, middle and last target layers."""
    L = wl.target.n_layers
    return sorted({0, 1, L // 2, L - 1, *wl.cond_layers})


@pytest.mark.timeout(1200)
@pytest.mark.parametrize("name,seqs,after", [("qwen3-8b-shape-b8", (0, 5), True),
                                              ("qwen3-14b-shape-b16", (11, 3), False)])
def test_batched_long_context_sampled(name, seqs, after):
    wl = get(name)
    t0 = time.time()
    W = make_weights(wl)
    prompts = make_prompts(wl)
    eng = engine_for(wl, W)
    eng.prefill(prompts, wl.new_tokens)
    lens = [len(p) for p in prompts]
    log(f"[{name}] gpu prefill of {len(prompts)} prompts ({min(lens)}..{max(lens)} tokens) {time.time() - t0:.1f}s")
    R = OracleRunner(OracleModel(wl, W, cache="f32"))
    RX = OracleRunner(OracleModel(wl, W, prec=Precision.for_dtype("f64"), cache="f32"))
    RX.m.W = R.m.W                                   # one weight cache for both
    s0, n, L = seqs[0], 24, wl.target.n_layers
    pre = R.prefill(prompts[s0][:n], wl.new_tokens)
    pre_x = RX.prefill(prompts[s0][:n], wl.new_tokens)
    rep = compare_prefill(eng, R, wl, [prompts[s0][:n]], [pre], TOL, layers=[0, 1, L // 2, L - 1],
                          exact_states=[pre_x], gpu_seqs=[s0])
    log(f"[{name}] seq {s0} prefix KV max err {rep.max_err} ({time.time() - t0:.1f}s)")
    states = [None] * wl.batch
    for b in seqs:
        st = R.m.new_state(prompts[b], wl.new_tokens)
        stv = eng.read(B.RT_T_STATE, b, (9,), np.int32)
        assert int(stv[0]) == lens[b]
        st.P, st.anchor, st.generated = int(stv[0]), int(stv[1]), [int(stv[1])]
        st.hD_prev = np.zeros((wl.block_size, wl.target.hidden))
        st.hT_prev = np.zeros((wl.block_size, wl.target.hidden))
        states[b] = st
    stages = {"target_layers": sampled_layers(wl)}
    rep = Report()
    # rounds 1 and 2: unforced; with A < B - 1 in round 1, round 2 conditions B - A - 1 rows
    run_teacher_forced(eng, R, wl, states, 2, TOL, rep=rep, exact=RX, stages=stages)
    log(f"[{name}] rounds 1-2: A {rep.accept} ({time.time() - t0:.1f}s)")
    # round 3: planted drafts -- a mismatch at block position 4 for seqs[0] (A = 3, then
    # B - 4 conditioned rows), the target's whole greedy continuation for seqs[1] (A = B: reset)
    k = 4
    drafts = planted_drafts(eng, wl, wl.batch, {seqs[0]: k, seqs[1]: None})
    run_teacher_forced(eng, R, wl, states, 1, TOL, forced=[drafts], rep=rep, exact=RX, stages=stages)
    st0 = eng.read(B.RT_T_STATE, seqs[0], (9,), np.int32)
    st1 = eng.read(B.RT_T_STATE, seqs[1], (9,), np.int32)
    a3 = [int(st0[7]), int(st1[7])]
    assert a3 == [k - 1, wl.B], f"planted acceptance lengths {a3}"
    assert (int(st0[2]), int(st0[3])) == (k, wl.B - k) and int(st1[3]) == 0, (st0, st1)
    log(f"[{name}] round 3 (planted): A {a3} ({time.time() - t0:.1f}s)")
    # round 4 (8B shape; the 14B shape stops after the planted round to bound the test's
    # time): seqs[0] conditioned on its shorter rejected suffix, seqs[1] on nothing
    if after:
        run_teacher_forced(eng, R, wl, states, 1, TOL, rep=rep, exact=RX, stages=stages)
    assert rep.conditioned >= 3, f"conditioned sequence rounds: {rep.conditioned}"
    assert rep.max_err["e_tilde"] > 0.0, "no conditioned row was compared"
    log(f"[{name}] seqs {seqs} 4 rounds: A {rep.accept}, conditioned {rep.conditioned}, max err {rep.max_err} "
        f"near-ties {rep.near_ties}/{rep.decisions}, per stage {rep.stage_near_ties}/{rep.stage_decisions} ({time.time() - t0:.1f}s)")
    eng.close()
