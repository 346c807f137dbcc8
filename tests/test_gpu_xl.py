"""GPU parity at the batched, long-context shapes: the Qwen3-8B shape with 8 ragged
sequences (prompts of 1024..8192 tokens) and the Qwen3-14B shape with 16 (8192..16384).

The whole batch runs on the GPU in the launch configuration the benchmark times; the
oracle checks sampled outputs one sequence at a time.  First the GPU prefill of a
sampled sequence on a causal prefix of its prompt (KV rows of the first tokens depend on
nothing later), then a round of the sampled sequences started from the GPU's KV caches
and carried state.  The oracle keeps float32 copies of the weights (exact for bf16)."""
import time

import numpy as np
import pytest

from oracle import OracleModel, OracleRunner, Precision
from workloads import get, make_prompts, make_weights

from gpu_parity import compare_prefill, engine_for, log, run_teacher_forced

pytestmark = pytest.mark.gpu
TOL = 2e-2


@pytest.mark.timeout(1200)
@pytest.mark.parametrize("name,seqs", [("qwen3-8b-shape-b8", (0, 5)), ("qwen3-14b-shape-b16", (11,))])
def test_batched_long_context_sampled(name, seqs):
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
        stv = eng.read(7, b, (8,), np.int32)
        assert int(stv[0]) == lens[b]
        st.P, st.anchor, st.generated = int(stv[0]), int(stv[1]), [int(stv[1])]
        st.hD_prev = np.zeros((wl.block_size, wl.target.hidden))
        st.hT_prev = np.zeros((wl.block_size, wl.target.hidden))
        states[b] = st
    rep = run_teacher_forced(eng, R, wl, states, 1, TOL, inject_kv=True, exact=RX)
    log(f"[{name}] seqs {seqs} round max err {rep.max_err} near-ties {rep.near_ties}/{rep.decisions} "
        f"({time.time() - t0:.1f}s)")
    eng.close()
