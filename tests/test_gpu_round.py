"""GPU parity of the ReTrace round against the oracle, through the C ABI."""
import numpy as np
import pytest

from oracle import OracleModel, OracleRunner, Precision
from workloads import get, make_prompts, make_weights

from gpu_parity import compare_prefill, engine_for, log, run_teacher_forced

pytestmark = pytest.mark.gpu

TOL = {"f32": 1e-4, "bf16": 2e-2}


def _setup(name, **over):
    wl = get(name, **over)
    W = make_weights(wl)
    prompts = make_prompts(wl)
    return wl, W, prompts


def _exact(wl, W, R):
    """A float64 runner sharing R's weights, for bf16 models of width >= 512: their
    end-to-end bf16 rounding noise reaches the fixed tolerance, so the end-to-end bounds
    are calibrated by the mixed-precision oracle's own distance from float64 arithmetic
    (as at the measured shapes); the per-stage checks keep the fixed tolerance."""
    if wl.dtype != "bf16" or wl.target.hidden < 512:
        return None
    RX = OracleRunner(OracleModel(wl, W, prec=Precision.for_dtype("f64")))
    RX.m.W = R.m.W
    return RX


@pytest.mark.parametrize("name", ["tiny-f32", "mini-bf16", "mini-bf16-ragged", "mini-bf16-gqa5", "mini-bf16-b4",
                                  "mini-bf16-w4096", "mini-bf16-b6", "mini-bf16-odd"])
def test_prefill_and_rounds_match_oracle(name):
    """Prefill KV, then six rounds, each checked end to end and stage by stage (every
    layer from the GPU's own input, both LM heads from the GPU's own operands)."""
    wl, W, prompts = _setup(name, norm_init="perturbed")
    log(f"[{name}] engine init")
    eng = engine_for(wl, W)
    R = OracleRunner(OracleModel(wl, W))
    log(f"[{name}] prefill")
    first = eng.prefill(prompts, wl.new_tokens)
    states = [R.prefill(p, wl.new_tokens) for p in prompts]
    assert list(first) == [st.anchor for st in states]
    tol = TOL[wl.dtype]
    rep = compare_prefill(eng, R, wl, prompts, states, tol)
    log(f"[{name}] prefill max err {rep.max_err}")
    rep = run_teacher_forced(eng, R, wl, states, 6, tol, exact=_exact(wl, W, R), stages={})
    log(f"[{name}] rounds {rep.rounds} max err {rep.max_err} p99.9 {rep.p999} "
        f"near-ties {rep.near_ties}/{rep.decisions}, per stage {rep.stage_near_ties}/{rep.stage_decisions}")
    assert rep.conditioned > 0, "no round carried a rejected suffix"
    eng.close()


@pytest.mark.parametrize("name,lens,batch", [("tiny-f32", (20, 600), 4), ("mini-bf16-ragged", (20, 900), 4),
                                             ("mini-bf16-b6", (20, 900), 7)])
def test_ragged_batch_key_splits_match_oracle(name, lens, batch):
    """A batch of very unequal contexts: the attention's key-split workgroups are shared
    out by context length (one split for the short sequences, several for the long
    ones, some workgroups idle), in the fp32 and the bf16 kernels; at seven sequences
    (112 rows, no fused q / k work) the slots split the concatenated chunks evenly and
    one slot may cover the end of a context and the start of the next ones."""
    wl, W, prompts = _setup(name, norm_init="perturbed", batch=batch, prompt_len=lens)
    log(f"[{name} ragged] prompts {[len(p) for p in prompts]}")
    eng = engine_for(wl, W)
    if batch > 4:   # the spanning plan wherever it is valid (debug flag 64)
        orig = eng.set_debug
        eng.set_debug = lambda f: orig(f | 64)
        eng.set_debug(0)
    R = OracleRunner(OracleModel(wl, W))
    first = eng.prefill(prompts, wl.new_tokens)
    states = [R.prefill(p, wl.new_tokens) for p in prompts]
    assert list(first) == [st.anchor for st in states]
    tol = TOL[wl.dtype]
    rep = compare_prefill(eng, R, wl, prompts, states, tol)
    log(f"[{name} ragged] prefill max err {rep.max_err}")
    rep = run_teacher_forced(eng, R, wl, states, 4, tol, exact=_exact(wl, W, R))
    log(f"[{name} ragged] rounds {rep.rounds} max err {rep.max_err} near-ties {rep.near_ties}/{rep.decisions}, per stage {rep.stage_near_ties}/{rep.stage_decisions}")
    eng.close()


@pytest.mark.parametrize("name,mode", [("tiny-f32", "raw_gated"), ("tiny-f32", "overwrite"),
                                       ("mini-bf16", "raw_gated"), ("mini-bf16", "overwrite"),
                                       ("mini-bf16-ragged", "off"), ("mini-bf16-b4", "raw_gated"),
                                       ("tiny-f32", "lowrank"), ("mini-bf16", "lowrank"),
                                       ("mini-bf16-ragged", "lowrank"), ("mini-bf16-b4", "lowrank")])
def test_ablation_conditioning_matches_oracle(name, mode):
    """The component-ablation drafters of Table 3 (raw gated fusion, overwrite), the
    low-rank deployment form of the conditioning path, and plain block drafting, round
    by round against the oracle run in the same mode."""
    wl, W, prompts = _setup(name, norm_init="perturbed", cond_mode=mode)
    log(f"[{name} {mode}] prefill")
    eng = engine_for(wl, W)
    R = OracleRunner(OracleModel(wl, W))
    first = eng.prefill(prompts, wl.new_tokens)
    states = [R.prefill(p, wl.new_tokens) for p in prompts]
    assert list(first) == [st.anchor for st in states]
    rep = run_teacher_forced(eng, R, wl, states, 6, TOL[wl.dtype], exact=_exact(wl, W, R))
    log(f"[{name} {mode}] rounds {rep.rounds} max err {rep.max_err} near-ties {rep.near_ties}/{rep.decisions}, per stage {rep.stage_near_ties}/{rep.stage_decisions}")
    eng.close()


def test_forced_split_k_matches_oracle():
    """Prefill GEMMs (128-row tiles) with every reduction split four ways across
    workgroups (last-arriver fixup)."""
    wl, W, prompts = _setup("mini-bf16", prompt_len=(300, 300), new_tokens=12, norm_init="perturbed")
    eng = engine_for(wl, W)
    R = OracleRunner(OracleModel(wl, W))
    eng.set_debug(4)
    first = eng.prefill(prompts, wl.new_tokens)
    states = [R.prefill(p, wl.new_tokens) for p in prompts]
    assert list(first) == [st.anchor for st in states]
    rep = compare_prefill(eng, R, wl, prompts, states, TOL[wl.dtype])
    # keep the split on for the rounds (debug flags 1|2 added by the parity loop)
    orig = eng.set_debug
    eng.set_debug = lambda f: orig(f | 4)
    rep = run_teacher_forced(eng, R, wl, states, 4, TOL[wl.dtype])
    log(f"[split-k] rounds max err {rep.max_err}")
    eng.close()


def test_long_prompt_chunked_prefill():
    """Prompt longer than one prefill pass: the wide (128-row tile) GEMM path, chunked
    prefill attention over earlier chunks, then rounds."""
    wl, W, prompts = _setup("mini-bf16", prompt_len=(700, 700), new_tokens=12, norm_init="perturbed")
    eng = engine_for(wl, W)
    R = OracleRunner(OracleModel(wl, W))
    log("[long prompt] prefill")
    first = eng.prefill(prompts, wl.new_tokens)
    states = [R.prefill(p, wl.new_tokens) for p in prompts]
    assert list(first) == [st.anchor for st in states]
    rep = compare_prefill(eng, R, wl, prompts, states, TOL[wl.dtype])
    log(f"[long prompt] prefill max err {rep.max_err}")
    rep = run_teacher_forced(eng, R, wl, states, 3, TOL[wl.dtype])
    log(f"[long prompt] rounds max err {rep.max_err}")
    eng.close()


def test_two_sequence_slab_kernel_matches_oracle():
    """Two sequences (32 round rows) of the 4096-wide mini model: the o and down k-slab
    partials run on the slab kernel with two 16-row groups of each slab's activations
    staged in LDS (one sequence runs one group); per stage and end to end."""
    wl, W, prompts = _setup("mini-bf16-w4096", norm_init="perturbed", batch=2, prompt_len=(40, 70))
    eng = engine_for(wl, W)
    R = OracleRunner(OracleModel(wl, W))
    first = eng.prefill(prompts, wl.new_tokens)
    states = [R.prefill(p, wl.new_tokens) for p in prompts]
    assert list(first) == [st.anchor for st in states]
    rep = run_teacher_forced(eng, R, wl, states, 4, TOL[wl.dtype], exact=_exact(wl, W, R), stages={})
    log(f"[w4096 batch 2] rounds {rep.rounds} max err {rep.max_err}")
    assert rep.conditioned > 0
    eng.close()
