"""State handed to the GPU from outside, through the C ABI: a round started from the
oracle's own prefill (KV rows of every layer and the round state written with
rt_debug_write into a model prefilled with other prompts) must match the oracle's round;
and a model built from host weight pointers must run rounds bit for bit like one built
from device pointers."""
import numpy as np
import pytest
import torch

from oracle import OracleModel, OracleRunner
from paper_2608_29748_amd import binding as B
from paper_2608_29748_amd.engine import RoundEngine
from workloads import get, make_prompts, make_weights, weight_specs

from gpu_parity import engine_for, keep_dtype, log, run_teacher_forced, store_to_f64

pytestmark = pytest.mark.gpu
TOL = {"f32": 1e-4, "bf16": 2e-2}


def to_store(x, wl):
    x32 = np.ascontiguousarray(np.asarray(x, np.float64).astype(np.float32))
    if wl.dtype == "bf16":
        bits = x32.view(np.uint32)
        assert not np.any(bits & 0xFFFF), "values are not bf16"
        return (bits >> 16).astype(np.uint16)
    return x32


@pytest.mark.parametrize("name", ["tiny-f32", "mini-bf16-ragged"])
def test_round_from_the_oracles_injected_state(name):
    wl = get(name, norm_init="perturbed")
    W = make_weights(wl)
    prompts = make_prompts(wl)
    R = OracleRunner(OracleModel(wl, W))
    states = [R.prefill(p, wl.new_tokens) for p in prompts]
    eng = engine_for(wl, W)
    other = [(p + 1 + i) % (wl.target.vocab - 1) for i, p in enumerate(prompts)]   # same lengths, other tokens
    eng.prefill(other, wl.new_tokens)
    s, et = wl.target, (np.uint16 if wl.dtype == "bf16" else np.float32)
    for b, st in enumerate(states):
        n = st.P
        for l in range(s.n_layers):
            for tid, src in ((B.RT_T_TARGET_K + l, st.tgt_k[l, :n]), (B.RT_T_TARGET_V + l, st.tgt_v[l, :n])):
                eng.write(tid, b, to_store(src, wl))
                back = eng.read(tid, b, (n, s.n_kv_heads, s.head_dim), et)
                assert np.array_equal(store_to_f64(back, wl), src), (b, l, tid)
        for l in range(wl.draft_layers):
            for tid, src in ((B.RT_T_DRAFT_K + l, st.ctx_k[l, :n]), (B.RT_T_DRAFT_V + l, st.ctx_v[l, :n])):
                eng.write(tid, b, to_store(src, wl))
        stv = eng.read(B.RT_T_STATE, b, (9,), np.int32)
        stv[0], stv[1], stv[5] = st.P, st.anchor, st.P
        eng.write(B.RT_T_STATE, b, stv)
    # the oracle keeps its own caches (inject_kv off): the GPU now holds the same values
    rep = run_teacher_forced(eng, R, wl, states, 4, TOL[wl.dtype])
    log(f"[{name} injected] rounds {rep.rounds} max err {rep.max_err} near-ties {rep.near_ties}/{rep.decisions}")
    assert rep.conditioned > 0
    eng.close()


def test_host_weight_pointers_build_the_same_model():
    wl = get("mini-bf16", norm_init="perturbed")
    W = make_weights(wl)
    prompts = make_prompts(wl)
    ref = engine_for(wl, W)
    cfg = ref.cfg
    host = [np.ascontiguousarray(W[n]) for n, _, _ in weight_specs(wl)]
    eng = RoundEngine.__new__(RoundEngine)
    eng.cfg, eng.device = cfg, torch.device("cuda", 0)
    eng.stream = torch.cuda.Stream(device=eng.device)
    nbytes = B.rt_workspace_bytes(cfg)
    eng.ws = torch.empty(nbytes + 256, dtype=torch.uint8, device=eng.device)
    base = eng.ws.data_ptr()
    eng.ws_ptr, eng.ws_bytes = base + (-base) % 256, nbytes
    torch.cuda.synchronize()
    eng.h = B.rt_init_models(cfg, [a.ctypes.data for a in host], eng.ws_ptr, eng.ws_bytes, eng.stream.cuda_stream)
    eng.n_seqs = 0
    assert list(ref.prefill(prompts, wl.new_tokens)) == list(eng.prefill(prompts, wl.new_tokens))
    kd, bk, d = keep_dtype(wl), wl.block_size, wl.target.hidden
    for t in range(3):
        a, b = ref.spec_round(), eng.spec_round()
        for x, y in zip(a, b):
            assert np.array_equal(x, y), (t, a, b)
        for tid in (B.RT_T_HD, B.RT_T_HT):
            assert np.array_equal(ref.read(tid, 0, (bk, d), kd).view(np.uint16), eng.read(tid, 0, (bk, d), kd).view(np.uint16))
    log("[host weights] 3 rounds equal bit for bit")
    ref.close()
    eng.close()
