"""Round semantics on the GPU through the C ABI: planted drafts with known
acceptance lengths, the carry / reset rule, losslessness against the oracle's
target-only greedy decode, budget clipping, graph replay, the W_v = 0 and
conditioning-off reductions, error statuses, and measurement calls that leave the
rounds unchanged."""
import numpy as np
import pytest

from oracle import OracleModel, OracleRunner
from paper_2608_29748_amd import binding as B
from workloads import get, make_prompts, make_weights

from gpu_parity import engine_for, log

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def tiny():
    wl = get("tiny-f32", norm_init="perturbed")
    W = make_weights(wl)
    prompt = make_prompts(wl)[0]
    truth = OracleRunner(OracleModel(wl, W)).ar_decode(prompt, wl.new_tokens + wl.block_size)
    return wl, W, prompt, truth


def test_planted_drafts_reset_rule_and_losslessness(tiny):
    wl, W, prompt, truth = tiny
    B_ = wl.B
    eng = engine_for(wl, W)
    first = eng.prefill([prompt], wl.new_tokens)
    gen = [int(first[0])]
    assert gen[0] == truth[0]
    for k in [1, 3, B_, None, 2, B_ - 1, 5]:
        draft = list(truth[len(gen):len(gen) + B_])
        if k is not None:
            draft[k - 1] = (draft[k - 1] + 1) % wl.target.vocab
        tok, n, a = eng.spec_round_forced(np.array([draft], np.int32))
        A = B_ if k is None else k - 1
        assert int(a[0]) == A, (k, a)
        assert int(n[0]) == A + 1
        gen += [int(x) for x in tok[0][: n[0]]]
        st = eng.read(B.RT_T_STATE, 0, (8,), np.int32)
        if A < B_ - 1:
            assert (st[2], st[3]) == (A + 1, B_ - A - 1), st
        else:
            assert st[3] == 0, st
        assert gen == truth[: len(gen)]
    while True:                                   # unforced to the end of the budget
        tok, n, a = eng.spec_round()
        if n[0] == 0:
            break
        gen += [int(x) for x in tok[0][: n[0]]]
    assert len(gen) == wl.new_tokens
    assert gen == truth[: wl.new_tokens], "GPU speculative output differs from target greedy decoding"
    eng.close()


def test_budget_clips_last_round(tiny):
    wl, W, prompt, truth = tiny
    eng = engine_for(wl, W)
    eng.prefill([prompt], 5)
    tok, n, a = eng.spec_round_forced(np.array([truth[1:1 + wl.B]], np.int32))
    assert int(a[0]) == wl.B and int(n[0]) == 4
    assert [int(x) for x in tok[0][:4]] == truth[1:5]
    tok, n, a = eng.spec_round()
    assert int(n[0]) == 0
    eng.close()


def _run(eng, rounds, forced=None):
    out = []
    for t in range(rounds):
        tok, n, a = eng.spec_round() if forced is None else eng.spec_round_forced(forced[t])
        out.append((tok.copy(), n.copy(), a.copy(), eng.read(B.RT_T_HD, 0, (eng.cfg.block_size, eng.cfg.hidden),
                                                              np.uint16).copy()))
    return out


def test_graph_replay_equals_eager_and_is_deterministic():
    wl = get("mini-bf16-ragged", norm_init="perturbed")
    W = make_weights(wl)
    prompts = make_prompts(wl)
    runs = []
    for flags in (0, 2, 0):
        eng = engine_for(wl, W)
        eng.set_debug(flags)
        eng.prefill(prompts, wl.new_tokens)
        runs.append(_run(eng, 5))
        eng.close()
    for other in runs[1:]:
        for (t0, n0, a0, h0), (t1, n1, a1, h1) in zip(runs[0], other):
            np.testing.assert_array_equal(t0, t1)
            np.testing.assert_array_equal(n0, n1)
            np.testing.assert_array_equal(h0, h1)


def test_wv_zero_equals_conditioning_off():
    """With W_v = 0 the gated residual vanishes (Eq.9), so every round must equal plain
    block drafting bit for bit."""
    wl = get("mini-bf16", norm_init="perturbed")
    W0 = make_weights(wl, wv_zero=True)
    prompts = make_prompts(wl)
    res = []
    for mode in (B.RT_COND_RETRACE, B.RT_COND_OFF):
        eng = engine_for(wl, W0, cond_mode=mode)
        eng.prefill(prompts, wl.new_tokens)
        rounds = []
        for _ in range(5):
            tok, n, a = eng.spec_round()
            et = eng.read(B.RT_T_ETILDE, 0, (wl.block_size, wl.target.hidden), np.float32)
            rounds.append((tok.copy(), et.copy()))
        res.append(rounds)
        eng.close()
    for (t0, e0), (t1, e1) in zip(*res):
        np.testing.assert_array_equal(t0, t1)
        np.testing.assert_array_equal(e0, e1)


def test_error_statuses(tiny):
    wl, W, prompt, _ = tiny
    eng = engine_for(wl, W)
    with pytest.raises(B.RetraceError) as ex:
        eng.spec_round()
    assert ex.value.code == B.RT_ERR_STATE
    bad = prompt.copy()
    bad[3] = wl.target.vocab
    with pytest.raises(B.RetraceError) as ex:
        eng.prefill([bad], 8)
    assert ex.value.code == B.RT_ERR_TOKEN
    with pytest.raises(B.RetraceError) as ex:
        eng.prefill([prompt], wl.max_seq_len)
    assert ex.value.code == B.RT_ERR_CAPACITY
    with pytest.raises(B.RetraceError) as ex:
        eng.prefill([prompt, prompt], 8)
    assert ex.value.code == B.RT_ERR_CAPACITY
    eng.prefill([prompt], 8)
    with pytest.raises(B.RetraceError) as ex:
        eng.spec_round_forced(np.full((1, wl.B), -1, np.int32))
    assert ex.value.code == B.RT_ERR_TOKEN
    eng.close()


def test_measurement_calls_leave_the_rounds_unchanged():
    """A profiled round is an ordinary round (same outputs, every launch counted once),
    and kernel replays of the scratch-writing classes change no KV and no carried state:
    the rounds that follow match an engine that was never measured, bit for bit."""
    wl = get("mini-bf16-ragged", norm_init="perturbed")
    W = make_weights(wl)
    prompts = make_prompts(wl)
    L, LD = wl.target.n_layers, wl.draft_layers
    runs = []
    for measured in (False, True):
        eng = engine_for(wl, W)
        eng.prefill(prompts, wl.new_tokens)
        out = _run(eng, 2)
        if measured:
            stats, stages, tok, n, a = eng.profile_round()
            by = {s["kind"]: s for s in stats}
            assert by["gemm_qkv"]["launches"] == L + LD
            assert by["gemm_gate_up"]["launches"] == L + LD
            assert by["attention"]["launches"] == L + LD
            assert by["gemm_cond"]["launches"] == 3
            assert all(s["ms"] > 0 for s in stats if s["launches"]), stats
            assert len(stages) == 7 and all(x >= 0 for x in stages)
            out.append((tok.copy(), n.copy(), a.copy(), eng.read(B.RT_T_HD, 0, (wl.block_size, wl.target.hidden),
                                                                 np.uint16).copy()))
            for kind in (B.RT_K_GEMM_QKV, B.RT_K_GEMM_O, B.RT_K_GEMM_GATE_UP, B.RT_K_GEMM_DOWN,
                         B.RT_K_GEMM_CONTEXT, B.RT_K_GEMM_COND, B.RT_K_ATTENTION, B.RT_K_ATTN_MERGE,
                         B.RT_K_LM_HEAD):
                r = eng.time_kernel(kind, 2)
                if kind == B.RT_K_ATTN_MERGE and r["launches"] == 0:   # one key split: no merge
                    continue
                assert r["launches"] > 0 and r["ms"] > 0 and r["bytes"] > 0, r
            for kind in (B.RT_K_NORM, B.RT_K_QKV_POST, B.RT_K_MISC):
                with pytest.raises(B.RetraceError) as ex:
                    eng.time_kernel(kind, 2)
                assert ex.value.code == B.RT_ERR_INVALID
        else:
            out += _run(eng, 1)
        out += _run(eng, 3)
        runs.append(out)
        eng.close()
    for (t0, n0, a0, h0), (t1, n1, a1, h1) in zip(*runs):
        np.testing.assert_array_equal(t0, t1)
        np.testing.assert_array_equal(n0, n1)
        np.testing.assert_array_equal(h0, h1)


def test_stream_read_probe():
    """The plain-read ceiling probe (non-temporal contiguous reads) runs on a device buffer,
    stays within it for every window and reports longer times for larger reads."""
    import torch
    buf = torch.zeros(128 << 20, dtype=torch.uint8, device="cuda")
    assert buf.data_ptr() % 256 == 0
    small = B.rt_stream_read(buf.data_ptr(), buf.numel(), 4 << 20, 512, 5)
    large = B.rt_stream_read(buf.data_ptr(), buf.numel(), 64 << 20, 512, 5)
    whole = B.rt_stream_read(buf.data_ptr(), buf.numel(), buf.numel(), 2048, 3)   # one window only
    torch.cuda.synchronize()
    log(f"stream probe: 4 MiB {small:.2f} us, 64 MiB {large:.2f} us, 128 MiB {whole:.2f} us")
    assert 0 < small < large < whole
    assert float(buf.sum()) == 0.0   # nothing was written
