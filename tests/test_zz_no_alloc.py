"""The allocation-free round (rt_spec_round_static: no graph instantiation, partial
results in the library's static scratch, outputs to device buffers) against
rt_spec_round on the same model and inputs: committed tokens, acceptance lengths,
round state and retained final states must be equal bit for bit, over consecutive calls
and again after a new prefill with a smaller batch (the static scratch then holds the
previous call's contents)."""
import numpy as np
import pytest
import torch

from paper_2608_29748_amd import binding as B
from workloads import ModelShape, get, make_prompts, make_weights

from gpu_parity import engine_for, keep_dtype, log

pytestmark = pytest.mark.gpu


def _static_round(eng):
    n, bk = eng.n_seqs, eng.cfg.block_size
    tok = torch.full((n, bk), -7, dtype=torch.int32, device=eng.device)
    nc = torch.full((n,), -7, dtype=torch.int32, device=eng.device)
    acc = torch.full((n,), -7, dtype=torch.int32, device=eng.device)
    torch.cuda.synchronize(eng.device)
    B.rt_spec_round_static(eng.h, tok.data_ptr(), nc.data_ptr(), acc.data_ptr())
    eng.stream.synchronize()
    return tok.cpu().numpy(), nc.cpu().numpy(), acc.cpu().numpy()


def _state(eng, wl):
    bk, d, kd = wl.block_size, wl.target.hidden, keep_dtype(wl)
    return [(eng.read(B.RT_T_STATE, b, (9,), np.int32), eng.read(B.RT_T_HD, b, (bk, d), kd).view(np.uint8),
             eng.read(B.RT_T_HT, b, (bk, d), kd).view(np.uint8)) for b in range(eng.n_seqs)]


@pytest.mark.parametrize("name,over", [("mini-bf16-b6", {}), ("mini-bf16", {}),
                                       ("tiny-f32", {"batch": 6, "prompt_len": (20, 80)})])
def test_static_round_equals_round(name, over):
    wl = get(name, norm_init="perturbed", **over)
    W = make_weights(wl)
    prompts = make_prompts(wl)
    ref = engine_for(wl, W)
    eng = engine_for(wl, W)
    with pytest.raises(B.RetraceError) as ei:
        _static_round(eng)
    assert ei.value.code == B.RT_ERR_STATE
    # two prefills: the whole batch, then fewer and shorter prompts (a smaller input)
    small = [p[: max(8, len(p) // 2)] for p in prompts[: max(1, len(prompts) // 3)]]
    for case, ps, rounds in (("batch", prompts, 3), ("smaller", small, 2)):
        assert list(ref.prefill(ps, wl.new_tokens)) == list(eng.prefill(ps, wl.new_tokens))
        for t in range(rounds):
            tok_r, n_r, a_r = ref.spec_round()
            tok_s, n_s, a_s = _static_round(eng)
            assert np.array_equal(tok_s, tok_r), (case, t, tok_s, tok_r)
            assert np.array_equal(n_s, n_r) and np.array_equal(a_s, a_r), (case, t, n_s, n_r, a_s, a_r)
            for b, (x, y) in enumerate(zip(_state(ref, wl), _state(eng, wl))):
                assert np.array_equal(x[0], y[0]), (case, t, b, x[0], y[0])
                assert np.array_equal(x[1], y[1]) and np.array_equal(x[2], y[2]), (case, t, b, "retained states")
        log(f"[{name}] {case}: {len(ps)} sequences, {rounds} rounds equal bit for bit")
    ref.close()
    eng.close()


def test_static_round_refuses_configurations_beyond_its_scratch():
    wl = get("mini-bf16", target=ModelShape(vocab=2048, hidden=2048, n_layers=1, n_q_heads=16, n_kv_heads=2,
                                            head_dim=128, ffn=512),
             draft_layers=1, cond_layers=(0,), batch=128, prompt_len=(16, 16), new_tokens=8)
    eng = engine_for(wl, make_weights(wl))
    with pytest.raises(B.RetraceError) as ei:
        _static_round(eng)
    assert ei.value.code == B.RT_ERR_CAPACITY, ei.value
    log(f"[static scratch] {ei.value}")
    eng.close()
