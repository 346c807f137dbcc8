"""Exact argmax ties go to the lowest token id (reading J: the paper does not say how
ties are broken) in both LM heads, on each of their paths: 16 rows (the head that
stages its activations in LDS), 32 rows, and 48 rows (the mid-size GEMM with the
argmax epilogue).

A tie is planted by copying the LM-head row of a token t that some row picks into a
lower, unused id t2: every logit of t2 then equals t's bit for bit (same operands, same
summation order), so wherever t was the maximum, t and t2 tie and t2 must win.  All
other tokens and every hidden state stay as in the unmodified run."""
import numpy as np
import pytest

from paper_2608_29748_amd import binding as B
from workloads import get, make_prompts, make_weights

from gpu_parity import engine_for, log

pytestmark = pytest.mark.gpu


def _round_tokens(wl, W, prompts):
    eng = engine_for(wl, W)
    first = eng.prefill(prompts, wl.new_tokens)
    eng.spec_round()
    bk = wl.block_size
    dt = np.stack([eng.read(B.RT_T_DRAFT_TOKENS, b, (bk,), np.int32)[1:] for b in range(wl.batch)])
    tt = np.stack([eng.read(B.RT_T_TARGET_TOKENS, b, (bk,), np.int32) for b in range(wl.batch)])
    eng.close()
    return np.asarray(first), dt, tt


def _tie(W, t, t2):
    W2 = dict(W)
    head = W["lm_head"].copy()
    head[t2] = head[t]
    W2["lm_head"] = head
    return W2


def _lower_unused(t, used):
    for t2 in range(t - 1, -1, -1):
        if t2 not in used:
            return t2
    return None


@pytest.mark.parametrize("batch", [1, 2, 3])
def test_exact_ties_pick_lowest_id(batch):
    wl = get("mini-bf16", batch=batch, prompt_len=(30, 60), norm_init="perturbed")
    W = make_weights(wl)
    prompts = make_prompts(wl)
    first, dt, tt = _round_tokens(wl, W, prompts)
    used = set(first.tolist()) | set(dt.ravel().tolist()) | set(tt.ravel().tolist())
    # drafter head: a draft token that is no sequence's anchor
    td = next(int(t) for t in dt.ravel() if int(t) not in set(first.tolist()) and _lower_unused(int(t), used) is not None)
    td2 = _lower_unused(td, used)
    f2, dt2, _ = _round_tokens(wl, _tie(W, td, td2), prompts)
    assert np.array_equal(f2, first)
    want = np.where(dt == td, td2, dt)
    log(f"[ties b{batch}] drafter: {td} duplicated into {td2}: {int((dt == td).sum())} rows tie")
    assert np.array_equal(dt2, want), (dt, dt2, td, td2)
    # verify head: a target token that is no anchor and no draft (drafts and their
    # verify inputs then stay as they were)
    tv = next(int(t) for t in tt.ravel() if int(t) not in set(first.tolist()) | set(dt.ravel().tolist())
              and _lower_unused(int(t), used) is not None)
    tv2 = _lower_unused(tv, used)
    f3, dt3, tt3 = _round_tokens(wl, _tie(W, tv, tv2), prompts)
    assert np.array_equal(f3, first) and np.array_equal(dt3, dt)
    want = np.where(tt == tv, tv2, tt)
    log(f"[ties b{batch}] verify: {tv} duplicated into {tv2}: {int((tt == tv).sum())} rows tie")
    assert np.array_equal(tt3, want), (tt, tt3, tv, tv2)
