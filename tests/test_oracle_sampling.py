"""Pins for the oracle's temperature sampling: the counter-based generator against
numpy's Philox4x64 bit generator, the filtered distribution's closed forms and a
hand-worked case, inverse-CDF sampling, the speculative-sampling rule's defining
property (committed tokens follow the target's filtered distribution exactly), and
planted mistakes that must break those pins."""
import copy
import dataclasses

import numpy as np
import pytest

import oracle.sampling as smp
from oracle import OracleModel, OracleRunner
from workloads import get, make_prompts, make_weights


# ------------------------------------------------------------ generator

@pytest.mark.parametrize("key,ctr", [((0, 0), (0, 0, 0, 0)), ((5, 7), (3, 0, 0, 0)),
                                     ((2**64 - 1, 12345), (2**64 - 2, 2**63, 17, 1)),
                                     ((42, 0), (1, 3, 2, 9))])
def test_philox_matches_numpy(key, ctr):
    """numpy's Philox (4x64, ten rounds) advances its counter before each block, so
    its first block is ours at counter + 1 (carry into the next word)."""
    bg = np.random.Philox(key=np.array(key, dtype=np.uint64), counter=np.array(ctr, dtype=np.uint64))
    got = [int(x) for x in bg.random_raw(8)]
    c = list(ctr)
    want = []
    for _ in range(2):
        for i in range(4):                      # 256-bit increment
            c[i] = (c[i] + 1) & smp.MASK64
            if c[i]:
                break
        want += smp.philox4x64_10(c, key)
    assert got == want


def test_uniform_range_and_bits():
    us = [smp.uniform(42, r, s, p, i) for r in range(3) for s in range(3) for p in range(1, 4) for i in range(4)]
    assert all(0.0 <= u < 1.0 for u in us)
    w = smp.philox4x64_10((1, 2, 3, 4), (42, 0))[0]
    assert smp.uniform(42, 1, 2, 3, 4) == (w >> 11) / 2.0 ** 53
    assert len(set(us)) == len(us)


# ------------------------------------------------------------ filtered distribution

def check_filtered(filt=smp.filtered):
    # hand-worked: logits [0, 2, 1, 2], T = 1, top-k 3 keeps ids 1, 3 (tie: lower id
    # first), 2 with probabilities e^2, e^2, e / (2e^2 + e); top-p 0.6 is reached at the
    # second: keep {1, 3} with 1/2 each
    d = filt(np.array([0.0, 2.0, 1.0, 2.0]), 1.0, 3, 0.6)
    assert list(d.ids) == [1, 3]
    np.testing.assert_allclose(d.probs, [0.5, 0.5], rtol=1e-15)
    d = filt(np.array([0.0, 2.0, 1.0, 2.0]), 1.0, 3, 0.9)
    e = np.exp(1.0)
    assert list(d.ids) == [1, 3, 2]
    np.testing.assert_allclose(d.probs, np.array([e * e, e * e, e]) / (2 * e * e + e), rtol=1e-14)
    # top-p applies to the renormalised top-k probabilities: [.3, .3, .2, .2] with top-k 3
    # renormalises to [.375, .375, .25], whose cumulative sum reaches 0.7 at the second
    d = filt(np.log(np.array([0.3, 0.3, 0.2, 0.2])), 1.0, 3, 0.7)
    assert list(d.ids) == [0, 1]
    np.testing.assert_allclose(d.probs, [0.5, 0.5], rtol=1e-14)
    # top-k 1 is the argmax (lowest id among equal maxima)
    d = filt(np.array([0.5, 3.0, -1.0, 3.0]), 1.0, 1, 0.95)
    assert list(d.ids) == [1] and list(d.probs) == [1.0]
    # top-p 1 over the whole vocabulary is the softmax, in decreasing order
    z = np.random.default_rng(0).standard_normal(50)
    d = filt(z, 1.0, 50, 1.0)
    ref = np.exp(z - z.max()) / np.exp(z - z.max()).sum()
    np.testing.assert_allclose(d.probs, ref[d.ids], rtol=1e-13)
    assert np.all(np.diff(d.probs) <= 0)
    # temperature 2 halves the logits
    d2, d1 = filt(z, 2.0, 20, 0.95), filt(z / 2.0, 1.0, 20, 0.95)
    assert list(d2.ids) == list(d1.ids)
    np.testing.assert_allclose(d2.probs, d1.probs, rtol=1e-14)


def test_filtered_distribution():
    check_filtered()


def test_sample_inverse_cdf():
    d = smp.Dist(ids=np.array([7, 3, 9]), probs=np.array([0.5, 0.25, 0.25]))
    assert smp.sample(d, 0.0) == 7
    assert smp.sample(d, 0.5) == 3            # first cumulative probability above u
    assert smp.sample(d, 0.7499) == 3
    assert smp.sample(d, 0.75) == 9
    assert smp.sample(d, 1.0 - 2 ** -53) == 9
    us = [smp.uniform(1, 0, 0, 1, i) for i in range(20000)]
    counts = np.bincount([smp.sample(d, u) for u in us], minlength=10)[[7, 3, 9]]
    chi2 = float(np.sum((counts - 20000 * d.probs) ** 2 / (20000 * d.probs)))
    assert chi2 < 13.8                        # 2 degrees of freedom, p = 0.001


# ------------------------------------------------------------ speculative sampling rule

def _dists():
    p = smp.Dist(ids=np.array([0, 1, 2, 3, 4]), probs=np.array([0.4, 0.25, 0.15, 0.12, 0.08]))
    q = smp.Dist(ids=np.array([2, 0, 5, 1]), probs=np.array([0.5, 0.2, 0.2, 0.1]))
    return p, q


def check_lossless(accept=smp.speculative_accept, n=60000):
    """Single-position block: draft y ~ q, then the rule; the committed token must be
    distributed as p whatever q is (chi-square over p's support plus q-only ids)."""
    p, q = _dists()
    out = np.zeros(8)
    for i in range(n):
        y = smp.sample(q, smp.uniform(9, i, 0, smp.U_DRAFT, 1))
        A, corr = accept([y], [q], [p, p], [smp.uniform(9, i, 0, smp.U_ACCEPT, 1)],
                         smp.uniform(9, i, 0, smp.U_RESAMPLE, 0))
        out[y if A == 1 else corr] += 1
    expect = np.zeros(8)
    expect[p.ids] = p.probs * n
    assert out[5] == 0 and out[6] == 0 and out[7] == 0   # never outside p's support
    sel = expect > 0
    chi2 = float(np.sum((out[sel] - expect[sel]) ** 2 / expect[sel]))
    assert chi2 < 18.5                                   # 4 degrees of freedom, p = 0.001


def test_speculative_sampling_is_lossless():
    check_lossless()


def test_speculative_accept_cases():
    p, q = _dists()
    # p >= q at the draft: always kept; all kept -> bonus from the last row
    A, corr = smp.speculative_accept([0], [smp.Dist(np.array([1, 0]), np.array([0.7, 0.3]))], [p, p], [0.999], 0.0)
    assert A == 1 and corr == 0
    # p < q at the draft: kept exactly when u < p / q (0.25 / 0.7)
    qq = smp.Dist(np.array([1, 0]), np.array([0.7, 0.3]))
    assert smp.speculative_accept([1], [qq], [p, p], [0.25 / 0.7 - 1e-12], 0.0)[0] == 1
    assert smp.speculative_accept([1], [qq], [p, p], [0.25 / 0.7 + 1e-12], 0.0)[0] == 0
    # draft outside p's support: always rejected, correction from p's residual
    A, corr = smp.speculative_accept([5], [q], [p, p], [0.0], 0.0)
    assert A == 0 and corr in (0, 1, 3, 4)
    # residual = normalised max(0, p - q) in p's order: ids 0 (0.2), 1 (0.15), 3, 4
    r = smp.residual(p, q)
    assert list(r.ids) == [0, 1, 3, 4]
    np.testing.assert_allclose(r.probs, np.array([0.2, 0.15, 0.12, 0.08]) / 0.55, rtol=1e-14)


def _swapped_ratio(y_hat, q, p, u_acc, u_res):
    for i, t in enumerate(y_hat):
        if not (u_acc[i] * p[i].prob(int(t)) < q[i].prob(int(t))):
            return i, smp.sample(smp.residual(p[i], q[i]), u_res)
    return len(y_hat), smp.sample(p[-1], u_res)


def _reversed_residual(y_hat, q, p, u_acc, u_res):
    for i, t in enumerate(y_hat):
        if not (u_acc[i] * q[i].prob(int(t)) < p[i].prob(int(t))):
            return i, smp.sample(smp.residual(q[i], p[i]), u_res)
    return len(y_hat), smp.sample(p[-1], u_res)


def _topk_after_topp(z, t, k, pp):
    d = smp.filtered(z, t, len(z), pp)
    n = min(k, len(d.ids))
    return smp.Dist(ids=d.ids[:n], probs=d.probs[:n] / d.probs[:n].sum())


@pytest.mark.parametrize("check,kw", [
    (check_lossless, {"accept": _swapped_ratio, "n": 20000}),
    (check_lossless, {"accept": _reversed_residual, "n": 20000}),
    (check_filtered, {"filt": _topk_after_topp}),
    (check_filtered, {"filt": lambda z, t, k, p: smp.filtered(z * t, 1.0, k, p)}),
])
def test_pins_catch_planted_mistakes(check, kw):
    with pytest.raises(AssertionError):
        check(**kw)


# ------------------------------------------------------------ whole rounds

def test_round_first_token_follows_target_distribution():
    """From one prefilled state, the first token committed by a sampled round has the
    target's filtered distribution at that position, whatever the drafter proposes
    (one round per seed, 400 seeds)."""
    wl = get("tiny-f32", norm_init="perturbed", temperature=1.0, top_k=20, top_p=0.95)
    W = make_weights(wl)
    prompt = make_prompts(wl)[0]
    R = OracleRunner(OracleModel(wl, W))
    st0 = R.prefill(prompt, 40)
    p1 = R.dist(R.verify(copy.deepcopy(st0), [0] * wl.B).logits[0])   # row 0 sees only the context
    counts = {}
    rejected = 0
    for seed in range(400):
        Rs = OracleRunner(OracleModel(dataclasses.replace(wl, sample_seed=seed), W))
        Rs.m.W = R.m.W
        st = copy.deepcopy(st0)
        rec = Rs.round(st)
        counts[rec.committed[0]] = counts.get(rec.committed[0], 0) + 1
        rejected += rec.A == 0
    assert set(counts) <= set(int(t) for t in p1.ids)
    obs = np.array([counts.get(int(t), 0) for t in p1.ids], float)
    exp = p1.probs * 400
    big = exp >= 5                          # pool the rare tail into one cell
    o = np.append(obs[big], obs[~big].sum())
    e = np.append(exp[big], exp[~big].sum())
    if e[-1] == 0:
        o, e = o[:-1], e[:-1]
    chi2 = float(np.sum((o - e) ** 2 / e))
    from scipy.stats import chi2 as chi2d
    assert chi2 < chi2d.ppf(0.999, len(e) - 1)
    assert rejected > 0                      # the residual path was exercised


def test_sampled_rounds_bookkeeping():
    """Sampled rounds keep the greedy bookkeeping: committed = drafts 1..A plus one
    token, carry / reset by A, budget clipping, the round counter advances."""
    wl = get("mini-bf16", norm_init="perturbed", temperature=1.0)
    W = make_weights(wl)
    R = OracleRunner(OracleModel(wl, W))
    st = R.prefill(make_prompts(wl)[0], 30)
    n = 0
    while not st.done:
        rec = R.round(st)
        n += 1
        assert st.rnd == n
        assert list(rec.committed[: rec.A]) == [int(t) for t in rec.y_hat[: rec.A]][: len(rec.committed)]
        assert st.cond_len == (wl.B - rec.A - 1 if rec.A < wl.B - 1 else 0)
    assert len(st.generated) == 30
