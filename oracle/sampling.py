"""Temperature sampling for speculative rounds -- TEST INFRASTRUCTURE ONLY (oracle).

The paper evaluates at temperature 1 with top-p 0.95 and top-k 20 (Section 5,
experimental setup) and relies on standard lossless speculative verification, whose
acceptance rule it does not restate.  This module writes out, in float64:

  * the counter-based random generator both sides use (Philox4x64 with ten rounds,
    from its published definition: two 64x64 -> 128-bit multiplies per round, the
    Weyl key schedule), so that random draws need not be passed in;
  * the filtered next-token distribution (temperature, then top-k, then top-p on the
    renormalised top-k probabilities, ties to the lowest id);
  * inverse-CDF sampling from such a distribution;
  * the speculative-sampling acceptance rule: draft token y_i drawn from the drafter's
    distribution q_i is kept with probability min(1, p_i(y_i) / q_i(y_i)); at the first
    rejection the correction is drawn from the normalised residual max(0, p_i - q_i);
    after B acceptances a bonus token is drawn from p_{B+1}.  The committed tokens are
    then distributed exactly as the target's own filtered sampling.

Counters: (round, sequence, purpose, position) with key (seed, 0); word 0 of the
output block gives the uniform (top 53 bits) / 2^53 in [0, 1).
"""
from __future__ import annotations

from dataclasses import dataclass
from typing import List, Sequence, Tuple

import numpy as np

MASK64 = (1 << 64) - 1
PHILOX_M = (0xD2E7470EE14C6C93, 0xCA5A826395121157)
PHILOX_W = (0x9E3779B97F4A7C15, 0xBB67AE8584CAA73B)

# purposes of a draw
U_DRAFT = 1      # sample the draft token at block position pos (1..B)
U_ACCEPT = 2     # acceptance test at block position pos (1..B)
U_RESAMPLE = 3   # correction (residual) or bonus token of a round
U_FIRST = 4      # the prefill's first token (round 0)
U_STEP = 5       # a target-only step


def philox4x64_10(counter: Sequence[int], key: Sequence[int]) -> List[int]:
    """One Philox4x64-10 block: four 64-bit words of counter, two of key."""
    c = [int(x) & MASK64 for x in counter]
    k = [int(x) & MASK64 for x in key]
    for _ in range(10):
        p0 = PHILOX_M[0] * c[0]
        p1 = PHILOX_M[1] * c[2]
        c = [(p1 >> 64) ^ c[1] ^ k[0], p1 & MASK64, (p0 >> 64) ^ c[3] ^ k[1], p0 & MASK64]
        k = [(k[0] + PHILOX_W[0]) & MASK64, (k[1] + PHILOX_W[1]) & MASK64]
    return c


def uniform(seed: int, rnd: int, seq: int, purpose: int, pos: int) -> float:
    """Uniform in [0, 1) for one draw: 53 random bits scaled by 2^-53 (exact in float64)."""
    w = philox4x64_10((rnd, seq, purpose, pos), (seed, 0))[0]
    return (w >> 11) * 2.0 ** -53


@dataclass
class Dist:
    """A filtered next-token distribution: ids in decreasing probability (ties by
    increasing id) and their probabilities, summing to one."""
    ids: np.ndarray
    probs: np.ndarray

    def prob(self, tok: int) -> float:
        hit = np.nonzero(self.ids == tok)[0]
        return float(self.probs[hit[0]]) if hit.size else 0.0


def filtered(logits: np.ndarray, temperature: float, top_k: int, top_p: float) -> Dist:
    """Softmax of logits / temperature restricted to the top_k largest logits (ties: lowest
    id first), renormalised, then cut to the shortest prefix whose cumulative probability
    reaches top_p (at least one token), renormalised again."""
    z = np.asarray(logits, np.float64)
    order = np.lexsort((np.arange(z.size), -z))[:top_k]      # by logit descending, id ascending
    s = z[order] / temperature
    w = np.exp(s - s[0])
    pk = w / w.sum()
    cum = np.cumsum(pk)
    n = int(np.searchsorted(cum, top_p, side="left")) + 1   # first index with cum >= top_p
    n = min(max(n, 1), len(order))
    p = pk[:n] / pk[:n].sum()
    return Dist(ids=order[:n].astype(np.int64), probs=p)


def sample(d: Dist, u: float) -> int:
    """Inverse CDF: the first token whose cumulative probability exceeds u."""
    cum = np.cumsum(d.probs)
    j = int(np.searchsorted(cum, u, side="right"))
    return int(d.ids[min(j, len(d.ids) - 1)])


def residual(p: Dist, q: Dist) -> Dist:
    """Normalised max(0, p - q) over p's support, in p's order (its support lies within
    p's: the weight is zero wherever p is)."""
    w = np.array([max(0.0, float(pp) - q.prob(int(t))) for t, pp in zip(p.ids, p.probs)])
    tot = w.sum()
    if tot <= 0.0:          # p == q on the support: no rejection can have happened
        return p
    keep = w > 0
    return Dist(ids=p.ids[keep], probs=w[keep] / tot)


def speculative_accept(y_hat: Sequence[int], q: Sequence[Dist], p: Sequence[Dist],
                       u_acc: Sequence[float], u_res: float) -> Tuple[int, int]:
    """Block acceptance for draft tokens y_hat[0..B-1] (block positions 1..B) with drafter
    distributions q[i] and target distributions p[i] (p has B+1 entries: position B+1 is
    the bonus row).  Returns (A, the correction or bonus token)."""
    B = len(y_hat)
    for i in range(B):
        t = int(y_hat[i])
        pq, qq = p[i].prob(t), q[i].prob(t)
        if not (u_acc[i] * qq < pq):          # keep with probability min(1, p/q)
            return i, sample(residual(p[i], q[i]), u_res)
    return B, sample(p[B], u_res)
