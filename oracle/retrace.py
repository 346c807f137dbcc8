"""Float64 reference of the ReTrace round (Section 4, Eq.3-9, Algorithm 1).

Round t, for one sequence whose committed context ends with the anchor at
position P (target KV and drafter context KV hold rows 0..P-1):

1. Conditioning (Eq.5-9).  If the previous round left a rejected suffix, its
   retained drafter states h^D and target states h^T are aligned to the new
   block (m_j = h^D_{r+j}, u_j = h^T_{r+j-1}, 1 <= j <= B-r, with r the previous
   first rejected position), corrected (c_j = W_c[m_j; u_j], r_j = m_j + beta c_j)
   and admitted into the mask inputs through the gated residual
   e~_j = e_j + (W_v r_j) * sigmoid(W_g[e_j; r_j]).  The anchor row and rows
   without an aligned state keep e_j.
2. Drafter forward on e~_{0:B} -> h^D_{0:B}, draft tokens y^_j = argmax of the
   LM head at row j, j = 1..B.
3. Verify: target forward of [anchor, y^_1..y^_B] at positions P..P+B ->
   h^T_{0:B}; the target's token for block position i is y^T_i = argmax of row i-1.
4. Accept: A = longest prefix with y^_i = y^T_i.  Commit y^_1..y^_A and the
   correction (bonus when A = B) y^T_{A+1}, clipped to the generation budget;
   the target keeps KV rows up to P+A (rollback), the drafter's context pathway
   appends rows 0..A, the new anchor is y^T_{A+1} at P+A+1.
5. Carry: if A < B-1, keep h^D and h^T (rounded to the retained format) with
   r = A+1 and B-r conditioned rows for the next round; otherwise nothing is
   carried (full acceptance, or rejection at the last position) -- the signal
   lives for exactly one round.

Ties in every argmax go to the lowest token id.  Losslessness: the committed
stream equals target-only greedy decoding (ar_decode).
"""
from __future__ import annotations

from dataclasses import dataclass
from typing import List, Optional, Sequence, Tuple

import numpy as np

from . import sampling as smp

from .model import DraftOut, OracleModel, SeqState, VerifyOut, sigmoid


def align_rejected(hD_prev: np.ndarray, hT_prev: np.ndarray, r: int, B: int):
    """Eq.5 and Eq.6.  Inputs are the previous round's retained states indexed by
    block row (0..B); returns (m, u), each [B+1][d] indexed by the next block's
    row j, zero for j = 0 and for j > B - r."""
    d = hD_prev.shape[1]
    m = np.zeros((B + 1, d))
    u = np.zeros((B + 1, d))
    for j in range(1, B - r + 1):
        m[j] = hD_prev[r + j]
        u[j] = hT_prev[r + j - 1]
    return m, u


def condition_inputs(e: np.ndarray, m: np.ndarray, u: np.ndarray, cond_len: int,
                     w_c: np.ndarray, w_v: np.ndarray, w_g: np.ndarray,
                     beta: float, mode: str = "retrace", lowrank=None) -> np.ndarray:
    """Eq.7 (correction), Eq.8 (corrected signal), Eq.9 (gated residual) for rows
    j = 1..cond_len.  Weight matrices are [out][in]; W_c's first d input columns
    act on m and W_g's first d on e.

    The component ablation (Section 5, Table 3; Appendix "Ablation Settings") uses the
    same aligned signal three ways: "retrace" corrects it (Eq.7-8) and adds it through
    the gate (Eq.9); "raw_gated" adds the raw aligned drafter state r_j = m_j through
    the same gate; "overwrite" replaces the conditioned mask inputs with m_j.

    "lowrank" is the deployment form of the conditioning path named in the appendix on
    concurrent serving (rank-64 rejected-suffix latents, input-side latent residual
    fusion, rank-32 target-aware correction), read as: latent z_j = A m_j, correction
    in latent space c_j = C_up C_down [m_j; u_j], rho_j = z_j + beta c_j, and
    e~_j = e_j + (V rho_j) * sigmoid(W_g[:, :d] e_j + G rho_j), with
    lowrank = (A, C_down, C_up, V, G).  It reduces to the full form when A = I,
    W_c = C_up C_down, W_v = V and W_g[:, d:] = G."""
    e_t = e.copy()
    d = e.shape[1]
    for j in range(1, cond_len + 1):
        if mode == "overwrite":
            e_t[j] = m[j]
            continue
        if mode == "lowrank":
            A, c_down, c_up, V, G = lowrank
            rho = A @ m[j] + beta * (c_up @ (c_down @ np.concatenate([m[j], u[j]])))
            gate = sigmoid(w_g[:, :d] @ e[j] + G @ rho)
            e_t[j] = e[j] + (V @ rho) * gate
            continue
        if mode == "raw_gated":
            rj = m[j]
        else:
            c = w_c @ np.concatenate([m[j], u[j]])
            rj = m[j] + beta * c
        gate = sigmoid(w_g @ np.concatenate([e[j], rj]))
        e_t[j] = e[j] + (w_v @ rj) * gate
    return e_t


def accept_length(draft: Sequence[int], target: Sequence[int]) -> int:
    """Number of leading block positions whose draft token equals the target's."""
    A = 0
    for a, b in zip(draft, target):
        if a != b:
            break
        A += 1
    return A


def argmax_rows(logits: np.ndarray) -> np.ndarray:
    """Per-row argmax; np.argmax returns the first maximum, i.e. the lowest id on ties."""
    return np.argmax(logits, axis=-1)


@dataclass
class RoundRecord:
    draft: DraftOut
    verify: VerifyOut
    y_hat: np.ndarray            # [B] draft tokens for block positions 1..B
    y_t: np.ndarray              # [B+1] target tokens for block positions 1..B+1
    A: int
    committed: List[int]
    cond_len: int                # rows conditioned in this round
    P: int                       # anchor position of this round


class OracleRunner:
    """Drives OracleModel through prefill, rounds and the target-only greedy decode."""

    def __init__(self, model: OracleModel):
        self.m = model
        self.wl = model.wl
        self.B = model.wl.B

    # -- prefill: prompt rows through the target, first token, drafter context
    @property
    def sampling(self) -> bool:
        return self.wl.temperature > 0.0

    def dist(self, logits_row) -> smp.Dist:
        return smp.filtered(logits_row, self.wl.temperature, self.wl.top_k, self.wl.top_p)

    def u(self, st: SeqState, rnd: int, purpose: int, pos: int) -> float:
        return smp.uniform(self.wl.sample_seed, rnd, st.seq, purpose, pos)

    def prefill(self, prompt, budget: int, seq: int = 0) -> SeqState:
        m = self.m
        st = m.new_state(prompt, budget)
        st.seq = seq
        out = m.target_forward(st, prompt, 0)
        if self.sampling:
            first = smp.sample(self.dist(out.logits[-1]), self.u(st, 0, smp.U_FIRST, 0))
        else:
            first = int(argmax_rows(out.logits[-1]))
        m.context_append(st, out.g, 0)
        d = self.wl.target.hidden
        st.P, st.anchor, st.generated = len(prompt), first, [first]
        st.hD_prev = np.zeros((self.B + 1, d))
        st.hT_prev = np.zeros((self.B + 1, d))
        st.r, st.cond_len = 0, 0
        return st

    # -- steps of one round, separately callable so a caller can override decisions
    def draft(self, st: SeqState) -> DraftOut:
        m, W = self.m, self.m.W
        e = m.block_inputs(st.anchor)
        if st.cond_len > 0 and self.wl.cond_mode != "off":
            mm, uu = align_rejected(st.hD_prev, st.hT_prev, st.r, self.B)
            lr = (tuple(W[f"retrace.lr_{n}"] for n in ("a", "c_down", "c_up", "v", "g"))
                  if self.wl.cond_mode == "lowrank" else None)
            e_t = condition_inputs(e, mm, uu, st.cond_len, W["retrace.w_c"], W["retrace.w_v"],
                                   W["retrace.w_g"], self.wl.beta, self.wl.cond_mode, lr)
        else:
            e_t = e.copy()
        e_t = m.prec.r(e_t)
        h, logits = m.drafter_forward(st, e_t)
        return DraftOut(e=e, e_tilde=e_t, h=h, logits=logits)

    def verify(self, st: SeqState, y_hat: Sequence[int]) -> VerifyOut:
        return self.m.target_forward(st, [st.anchor] + [int(t) for t in y_hat], st.P)

    def commit(self, st: SeqState, y_hat, y_t, d: DraftOut, v: VerifyOut) -> Tuple[int, List[int]]:
        """Greedy acceptance: the longest prefix of drafts equal to the target's argmax."""
        A = accept_length(y_hat, y_t[: self.B])
        return self.commit_tokens(st, y_hat, A, int(y_t[A]), d, v)

    def commit_tokens(self, st: SeqState, y_hat, A: int, corr: int, d: DraftOut,
                      v: VerifyOut) -> Tuple[int, List[int]]:
        """Commits drafts 1..A and the correction / bonus token corr, rolls the target
        cache back, extends the drafter context and applies the carry / reset rule."""
        B = self.B
        st.rnd += 1
        new = [int(t) for t in y_hat[:A]] + [int(corr)]
        new = new[: max(0, st.budget - len(st.generated))]
        st.generated.extend(new)
        # rollback: target rows P+A+1..P+B were computed for rejected tokens
        st.tgt_k[:, st.P + A + 1: st.P + B + 1] = 0.0
        st.tgt_v[:, st.P + A + 1: st.P + B + 1] = 0.0
        self.m.context_append(st, v.g[: A + 1], st.P)
        st.P += A + 1
        st.anchor = int(corr)
        if A < B - 1:
            st.r = A + 1
            st.cond_len = B - st.r
            st.hD_prev = self.m.prec.k(d.h)
            st.hT_prev = self.m.prec.k(v.h)
        else:
            st.r, st.cond_len = 0, 0
            st.hD_prev = np.zeros_like(st.hD_prev)
            st.hT_prev = np.zeros_like(st.hT_prev)
        return A, new

    def round(self, st: SeqState, forced_draft: Optional[Sequence[int]] = None) -> RoundRecord:
        if self.sampling:
            return self.sample_round(st, forced_draft)
        P, cond_len = st.P, st.cond_len
        d = self.draft(st)
        y_hat = (np.asarray(forced_draft, dtype=np.int64) if forced_draft is not None
                 else argmax_rows(d.logits[1:]))
        v = self.verify(st, y_hat)
        y_t = argmax_rows(v.logits)
        A, new = self.commit(st, y_hat, y_t, d, v)
        return RoundRecord(draft=d, verify=v, y_hat=y_hat, y_t=y_t, A=A, committed=new,
                           cond_len=cond_len, P=P)

    def sample_round(self, st: SeqState, forced_draft: Optional[Sequence[int]] = None) -> RoundRecord:
        """A round under temperature sampling: drafts drawn from the drafter's filtered
        distributions, speculative-sampling acceptance against the target's."""
        P, cond_len, B = st.P, st.cond_len, self.B
        rnd = st.rnd + 1
        d = self.draft(st)
        q = [self.dist(d.logits[i]) for i in range(1, B + 1)]
        if forced_draft is not None:
            y_hat = np.asarray(forced_draft, dtype=np.int64)
        else:
            y_hat = np.array([smp.sample(q[i - 1], self.u(st, rnd, smp.U_DRAFT, i)) for i in range(1, B + 1)],
                             dtype=np.int64)
        v = self.verify(st, y_hat)
        p = [self.dist(v.logits[i]) for i in range(B + 1)]
        u_acc = [self.u(st, rnd, smp.U_ACCEPT, i) for i in range(1, B + 1)]
        A, corr = smp.speculative_accept(y_hat, q, p, u_acc, self.u(st, rnd, smp.U_RESAMPLE, 0))
        A, new = self.commit_tokens(st, y_hat, A, corr, d, v)
        return RoundRecord(draft=d, verify=v, y_hat=y_hat, y_t=argmax_rows(v.logits), A=A, committed=new,
                           cond_len=cond_len, P=P)

    def spec_decode(self, prompt, budget: int, max_rounds: Optional[int] = None):
        st = self.prefill(prompt, budget)
        recs = []
        while not st.done and (max_rounds is None or len(recs) < max_rounds):
            recs.append(self.round(st))
        return st.generated, recs, st

    # -- references
    def ar_decode(self, prompt, n_new: int, seq: int = 0) -> List[int]:
        """Target-only decoding, one row per step, n_new tokens: greedy, or under
        temperature sampling with the step index as the draw's round."""
        m = self.m
        st = m.new_state(prompt, n_new)
        st.seq = seq
        pick = ((lambda row, k: smp.sample(self.dist(row), self.u(st, k, smp.U_STEP if k else smp.U_FIRST, 0)))
                if self.sampling else (lambda row, k: int(argmax_rows(row))))
        out = m.target_forward(st, prompt, 0)
        tok = pick(out.logits[-1], 0)
        toks, pos = [tok], len(prompt)
        while len(toks) < n_new:
            out = m.target_forward(st, [tok], pos)
            tok = pick(out.logits[-1], len(toks))
            toks.append(tok)
            pos += 1
        return toks

    def logits_nocache(self, tokens) -> np.ndarray:
        """Target logits of every row of `tokens`, recomputed from an empty cache."""
        st = self.m.new_state(tokens, 0)
        return self.m.target_forward(st, tokens, 0).logits
