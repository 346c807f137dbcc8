"""Float64 reference of the target (Qwen3-style decoder) and the block drafter.

Target: Qwen3 decoder layers -- RMSNorm (eps 1e-6), q/k/v projections, per-head
q-norm and k-norm, rotate-half RoPE (theta 1e6), grouped-query softmax
attention with scale 1/sqrt(head_dim), o-projection, RMSNorm, SwiGLU MLP; final
RMSNorm and an LM head untied from the embedding.  Block verification runs the
B+1 rows [anchor, draft_1..draft_B] at absolute positions P..P+B, causally
over the cached context plus the block (Section 2 / Alg.1 Verify).

Drafter (DFlash-style, the paper's drafter backbone; its internals are not
defined in the paper -- parity unpinned against the paper): layers of the
target's width and form.  Context pathway: the target's residual states after
each conditioning layer are concatenated, projected by fc (n_c*d -> d) and
RMS-normalised; every drafter layer projects that feature with its own W_k
(k-norm, RoPE at the absolute position) and W_v into a context KV cache.  The
block of B+1 rows (anchor embedding followed by B mask embeddings, after
conditioning) attends to the context keys and to all block keys (no causal
mask inside the block); its final RMSNorm output h^D feeds the shared LM head,
and row j proposes the token at position P+j.

RoPE convention: inv_freq_i is theta**(-2i/hd) rounded to float32, the angle is
the float32-rounded product position*inv_freq_i, and cos/sin are evaluated
exactly on that angle.
"""
from __future__ import annotations

from dataclasses import dataclass, field
from typing import Dict, List, Optional

import numpy as np

from workloads import Workload
from workloads.generate import as_f32

from .numerics import Precision, round_f32


# ---------------------------------------------------------------- layer math

def rms_norm(x: np.ndarray, w: np.ndarray, eps: float) -> np.ndarray:
    """x / sqrt(mean(x^2) + eps) * w over the last axis."""
    return x / np.sqrt(np.mean(x * x, axis=-1, keepdims=True) + eps) * w


def silu(x: np.ndarray) -> np.ndarray:
    return x / (1.0 + np.exp(-x))


def sigmoid(x: np.ndarray) -> np.ndarray:
    return 1.0 / (1.0 + np.exp(-x))


def rope_inv_freq(head_dim: int, theta: float) -> np.ndarray:
    i = np.arange(head_dim // 2, dtype=np.float64)
    return round_f32(theta ** (-2.0 * i / head_dim))


def rope_angles(positions: np.ndarray, head_dim: int, theta: float) -> np.ndarray:
    """[n, head_dim/2] float32-rounded angles position * inv_freq."""
    pos = np.asarray(positions, dtype=np.float64)
    return round_f32(pos[:, None] * rope_inv_freq(head_dim, theta)[None, :])


def apply_rope(x: np.ndarray, positions: np.ndarray, theta: float) -> np.ndarray:
    """Rotate-half RoPE on x[n, heads, hd]: (x1, x2) -> (x1 cos - x2 sin, x2 cos + x1 sin)."""
    hd = x.shape[-1]
    ang = rope_angles(positions, hd, theta)[:, None, :]
    cos, sin = np.cos(ang), np.sin(ang)
    x1, x2 = x[..., : hd // 2], x[..., hd // 2:]
    return np.concatenate([x1 * cos - x2 * sin, x2 * cos + x1 * sin], axis=-1)


def attention(q: np.ndarray, k: np.ndarray, v: np.ndarray, q_pos: np.ndarray,
              k_pos: np.ndarray, causal: bool) -> np.ndarray:
    """Grouped-query softmax attention.  q[n, Hq, hd], k/v[T, Hkv, hd]; query head h
    reads kv head h // (Hq/Hkv).  causal: key position must not exceed the query's.
    The probabilities are the plain softmax of the scaled scores (no storage rounding:
    only the stored output is rounded)."""
    n, hq, hd = q.shape
    group = hq // k.shape[1]
    out = np.empty_like(q)
    visible = (k_pos[None, :] <= q_pos[:, None]) if causal else np.ones((n, len(k_pos)), bool)
    for h in range(hq):
        kh = h // group
        s = (q[:, h, :] @ k[:, kh, :].T) / np.sqrt(hd)
        s = np.where(visible, s, -np.inf)
        s = s - s.max(axis=1, keepdims=True)
        p = np.exp(s)
        p /= p.sum(axis=1, keepdims=True)
        out[:, h, :] = p @ v[:, kh, :]
    return out


# ---------------------------------------------------------------- weights

class Weights:
    """Float64 views of the stored tensors, converted on first use.  cache=True keeps
    the float64 copies; cache="f32" keeps float32 copies (exact for bf16 and fp32
    storage) and widens them on every use, at half the memory; cache=False keeps
    nothing."""

    def __init__(self, stored: Dict[str, np.ndarray], cache=True):
        self.stored = stored
        self.cache = cache
        self._f64: Dict[str, np.ndarray] = {}

    def __getitem__(self, name: str) -> np.ndarray:
        w = self._f64.get(name)
        if w is None:
            w32 = as_f32(self.stored[name])
            if self.cache == "f32":
                self._f64[name] = w32
                return w32.astype(np.float64)
            w = w32.astype(np.float64)
            if self.cache:
                self._f64[name] = w
        elif w.dtype != np.float64:
            return w.astype(np.float64)
        return w

    def rows(self, name: str, idx) -> np.ndarray:
        return as_f32(self.stored[name][idx]).astype(np.float64)


# ---------------------------------------------------------------- state

@dataclass
class SeqState:
    """Everything one sequence carries between rounds."""
    prompt: np.ndarray
    tgt_k: np.ndarray            # [L][max_len][Hkv][hd]
    tgt_v: np.ndarray
    ctx_k: np.ndarray            # [L_D][max_len][Hkv][hd]
    ctx_v: np.ndarray
    P: int = 0                   # anchor position = number of valid target KV rows
    anchor: int = -1
    generated: List[int] = field(default_factory=list)
    budget: int = 0
    hD_prev: Optional[np.ndarray] = None   # retained [B+1][d] drafter final states
    hT_prev: Optional[np.ndarray] = None   # retained [B+1][d] target final states
    r: int = 0                   # first rejected block position of the last round
    cond_len: int = 0            # number of conditioned rows for the next draft
    seq: int = 0                 # batch position (selects the sequence's random draws)
    rnd: int = 0                 # rounds (or target-only steps) completed

    @property
    def done(self) -> bool:
        return len(self.generated) >= self.budget


@dataclass
class DraftOut:
    e: np.ndarray                # [B+1][d] plain drafter inputs
    e_tilde: np.ndarray          # [B+1][d] conditioned inputs
    h: np.ndarray                # [B+1][d] final-norm states h^D
    logits: np.ndarray           # [B+1][V]


@dataclass
class VerifyOut:
    h: np.ndarray                # [B+1][d] final-norm states h^T
    g: np.ndarray                # [B+1][n_c*d] captured conditioning-layer states
    logits: np.ndarray           # [B+1][V]


# ---------------------------------------------------------------- model

class OracleModel:
    def __init__(self, wl: Workload, stored: Dict[str, np.ndarray],
                 prec: Optional[Precision] = None, cache=True):
        self.wl = wl
        self.s = wl.target
        self.W = Weights(stored, cache)
        self.prec = prec or Precision.for_dtype(wl.dtype)
        self.eps = wl.rms_eps
        self.theta = wl.rope_theta

    # -- one decoder layer, split so the drafter can splice in its context keys
    def _qkv(self, pre: str, x: np.ndarray, pos: np.ndarray):
        s, W, P = self.s, self.W, self.prec
        n = x.shape[0]
        h = P.a(rms_norm(x, W[f"{pre}.input_norm"], self.eps))
        q = (h @ W[f"{pre}.q_proj"].T).reshape(n, s.n_q_heads, s.head_dim)
        k = (h @ W[f"{pre}.k_proj"].T).reshape(n, s.n_kv_heads, s.head_dim)
        v = (h @ W[f"{pre}.v_proj"].T).reshape(n, s.n_kv_heads, s.head_dim)
        q = P.a(apply_rope(rms_norm(q, W[f"{pre}.q_norm"], self.eps), pos, self.theta))
        k = P.a(apply_rope(rms_norm(k, W[f"{pre}.k_norm"], self.eps), pos, self.theta))
        return q, k, P.a(v)

    # -- the rest of a decoder layer, one storage point per step
    def attn_out(self, q, keys, vals, q_pos, k_pos, causal: bool) -> np.ndarray:
        """Attention output rows [n][Hq*hd], rounded to the storage type."""
        return self.prec.a(attention(q, keys, vals, q_pos, k_pos, causal)).reshape(q.shape[0], -1)

    def o_residual(self, pre: str, x, o) -> np.ndarray:
        """Residual after the attention block: x + o W_o^T."""
        return self.prec.r(x + o @ self.W[f"{pre}.o_proj"].T)

    def mlp_input(self, pre: str, x) -> np.ndarray:
        """Post-attention RMSNorm, rounded to the storage type."""
        return self.prec.a(rms_norm(x, self.W[f"{pre}.post_norm"], self.eps))

    def swiglu(self, pre: str, h) -> np.ndarray:
        """SwiGLU product silu(h W_gate^T) * (h W_up^T), rounded to the storage type."""
        W = self.W
        return self.prec.a(silu(h @ W[f"{pre}.gate_proj"].T) * (h @ W[f"{pre}.up_proj"].T))

    def down_residual(self, pre: str, x, a) -> np.ndarray:
        """Layer output: x + a W_down^T."""
        return self.prec.r(x + a @ self.W[f"{pre}.down_proj"].T)

    def _attn_mlp(self, pre: str, x, q, keys, vals, q_pos, k_pos, causal: bool):
        x = self.o_residual(pre, x, self.attn_out(q, keys, vals, q_pos, k_pos, causal))
        return self.down_residual(pre, x, self.swiglu(pre, self.mlp_input(pre, x)))

    def lm_logits(self, h: np.ndarray) -> np.ndarray:
        return self.prec.a(h) @ self.W["lm_head"].T

    def new_state(self, prompt: np.ndarray, budget: int) -> SeqState:
        s, wl = self.s, self.wl
        T = len(prompt) + budget + wl.block_size
        z = lambda L: np.zeros((L, T, s.n_kv_heads, s.head_dim))
        return SeqState(prompt=np.asarray(prompt), tgt_k=z(s.n_layers), tgt_v=z(s.n_layers),
                        ctx_k=z(wl.draft_layers), ctx_v=z(wl.draft_layers), budget=budget)

    # -- target
    def target_layer(self, st: SeqState, l: int, x: np.ndarray, pos0: int) -> np.ndarray:
        """Target decoder layer l on residual rows x at positions pos0..: writes their
        K/V into st's cache at layer l (rows at and beyond pos0 are overwritten) and
        attends causally to cache rows 0..pos.  Returns the layer's output residual."""
        n = x.shape[0]
        pos = pos0 + np.arange(n)
        pre = f"target.{l}"
        q, k, v = self._qkv(pre, x, pos)
        st.tgt_k[l, pos0:pos0 + n] = k
        st.tgt_v[l, pos0:pos0 + n] = v
        end = pos0 + n
        return self._attn_mlp(pre, x, q, st.tgt_k[l, :end], st.tgt_v[l, :end], pos,
                              np.arange(end), causal=True)

    def target_forward(self, st: SeqState, tokens, pos0: int) -> VerifyOut:
        """Run rows `tokens` at positions pos0.. through the target, writing their K/V
        into st's cache (rows at and beyond pos0 are overwritten), attending causally
        to cache rows 0..pos."""
        s, W, P = self.s, self.W, self.prec
        tokens = np.asarray(tokens)
        x = P.r(W.rows("embed", tokens))
        g = []
        for l in range(s.n_layers):
            x = self.target_layer(st, l, x, pos0)
            if l in self.wl.cond_layers:
                g.append(P.a(x))
        h = rms_norm(x, W["target.final_norm"], self.eps)
        return VerifyOut(h=h, g=np.concatenate(g, axis=-1), logits=self.lm_logits(h))

    # -- drafter
    def context_append(self, st: SeqState, g: np.ndarray, pos0: int) -> None:
        """Project captured target states g[n][n_c*d] for positions pos0.. into the
        drafter's per-layer context K/V."""
        s, W, P = self.s, self.W, self.prec
        n = g.shape[0]
        pos = pos0 + np.arange(n)
        f = P.a(rms_norm(g @ W["draft.fc"].T, W["draft.hidden_norm"], self.eps))
        for l in range(self.wl.draft_layers):
            pre = f"draft.{l}"
            k = (f @ W[f"{pre}.k_proj"].T).reshape(n, s.n_kv_heads, s.head_dim)
            v = (f @ W[f"{pre}.v_proj"].T).reshape(n, s.n_kv_heads, s.head_dim)
            st.ctx_k[l, pos0:pos0 + n] = P.a(apply_rope(rms_norm(k, W[f"{pre}.k_norm"], self.eps),
                                                       pos, self.theta))
            st.ctx_v[l, pos0:pos0 + n] = P.a(v)

    def drafter_layer(self, st: SeqState, l: int, x: np.ndarray) -> np.ndarray:
        """Drafter layer l on the block's residual rows x at positions P..P+B: queries
        attend to context rows 0..P-1 of st's drafter cache and to every block row."""
        n = x.shape[0]
        pos = st.P + np.arange(n)
        pre = f"draft.{l}"
        q, k, v = self._qkv(pre, x, pos)
        keys = np.concatenate([st.ctx_k[l, :st.P], k], axis=0)
        vals = np.concatenate([st.ctx_v[l, :st.P], v], axis=0)
        return self._attn_mlp(pre, x, q, keys, vals, pos, np.concatenate([np.arange(st.P), pos]),
                              causal=False)

    def drafter_forward(self, st: SeqState, e_tilde: np.ndarray):
        """Block of B+1 conditioned rows at positions P..P+B over context rows 0..P-1."""
        x = self.prec.r(e_tilde)
        for l in range(self.wl.draft_layers):
            x = self.drafter_layer(st, l, x)
        h = rms_norm(x, self.W["draft.final_norm"], self.eps)
        return h, self.lm_logits(h)

    def block_inputs(self, anchor: int) -> np.ndarray:
        """e_{0:B}: the anchor's embedding followed by B mask-token embeddings."""
        wl = self.wl
        toks = np.array([anchor] + [wl.mask_token_id] * wl.B)
        return self.W.rows("embed", toks)
