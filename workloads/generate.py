"""Seeded weight and prompt generators (inputs only; no model arithmetic).

Weights: every linear / embedding tensor is N(0, init_std) drawn in float32 from
numpy's PCG64, one independent stream per (seed, tensor index, chunk index), then
rounded to nearest-even bfloat16 for bf16 workloads (kept float32 for f32 ones).
RMSNorm weights are 1 ("ones") or 1 + 0.1 N(0,1) ("perturbed", used by tests so a
dropped norm-weight multiply is visible).  Prompts: per-sequence lengths uniform
in the inclusive prompt range, token ids uniform over the vocabulary.
"""
from __future__ import annotations

import concurrent.futures as _cf
import os
from typing import Dict, Iterable, List, Optional, Tuple

import numpy as np

from .configs import Workload

CHUNK = 1 << 22
PROMPT_STREAM = 1_000_000


def _layer_specs(prefix: str, s, d: int) -> List[Tuple[str, Tuple[int, ...], str]]:
    q, kv, hd, f = s.n_q_heads * s.head_dim, s.n_kv_heads * s.head_dim, s.head_dim, s.ffn
    return [
        (f"{prefix}.input_norm", (d,), "norm"),
        (f"{prefix}.q_proj", (q, d), "linear"),
        (f"{prefix}.k_proj", (kv, d), "linear"),
        (f"{prefix}.v_proj", (kv, d), "linear"),
        (f"{prefix}.q_norm", (hd,), "norm"),
        (f"{prefix}.k_norm", (hd,), "norm"),
        (f"{prefix}.o_proj", (d, q), "linear"),
        (f"{prefix}.post_norm", (d,), "norm"),
        (f"{prefix}.gate_proj", (f, d), "linear"),
        (f"{prefix}.up_proj", (f, d), "linear"),
        (f"{prefix}.down_proj", (d, f), "linear"),
    ]


LOWRANK_LATENT = 64   # rank of the rejected-suffix latents (appendix, concurrent serving)
LOWRANK_CORR = 32     # rank of the target-aware correction


def weight_specs(wl: Workload) -> List[Tuple[str, Tuple[int, ...], str]]:
    """Canonical tensor order: (name, shape [out, in], kind).  Linear weights are
    stored [out][in] row-major.  The drafter shares the target's embedding and LM
    head; the target's LM head is untied from its embedding."""
    s, d = wl.target, wl.target.hidden
    specs = [("embed", (s.vocab, d), "linear")]
    for l in range(s.n_layers):
        specs += _layer_specs(f"target.{l}", s, d)
    specs += [("target.final_norm", (d,), "norm"), ("lm_head", (s.vocab, d), "linear")]
    specs += [("draft.fc", (d, len(wl.cond_layers) * d), "linear"),
              ("draft.hidden_norm", (d,), "norm")]
    for l in range(wl.draft_layers):
        specs += _layer_specs(f"draft.{l}", s, d)
    specs += [("draft.final_norm", (d,), "norm")]
    specs += [("retrace.w_c", (d, 2 * d), "linear"), ("retrace.w_v", (d, d), "linear"),
              ("retrace.w_g", (d, 2 * d), "linear")]
    if wl.cond_mode == "lowrank":   # the low-rank conditioning path's factors
        specs += [("retrace.lr_a", (LOWRANK_LATENT, d), "linear"),
                  ("retrace.lr_c_down", (LOWRANK_CORR, 2 * d), "linear"),
                  ("retrace.lr_c_up", (LOWRANK_LATENT, LOWRANK_CORR), "linear"),
                  ("retrace.lr_v", (d, LOWRANK_LATENT), "linear"),
                  ("retrace.lr_g", (d, LOWRANK_LATENT), "linear")]
    return specs


def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round float32 to the nearest bfloat16 (ties to even); returns uint16 bit patterns."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    r = (u >> np.uint32(16)) & np.uint32(1)
    return ((u + np.uint32(0x7FFF) + r) >> np.uint32(16)).astype(np.uint16)


def bf16_bits_to_f32(b: np.ndarray) -> np.ndarray:
    return (np.asarray(b, dtype=np.uint16).astype(np.uint32) << np.uint32(16)).view(np.float32)


def as_f32(arr: np.ndarray) -> np.ndarray:
    """Float32 values of a stored tensor (bf16 bit patterns are widened exactly)."""
    return bf16_bits_to_f32(arr) if arr.dtype == np.uint16 else arr


def _normal_chunk(seed: int, t_idx: int, c_idx: int, n: int) -> np.ndarray:
    g = np.random.Generator(np.random.PCG64(np.random.SeedSequence([seed, t_idx, c_idx])))
    return g.standard_normal(n, dtype=np.float32)


def make_weights(wl: Workload, names: Optional[Iterable[str]] = None, threads: Optional[int] = None,
                 wv_zero: bool = False) -> Dict[str, np.ndarray]:
    """Generate the workload's weights (all of them, or the named subset; any subset
    equals the same tensors of the full set).  bf16 workloads return uint16 bf16 bit
    patterns, f32 workloads float32 arrays.  wv_zero=True zeroes the gated-residual
    value projection W_v, the initialisation under which the conditioned drafter
    input equals the plain one."""
    specs = weight_specs(wl)
    want = None if names is None else set(names)
    bf16 = wl.dtype == "bf16"
    out: Dict[str, np.ndarray] = {}
    jobs = []
    for t_idx, (name, shape, kind) in enumerate(specs):
        if want is not None and name not in want:
            continue
        n = int(np.prod(shape))
        arr = np.empty(n, dtype=np.uint16 if bf16 else np.float32)
        out[name] = arr
        if kind == "norm":
            if wl.norm_init == "ones":
                v = np.ones(n, dtype=np.float32)
            else:
                v = 1.0 + 0.1 * _normal_chunk(wl.seed, t_idx, 0, n)
            arr[:] = f32_to_bf16_bits(v) if bf16 else v
            continue
        if wv_zero and name == "retrace.w_v":
            arr[:] = 0
            continue
        for c_idx, lo in enumerate(range(0, n, CHUNK)):
            jobs.append((arr, t_idx, c_idx, lo, min(n, lo + CHUNK)))

    std = np.float32(wl.init_std)

    def run(job):
        arr, t_idx, c_idx, lo, hi = job
        v = _normal_chunk(wl.seed, t_idx, c_idx, hi - lo) * std
        arr[lo:hi] = f32_to_bf16_bits(v) if bf16 else v

    nthr = threads or min(16, os.cpu_count() or 1)
    if len(jobs) > 1 and nthr > 1:
        with _cf.ThreadPoolExecutor(nthr) as ex:
            list(ex.map(run, jobs))
    else:
        for j in jobs:
            run(j)
    shapes = {name: shape for name, shape, _ in specs}
    return {k: v.reshape(shapes[k]) for k, v in out.items()}


def make_prompts(wl: Workload) -> List[np.ndarray]:
    """Per-sequence prompt token ids (int32), lengths uniform in wl.prompt_len."""
    g = np.random.Generator(np.random.PCG64(np.random.SeedSequence([wl.seed, PROMPT_STREAM])))
    lo, hi = wl.prompt_len
    lens = g.integers(lo, hi, endpoint=True, size=wl.batch)
    return [g.integers(0, wl.target.vocab, size=int(n)).astype(np.int32) for n in lens]
