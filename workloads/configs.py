"""Workload presets: model shapes, block size, batch, prompt mix and seeds.

The five named workloads follow the synthetic configurations the method is
measured on (a tiny fp32 model and Qwen3-0.6B/4B/8B/14B-shaped bf16 models);
the small extra presets exist only to keep CPU tests fast.
"""
from __future__ import annotations

import math
from dataclasses import dataclass, replace
from typing import Tuple


@dataclass(frozen=True)
class ModelShape:
    vocab: int
    hidden: int
    n_layers: int
    n_q_heads: int
    n_kv_heads: int
    head_dim: int
    ffn: int


def cond_layer_ids(n_layers: int, n_cond: int) -> Tuple[int, ...]:
    """Evenly spaced target layers whose outputs feed the drafter's context path.

    floor(linspace(1, L-2, n)): reproduces the given {1, 13, 26} for a 28-layer
    target and gives {1, 9, 17, 25, 34} for 36 layers, {1, 10, 19, 28, 38} for 40.
    """
    if n_cond == 1:
        return (1,)
    lo, hi = 1, n_layers - 2
    return tuple(math.floor(lo + (hi - lo) * i / (n_cond - 1)) for i in range(n_cond))


@dataclass(frozen=True)
class Workload:
    name: str
    dtype: str                      # "f32" or "bf16": weight / activation storage type
    target: ModelShape
    draft_layers: int
    cond_layers: Tuple[int, ...]
    block_size: int                 # rows per draft block incl. the anchor; B = block_size-1
    batch: int
    prompt_len: Tuple[int, int]     # inclusive range; equal ends = fixed length
    new_tokens: int                 # generation budget per sequence, first token included
    seed: int
    rope_theta: float = 1.0e6
    rms_eps: float = 1.0e-6
    page_size: int = 16
    beta: float = 1.0
    cond_mode: str = "retrace"      # "retrace" (corrected, gated), "raw_gated", "overwrite", "lowrank", "off"
    temperature: float = 0.0        # 0: greedy; > 0: speculative sampling with top-k / top-p
    top_k: int = 20
    top_p: float = 0.95
    sample_seed: int = 42
    init_std: float = 0.02
    norm_init: str = "ones"         # "ones" or "perturbed" (1 + 0.1 N(0,1)); tests use both

    @property
    def B(self) -> int:
        return self.block_size - 1

    @property
    def mask_token_id(self) -> int:
        return self.target.vocab - 1

    @property
    def max_prompt(self) -> int:
        return self.prompt_len[1]

    @property
    def max_seq_len(self) -> int:
        # prompt + budget + one full block of scratch rows for the last verify
        return self.prompt_len[1] + self.new_tokens + self.block_size

    def with_(self, **kw) -> "Workload":
        return replace(self, **kw)


def _qwen(vocab, hidden, layers, hq, hkv, ffn):
    return ModelShape(vocab=vocab, hidden=hidden, n_layers=layers, n_q_heads=hq,
                      n_kv_heads=hkv, head_dim=128, ffn=ffn)


PRESETS = {
    # Tiny fp32 model: 2 target layers, 1 drafter layer conditioned on layers {0,1}.
    "tiny-f32": Workload(
        name="tiny-f32", dtype="f32",
        target=ModelShape(vocab=1024, hidden=256, n_layers=2, n_q_heads=4, n_kv_heads=2,
                          head_dim=64, ffn=688),
        draft_layers=1, cond_layers=(0, 1), block_size=8, batch=1, prompt_len=(64, 64),
        new_tokens=128, seed=0),
    "qwen3-0.6b-shape": Workload(
        name="qwen3-0.6b-shape", dtype="bf16", target=_qwen(151936, 1024, 28, 16, 8, 3072),
        draft_layers=3, cond_layers=(1, 13, 26), block_size=16, batch=1,
        prompt_len=(512, 512), new_tokens=256, seed=1),
    "qwen3-4b-shape": Workload(
        name="qwen3-4b-shape", dtype="bf16", target=_qwen(151936, 2560, 36, 32, 8, 9728),
        draft_layers=5, cond_layers=cond_layer_ids(36, 5), block_size=16, batch=1,
        prompt_len=(4096, 4096), new_tokens=512, seed=2),
    "qwen3-8b-shape-b8": Workload(
        name="qwen3-8b-shape-b8", dtype="bf16", target=_qwen(151936, 4096, 36, 32, 8, 12288),
        draft_layers=5, cond_layers=cond_layer_ids(36, 5), block_size=16, batch=8,
        prompt_len=(1024, 8192), new_tokens=256, seed=3),
    "qwen3-14b-shape-b16": Workload(
        name="qwen3-14b-shape-b16", dtype="bf16", target=_qwen(151936, 5120, 40, 40, 8, 17408),
        draft_layers=5, cond_layers=cond_layer_ids(40, 5), block_size=16, batch=16,
        prompt_len=(8192, 16384), new_tokens=128, seed=4),
    # Concurrent serving at the Qwen3-4B shape (Appendix, concurrent serving): short
    # math-word-problem prompts (96..320 tokens), up to 1024 new tokens, 16-token blocks;
    # the batch (client concurrency 1..32) is set per run.
    "qwen3-4b-serve": Workload(
        name="qwen3-4b-serve", dtype="bf16", target=_qwen(151936, 2560, 36, 32, 8, 9728),
        draft_layers=5, cond_layers=cond_layer_ids(36, 5), block_size=16, batch=1,
        prompt_len=(96, 320), new_tokens=1024, seed=5),
    # Small bf16 models for fast CPU/GPU tests (not measured workloads).
    "mini-bf16": Workload(
        name="mini-bf16", dtype="bf16",
        target=ModelShape(vocab=2048, hidden=256, n_layers=3, n_q_heads=4, n_kv_heads=2,
                          head_dim=64, ffn=512),
        draft_layers=2, cond_layers=(0, 1, 2), block_size=16, batch=1, prompt_len=(40, 40),
        new_tokens=48, seed=7),
    "mini-bf16-ragged": Workload(
        name="mini-bf16-ragged", dtype="bf16",
        target=ModelShape(vocab=2048, hidden=256, n_layers=3, n_q_heads=8, n_kv_heads=2,
                          head_dim=64, ffn=512),
        draft_layers=2, cond_layers=(0, 2), block_size=16, batch=3, prompt_len=(17, 70),
        new_tokens=40, seed=8),
    # Four sequences (64 round rows) over a 1024-wide model: the mid-size GEMM path with
    # k slabs (reductions of 32..64 k tiles), including the fp32-operand conditioning GEMMs
    "mini-bf16-b4": Workload(
        name="mini-bf16-b4", dtype="bf16",
        target=ModelShape(vocab=2048, hidden=1024, n_layers=2, n_q_heads=8, n_kv_heads=2,
                          head_dim=128, ffn=2048),
        draft_layers=1, cond_layers=(0, 1), block_size=16, batch=4, prompt_len=(30, 90),
        new_tokens=40, seed=10),
    # Six ragged sequences (96 round rows): every round GEMM on the mid-size kernel (q|k|v
    # k-slab partials summed by qkv_post, deferred o / down slabs folded by the norm,
    # fp32-operand conditioning GEMMs), batched conditioning gathers and one attention
    # row block per sequence and KV head
    "mini-bf16-b6": Workload(
        name="mini-bf16-b6", dtype="bf16",
        target=ModelShape(vocab=2048, hidden=512, n_layers=2, n_q_heads=8, n_kv_heads=2,
                          head_dim=64, ffn=1024),
        draft_layers=2, cond_layers=(0, 1), block_size=16, batch=6, prompt_len=(20, 200),
        new_tokens=40, seed=12),
    # Ten sequences (160 round rows: 256-row tiles of the mid-size kernel with the fragment
    # double buffer) at widths with odd k-tile counts (hidden 544 = 17 k tiles, FFN 1040
    # padded to 33), so that k walks and k slabs of odd length end on the single step
    "mini-bf16-odd": Workload(
        name="mini-bf16-odd", dtype="bf16",
        target=ModelShape(vocab=2048, hidden=544, n_layers=2, n_q_heads=4, n_kv_heads=2,
                          head_dim=64, ffn=1040),
        draft_layers=1, cond_layers=(0, 1), block_size=16, batch=10, prompt_len=(20, 80),
        new_tokens=40, seed=13),
    # Width 4096 at batch 1 (as the Qwen3-8B shape): the LM head stages 128 KiB of
    # activations per workgroup; q and kv widths below the model width
    "mini-bf16-w4096": Workload(
        name="mini-bf16-w4096", dtype="bf16",
        target=ModelShape(vocab=2048, hidden=4096, n_layers=2, n_q_heads=4, n_kv_heads=2,
                          head_dim=128, ffn=512),
        draft_layers=1, cond_layers=(0, 1), block_size=16, batch=1, prompt_len=(40, 40),
        new_tokens=40, seed=11),
    # GQA group of 5 (80 query rows per 16-token block, as at the Qwen3-14B shape), hd 128
    "mini-bf16-gqa5": Workload(
        name="mini-bf16-gqa5", dtype="bf16",
        target=ModelShape(vocab=2048, hidden=256, n_layers=2, n_q_heads=10, n_kv_heads=2,
                          head_dim=128, ffn=512),
        draft_layers=1, cond_layers=(0, 1), block_size=16, batch=2, prompt_len=(90, 150),
        new_tokens=40, seed=9),
}


def get(name: str, **overrides) -> Workload:
    wl = PRESETS[name]
    return wl.with_(**overrides) if overrides else wl
