"""CPU oracle of one ReTrace speculative-decoding round -- TEST INFRASTRUCTURE ONLY.

A plain, slow, float64 reference of what the GPU path computes: the Qwen3-style
target, the DFlash-style block drafter, rejected-trajectory conditioning
(Eq.5-9), greedy prefix acceptance with KV rollback, and the plain target-only
greedy decode whose output the speculative loop must reproduce token for token.
Only the test suite, the smoke check and the benchmark's CPU-baseline leg may
import it; the product path never does.  It shares no code with the HIP path:
its only inputs are the seeded arrays from ``workloads``.

Parity status per part (what pins each one lives in tests/test_oracle_*.py):
  numerics, RMSNorm, RoPE, SwiGLU, attention ....... closed forms / library cross-checks
  target (Qwen3-style) forward ..................... transformers' Qwen3 on CPU, brute force
  conditioning (Eq.5-9) ............................ special-case closed forms, Fig.3 indices,
                                                     W_v = 0 and beta = 0 reductions
  ablation and low-rank conditioning forms ......... closed forms; the low-rank form (a
                                                     reading of one sentence of the paper)
                                                     is pinned only by its reduction to the
                                                     full form: parity unpinned against the
                                                     paper
  acceptance / rollback / losslessness ............. target-only greedy decode, planted drafts
  temperature sampling (sampling.py) ............... Philox4x64-10 against numpy's generator,
                                                     filtered-distribution closed forms, the
                                                     speculative-sampling rule's output
                                                     distribution (chi-square), whole rounds
  drafter internals (DFlash context pathway) ....... parity unpinned against the paper (the
                                                     paper does not define the DFlash
                                                     architecture); only internal-consistency
                                                     pins (cached vs recomputed context,
                                                     empty-context reduction to a Qwen3 layer)
"""
from .numerics import Precision, round_bf16, round_f16, round_f32
from .model import OracleModel, SeqState, DraftOut, VerifyOut
from .retrace import (align_rejected, condition_inputs, accept_length, RoundRecord,
                      OracleRunner)
from . import sampling

__all__ = ["Precision", "round_bf16", "round_f16", "round_f32", "OracleModel", "SeqState",
           "DraftOut", "VerifyOut", "align_rejected", "condition_inputs", "accept_length",
           "RoundRecord", "OracleRunner"]
