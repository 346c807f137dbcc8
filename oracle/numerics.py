"""Rounding to the storage formats of the mixed-precision contract (oracle side).

Each function takes float64 values and returns the float64 value of the nearest
representable number of the named IEEE-754 binary format, ties to even, with
gradual underflow and overflow to infinity.  The arithmetic between these
storage points stays in float64.
"""
from __future__ import annotations

from dataclasses import dataclass

import numpy as np


def _round_binary(x, sig_bits: int, emin: int, max_finite: float) -> np.ndarray:
    """Nearest value with `sig_bits` significand bits (hidden bit included) and
    smallest normal exponent `emin`; below 2**emin the spacing stays 2**(emin-sig_bits+1)."""
    x = np.asarray(x, dtype=np.float64)
    _, e = np.frexp(x)                              # |x| in [2**(e-1), 2**e)
    q = np.maximum(e - sig_bits, emin - sig_bits + 1)  # exponent of one unit in the last place
    r = np.ldexp(np.rint(np.ldexp(x, -q)), q)       # np.rint rounds half to even
    return np.where(np.abs(r) > max_finite, np.copysign(np.inf, x), r)


def round_bf16(x) -> np.ndarray:
    """bfloat16: 8 significand bits, exponent range of float32."""
    return _round_binary(x, 8, -126, float.fromhex("0x1.fe00000000000p+127"))


def round_f16(x) -> np.ndarray:
    """IEEE binary16: 11 significand bits, normal range from 2**-14 to 65504."""
    return _round_binary(x, 11, -14, 65504.0)


def round_f32(x) -> np.ndarray:
    """IEEE binary32: 24 significand bits."""
    return _round_binary(x, 24, -126, float.fromhex("0x1.fffffe0000000p+127"))


_ROUND = {"bf16": round_bf16, "f16": round_f16, "f32": round_f32,
          "f64": lambda x: np.asarray(x, dtype=np.float64)}


@dataclass(frozen=True)
class Precision:
    """Where values are stored in reduced precision.

    act:   GEMM A-operands (normed activations, attention output, SwiGLU product,
           the captured conditioning-layer states, q before attention) and the K/V cache.
    resid: the residual stream (and the conditioned drafter input it starts from).
    keep:  the retained drafter/target final states carried to the next round
           (FP16 for the bf16 models, following the paper's configuration table).
    """
    act: str = "bf16"
    resid: str = "f32"
    keep: str = "f16"

    @staticmethod
    def for_dtype(dtype: str) -> "Precision":
        if dtype == "bf16":
            return Precision("bf16", "f32", "f16")
        if dtype == "f32":
            return Precision("f32", "f32", "f32")
        if dtype == "f64":
            return Precision("f64", "f64", "f64")
        raise ValueError(dtype)

    def a(self, x):
        return _ROUND[self.act](x)

    def r(self, x):
        return _ROUND[self.resid](x)

    def k(self, x):
        return _ROUND[self.keep](x)
