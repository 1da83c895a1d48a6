"""Error measures and bounds of the parity tests (plain NumPy; no GPU needed).

Two measures of a tensor ``got`` against the oracle's ``ref``:

* max-norm relative error ``max_i |g_i - r_i| / max_i |r_i|``;
* element-wise relative error with an RMS floor,
  ``max_i |g_i - r_i| / max(|r_i|, rms(r))`` (the floor keeps values near zero
  from dominating).

Bounds (1e-4 for float32, 2e-2 for bfloat16):

* One block on the same input (``blocks=1``): both measures at the bound.
  Derivation for bf16: an implementation that accumulates in float32 instead
  of float64 rounds the same values to bf16 at the same points, but any last
  bit of difference before a rounding point can flip that rounding by one
  unit in the last place somewhere in a large tensor. Of a block's rounding
  points, two lie on the residual path that carries the output's magnitude:
  ``H = X + O W_o^T + b_o`` and the block output ``H + MLP(H)``. One unit in
  the last place of a bf16 value is at most 2^-7 of its magnitude, so two
  flips move an output element by at most 2 x 2^-7 = 1.56e-2 of itself. The
  rest of a correct block's error (accumulation order, the softmax weights
  rounded against a different running maximum, flips at the LayerNorm,
  Q/K/V, attention-output and GELU rounding points, which enter the output
  only through a product with weights of standard deviation <= 0.08) is far
  smaller, so 2e-2 holds with room and an indexing or algebra mistake
  (a dropped key range, a wrong scale, a wrong head) does not fit under it
  (tests/test_parity_gate.py).
* A stack of ``blocks`` blocks: the max-norm bound as for one block; the
  element-wise bound grows by one block's bound per block the rows pass
  through, since each block adds at most its own flips to what it inherits
  through the residual connection (whose gain is ~1 at these weight scales).
"""
from __future__ import annotations

import numpy as np

TOL = {"fp32": 1e-4, "bf16": 2e-2}


def max_rel_err(got, ref) -> float:
    """max_i |g_i - r_i| / max_i |r_i|: relative error in the max norm."""
    got = np.asarray(got, np.float64)
    ref = np.asarray(ref, np.float64)
    if ref.size == 0:
        return 0.0
    den = np.max(np.abs(ref))
    return float(np.max(np.abs(got - ref)) / (den if den > 0 else 1.0))


def elem_rel_err(got, ref) -> float:
    """max_i |g_i - r_i| / max(|r_i|, rms(r)): element-wise relative error with an RMS floor."""
    got = np.asarray(got, np.float64)
    ref = np.asarray(ref, np.float64)
    if ref.size == 0:
        return 0.0
    rms = np.sqrt(np.mean(ref ** 2))
    den = np.maximum(np.abs(ref), rms if rms > 0 else 1.0)
    return float(np.max(np.abs(got - ref) / den))


def elem_tol(dtype: str, blocks: int) -> float:
    """Element-wise bound after ``blocks`` blocks (see the module docstring)."""
    if blocks < 1:
        raise ValueError("blocks must be >= 1")
    return TOL[dtype] * blocks


def check(got, ref, dtype: str, blocks: int):
    """(passes, max-norm error, element-wise error, element-wise bound)."""
    e1, e2 = max_rel_err(got, ref), elem_rel_err(got, ref)
    lim = elem_tol(dtype, blocks)
    return (e1 <= TOL[dtype] and e2 <= lim), e1, e2, lim
