"""Per-element tolerance for decode attention against the float64 oracle.

The kernels evaluate softmax attention in float32 from bfloat16 q, K and V
(every product of two bfloat16 values is exact in float32).  With u = 2^-24
(float32's unit roundoff), the error of an output element o[r, h, d] has
three sources, each scaled by a quantity the oracle returns beside the output
(``oracle.attention.decode_attention_scales``):

* Relative errors delta_t in the softmax weights move o by
  sum_t p_t delta_t (V_t,d - o_d).  For rounding errors that are independent
  across tokens, this has spread |delta| * w2, w2 = sqrt(sum p^2 (V - o)^2).
  A weight's relative error is bounded by
    - its score's error: a score is a sum of head_dim exact products reached
      through at most N_S = 16 roundings (four dot2 or MFMA accumulations,
      four cross-lane adds, the scale), each off by at most u times the sum
      of absolute products, s1, independently: spread sqrt(N_S) * u * s1;
      after normalisation by the sum of weights, twice that;
    - the exponential, the rescale factors and the scale product: 4 u;
    - in the matrix-core pass, the weight enters P.V as bf16(P) + bf16(P -
      bf16(P)), a relative 2^-16.
* The weighted sums of V and of the weights themselves accumulate in float32
  along chains of at most N_A = min(split, T) + ceil(T / split) + 64
  additions: at most one per token of a split in any lane's chain (the vector
  pass's lanes
  take split / 8 tokens or fewer; the matrix-core pass's 32-token tiles take
  split / 128 x 2 MFMAs of 32 products each), one per split in the merge,
  and 64 for the row, wave and set merges.  Every partial sum is bounded by
  w1 = sum p |V|, so rounding errors of size u per addition, independent,
  spread to u * sqrt(N_A) * w1.

The tolerance is KAPPA times the sum of the two spreads.  The rounding
errors above are bounded by, and roughly uniform within, their bounds, so
the spreads over-state a standard deviation by sqrt(3): KAPPA = 5 is about
nine standard deviations of a sum of such errors.  This is a statistical bound
and holds for the seeded random data of the tests: the rounding errors do not
correlate with V there.

The bound is tight enough to reject kernels with the errors the tests guard
against (``tests/test_oracle_attention.py`` checks, in numpy, that it rejects
weights carried as bf16(P) alone and a 32-token tile left out of a 32,000-token
request, and accepts a float32 emulation of the kernels' arithmetic).
"""

from __future__ import annotations

import numpy as np

U = 2.0 ** -24     # float32 unit roundoff (round to nearest)
P_SPLIT = 2.0 ** -16  # relative error of a weight carried as two bfloat16 parts
N_S = 16           # roundings in one score
KAPPA = 5.0


def matrix_core_pass(q_heads: int, kv_heads: int, head_dim: int) -> bool:
    """Whether the library runs pass 1 on the matrix cores for this shape."""
    return head_dim == 128 and q_heads // kv_heads == 8


def accumulation_chain(T, split: int) -> np.ndarray:
    """N_A per request: the longest chain of float32 additions an output's
    sums go through."""
    T = np.asarray(T, dtype=np.float64)
    return np.minimum(split, T) + np.ceil(T / split) + 64


def tolerance(w1, w2, s1, lens, split: int, matrix_core: bool) -> np.ndarray:
    """Per-element bound on |kernel - oracle| for outputs (n, Hq, Dh), from
    the oracle's scales w1, w2 (n, Hq, Dh), s1 (n, Hq), the requests' token
    counts and the split length the kernel ran with."""
    w1, w2, s1 = np.asarray(w1), np.asarray(w2), np.asarray(s1)
    eps_w = 2 * np.sqrt(N_S) * U * s1[:, :, None] + 4 * U + (P_SPLIT if matrix_core else 0.0)
    n_a = accumulation_chain(lens, split)[:, None, None]
    return KAPPA * (eps_w * w2 + U * np.sqrt(n_a) * w1)


def check(got, want, w1, w2, s1, lens, split: int, matrix_core: bool):
    """Assert every element is within its bound; returns (max error, max
    error / bound)."""
    got, want = np.asarray(got, dtype=np.float64), np.asarray(want, dtype=np.float64)
    tol = tolerance(w1, w2, s1, lens, split, matrix_core)
    err = np.abs(got - want)
    assert np.all(np.isfinite(got)), "non-finite output"
    ratio = err / np.maximum(tol, np.finfo(np.float64).tiny)
    worst = np.unravel_index(int(np.argmax(ratio)), ratio.shape)
    assert np.all(err <= tol), (f"element {worst}: error {err[worst]:.3e} above its bound "
                                f"{tol[worst]:.3e} (w1 {w1[worst]:.3e}, w2 {w2[worst]:.3e})")
    return float(err.max()), float(ratio.max())
