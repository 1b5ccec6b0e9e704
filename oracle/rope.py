"""Oracle: rotary position embedding (RoPE), float64.

TEST INFRASTRUCTURE ONLY (see ``oracle/__init__.py``).

The paper applies RoPE to queries and keys of every head before attention
and runs it in place, fused, to avoid the memory spike of an fp32 copy
(Section 4, "Implementation"; the embedding itself is RoFormer's).  The
definition written out here:

* A head vector x of even width d is split into d/2 coordinate pairs.  Pair
  e (0 <= e < d/2) has frequency theta_e = base^(-2e/d).
* At sequence position p the pair is rotated by the angle p * theta_e:
      y_a = x_a cos(p theta_e) - x_b sin(p theta_e)
      y_b = x_b cos(p theta_e) + x_a sin(p theta_e)
  i.e. (y_a + i y_b) = (x_a + i x_b) exp(i p theta_e).
* Pairing (reading taken here): pair e is the coordinates (e, e + d/2), the
  "rotate half" layout of the Llama-3 and Qwen-3 implementations the paper
  trains and of the fused kernel it calls.  RoFormer's own layout pairs
  (2e, 2e + 1); the two differ only by a fixed permutation of head
  coordinates, which projection weights absorb.
* The inverse (the transpose of the rotation) turns by -p theta_e; it maps a
  gradient with respect to the rotated vector back to the unrotated one.

Angles are formed as p * theta_e in float64 and reduced by numpy's cos/sin;
no table, no fp32 step.
"""

import numpy as np


def rope_theta(d, base):
    """Frequencies theta_e = base^(-2e/d), e = 0 .. d/2 - 1."""
    if d % 2:
        raise ValueError("head width must be even")
    e = np.arange(d // 2, dtype=np.float64)
    return np.float64(base) ** (-2.0 * e / d)


def rope(x, pos, base, inverse=False):
    """Rotate x [S, H, d] (float64 copy) at positions pos [S] (integers).

    Returns y [S, H, d]; with ``inverse`` the rotation by minus the angle."""
    x = np.asarray(x, np.float64)
    S, H, d = x.shape
    pos = np.asarray(pos, np.float64).reshape(S)
    ang = pos[:, None] * rope_theta(d, base)[None, :]          # [S, d/2]
    if inverse:
        ang = -ang
    c = np.cos(ang)[:, None, :]
    s = np.sin(ang)[:, None, :]
    half = d // 2
    xa, xb = x[..., :half], x[..., half:]
    return np.concatenate([xa * c - xb * s, xb * c + xa * s], axis=-1)
