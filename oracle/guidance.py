"""Oracle: first-frame key enhancement (float64, plain NumPy).

TEST INFRASTRUCTURE ONLY -- see the package docstring.

Sec. 3.4 "Guidance Enhancement", Eq. (1): after the QKV projection of a
self-attention layer, the keys of the first frame's tokens are multiplied by
a step-dependent factor beta, Q and V are left as they are:

    K[:, 0:N0, :, :]  <-  beta * K[:, 0:N0, :, :],    N0 = H_patch * W_patch

(the tokens of the first latent frame come first in the [B, S, H, D] token
order).  Everything downstream of the projection then sees the scaled keys:
the block-masked attention (``attention.attention``), the pooled-score mask
predictor (``mask``) and the true block mass (``mass``) are simply applied to
``enhance_first_frame_keys(K, N0, beta)``.  Because a logit is linear in its
key, this is the same as multiplying the logits z_rc of the keys c < N0 by
beta, which is how the GPU path applies it.

The schedule of beta over sampling steps is not printed in the paper; here
beta is a plain argument (reading listed with the others in the design
notes).
"""

from __future__ import annotations

import numpy as np


def first_frame_tokens(grid) -> int:
    """N0 = H_patch * W_patch for a latent grid (T, H_patch, W_patch)."""
    _, hp, wp = grid
    return int(hp) * int(wp)


def enhance_first_frame_keys(k, n_first: int, beta: float) -> np.ndarray:
    """Eq. (1) on a copy of ``k [B, S, H, D]`` (float64)."""
    out = np.array(k, dtype=np.float64, copy=True)
    if not 0 <= n_first <= out.shape[1]:
        raise ValueError("n_first must lie in [0, S]")
    out[:, :n_first] *= float(beta)
    return out
