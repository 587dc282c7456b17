"""Budget allocation, the second half of Algorithm 1 (Section 4.4), in Python floats.

1. Min-max normalisation (Eq. sensitivity-normalization): s_hat = (s - s_min) /
   (s_max - s_min); a constant profile gives s_hat = 0 everywhere.  Algorithm 1
   adds an epsilon to the denominator; the equation does not.  ``eps`` selects
   (default 0, the equation with its constant-profile branch).
2. Exponential mapping (Eq. sensitivity-mapping): w_tilde = exp(log r * s_hat) =
   r ** s_hat, r >= 1.
3. ClipNormalize (Eq. weight-normalization): clip to [1/gamma, gamma] once, then
   rescale to mean one.  gamma <= 0 or infinite means no clipping (the paper
   gives gamma no value).
4. Integer budgets (Eq. layer-budget): b = round(B / |A| * w).  Independent
   rounding does not keep sum(b) = B (Eq. global-budget), so the default reading is
   largest-remainder apportionment: q = B w / |A| snapped to multiples of 2**-20,
   b = floor(q), then the B - sum(floor(q)) leftover units go to the largest
   fractional parts, ties to the larger s and then the lower index.  ``rounding=
   "nearest_even"`` gives the literal per-layer rounding instead.
"""
from __future__ import annotations

import math
from typing import List, Optional, Sequence, Tuple

SNAP = 2.0 ** 20


def normalize(s: Sequence[float], eps: float = 0.0) -> List[float]:
    s_min, s_max = min(s), max(s)
    if s_max == s_min:
        return [0.0 for _ in s]
    return [(x - s_min) / (s_max - s_min + eps) for x in s]


def exp_map(s_hat: Sequence[float], r: float) -> List[float]:
    lr = math.log(r)
    return [math.exp(lr * x) for x in s_hat]


def clip_normalize(w: Sequence[float], gamma: Optional[float]) -> List[float]:
    if gamma is not None and gamma > 0 and math.isfinite(gamma):
        c = [min(max(x, 1.0 / gamma), gamma) for x in w]
    else:
        c = list(w)
    mean = sum(c) / len(c)
    return [x / mean for x in c]


def integer_budgets(w: Sequence[float], s: Sequence[float], B: int, rounding: str = "largest_remainder") -> List[int]:
    n = len(w)
    q = [B * x / n for x in w]
    if rounding == "nearest_even":
        return [int(round(x)) for x in q]
    q = [math.floor(x * SNAP + 0.5) / SNAP for x in q]
    b = [int(math.floor(x)) for x in q]
    left = B - sum(b)
    order = sorted(range(n), key=lambda i: (-(q[i] - b[i]), -s[i], i))
    for k in range(left):
        b[order[k % n]] += 1
    return b


def layer_budgets(s: Sequence[float], B: int, r: float, gamma: Optional[float] = None, eps: float = 0.0,
                  rounding: str = "largest_remainder") -> Tuple[List[float], List[int]]:
    """Algorithm 1, allocation half: returns (w, b)."""
    if len(s) == 0:
        raise ValueError("empty profile")
    if r < 1.0:
        raise ValueError("r must be >= 1")
    if B < 0:
        raise ValueError("B must be >= 0")
    if gamma is not None and 0 < gamma < 1.0:
        raise ValueError("gamma must be >= 1")
    if any(not math.isfinite(x) for x in s):
        raise ValueError("non-finite sensitivity")
    w = clip_normalize(exp_map(normalize(s, eps), r), gamma)
    return w, integer_budgets(w, s, B, rounding)
