"""Gaussian noise for the Value perturbation (Section 4.3, Eq. value-perturbation).

The paper draws epsilon ~ N(0, I) per (sequence i, layer l, KV head h, position u)
and names no generator.  The reading taken here is a counter-based generator so
that the GPU and this oracle can regenerate the identical draw independently:

* Philox4x32-10 (Salmon, Moraes, Dror, Shaw, "Parallel Random Numbers: As Easy
  as 1, 2, 3", SC'11): a 4x32-bit counter and a 2x32-bit key, ten rounds of two
  32x32->64 multiplications (constants 0xD2511F53 and 0xCD9E8D57) with a Weyl
  key schedule (increments 0x9E3779B9, 0xBB67AE85).
* counter = (u, g | h << 16, l, i) where g = j // 4 indexes the group of four
  coordinates j of the head_dim vector that one Philox block feeds; key = (seed
  mod 2**32, seed >> 32).  The draw does not depend on alpha (common random
  numbers across perturbation strengths).
* each 32-bit word x becomes a uniform U = (2 * (x >> 9) + 1) * 2**-24, exactly
  representable in fp32 and strictly inside (0, 1);
* Box-Muller (Box & Muller 1958): from (U0, U1) the pair
  sqrt(-2 ln U0) * (cos 2 pi U1, sin 2 pi U1) gives coordinates 4g, 4g+1, and
  (U2, U3) gives 4g+2, 4g+3.  Evaluated in float64, rounded to float32.
"""
from __future__ import annotations

import numpy as np

_M0 = np.uint64(0xD2511F53)
_M1 = np.uint64(0xCD9E8D57)
_W0 = np.uint64(0x9E3779B9)
_W1 = np.uint64(0xBB67AE85)
_MASK = np.uint64(0xFFFFFFFF)


def philox4x32_10(ctr: np.ndarray, key) -> np.ndarray:
    """Philox4x32 with 10 rounds.  ``ctr``: uint32 [..., 4]; ``key``: two uint32.

    One round maps (c0, c1, c2, c3) to
    (hi(M1*c2) ^ c1 ^ k0, lo(M1*c2), hi(M0*c0) ^ c3 ^ k1, lo(M0*c0));
    the key is bumped by the Weyl constants between rounds.
    """
    ctr = np.asarray(ctr, dtype=np.uint32)
    c0 = ctr[..., 0].astype(np.uint64)
    c1 = ctr[..., 1].astype(np.uint64)
    c2 = ctr[..., 2].astype(np.uint64)
    c3 = ctr[..., 3].astype(np.uint64)
    k0 = np.uint64(int(key[0]) & 0xFFFFFFFF)
    k1 = np.uint64(int(key[1]) & 0xFFFFFFFF)
    for r in range(10):
        if r > 0:
            k0 = (k0 + _W0) & _MASK
            k1 = (k1 + _W1) & _MASK
        p0 = _M0 * c0
        p1 = _M1 * c2
        hi0, lo0 = p0 >> np.uint64(32), p0 & _MASK
        hi1, lo1 = p1 >> np.uint64(32), p1 & _MASK
        c0, c1, c2, c3 = (hi1 ^ c1 ^ k0), lo1, (hi0 ^ c3 ^ k1), lo0
    return np.stack([c0, c1, c2, c3], axis=-1).astype(np.uint32)


def uniforms(words: np.ndarray) -> np.ndarray:
    """32-bit words -> uniforms in (0, 1), (2 * (x >> 9) + 1) * 2**-24 (exact in fp32)."""
    w = np.asarray(words, dtype=np.uint32).astype(np.float64)
    top = np.floor(w / 512.0)          # x >> 9
    return (2.0 * top + 1.0) * 2.0 ** -24


def box_muller(u: np.ndarray) -> np.ndarray:
    """[..., 4] uniforms -> [..., 4] standard normals (float64)."""
    r0 = np.sqrt(-2.0 * np.log(u[..., 0]))
    r1 = np.sqrt(-2.0 * np.log(u[..., 2]))
    t0 = 2.0 * np.pi * u[..., 1]
    t1 = 2.0 * np.pi * u[..., 3]
    return np.stack([r0 * np.cos(t0), r0 * np.sin(t0), r1 * np.cos(t1), r1 * np.sin(t1)], axis=-1)


def value_noise(seed: int, seq: int, layer: int, n_kv_heads: int, positions: np.ndarray,
                head_dim: int) -> np.ndarray:
    """epsilon[u, h, j] for the given positions u (within sequence ``seq``): float32
    [len(positions), n_kv_heads, head_dim]."""
    if head_dim % 4 != 0:
        raise ValueError("head_dim must be a multiple of 4")
    pos = np.asarray(positions, dtype=np.uint64)
    G = head_dim // 4
    h = np.arange(n_kv_heads, dtype=np.uint64)
    g = np.arange(G, dtype=np.uint64)
    ctr = np.empty((len(pos), n_kv_heads, G, 4), dtype=np.uint32)
    ctr[..., 0] = pos[:, None, None]
    ctr[..., 1] = (g[None, None, :] | (h[None, :, None] << np.uint64(16)))
    ctr[..., 2] = np.uint32(layer)
    ctr[..., 3] = np.uint32(seq)
    key = (seed & 0xFFFFFFFF, (seed >> 32) & 0xFFFFFFFF)
    z = box_muller(uniforms(philox4x32_10(ctr, key)))
    return z.reshape(len(pos), n_kv_heads, head_dim).astype(np.float32)
