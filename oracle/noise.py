"""Coordinate-bound noise re-injection (paper Section 3.2, Stages 2 and 3;
Section 3.3.3), fp64.

TEST INFRASTRUCTURE ONLY (see the package docstring).

The paper re-injects noise that is bound to spatial coordinates when the
resolution changes (Stage 1 -> 2 into the mixed-resolution sequence, Stage
2 -> 3 into the full grid) and defers the details to prior practice.  The
reading used here:

* The noise is a fixed standard-normal field over the target (high-res)
  grid: at high-res pixel p (raster index y W_hr + x) and latent channel c it
  is eps(p, c), the same value at every re-injection.  The initial noise of
  Section 3.2 (drawn at the target resolution, then downsampled) is this
  field too.
* A low-resolution token stands for a 2x2 block of pixels; its noise is the
  sum of its four children's noise halved, which is again standard normal
  and consistent with the children (their mean, scaled to unit variance).
* Re-injection at noise level t moves the flow-matching interpolant to t:
  x <- (1 - t) x + t eps, with x the estimate of the clean latent at the
  boundary.
* eps is drawn from a counter-based generator so that any pixel's noise can
  be produced independently and identically on both sides: Philox-4x32 with
  10 rounds (Salmon, Moraes, Dror and Shaw, "Parallel random numbers: as easy
  as 1, 2, 3", SC 2011), counter (p, c // 4, 0, 0), key (seed mod 2^32,
  seed div 2^32); its four 32-bit words become four normals by the
  Box-Muller transform on pairs of uniforms u = (floor(w / 2^8) + 1/2) 2^-24
  (words 0 and 1 give channels 4j and 4j + 1 as r cos(2 pi u1) and
  r sin(2 pi u1) with r = sqrt(-2 ln u0); words 2 and 3 give 4j + 2 and
  4j + 3).
"""
from __future__ import annotations

import numpy as np

# Philox-4x32 constants (Salmon et al. 2011): round multipliers and Weyl key increments.
PHILOX_M0 = 0xD2511F53
PHILOX_M1 = 0xCD9E8D57
PHILOX_W0 = 0x9E3779B9
PHILOX_W1 = 0xBB67AE85
MASK32 = 0xFFFFFFFF


def philox4x32_10(ctr, key):
    """Philox-4x32 with 10 rounds on counters ctr [n, 4] (uint32) under the
    key (k0, k1); returns [n, 4] uint32.

    A round multiplies word 0 by M0 and word 2 by M1 (64-bit products split
    into high and low halves) and forms (hi(M1 x2) ^ x1 ^ k0, lo(M1 x2),
    hi(M0 x0) ^ x3 ^ k1, lo(M0 x0)); the key is bumped by (W0, W1) between
    rounds.
    """
    x = np.asarray(ctr, dtype=np.uint64).reshape(-1, 4) & MASK32
    x0, x1, x2, x3 = (x[:, i].copy() for i in range(4))
    k0, k1 = np.uint64(int(key[0]) & MASK32), np.uint64(int(key[1]) & MASK32)
    m0, m1 = np.uint64(PHILOX_M0), np.uint64(PHILOX_M1)
    mask, sh = np.uint64(MASK32), np.uint64(32)
    for r in range(10):
        if r:
            k0 = (k0 + np.uint64(PHILOX_W0)) & mask
            k1 = (k1 + np.uint64(PHILOX_W1)) & mask
        p0 = m0 * x0
        p1 = m1 * x2
        hi0, lo0 = p0 >> sh, p0 & mask
        hi1, lo1 = p1 >> sh, p1 & mask
        x0, x1, x2, x3 = hi1 ^ x1 ^ k0, lo1, hi0 ^ x3 ^ k1, lo0
    return np.stack([x0, x1, x2, x3], axis=1).astype(np.uint32)


def uniform24(words):
    """32-bit words -> uniforms in (0, 1): (floor(w / 2^8) + 1/2) 2^-24."""
    w = np.asarray(words, dtype=np.uint64)
    return ((w >> np.uint64(8)).astype(np.float64) + 0.5) * 2.0 ** -24


def box_muller(words):
    """[n, 4] words -> [n, 4] standard normals (pairs (0, 1) and (2, 3))."""
    u = uniform24(words)
    out = np.empty(u.shape)
    for a in (0, 2):
        r = np.sqrt(-2.0 * np.log(u[:, a]))
        th = 2.0 * np.pi * u[:, a + 1]
        out[:, a] = r * np.cos(th)
        out[:, a + 1] = r * np.sin(th)
    return out


def _key(seed: int):
    return (seed & MASK32, (seed >> 32) & MASK32)


def pixel_noise_bits(pixels, C: int, seed: int):
    """Philox words of the noise at high-res raster pixels [n]: [n, C] uint32
    (channel c is word c % 4 of counter (p, c // 4, 0, 0))."""
    if C % 4:
        raise ValueError("C must be a multiple of 4")
    p = np.asarray(pixels, dtype=np.int64).reshape(-1)
    j = np.arange(C // 4, dtype=np.int64)
    ctr = np.zeros((p.size, C // 4, 4), dtype=np.uint64)
    ctr[:, :, 0] = p[:, None]
    ctr[:, :, 1] = j[None, :]
    return philox4x32_10(ctr.reshape(-1, 4), _key(seed)).reshape(p.size, C)


def pixel_noise(pixels, C: int, seed: int):
    """eps(p, c) at high-res raster pixels [n]: [n, C] fp64."""
    bits = pixel_noise_bits(pixels, C, seed)
    return box_muller(bits.reshape(-1, 4)).reshape(bits.shape)


def block_noise(blocks, W_lr: int, C: int, seed: int):
    """Noise of low-res tokens [n] (raster index on the H_lr x W_lr grid):
    the sum of their four high-res children's noise, halved."""
    b = np.asarray(blocks, dtype=np.int64).reshape(-1)
    r, c = b // W_lr, b % W_lr
    W_hr = 2 * W_lr
    acc = np.zeros((b.size, C))
    for dr in (0, 1):
        for dc in (0, 1):
            acc += pixel_noise((2 * r + dr) * W_hr + 2 * c + dc, C, seed)
    return acc / 2.0


def halfunit_noise(pos, W_hr: int, C: int, seed: int):
    """Noise of the rows of a sequence from their positions in half units
    (frame, Y, X) = (frame, 2y, 2x): a row at even (Y, X) is the high-res
    pixel (Y / 2, X / 2); a row at odd (Y, X) = (4r + 1, 4c + 1) is the
    centre of low-res block (r, c) and takes that block's noise."""
    pos = np.asarray(pos, dtype=np.int64).reshape(-1, 3)
    Y, X = pos[:, 1], pos[:, 2]
    out = np.empty((pos.shape[0], C))
    even = (Y % 2 == 0) & (X % 2 == 0)
    odd = (Y % 2 == 1) & (X % 2 == 1)
    if not np.all(even | odd):
        raise ValueError("positions must be pixel (even, even) or block centre (odd, odd) in half units")
    if even.any():
        out[even] = pixel_noise((Y[even] // 2) * W_hr + X[even] // 2, C, seed)
    if odd.any():
        W_lr = W_hr // 2
        out[odd] = block_noise(((Y[odd] - 1) // 4) * W_lr + (X[odd] - 1) // 4, W_lr, C, seed)
    return out


def reinject(x, eps, t: float):
    """The flow-matching interpolant at noise level t: (1 - t) x + t eps."""
    return (1.0 - float(t)) * np.asarray(x, dtype=np.float64) + float(t) * np.asarray(eps, dtype=np.float64)
