"""Shared orthogonal rotation R, "implemented by SRHT".

Paper: Sec. "Preprocessing", step (1) Normalize & rotate, and the Appendix
remark "SRHT vs. Haar".  The paper names the transform but gives no
construction; the reading used here is one round of a subsampling-free
randomized Hadamard transform

    R = H_D diag(s) / sqrt(D),

with H_D the natural-order (Sylvester) Walsh-Hadamard matrix,
H[i, j] = (-1)^{popcount(i & j)}, and s in {+1, -1}^D random signs.  R is
orthogonal because H H^T = D I.  The signs are an input everywhere; a seeded
generator is provided (`seeded_signs`): s_j = -1 iff the top bit of the first
SplitMix64 output from state seed + j is set.
"""

import numpy as np


def hadamard(D):
    """Dense Sylvester Hadamard matrix of order D (a power of two), entries +-1."""
    if D < 1 or D & (D - 1):
        raise ValueError("D must be a power of two")
    i = np.arange(D)
    bits = np.bitwise_and.outer(i, i)
    popc = np.zeros_like(bits)
    while bits.any():
        popc += bits & 1
        bits >>= 1
    return np.where(popc % 2 == 0, 1.0, -1.0)


def srht_matrix(signs):
    """R = H diag(s) / sqrt(D) as a dense float64 matrix."""
    s = np.asarray(signs, dtype=np.float64)
    D = s.shape[0]
    return hadamard(D) * s[None, :] / np.sqrt(D)


def fwht(x):
    """Unnormalised fast Walsh-Hadamard transform along the last axis: returns H x.

    Butterflies (a, b) -> (a + b, a - b) over strides 1, 2, 4, ..., D/2 in
    natural order.  Applied to float64 copies of float16 data every partial
    sum is an integer multiple of 2^-24 below 2^47 in magnitude, so every
    addition is exact and the result does not depend on the order of the
    butterflies.
    """
    y = np.array(x, dtype=np.float64, copy=True)
    D = y.shape[-1]
    h = 1
    while h < D:
        y = y.reshape(y.shape[:-1] + (D // (2 * h), 2, h))
        a = y[..., 0, :].copy()
        b = y[..., 1, :].copy()
        y[..., 0, :] = a + b
        y[..., 1, :] = a - b
        y = y.reshape(y.shape[:-3] + (D,))
        h *= 2
    return y


_MASK64 = (1 << 64) - 1


def splitmix64(state):
    """First output of the SplitMix64 generator (Steele, Lea, Flood, "Fast
    splittable pseudorandom number generators", 2014) started at `state`:
    advance the state by the golden-ratio increment, then mix it."""
    z = (state + 0x9E3779B97F4A7C15) & _MASK64
    z = ((z ^ (z >> 30)) * 0xBF58476D1CE4E5B9) & _MASK64
    z = ((z ^ (z >> 27)) * 0x94D049BB133111EB) & _MASK64
    return z ^ (z >> 31)


def seeded_signs(seed, D):
    """s_j = -1 if bit 63 of splitmix64(seed + j) is set, else +1 (int8)."""
    return np.array([-1 if splitmix64((seed + j) & _MASK64) >> 63 else 1 for j in range(D)],
                    dtype=np.int8)
