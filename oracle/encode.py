"""Key summarisation: centroid ids, 4-bit direction codes and weights w.

Paper: Sec. "Prefill Phase" -- Preprocessing steps (1)-(3), "Assign
Directions to Centroids" (Eqs. omega_centers, dir_assign), "Low-Bit Rerank
Metadata" (Eqs. correct_term, scaling_factor); Appendix "RSQ-IP Reranking
from 4-Bit Key Summaries" Step 1 (Eq. rsqip_sign_mag_code) and Step 2
(Eq. alpha_def); Alg. 1, encode part.

Two forms are given.

``encode_paper`` takes the paper's steps literally in float64:
    k_hat = k / ||k||;  k_tilde = R k_hat;  split into B blocks of m;
    r_b = ||k_tilde_b||;  u_b = k_tilde_b / r_b;
    id_b = argmax_{omega in {+-1/sqrt m}^m} <u_b, omega>     (brute force)
    s_j = sign(u_j);  t_j = bucketize_tau(|u_j|);  v_j = s_j a[t_j]
    alpha_b = <v_b, u_b>;  w_b = ||k|| r_b / alpha_b.

``encode`` is the same computation on the scaled vector y = H (s (.) k),
which equals sqrt(D) ||k|| k_tilde: the positive factor sqrt(D) ||k|| is
never formed because every decision and output is invariant to it or
cancels it exactly:
    u_b = y_b / sqrt(S_b)            with S_b = sum_j y_{b,j}^2
    id_b bit j = [y_{b,j} < 0]       (argmax over Omega is the sign pattern)
    t_j  = #{t : y_j^2 >= tau_t^2 S_b}   (|u_j| >= tau_t, squared)
    alpha_b = A_b / sqrt(S_b)        with A_b = sum_j a[t_j] |y_{b,j}|
    w_b  = ||k|| r_b / alpha_b = S_b / (sqrt(D) A_b),  stored as W_b = sqrt(D) w_b.
y is exact in float64 (see rotation.fwht); the remaining float64 operations
are taken in a fixed order without fused multiply-adds:
    Y_j = fl(y_j * y_j);  S_b = ((Y0+Y1)+(Y2+Y3))+((Y4+Y5)+(Y6+Y7)) (generalised
    to a pairwise tree for any power-of-two m);  T_t = fl(tau_t * tau_t);
    t_j = #{t : Y_j >= fl(T_t * S_b)} (0 when S_b = 0);  A_b = same tree over fl(a[t_j] * |y_j|);
    W_b = float32(fl(S_b / A_b)).
This is the bit-exact definition the GPU encoder is compared against.

Ablation variants (Sec. "Ablation Studies", Sec. "Low-Bit Rerank Metadata"):
  * ``rotate=False`` drops the rotation (R = I): y = k, the ids are the sign
    patterns of the raw subspaces and W_b = ||k_b|| / alpha_b = w_b (the
    scale factor sqrt(D) belongs to the rotated form only);
  * ``alpha_correction=False`` drops the correction of Eq. correct_term:
    w_b = ||k|| r_b, i.e. W_b = float32(sqrt(S_b)) (IEEE square root).

Conventions (readings where the paper is silent):
  * bit j of id_b is coordinate j of subspace b, set when that coordinate is
    negative; a zero coordinate counts as positive (it is the smallest id
    among the tied argmax centroids);
  * magnitude bins are half-open [tau_t, tau_{t+1});
  * an all-zero subspace (S_b = 0) gets id 0, bins 0 and W_b = 0;
  * the 4-bit code is (sign << 3) | t with sign = 1 for negative.
"""

import numpy as np

from .rotation import fwht, srht_matrix


def _tree_sum(x):
    """Pairwise sum over the last axis (length a power of two) in fixed order."""
    while x.shape[-1] > 1:
        x = x[..., 0::2] + x[..., 1::2]
    return x[..., 0]


def centroid_set(m):
    """Omega = {+-1/sqrt(m)}^m; row c has coordinate j negative iff bit j of c is set."""
    c = np.arange(2 ** m)[:, None]
    j = np.arange(m)[None, :]
    neg = (c >> j) & 1
    return np.where(neg == 1, -1.0, 1.0) / np.sqrt(m)


def assign_centroid_bruteforce(u):
    """argmax over all of Omega of <u, omega> (Eq. dir_assign), ties -> smallest id."""
    u = np.asarray(u, dtype=np.float64)
    m = u.shape[-1]
    omega = centroid_set(m)
    return np.argmax(u @ omega.T, axis=-1)


def encode_paper(K, signs, tau, a, n_subspaces, rotate=True, alpha_correction=True):
    """Literal float64 encode of keys K [n, D].

    Returns dict with ids [n,B] (int), sign [n,D] (+-1), bins [n,D] (0..7),
    r [n,B], u [n,D], alpha [n,B], w [n,B], norm [n].
    """
    K = np.asarray(K, dtype=np.float64)
    n, D = K.shape
    B = n_subspaces
    m = D // B
    R = srht_matrix(signs) if rotate else np.eye(D)
    norm = np.sqrt(np.sum(K * K, axis=1))
    safe = np.where(norm > 0, norm, 1.0)
    k_hat = K / safe[:, None]
    k_tilde = k_hat @ R.T
    blocks = k_tilde.reshape(n, B, m)
    r = np.sqrt(np.sum(blocks * blocks, axis=2))
    u = blocks / np.where(r > 0, r, 1.0)[:, :, None]
    ids = assign_centroid_bruteforce(u)
    ids = np.where(r > 0, ids, 0)
    sgn = np.where(u < 0, -1.0, 1.0)
    bins = np.zeros(u.shape, dtype=np.int64)
    for t in tau:
        bins += (np.abs(u) >= t)
    v = sgn * np.asarray(a)[bins]
    alpha = np.sum(v * u, axis=2)
    corr = np.where(alpha != 0, alpha, 1.0) if alpha_correction else 1.0
    w = np.where(r > 0, norm[:, None] * r / corr, 0.0)
    return dict(ids=ids, sign=sgn.reshape(n, D), bins=bins.reshape(n, D), r=r,
                u=u.reshape(n, D), alpha=alpha, w=w, norm=norm)


def encode(K, signs, tau, a, n_subspaces, rotate=True, alpha_correction=True):
    """Bit-exact float64 encode of float16 keys K [n, D] (scaled form, see module doc).

    Returns (ids uint8 [n,B], codes uint8 [n,D] with (sign<<3)|t, W float32 [n,B]).
    """
    K = np.asarray(K)
    n, D = K.shape
    B = n_subspaces
    m = D // B
    s = np.asarray(signs, dtype=np.float64)
    y = (fwht(K.astype(np.float64) * s[None, :]) if rotate else K.astype(np.float64)).reshape(n, B, m)
    neg = y < 0
    ids = np.zeros((n, B), dtype=np.int64)
    for j in range(m):
        ids |= neg[:, :, j].astype(np.int64) << j
    Y = y * y
    S = _tree_sum(Y)
    T = np.asarray(tau, dtype=np.float64) * np.asarray(tau, dtype=np.float64)
    bins = np.zeros(y.shape, dtype=np.int64)
    live = (S > 0)[:, :, None]  # an all-zero subspace keeps bins 0
    for Tt in T:
        bins += (Y >= (Tt * S)[:, :, None]) & live
    lev = np.asarray(a, dtype=np.float64)[bins]
    A = _tree_sum(lev * np.abs(y))
    with np.errstate(divide="ignore", invalid="ignore"):
        if alpha_correction:
            W = np.where(S > 0, S / np.where(A > 0, A, 1.0), 0.0)
        else:
            W = np.sqrt(S)
    codes = (neg.astype(np.int64) << 3) | bins
    return (ids.astype(np.uint8), codes.reshape(n, D).astype(np.uint8),
            W.astype(np.float32))


def cluster_counts(ids, m):
    """counts[b][c] = #{i : id_{i,b} = c} over the keys given (ids [n, B])."""
    ids = np.asarray(ids, dtype=np.int64)
    B = ids.shape[1]
    out = np.zeros((B, 2 ** m), dtype=np.int64)
    for b in range(B):
        out[b] = np.bincount(ids[:, b], minlength=2 ** m)
    return out


def dequantize(codes, a):
    """v_j = s_j a[t_j] from 4-bit codes ((sign<<3)|t)."""
    codes = np.asarray(codes, dtype=np.int64)
    sgn = np.where((codes >> 3) & 1, -1.0, 1.0)
    return sgn * np.asarray(a, dtype=np.float64)[codes & 7]
