"""Decode-time two-stage retrieval for one query head.

Paper: Sec. "Retrieval" (coarse candidate generation, candidate reranking),
Appendix "Coarse Candidate Generation (Collision Ratio and Multi-Tier
Weights)" with Eq. collision_score and the "Top-beta selection with
small-range integer scores" paragraph, Appendix "RSQ-IP Reranking from 4-Bit
Key Summaries" (Eqs. rsqip_cosine, rsqip_raw, rsqip_raw_weighted), and
Alg. 1 (decode part).

Query transform.  q_hat = q/||q||, q_tilde = R q_hat.  With
R = H diag(s)/sqrt(D) this is q_tilde = z / (sqrt(D) ||q||), z = H (s (.) q);
z is exact in float64 for float16 q.

Stage I (readings where the paper leaves the granularity open):
  * the centroid proxy of cluster c in subspace b is <q_tilde_b, omega_c>; it
    is a positive multiple of sum_j (-1)^{bit_j(c)} z_{b,j}, an exact float64
    sum, so the cluster order is exact;
  * clusters are ranked by (proxy descending, centroid id ascending);
    P(c) = number of keys in clusters ranked before c;
  * "top clusters covering ratio rho": whole clusters are admitted while
    P(c) < C_rho, with C_rho the collision budget (ceil(rho n));
  * tiers: with percentiles (5, 15, 30, 50, 75, 100) the cut of tier l is
    ceil(pct_l C_rho / 100) (integer arithmetic); an admitted cluster takes
    the first tier whose cut exceeds P(c), with weights (6, 5, 4, 3, 2, 1);
    other clusters score 0;
  * S_i = sum_b bonus_b(id_{i,b}), an integer in [0, 6B].
Selection: C = min(n_cand, n) keys by S descending, ties at the threshold
taken in ascending key index ("deterministic truncation"); the candidate
list is returned in ascending key index.

Stage II: s_hat_i = ||q|| sum_b w_{i,b} <v_{i,b}, q_tilde_b>, with the stored
W (float32) giving w = W / sqrt(D).  Final top-k: (s_hat descending, key
index ascending); short lists are padded with index -1.

Ablation variants (Sec. "Ablation Studies"; App. "Coarse Candidate
Generation", the binary 0/1 collision the tiers replace):
  * ``binary=True``: every admitted cluster scores 1 (S_i in [0, B]);
  * ``rotate=False``: R = I, so q_tilde = q/||q||; the transform returns
    z = D q so that z / D = q keeps the scaled estimator's form, and the
    stored W of an unrotated index is w itself (no sqrt(D) factor).
"""

import numpy as np

from .encode import centroid_set, dequantize
from .rotation import fwht, srht_matrix

TIER_WEIGHTS = (6, 5, 4, 3, 2, 1)
TIER_PERCENTILES = (5, 15, 30, 50, 75, 100)


def query_transform(q, signs, rotate=True):
    """z = H (s (.) q) = sqrt(D) ||q|| q_tilde, exact in float64 for float16 q.
    Without the rotation: z = D q (exact: D is a power of two)."""
    q = np.asarray(q).astype(np.float64)
    if not rotate:
        return q * q.shape[0]
    s = np.asarray(signs, dtype=np.float64)
    return fwht(q * s)


def centroid_proxy(z_b):
    """sum_j (-1)^{bit_j(c)} z_{b,j} for every centroid c (a positive multiple of q_tilde_b . omega_c)."""
    m = z_b.shape[-1]
    return z_b @ (centroid_set(m) * np.sqrt(m)).T


def cluster_order(proxy):
    """Cluster ids ranked by (proxy descending, id ascending)."""
    ids = np.arange(proxy.shape[0])
    return np.lexsort((ids, -proxy))


def tier_cuts(n_collide):
    """Key-count cut of each tier: ceil(pct * C_rho / 100), integer arithmetic."""
    return tuple((p * int(n_collide) + 99) // 100 for p in TIER_PERCENTILES)


def tier_bonus(start, cuts, binary=False):
    """Weight of the first tier whose cut exceeds the cluster start rank, else 0.
    Binary collisions: 1 for every admitted cluster (start below C_rho)."""
    if binary:
        return 1 if start < cuts[-1] else 0
    for w, c in zip(TIER_WEIGHTS, cuts):
        if start < c:
            return w
    return 0


def collision_scores_per_key(ids, z, n_collide, m, binary=False):
    """Eq. collision_score evaluated from its definition, key by key.

    In each subspace the keys are ranked by their cluster's proxy (ties by
    cluster id, then key index); a cluster's start rank is the rank of its
    first key; every key of the cluster gets that cluster's tier bonus.
    """
    ids = np.asarray(ids, dtype=np.int64)
    n, B = ids.shape
    cuts = tier_cuts(n_collide)
    S = np.zeros(n, dtype=np.int64)
    zb = np.asarray(z, dtype=np.float64).reshape(B, m)
    keys = np.arange(n)
    for b in range(B):
        prox = centroid_proxy(zb[b])[ids[:, b]]
        order = np.lexsort((keys, ids[:, b], -prox))
        rank = np.empty(n, dtype=np.int64)
        rank[order] = keys
        start = {}
        for i in range(n):
            c = ids[i, b]
            start[c] = min(start.get(c, n), rank[i])
        bonus = {c: tier_bonus(p, cuts, binary) for c, p in start.items()}
        S += np.array([bonus[c] for c in ids[:, b]], dtype=np.int64)
    return S


def collision_lut(counts, z, n_collide, m, binary=False):
    """Per-subspace bonus table lut[b][c] from cluster counts (the form the GPU uses)."""
    counts = np.asarray(counts, dtype=np.int64)
    B = counts.shape[0]
    cuts = tier_cuts(n_collide)
    zb = np.asarray(z, dtype=np.float64).reshape(B, m)
    lut = np.zeros((B, 2 ** m), dtype=np.int64)
    for b in range(B):
        order = cluster_order(centroid_proxy(zb[b]))
        start = np.concatenate(([0], np.cumsum(counts[b][order])[:-1]))
        for c, p in zip(order, start):
            lut[b, c] = tier_bonus(p, cuts, binary)
    return lut


def collision_scores_from_lut(ids, lut):
    """S_i = sum_b lut[b][id_{i,b}]."""
    ids = np.asarray(ids, dtype=np.int64)
    B = ids.shape[1]
    return np.sum(np.asarray(lut)[np.arange(B)[None, :], ids], axis=1)


def select_candidates(S, n_cand):
    """Top-min(C, n) keys by S, ties by ascending index; returned in ascending index."""
    S = np.asarray(S, dtype=np.int64)
    n = S.shape[0]
    C = min(int(n_cand), n)
    order = np.lexsort((np.arange(n), -S))
    return np.sort(order[:C])


def selection_threshold(S, n_cand):
    """(theta, #{S > theta}, quota of S == theta keys) of the bucket selection."""
    S = np.asarray(S, dtype=np.int64)
    C = min(int(n_cand), S.shape[0])
    if C == 0:
        return None, 0, 0
    theta = int(np.sort(S)[::-1][C - 1])
    gt = int(np.sum(S > theta))
    return theta, gt, C - gt


def rsqip_scores(q, codes, W, signs, a, n_subspaces, rotate=True):
    """Eq. rsqip_raw_weighted for the keys whose (codes [c,D], W [c,B]) are given."""
    q = np.asarray(q).astype(np.float64)
    D = q.shape[0]
    B = n_subspaces
    m = D // B
    qn = np.sqrt(np.sum(q * q))
    if qn == 0:
        return np.zeros(np.asarray(codes).shape[0])
    q_tilde = (srht_matrix(signs) @ (q / qn)) if rotate else q / qn
    v = dequantize(codes, a).reshape(-1, B, m)
    w = np.asarray(W, dtype=np.float64) / (np.sqrt(D) if rotate else 1.0)
    ip = np.einsum("cbj,bj->cb", v, q_tilde.reshape(B, m))
    return qn * np.sum(w * ip, axis=1)


def topk(cand, scores, k):
    """k best (score descending, index ascending); pads with (-1, -inf)."""
    cand = np.asarray(cand, dtype=np.int64)
    scores = np.asarray(scores, dtype=np.float64)
    order = np.lexsort((cand, -scores))[:k]
    idx = np.full(k, -1, dtype=np.int64)
    sc = np.full(k, -np.inf)
    idx[:order.shape[0]] = cand[order]
    sc[:order.shape[0]] = scores[order]
    return idx, sc


def retrieve_head(q, ids, codes, W, counts, signs, a, n_subspaces,
                  n_cand, n_collide, top_k, rotate=True, binary=False):
    """Alg. 1 decode for one query head over the n keys of its KV head.

    Returns dict(z, lut, S, cand, cand_scores, idx, scores).
    """
    D = np.asarray(q).shape[0]
    m = D // n_subspaces
    z = query_transform(q, signs, rotate)
    lut = collision_lut(counts, z, n_collide, m, binary)
    S = collision_scores_from_lut(ids, lut)
    cand = select_candidates(S, n_cand)
    cs = rsqip_scores(q, np.asarray(codes)[cand], np.asarray(W)[cand], signs, a,
                      n_subspaces, rotate)
    idx, sc = topk(cand, cs, top_k)
    return dict(z=z, lut=lut, S=S, cand=cand, cand_scores=cs, idx=idx, scores=sc)


def exact_topk(K, q, k):
    """Reference TopK(q) by float64 <k_i, q>, ties -> lower index."""
    s = np.asarray(K, dtype=np.float64) @ np.asarray(q, dtype=np.float64)
    return np.lexsort((np.arange(s.shape[0]), -s))[:k]


def recall(selected, reference):
    """|selected & reference| / |reference| (ignoring -1 padding)."""
    sel = set(int(i) for i in np.asarray(selected) if i >= 0)
    ref = [int(i) for i in np.asarray(reference)]
    return len(sel.intersection(ref)) / max(1, len(ref))
