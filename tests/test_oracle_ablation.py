"""Pins of the oracle's ablation variants (Sec. "Ablation Studies"): no rotation, no
alpha-correction, binary (0/1) collisions.  Each variant is checked against a closed
form or a brute-force definition, not against its own formula."""

import numpy as np
import pytest

import workloads
from oracle import encode, quantizer, retrieve, rotation

TAU, A, _ = quantizer.lloyd_max(8)
D, B, M = 128, 16, 8


def _keys(n=400, seed=31):
    return workloads.head_keys(seed, 0, 0, n)


def test_unrotated_ids_are_the_argmax_over_omega_of_the_raw_subspaces():
    K = _keys()
    signs = workloads.rotation_signs(1)
    ids, codes, W = encode.encode(K, signs, TAU, A, B, rotate=False)
    kb = K.astype(np.float64).reshape(-1, B, M)
    u = kb / np.linalg.norm(kb, axis=2, keepdims=True)
    np.testing.assert_array_equal(ids, encode.assign_centroid_bruteforce(u))
    # the signs do not enter an unrotated encode
    ids2, codes2, W2 = encode.encode(K, -signs, TAU, A, B, rotate=False)
    np.testing.assert_array_equal(ids, ids2)
    np.testing.assert_array_equal(W.view(np.uint32), W2.view(np.uint32))


def test_unrotated_literal_and_scaled_forms_agree():
    K = _keys(300, 32)
    signs = workloads.rotation_signs(2)
    lit = encode.encode_paper(K, signs, TAU, A, B, rotate=False)
    ids, codes, W = encode.encode(K, signs, TAU, A, B, rotate=False)
    np.testing.assert_array_equal(ids, lit["ids"])
    np.testing.assert_array_equal(codes & 7, lit["bins"])
    # without the rotation the stored W is w itself
    np.testing.assert_allclose(W.astype(np.float64), lit["w"], rtol=1e-6)


def test_uncorrected_weight_is_the_rotated_subspace_norm():
    K = _keys(300, 33)
    signs = workloads.rotation_signs(3)
    _, _, W = encode.encode(K, signs, TAU, A, B, alpha_correction=False)
    y = (K.astype(np.float64) @ rotation.srht_matrix(signs).T) * np.sqrt(D)  # sqrt(D) R k = H (s (.) k)
    ref = np.linalg.norm(y.reshape(-1, B, M), axis=2)
    np.testing.assert_allclose(W.astype(np.float64), ref, rtol=2 ** -23)
    lit = encode.encode_paper(K, signs, TAU, A, B, alpha_correction=False)
    np.testing.assert_allclose(W.astype(np.float64), np.sqrt(D) * lit["w"], rtol=1e-6)


@pytest.mark.parametrize("rotate", [True, False])
def test_self_estimate_with_and_without_the_correction(rotate):
    """s_hat(k, k) = ||k||^2 exactly with the correction (q_tilde parallel to u in every
    subspace); without it s_hat(k, k) = ||k||^2 sum_b r_b^2 alpha_b, below ||k||^2 on
    average (alpha_b can exceed 1 for one key: a level a[t] may lie above |u_j|)."""
    K = _keys(60, 34)
    signs = workloads.rotation_signs(4)
    lit = encode.encode_paper(K, signs, TAU, A, B, rotate=rotate)
    _, codes, W = encode.encode(K, signs, TAU, A, B, rotate=rotate)
    _, codes_u, W_u = encode.encode(K, signs, TAU, A, B, rotate=rotate, alpha_correction=False)
    ratios = []
    for i in range(K.shape[0]):
        k = K[i]
        n2 = float(np.sum(k.astype(np.float64) ** 2))
        s = retrieve.rsqip_scores(k, codes[i:i + 1], W[i:i + 1].astype(np.float64), signs, A, B, rotate)[0]
        assert abs(s - n2) <= 1e-6 * n2
        su = retrieve.rsqip_scores(k, codes_u[i:i + 1], W_u[i:i + 1].astype(np.float64), signs, A, B, rotate)[0]
        closed = n2 * float(np.sum(lit["r"][i] ** 2 * lit["alpha"][i]))
        assert abs(su - closed) <= 1e-6 * n2
        ratios.append(su / s)
    assert np.mean(ratios) < 1.0


def test_unrotated_query_transform_and_proxy_order():
    q = workloads.head_keys(35, 0, 0, 1)[0]
    z = retrieve.query_transform(q, workloads.rotation_signs(5), rotate=False)
    np.testing.assert_array_equal(z, q.astype(np.float64) * D)
    omega = encode.centroid_set(M)
    for b in range(B):
        qb = q.astype(np.float64)[M * b:M * (b + 1)]
        ref = np.lexsort((np.arange(256), -(omega @ qb)))
        np.testing.assert_array_equal(retrieve.cluster_order(retrieve.centroid_proxy(z[M * b:M * (b + 1)])), ref)


def _head(n=1500, seed=36):
    K = workloads.head_keys(seed, 0, 0, n)
    signs = workloads.rotation_signs(seed)
    ids, codes, W = encode.encode(K, signs, TAU, A, B)
    counts = encode.cluster_counts(ids, M)
    q = workloads.needle_queries(K, seed, 0, 0, 1)[0][0]
    return K, signs, ids, codes, W, counts, q


@pytest.mark.parametrize("n_collide", [50, 300, 1500, 5000])
def test_binary_collisions_mark_the_admitted_clusters(n_collide):
    K, signs, ids, codes, W, counts, q = _head()
    z = retrieve.query_transform(q, signs)
    tiers = retrieve.collision_lut(counts, z, n_collide, M)
    binary = retrieve.collision_lut(counts, z, n_collide, M, binary=True)
    np.testing.assert_array_equal(binary, (tiers > 0).astype(np.int64))
    S = retrieve.collision_scores_from_lut(ids, binary)
    np.testing.assert_array_equal(S, retrieve.collision_scores_per_key(ids, z, n_collide, M, binary=True))
    assert S.min() >= 0 and S.max() <= B
    if n_collide >= ids.shape[0]:
        assert np.all(S == B)  # every cluster is admitted


def test_binary_collisions_brute_force_on_a_tiny_head():
    # n = 40 keys: a cluster is admitted iff fewer than C_rho keys sit in clusters ranked before it
    K, signs, ids, codes, W, counts, q = _head(40, 37)
    ids = ids.astype(np.int64)
    z = retrieve.query_transform(q, signs)
    omega = encode.centroid_set(M)
    for n_collide in (1, 7, 20, 39):
        S = np.zeros(40, dtype=np.int64)
        for b in range(B):
            prox = omega @ z[M * b:M * (b + 1)]
            for i in range(40):
                c = ids[i, b]
                before = sum(1 for j in range(40)
                             if (prox[ids[j, b]], -ids[j, b]) > (prox[c], -c))
                S[i] += 1 if before < n_collide else 0
        lut = retrieve.collision_lut(encode.cluster_counts(ids, M), z, n_collide, M, binary=True)
        np.testing.assert_array_equal(retrieve.collision_scores_from_lut(ids, lut), S)
