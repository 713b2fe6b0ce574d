"""Pins of the oracle's rotation and key encoder (Sec. "Prefill Phase", Alg. 1 encode)."""

import json
import os

import numpy as np
import pytest

import workloads
from oracle import encode, quantizer, rotation

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def test_hadamard_small_and_orthogonal():
    np.testing.assert_array_equal(rotation.hadamard(2), [[1, 1], [1, -1]])
    np.testing.assert_array_equal(rotation.hadamard(4)[3], [1, -1, -1, 1])
    for D in (2, 8, 32, 128):
        H = rotation.hadamard(D)
        np.testing.assert_array_equal(H @ H.T, D * np.eye(D))


def test_srht_orthogonal_and_preserves_inner_products():
    s = workloads.rotation_signs(3)
    R = rotation.srht_matrix(s)
    np.testing.assert_allclose(R @ R.T, np.eye(128), atol=1e-14)
    rng = np.random.default_rng(0)
    x, y = rng.standard_normal((2, 128))
    assert abs((R @ x) @ (R @ y) - x @ y) < 1e-12


def test_fwht_equals_dense_and_is_exact_on_float16():
    rng = np.random.default_rng(1)
    x = rng.standard_normal((5, 128))
    np.testing.assert_allclose(rotation.fwht(x), x @ rotation.hadamard(128).T, atol=1e-12)
    # float16 inputs span the full exponent range; the transform must equal
    # exact integer arithmetic in units of 2^-24.
    k = (rng.standard_normal((50, 128)) * np.exp2(rng.integers(-20, 14, size=(50, 128)))).astype(np.float16)
    k[k == np.inf] = 60000
    k[k == -np.inf] = -60000
    ints = (k.astype(np.float64) * 2.0 ** 24).astype(np.int64)
    assert np.all(ints.astype(np.float64) == k.astype(np.float64) * 2.0 ** 24)
    H = rotation.hadamard(128).astype(np.int64)
    exact = ints @ H.T
    got = rotation.fwht(k)
    assert np.all(got * 2.0 ** 24 == exact.astype(np.float64))


def test_paper_worked_example_m3():
    g = json.load(open(os.path.join(GOLDEN, "centroid_m3.json")))
    omega = encode.centroid_set(g["m"])
    assert omega.shape == (g["n_centres"], g["m"])
    np.testing.assert_allclose(np.abs(omega), g["centre_coordinate_abs"], rtol=1e-15)
    for ex in g["examples"]:
        u = np.array(ex["u_direction"]) / np.linalg.norm(ex["u_direction"])
        c = int(encode.assign_centroid_bruteforce(u[None, :])[0])
        np.testing.assert_allclose(omega[c], ex["assigned"], rtol=1e-15)
        assert [(c >> j) & 1 for j in range(3)] == ex["id_bits_negative"]


def test_bruteforce_argmax_is_the_sign_pattern():
    rng = np.random.default_rng(2)
    u = rng.standard_normal((4000, 8))
    c = encode.assign_centroid_bruteforce(u)
    bits = sum(((u[:, j] < 0).astype(np.int64) << j) for j in range(8))
    np.testing.assert_array_equal(c, bits)


def _keys(n=600, seed=5):
    return workloads.head_keys(seed, 0, 0, n), workloads.rotation_signs(seed)


def test_literal_and_scaled_encode_agree():
    K, s = _keys()
    tau, a, _ = quantizer.lloyd_max(8)
    lit = encode.encode_paper(K, s, tau, a, 16)
    ids, codes, W = encode.encode(K, s, tau, a, 16)
    np.testing.assert_array_equal(ids, lit["ids"])
    # bins may differ only where |u_j| sits within 1e-12 of a threshold
    bins = codes & 7
    sgn = np.where(codes >> 3, -1.0, 1.0)
    np.testing.assert_array_equal(sgn, lit["sign"])
    near = np.min(np.abs(np.abs(lit["u"])[..., None] - tau[None, None, :]), axis=-1) < 1e-12
    assert np.all((bins == lit["bins"]) | near)
    assert np.sum(bins != lit["bins"]) == 0
    # W = sqrt(D) w, then rounded to float32
    np.testing.assert_allclose(W.astype(np.float64), np.sqrt(128) * lit["w"], rtol=1e-7)


def test_alpha_and_weight_definitions():
    K, s = _keys(200)
    tau, a, _ = quantizer.lloyd_max(8)
    lit = encode.encode_paper(K, s, tau, a, 16)
    u = lit["u"].reshape(-1, 16, 8)
    # u_b is a unit vector and k_tilde_b = r_b u_b recomposes ||k|| k_hat rotated
    np.testing.assert_allclose(np.sum(u * u, axis=2), 1.0, atol=1e-13)
    R = rotation.srht_matrix(s)
    kt = (K.astype(np.float64) @ R.T) / lit["norm"][:, None]
    np.testing.assert_allclose((lit["r"][:, :, None] * u).reshape(-1, 128), kt, atol=1e-13)
    # 0 < alpha <= ||v||, and w > 0
    v = encode.dequantize((np.where(lit["sign"] < 0, 8, 0) + lit["bins"]), a).reshape(-1, 16, 8)
    assert np.all(lit["alpha"] > 0)
    assert np.all(lit["alpha"] <= np.linalg.norm(v, axis=2) + 1e-15)
    assert np.all(lit["w"] > 0)


def test_encode_scale_invariance_and_zero_key():
    K, s = _keys(300)
    tau, a, _ = quantizer.lloyd_max(8)
    ids, codes, W = encode.encode(K, s, tau, a, 16)
    K2 = (K.astype(np.float32) * 4).astype(np.float16)  # exact power-of-two scaling
    ids2, codes2, W2 = encode.encode(K2, s, tau, a, 16)
    np.testing.assert_array_equal(ids, ids2)
    np.testing.assert_array_equal(codes, codes2)
    # w = ||k|| r_b / alpha_b is positively homogeneous of degree 1 in k
    np.testing.assert_array_equal(4 * W, W2)
    Z = np.zeros((3, 128), dtype=np.float16)
    idz, cz, wz = encode.encode(Z, s, tau, a, 16)
    assert not idz.any() and not cz.any() and not wz.any()


def test_cluster_counts():
    K, s = _keys(500)
    tau, a, _ = quantizer.lloyd_max(8)
    ids, _, _ = encode.encode(K, s, tau, a, 16)
    cnt = encode.cluster_counts(ids, 8)
    assert cnt.shape == (16, 256)
    np.testing.assert_array_equal(cnt.sum(axis=1), 500)
    for b in (0, 7, 15):
        for c in np.unique(ids[:, b])[:5]:
            assert cnt[b, c] == np.sum(ids[:, b] == c)


def test_seeded_signs_follow_splitmix64():
    # SplitMix64's first two outputs from state 0, as published with the generator.
    assert rotation.splitmix64(0) == 0xE220A8397B1DCDAF
    assert rotation.splitmix64(0x9E3779B97F4A7C15) == 0x6E789E6AA1B965F4
    s = rotation.seeded_signs(41, 256)
    assert s.dtype == np.int8 and set(np.unique(s)) <= {-1, 1}
    # sign j depends on seed + j only
    np.testing.assert_array_equal(rotation.seeded_signs(42, 255), s[1:])
    # balanced: over 64 seeds x 128 signs the fraction of -1 is within 4 sigma of 1/2
    frac = np.mean([rotation.seeded_signs(7000 + t, 128) == -1 for t in range(64)])
    assert abs(frac - 0.5) < 4 * 0.5 / np.sqrt(64 * 128)
