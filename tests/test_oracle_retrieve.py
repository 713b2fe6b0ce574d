"""Pins of the oracle's decode-time retrieval (Stage I, selection, RSQ-IP, top-k, attention)."""

import json
import os

import numpy as np
import pytest

import workloads
from oracle import attention, encode, quantizer, retrieve, rotation

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")
TAU, A, _ = quantizer.lloyd_max(8)


# ---------------------------------------------------------------- Stage I

def test_tier_cuts():
    assert retrieve.tier_cuts(100) == (5, 15, 30, 50, 75, 100)
    assert retrieve.tier_cuts(10) == (1, 2, 3, 5, 8, 10)
    assert retrieve.tier_cuts(16384) == (820, 2458, 4916, 8192, 12288, 16384)


def test_hand_worked_tiers_m2():
    g = json.load(open(os.path.join(GOLDEN, "tiers_m2.json")))
    z = np.array(g["z"])
    cases = [dict(n_collide=g["n_collide"], cuts=g["cuts"], lut=g["lut"])] + g["cases_more"]
    counts = np.array(g["counts"])
    for case in cases:
        assert list(retrieve.tier_cuts(case["n_collide"])) == case["cuts"]
        lut = retrieve.collision_lut(counts, z, case["n_collide"], g["m"])
        np.testing.assert_array_equal(lut, case["lut"])
        # the same scores from the per-key definition on keys laid out by the counts
        ids = np.repeat(np.arange(4), counts[0])[:, None]
        ids = ids[np.random.default_rng(0).permutation(ids.shape[0])]
        S = retrieve.collision_scores_per_key(ids, z, case["n_collide"], g["m"])
        np.testing.assert_array_equal(S, np.array(case["lut"][0])[ids[:, 0]])


def _head(n=1500, seed=11, nq=3):
    K = workloads.head_keys(seed, 0, 0, n)
    s = workloads.rotation_signs(seed)
    ids, codes, W = encode.encode(K, s, TAU, A, 16)
    Q, needles = workloads.needle_queries(K, seed, 0, 0, nq)
    return K, s, ids, codes, W, Q, needles


@pytest.mark.parametrize("n_collide", [1, 37, 300, 1500, 5000])
def test_per_key_definition_equals_lut_form(n_collide):
    K, s, ids, codes, W, Q, _ = _head()
    cnt = encode.cluster_counts(ids, 8)
    for q in Q:
        z = retrieve.query_transform(q, s)
        S1 = retrieve.collision_scores_per_key(ids, z, n_collide, 8)
        lut = retrieve.collision_lut(cnt, z, n_collide, 8)
        S2 = retrieve.collision_scores_from_lut(ids, lut)
        np.testing.assert_array_equal(S1, S2)
        assert S1.min() >= 0 and S1.max() <= 6 * 16
        if n_collide >= ids.shape[0]:
            assert S1.min() >= 16  # every cluster admitted -> at least weight 1 per subspace


def test_identical_keys_all_score_max():
    K = np.tile(workloads.head_keys(3, 0, 0, 1), (50, 1))
    s = workloads.rotation_signs(3)
    ids, _, _ = encode.encode(K, s, TAU, A, 16)
    q = workloads.head_keys(4, 0, 0, 1)[0]
    z = retrieve.query_transform(q, s)
    S = retrieve.collision_scores_per_key(ids, z, 10, 8)
    np.testing.assert_array_equal(S, 96)


def test_proxy_ranking_matches_paper_proxy():
    # ranking by the exact scaled proxy equals ranking by <q_tilde_b, omega_c>
    _, s, _, _, _, Q, _ = _head(nq=2)
    R = rotation.srht_matrix(s)
    omega = encode.centroid_set(8)
    for q in Q:
        qf = q.astype(np.float64)
        q_tilde = R @ (qf / np.linalg.norm(qf))
        z = retrieve.query_transform(q, s)
        for b in range(16):
            p_paper = omega @ q_tilde[8 * b:8 * b + 8]
            p_ours = retrieve.centroid_proxy(z[8 * b:8 * b + 8])
            np.testing.assert_allclose(p_ours / (np.sqrt(8) * np.sqrt(128) * np.linalg.norm(qf)),
                                       p_paper, atol=1e-13)
            o = retrieve.cluster_order(p_ours)
            assert np.all(np.diff(p_paper[o]) <= 1e-12)



def test_cluster_order_from_pair_representatives():
    # The query kernel ranks the 256 centroids of a subspace from one sort of 128 keys:
    # flipping every sign of centroid c gives c ^ 255 with the negated proxy, so of each
    # pair the member with the larger proxy (c itself when the proxy is 0) sorted by
    # (|proxy| desc, id asc) takes ranks 0..127 and its partner rank 255 - i.  That
    # order must be the oracle's (proxy desc, ties by the lower id), ties included.
    rng = np.random.default_rng(17)
    for trial in range(400):
        kind = trial % 4
        if kind == 0:
            zb = rng.standard_normal(8)
        elif kind == 1:
            zb = rng.integers(-2, 3, size=8).astype(np.float64)   # many exact ties and zeros
        elif kind == 2:
            zb = np.zeros(8)
            zb[rng.integers(0, 8)] = 1.0                          # half the proxies equal
        else:
            zb = np.zeros(8)                                      # every proxy 0
        prox = retrieve.centroid_proxy(zb)
        np.testing.assert_array_equal(prox[np.arange(256) ^ 255], -prox)
        reps = sorted((-abs(prox[c]), c ^ 255 if prox[c] < 0 else c) for c in range(128))
        rank = np.empty(256, dtype=np.int64)
        for i, (_, rep) in enumerate(reps):
            rank[rep] = i
            rank[rep ^ 255] = 255 - i
        np.testing.assert_array_equal(np.argsort(rank), retrieve.cluster_order(prox))

# ---------------------------------------------------------------- selection

def test_hand_worked_selection():
    g = json.load(open(os.path.join(GOLDEN, "select_small.json")))
    for case in g["cases"]:
        cand = retrieve.select_candidates(g["S"], case["C"])
        assert list(cand) == case["cand"]
        theta, gt, quota = retrieve.selection_threshold(g["S"], case["C"])
        assert theta == case["theta"]


def test_selection_properties():
    rng = np.random.default_rng(3)
    for n, C in [(1, 1), (10, 3), (1000, 100), (1000, 1000), (500, 900), (2000, 1)]:
        S = rng.integers(0, 97, size=n)
        S[rng.integers(0, n, size=n // 3)] = 40  # many ties
        cand = retrieve.select_candidates(S, C)
        assert cand.shape[0] == min(C, n)
        assert np.all(np.diff(cand) > 0)
        out = np.setdiff1d(np.arange(n), cand)
        if out.size and cand.size:
            assert S[cand].min() >= S[out].max()
            theta = S[cand].min()
            tied_out = out[S[out] == theta]
            tied_in = cand[S[cand] == theta]
            if tied_out.size:
                assert tied_in.max() < tied_out.min()


# ---------------------------------------------------------------- RSQ-IP

def test_estimator_self_inner_product_is_exact():
    # q = k: <v_b, q_tilde_b> = r_b alpha_b so s_hat = ||k||^2 sum_b r_b^2 = ||k||^2.
    K, s, ids, codes, W, _, _ = _head(300)
    lit = encode.encode_paper(K, s, TAU, A, 16)
    Wlit = np.sqrt(128) * lit["w"]
    for i in range(0, 300, 17):
        sh = retrieve.rsqip_scores(K[i], codes[i:i + 1], Wlit[i:i + 1], s, A, 16)[0]
        k = K[i].astype(np.float64)
        assert abs(sh - k @ k) <= 1e-12 * (k @ k)


def test_estimator_linear_in_q_and_zero_cases():
    K, s, ids, codes, W, Q, _ = _head(200, nq=2)
    q1, q2 = Q.astype(np.float64)
    f = lambda q: retrieve.rsqip_scores(q, codes, W, s, A, 16)
    np.testing.assert_allclose(f(q1 + q2), f(q1) + f(q2), rtol=1e-10, atol=1e-9)
    np.testing.assert_allclose(f(-2.5 * q1), -2.5 * f(q1), rtol=1e-12, atol=1e-10)
    assert np.all(f(np.zeros(128)) == 0)
    _, cz, wz = encode.encode(np.zeros((2, 128), np.float16), s, TAU, A, 16)
    assert np.all(retrieve.rsqip_scores(q1, cz, wz, s, A, 16) == 0)


def test_alignment_correction_removes_shrinkage():
    # "quantization typically shrinks this alignment, causing a systematic
    # underestimation" (Sec. Low-Bit Rerank Metadata): the corrected estimator
    # is unbiased on near-parallel pairs, the uncorrected one is biased low.
    K, s, ids, codes, W, Q, _ = _head(3000, seed=21, nq=1)
    lit = encode.encode_paper(K, s, TAU, A, 16)
    rng = np.random.default_rng(5)
    ratios_c, ratios_u = [], []
    for i in range(0, 3000, 10):
        q = K[i].astype(np.float64) + 0.5 * rng.standard_normal(128)
        exact = K[i].astype(np.float64) @ q
        c = retrieve.rsqip_scores(q, codes[i:i + 1], W[i:i + 1], s, A, 16)[0]
        Wu = np.sqrt(128) * lit["w"][i:i + 1] * lit["alpha"][i:i + 1]
        u = retrieve.rsqip_scores(q, codes[i:i + 1], Wu, s, A, 16)[0]
        ratios_c.append(c / exact)
        ratios_u.append(u / exact)
    assert abs(np.mean(ratios_c) - 1) < 2e-3
    assert np.mean(ratios_u) < 0.997


def test_estimator_tracks_exact_scores():
    K, s, ids, codes, W, Q, _ = _head(2000, nq=4)
    for q in Q:
        exact = K.astype(np.float64) @ q.astype(np.float64)
        est = retrieve.rsqip_scores(q, codes, W, s, A, 16)
        assert np.corrcoef(exact, est)[0, 1] > 0.99


# ---------------------------------------------------------------- top-k / attention

def test_topk_order_ties_and_padding():
    idx, sc = retrieve.topk([4, 9, 2, 7], [1.0, 3.0, 3.0, -1.0], 3)
    assert list(idx) == [2, 9, 4] and list(sc) == [3.0, 3.0, 1.0]
    idx, sc = retrieve.topk([5], [0.5], 3)
    assert list(idx) == [5, -1, -1]


def test_attention_closed_forms():
    v = np.arange(8.0).reshape(2, 4)
    K = np.array([[0.0, 0.0], [np.log(3.0), 0.0]])
    o = attention.sparse_attention(np.array([1.0, 0.0]), K, v, [0, 1])
    np.testing.assert_allclose(o, 0.25 * v[0] + 0.75 * v[1], rtol=1e-15)
    np.testing.assert_allclose(attention.sparse_attention([1.0, 0.0], K, v, [1, -1]), v[1])
    Ke = np.ones((5, 2))
    Ve = np.random.default_rng(0).standard_normal((5, 4))
    np.testing.assert_allclose(attention.full_attention([1.0, 2.0], Ke, Ve), Ve.mean(axis=0),
                               atol=1e-15)
    assert not attention.sparse_attention([1.0, 0.0], K, v, [-1, -1]).any()


def test_full_budget_retrieval_reproduces_full_attention():
    # C = n and k = n: the candidate set is every key, so Eq. approx_output
    # equals Eq. full_attention.
    n = 300
    K, s, ids, codes, W, Q, _ = _head(n, nq=2)
    V = workloads.head_values(11, 0, 0, n)
    cnt = encode.cluster_counts(ids, 8)
    for q in Q:
        r = retrieve.retrieve_head(q, ids, codes, W, cnt, s, A, 16, n, n, n)
        assert sorted(r["idx"]) == list(range(n))
        o1 = attention.sparse_attention(q, K, V, r["idx"], scale=1 / np.sqrt(128))
        o2 = attention.full_attention(q, K, V, scale=1 / np.sqrt(128))
        np.testing.assert_allclose(o1, o2, rtol=1e-12, atol=1e-12)


def test_needles_are_found():
    cfg = workloads.CONFIGS["tiny"]
    K, V = workloads.layer_kv(cfg)
    Q, needles = workloads.layer_queries(cfg, K)
    s = workloads.rotation_signs(cfg.seed)
    ids, codes, W = encode.encode(K[0, 0], s, TAU, A, 16)
    cnt = encode.cluster_counts(ids, 8)
    hits = 0
    for h in range(cfg.n_q_heads):
        q = Q[0, h]
        ref = retrieve.exact_topk(K[0, 0], q, cfg.top_k)
        assert needles[0, h] in ref  # the generator plants a findable needle
        r = retrieve.retrieve_head(q, ids, codes, W, cnt, s, A, 16, cfg.n_cand,
                                   cfg.n_collide, cfg.top_k)
        hits += needles[0, h] in r["idx"]
        assert retrieve.recall(r["idx"], ref) > 0.5
    assert hits == cfg.n_q_heads


def test_exact_topk_brute_force_and_ties():
    # exact_topk against a plain Python selection: scores summed term by term in float64,
    # then repeatedly the largest remaining score, the lower index on ties
    r = np.random.default_rng(5)
    K = r.standard_normal((40, 6)).astype(np.float16)
    K[7] = K[3]            # equal keys tie: the lower index comes first
    K[20] = K[3]
    q = r.standard_normal(6).astype(np.float16)
    scores = [sum(float(K[i, j]) * float(q[j]) for j in range(6)) for i in range(40)]
    left, want = list(range(40)), []
    for _ in range(12):
        best = max(left, key=lambda i: (scores[i], -i))
        want.append(best)
        left.remove(best)
    got = [int(i) for i in retrieve.exact_topk(K, q, 12)]
    assert got == want
    if 3 in want:
        assert want.index(3) < want.index(7) < want.index(20)
    # k above n returns every key, best first
    assert sorted(int(i) for i in retrieve.exact_topk(K, q, 100)) == list(range(40))


def test_recall_counts_hits_over_the_reference():
    assert retrieve.recall([4, 1, -1, -1], [1, 2, 3]) == pytest.approx(1 / 3)
    assert retrieve.recall([3, 2, 1], [1, 2, 3]) == 1.0
    assert retrieve.recall([3, 3, 3, -1], [3, 4]) == 0.5      # a repeated index counts once
    assert retrieve.recall([-1, -1], [0, 1]) == 0.0            # padding is never a hit
    assert retrieve.recall([5], []) == 0.0                     # empty reference
    assert retrieve.recall(np.array([9, 8, 7], np.int32), np.array([7, 8, 9, 10])) == 0.75
