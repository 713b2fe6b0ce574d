"""Pins of the oracle's decode-time KV regions and window attention (Sec. "Buffer Update")."""

import json
import os

import numpy as np
import pytest

from oracle import attention, window

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _state(R):
    return dict(sink=R.sink, retrieval=R.retrieval, local=R.local, buffer=R.buffer)


def test_hand_traced_regions():
    g = json.load(open(os.path.join(GOLDEN, "window_regions_small.json")))
    for case in g["cases"]:
        R = window.after_prefill(case["P"], case["sink"], case["local"], case["m"])
        for step in case["steps"]:
            if step["t"] > 0:
                ev = window.decode_step(R)
                assert ev == step["evicted"], (case["P"], step["t"])
            st = _state(R)
            for name in ("sink", "retrieval", "local", "buffer"):
                assert st[name] == step[name], (case["P"], step["t"], name)


@pytest.mark.parametrize("P,sink,local,m", [(2000, 128, 512, 256), (2000, 128, 512, 512), (700, 128, 512, 256),
                                            (100, 128, 512, 64), (3000, 0, 512, 1), (1000, 16, 8, 32)])
def test_region_invariants_over_a_long_decode(P, sink, local, m):
    R = window.after_prefill(P, sink, local, m)
    n_retr = len(R.retrieval)
    for t in range(1, 1500):
        before = list(R.local)
        ev = window.decode_step(R)
        T = P + t
        # the four regions tile [0, T) in order
        assert R.sink + R.retrieval + R.local + R.buffer == list(range(T))
        assert len(R.sink) == min(sink, P)
        assert len(R.buffer) == t % m and len(R.buffer) < m
        if ev:
            # Retrieval grows by exactly what was evicted: the oldest tokens of Local + Buffer
            assert ev == (before + list(range(T - m, T)))[:len(ev)]
            n_retr += len(ev)
        assert len(R.retrieval) == n_retr
        assert len(R.local) <= local
        if P >= sink + local:
            assert len(R.local) == local  # Local is always full once the prompt filled it
            if t % m == 0:
                assert len(ev) == m


def test_per_step_update_keeps_local_exact():
    # m = 1: every new token is promoted at once, so Local is always the `local` newest tokens
    R = window.after_prefill(1000, 128, 512, 1)
    for t in range(1, 300):
        ev = window.decode_step(R)
        T = 1000 + t
        assert R.local == list(range(T - 512, T)) and R.buffer == []
        assert ev == [T - 513]


def _kv(n, seed=3, D=16):
    r = np.random.default_rng(seed)
    return r.standard_normal((n, D)), r.standard_normal((n, D)), r.standard_normal(D)


def test_window_attention_with_every_retrieval_row_is_full_attention():
    K, V, q = _kv(900)
    R = window.after_prefill(600, 32, 128, 64)
    for _ in range(300):
        window.decode_step(R)
    assert R.length == 900
    o = window.window_attention(q, K, V, window.dense_rows(R), R.retrieval, scale=0.25)
    np.testing.assert_allclose(o, attention.full_attention(q, K, V, scale=0.25), rtol=1e-12, atol=1e-12)


def test_window_attention_equal_scores_average_the_values():
    K, V, _ = _kv(300)
    q = np.zeros(K.shape[1])
    dense = list(range(0, 10)) + list(range(250, 300))
    retrieved = [40, 77, -1, 123]
    o = window.window_attention(q, K, V, dense, retrieved)
    rows = dense + [40, 77, 123]
    np.testing.assert_allclose(o, V[rows].mean(axis=0), rtol=1e-13, atol=1e-13)


def test_window_attention_without_dense_rows_is_sparse_attention():
    K, V, q = _kv(200, seed=5)
    idx = [5, 17, 99, -1, 150]
    np.testing.assert_array_equal(window.window_attention(q, K, V, [], idx, 0.5),
                                  attention.sparse_attention(q, K, V, idx, 0.5))
