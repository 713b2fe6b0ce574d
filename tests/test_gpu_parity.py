"""GPU parity of the HIP path (through the C ABI) with the CPU oracle.

Bit-exact: centroid ids, 4-bit codes, W, cluster counts, the query transform
rounded to float, the bonus tables, collision scores, the selection threshold
and the candidate lists.  Within the stated tolerances: RSQ-IP estimates,
the top-k sets and the attention output (see tests/parity.py)."""

import numpy as np
import pytest
import torch

import paper_2602_07721_amd as pk
import workloads
from oracle import attention as oatt
from oracle import retrieve as oret

from parity import (SLOT, GpuRun, check_attention, check_head, check_index, decode_rec,
                    oracle_group)

pytestmark = pytest.mark.gpu
SCALE = 1.0 / np.sqrt(128.0)


def _inputs(cfg, n=None, batch=None, step=0):
    n = cfg.n if n is None else n
    wc = workloads.Config(**{**cfg.__dict__, "n": n, "batch": batch or cfg.batch})
    K, V = workloads.layer_kv(wc)
    Q, needles = workloads.layer_queries(wc, K, step=step)
    return wc, K, V, Q, needles, workloads.rotation_signs(cfg.seed)


def _full_check(wc, K, V, Q, signs, budget, capacity=None, attention=True):
    run = GpuRun(K, V, Q, signs, wc.q_per_kv, budget, SCALE, capacity=capacity).retrieve()
    inter = run.intermediates()
    o_gpu = run.attend() if attention else None
    gids, grec, gcnt = run.host_index()
    b, hkv, n, _ = K.shape
    results = {}
    for s in range(b):
        for h in range(hkv):
            orc = oracle_group(K[s, h], signs)
            check_index(gids[s, h], grec[s, h], gcnt[s, h], orc)
            for g in range(wc.q_per_kv):
                hq = h * wc.q_per_kv + g
                r = check_head(inter, s, h, g, wc.q_per_kv, Q[s, hq], orc, signs, budget, n)
                if attention:
                    check_attention(o_gpu[s, hq], Q[s, hq], K[s, h], V[s, h], inter["idx"][s, hq], SCALE)
                results[(s, hq)] = r
    return run, inter, results


def test_tiny_single_head_full_pipeline():
    cfg = workloads.CONFIGS["tiny"]
    wc, K, V, Q, needles, signs = _inputs(cfg)
    print(f"case tiny n={wc.n}", flush=True)
    budget = pk.Budget(cfg.n_cand, cfg.n_collide, cfg.top_k)
    run, inter, res = _full_check(wc, K, V, Q, signs, budget)
    hits = sum(int(needles[0, h]) in set(inter["idx"][0, h].tolist()) for h in range(wc.n_q_heads))
    assert hits == wc.n_q_heads


def test_layer32k_all_heads():
    cfg = workloads.CONFIGS["layer32k"]
    wc, K, V, Q, needles, signs = _inputs(cfg)
    print(f"case layer32k n={wc.n}", flush=True)
    budget = pk.Budget(cfg.n_cand, cfg.n_collide, cfg.top_k)
    _full_check(wc, K, V, Q, signs, budget)


EDGE = [
    # name, batch, hkv, G, n, (C, C_rho, k)
    ("n1", 1, 1, 4, 1, (512, 1024, 64)),
    ("n_below_C", 1, 2, 4, 100, (512, 1024, 64)),
    ("k_eq_C_eq_n", 1, 1, 4, 64, (64, 64, 64)),
    ("ragged_two_chunks", 1, 1, 4, 4099, (512, 1024, 64)),
    ("g3_batch2", 2, 2, 3, 9000, (700, 1500, 100)),
    ("g6_two_quads", 1, 2, 6, 5000, (400, 800, 50)),
    ("g1", 1, 3, 1, 3001, (300, 300, 30)),
    ("tiny_collide_budget", 1, 1, 4, 2000, (200, 1, 20)),
    ("collide_budget_above_n", 1, 1, 4, 2000, (200, 100000, 20)),
    ("k_odd_ragged", 1, 1, 2, 777, (333, 555, 77)),
    ("big_C", 1, 1, 2, 40000, (10000, 20000, 300)),         # two-pass top-k: 3 slices of 4096
    ("huge_C", 1, 1, 1, 70000, (40000, 60000, 2048)),       # 10 slices, final pass over 20480 winners
    ("C_20000", 1, 1, 2, 40000, (20000, 30000, 1000)),      # 5 slices, final pass over 5000
    ("many_chunks", 1, 1, 1, 300000, (4096, 8192, 256)),    # 74 chunks: multi-wave chunk prefix
    # the threshold kernel loads 2, 4, 8 or 16 chunks per wave and round: 49 chunks take
    # the 4-chunk form; past 256 chunks the 16-chunk form loops and re-reads the chunk
    # counts at theta from memory
    ("chunks_49", 1, 1, 2, 200000, (2048, 4096, 128)),
    # 64 chunks, the most whose bases one wave scans from the loaded registers
    ("chunks_64_ragged", 1, 1, 1, 262000, (4096, 8192, 256)),
    ("chunks_269_two_rounds", 1, 1, 1, 1100000, (8192, 16384, 256)),
    # fewer than 32 score rows (quads of query heads): the scan keeps its plain block order
    ("rows8_ragged", 1, 8, 4, 5000, (512, 1024, 64)),
    ("rows8_two_quads_ragged", 1, 4, 8, 4099, (300, 700, 40)),
    ("rows16_one_chunk", 2, 8, 3, 100, (64, 80, 16)),
    # 32 or more score rows, a multiple of 8: the scan hands each XCD whole rows
    # (rows = x mod 8), here with a ragged last chunk
    ("rows32_xcd_ragged", 4, 8, 4, 5000, (512, 1024, 64)),
    ("rows32_two_quads_3key_tail", 4, 4, 8, 4099, (300, 700, 40)),
    ("rows48_partial_quads_ragged", 3, 8, 6, 9000, (700, 1500, 100)),
]


@pytest.mark.parametrize("name,batch,hkv,G,n,bud", EDGE, ids=[e[0] for e in EDGE])
def test_edge_shapes(name, batch, hkv, G, n, bud):
    print(f"case {name} batch={batch} hkv={hkv} G={G} n={n} budget={bud}", flush=True)
    wc = workloads.Config(name, batch=batch, n_kv_heads=hkv, q_per_kv=G, n=n, n_cand=bud[0],
                          n_collide=bud[1], top_k=bud[2], seed=101 + len(name))
    K, V = workloads.layer_kv(wc)
    Q, _ = workloads.layer_queries(wc, K)
    signs = workloads.rotation_signs(wc.seed)
    _full_check(wc, K, V, Q, signs, pk.Budget(*bud), capacity=n + 37)


RECOUNT = [
    # name, batch, hkv, G, n, (C, C_rho, k)
    ("ragged_two_chunks", 1, 1, 4, 4099, (512, 1024, 64)),
    ("g6_two_quads", 1, 2, 6, 5000, (400, 800, 50)),
    ("k_odd_ragged", 1, 1, 2, 777, (333, 555, 77)),
    ("many_chunks", 1, 1, 1, 300000, (4096, 8192, 256)),
    ("rows32_xcd_ragged", 4, 8, 4, 5000, (512, 1024, 64)),
]


@pytest.mark.parametrize("name,batch,hkv,G,n,bud", RECOUNT, ids=[e[0] for e in RECOUNT])
def test_exact_recount_path(name, batch, hkv, G, n, bud):
    # With PARISKV_EXACT_RECOUNT the scan histograms nothing and every threshold comes
    # from the recount over the stored scores: the oracle must still match in full,
    # and the outputs must equal those of the ordinary call bit for bit.
    print(f"case recount {name} batch={batch} hkv={hkv} G={G} n={n} budget={bud}", flush=True)
    wc = workloads.Config(name, batch=batch, n_kv_heads=hkv, q_per_kv=G, n=n, n_cand=bud[0],
                          n_collide=bud[1], top_k=bud[2], seed=101 + len(name))
    K, V = workloads.layer_kv(wc)
    Q, _ = workloads.layer_queries(wc, K)
    signs = workloads.rotation_signs(wc.seed)
    run, inter, _ = _full_check(wc, K, V, Q, signs, pk.Budget(*bud, flags=pk.EXACT_RECOUNT), capacity=n + 37)
    assert np.all(inter["thresh"][..., 5] == 1)
    plain = GpuRun(K, V, Q, signs, G, pk.Budget(*bud), SCALE, capacity=n + 37).retrieve()
    pi = plain.intermediates()
    for k in ("cand", "cand_score", "idx", "score"):
        np.testing.assert_array_equal(inter[k].view(np.uint32), pi[k].view(np.uint32))
    np.testing.assert_array_equal(inter["thresh"][..., :4], pi["thresh"][..., :4])


@pytest.mark.parametrize("n,bud", [(12000, (10000, 20000, 300)), (24000, (20000, 30000, 600))],
                         ids=["C10000_16_per_thread", "C20000_32_per_thread"])
def test_many_rows_one_pass_top_k(n, bud):
    # 256 score rows (2 sequences x 32 KV heads x 4 query heads): candidate lists of
    # 8193..32768 go through the one-pass top-k with 16 or 32 keys per thread.  Three
    # whole groups through the oracle, invariants on every head.
    wc = workloads.Config("rows256", batch=2, n_kv_heads=32, q_per_kv=4, n=n, n_cand=bud[0],
                          n_collide=bud[1], top_k=bud[2], seed=131)
    print(f"case many rows n={n} budget={bud}", flush=True)
    K, V = workloads.layer_kv(wc, threads=16)
    Q, _ = workloads.layer_queries(wc, K)
    signs = workloads.rotation_signs(wc.seed)
    budget = pk.Budget(*bud)
    run = GpuRun(K, V, Q, signs, 4, budget, SCALE)
    assert pk.workspace_layout(run.cfg, 2, n, budget)["topk_parts"] == 1
    o_gpu = run.retrieve_attend()
    inter = run.intermediates()
    gids, grec, gcnt = run.host_index()
    for s, h in ((0, 0), (1, 17), (1, 31)):
        orc = oracle_group(K[s, h], signs)
        check_index(gids[s, h], grec[s, h], gcnt[s, h], orc)
        for g in range(4):
            check_head(inter, s, h, g, 4, Q[s, h * 4 + g], orc, signs, budget, n)
            check_attention(o_gpu[s, h * 4 + g], Q[s, h * 4 + g], K[s, h], V[s, h], inter["idx"][s, h * 4 + g], SCALE)
    C = budget.n_cand
    cand = inter["cand"][:, :, :C]
    assert np.all(np.diff(cand, axis=-1) > 0) and np.all(np.diff(inter["idx"], axis=-1) > 0)
    # every head's winners are among its candidates, with estimates no lower than any
    # candidate left out (ties at the k-th estimate aside)
    for c_row, i_row, e_row, s_row in zip(cand.reshape(-1, C), inter["idx"].reshape(-1, budget.top_k),
                                          inter["cand_score"][:, :, :C].reshape(-1, C),
                                          inter["score"].reshape(-1, budget.top_k)):
        win = np.isin(c_row, i_row)
        assert win.sum() == budget.top_k
        assert e_row[~win].max() <= s_row.min()


def test_degenerate_keys_and_queries():
    # duplicates (ties in S and in the estimates), zero keys, a zero query,
    # and one giant cluster (positive multiples of one key).
    wc = workloads.Config("degenerate", batch=1, n_kv_heads=2, q_per_kv=4, n=3000, n_cand=300,
                          n_collide=600, top_k=40, seed=77)
    K, V = workloads.layer_kv(wc)
    K[0, 0, 1000:1500] = K[0, 0, 10]                 # 500 identical keys
    K[0, 0, 1500:1520] = 0                            # zero keys
    base = K[0, 1, 5].astype(np.float32)
    K[0, 1] = (base[None, :] * np.linspace(0.5, 2.0, 3000, dtype=np.float32)[:, None]).astype(np.float16)
    Q, _ = workloads.layer_queries(wc, K)
    Q[0, 1] = 0                                       # zero query
    Q[0, 2] = K[0, 0, 10]                             # query equal to the duplicated key
    signs = workloads.rotation_signs(wc.seed)
    print("case degenerate", flush=True)
    _full_check(wc, K, V, Q, signs, pk.Budget(300, 600, 40))


def test_keys_spanning_the_float16_range():
    # Key coordinates from the subnormals to 65504 in one key: the float64 transform,
    # codes, weights and collision scores must still match the oracle bit for bit.
    wc = workloads.Config("wide_range", batch=1, n_kv_heads=2, q_per_kv=4, n=2500, n_cand=250,
                          n_collide=500, top_k=32, seed=91)
    rng = np.random.default_rng(91)
    K = rng.standard_normal((1, 2, wc.n, 128)) * np.exp2(rng.integers(-26, 16, size=(1, 2, wc.n, 128)))
    K = np.clip(K, -65504.0, 65504.0).astype(np.float16)
    K[0, 0, :50] = np.float16(65504.0)      # the largest finite value in every coordinate
    K[0, 1, :50] = np.float16(2.0 ** -24)   # the smallest subnormal
    V = rng.standard_normal((1, 2, wc.n, 128)).astype(np.float16)
    Q = rng.standard_normal((1, 8, 128)).astype(np.float16)
    signs = workloads.rotation_signs(wc.seed)
    print("case wide_range", flush=True)
    _full_check(wc, K, V, Q, signs, pk.Budget(250, 500, 32), attention=False)


def test_full_budget_reproduces_full_attention():
    # C = n and k = n: every key is selected, so the sparse output is full attention.
    wc = workloads.Config("full", batch=1, n_kv_heads=2, q_per_kv=4, n=512, n_cand=512,
                          n_collide=512, top_k=512, seed=9)
    K, V = workloads.layer_kv(wc)
    Q, _ = workloads.layer_queries(wc, K)
    signs = workloads.rotation_signs(wc.seed)
    print("case full-budget", flush=True)
    run = GpuRun(K, V, Q, signs, 4, pk.Budget(512, 512, 512), SCALE).retrieve()
    o = run.attend()
    idx = run.out_idx.cpu().numpy()
    for hq in range(8):
        assert sorted(idx[0, hq].tolist()) == list(range(512))
        ref = oatt.full_attention(Q[0, hq], K[0, hq // 4], V[0, hq // 4], scale=SCALE)
        d = np.abs(o[0, hq] - ref)
        assert d.max() <= 2e-3 * np.abs(ref).max()


def test_repeat_runs_are_bit_identical():
    cfg = workloads.CONFIGS["layer32k"]
    wc, K, V, Q, _, signs = _inputs(cfg, n=20000)
    print("case determinism", flush=True)
    budget = pk.Budget(cfg.n_cand, cfg.n_collide, cfg.top_k)
    run = GpuRun(K, V, Q, signs, wc.q_per_kv, budget, SCALE).retrieve()
    a = run.intermediates()
    oa = run.attend()
    ids_a, rec_a, cnt_a = run.host_index()
    pk.encode(run.cfg, run.index, run.K)
    run.retrieve()
    b = run.intermediates()
    ob = run.attend()
    ids_b, rec_b, cnt_b = run.host_index()
    # S rows are padded to a multiple of 64; only the first n entries are defined.
    np.testing.assert_array_equal(a["S"][..., :run.n], b["S"][..., :run.n])
    for k in ("lut", "thresh", "cand", "cand_score", "idx", "score"):
        np.testing.assert_array_equal(a[k], b[k])
    np.testing.assert_array_equal(oa, ob)
    np.testing.assert_array_equal(ids_a, ids_b)
    np.testing.assert_array_equal(rec_a, rec_b)
    np.testing.assert_array_equal(cnt_a, cnt_b)


def test_append_equals_bulk_encode():
    wc = workloads.Config("append", batch=2, n_kv_heads=2, q_per_kv=4, n=3000, n_cand=256,
                          n_collide=512, top_k=32, seed=55)
    K, V = workloads.layer_kv(wc)
    Q, _ = workloads.layer_queries(wc, K)
    signs = workloads.rotation_signs(wc.seed)
    print("case append", flush=True)
    budget = pk.Budget(256, 512, 32)
    bulk = GpuRun(K, V, Q, signs, 4, budget, SCALE).retrieve()
    inc = GpuRun(K[:, :, :2000].copy(), V, Q, signs, 4, budget, SCALE, capacity=3000)
    n_cur = 2000
    for t in (1, 1, 5, 300, 693):
        chunk = torch.from_numpy(np.ascontiguousarray(K[:, :, n_cur:n_cur + t])).cuda()
        pk.append(inc.cfg, inc.index, chunk, n_cur)
        n_cur += t
    assert n_cur == 3000
    inc.n = 3000
    inc.retrieve()
    for x, y in zip(bulk.host_index(), inc.host_index()):
        np.testing.assert_array_equal(x, y)
    a, b = bulk.intermediates(), inc.intermediates()
    np.testing.assert_array_equal(a["S"][..., :3000], b["S"][..., :3000])
    for k in ("lut", "cand", "idx", "score"):
        np.testing.assert_array_equal(a[k], b[k])


def test_streaming_decode_steps_match_the_oracle():
    # Prefill, then decode steps that append 1..55 keys per (sequence, KV head) and
    # retrieve with budgets that grow with n: every step is checked in full against
    # the oracle run on all keys cached so far.
    wc = workloads.Config("stream", batch=1, n_kv_heads=2, q_per_kv=4, n=2600, n_cand=1,
                          n_collide=1, top_k=32, seed=66)
    K, V = workloads.layer_kv(wc)
    signs = workloads.rotation_signs(wc.seed)
    n0 = 2500
    print("case streaming decode", flush=True)
    run = GpuRun(K[:, :, :n0].copy(), V, K[:, :, 0, :].repeat(4, axis=1), signs, 4,
                 pk.Budget(1, 1, 1), SCALE, capacity=wc.n)
    run.K = torch.from_numpy(np.ascontiguousarray(K)).cuda()  # attention reads the full cache
    n_cur = n0
    for step, t in enumerate((1, 3, 1, 40, 55)):
        chunk = torch.from_numpy(np.ascontiguousarray(K[:, :, n_cur:n_cur + t])).cuda()
        pk.append(run.cfg, run.index, chunk, n_cur)
        n_cur += t
        C = -(-n_cur // 8)
        budget = pk.Budget(C, 2 * C, 32)
        Kc = np.ascontiguousarray(K[:, :, :n_cur])
        Q, _ = workloads.layer_queries(wc, Kc, step=step)
        run.Q = torch.from_numpy(np.ascontiguousarray(Q)).cuda()
        run.budget, run.n = budget, n_cur
        run.retrieve()
        inter = run.intermediates()
        o_gpu = run.attend()
        gids, grec, gcnt = run.host_index()
        for h in range(wc.n_kv_heads):
            orc = oracle_group(Kc[0, h], signs)
            check_index(gids[0, h], grec[0, h], gcnt[0, h], orc)
            for g in range(wc.q_per_kv):
                hq = h * wc.q_per_kv + g
                check_head(inter, 0, h, g, wc.q_per_kv, Q[0, hq], orc, signs, budget, n_cur)
                check_attention(o_gpu[0, hq], Q[0, hq], Kc[0, h], V[0, h, :n_cur], inter["idx"][0, hq],
                                SCALE)
    assert n_cur == wc.n


def test_drift_decode_at_full_width_sampled():
    # The drift workload at its own width (4 sequences x 8 KV heads x 4 query heads, a
    # 32768-key prefill) after appends of 1, 255 and 256 drifted keys, retrieved and
    # attended with the fused call and C = ceil(n/16): two whole groups through the
    # oracle (grown index, Stage I/II, top-k, attention), invariants on every head.
    wc = workloads.CONFIGS["drift"]
    total = wc.extra["decode_steps"]
    extra = 512
    print("case drift full width", flush=True)
    K0, V0 = workloads.layer_kv(wc, threads=16)
    b, hkv, n0, D = K0.shape
    K = np.empty((b, hkv, n0 + extra, D), np.float16)
    V = np.empty_like(K)
    K[:, :, :n0], V[:, :, :n0] = K0, V0
    rng = np.random.default_rng(wc.seed)
    for s_ in range(b):
        for h in range(hkv):
            K[s_, h, n0:] = workloads.drift_keys(wc.seed, s_, h, 0, extra, total)
            V[s_, h, n0:] = rng.standard_normal((extra, D)).astype(np.float16)
    signs = workloads.rotation_signs(wc.seed)
    g = wc.q_per_kv
    run = GpuRun(K0, None, np.zeros((b, hkv * g, D), np.float16), signs, g, pk.Budget(1, 1, 1), SCALE,
                 capacity=n0 + extra)
    n_cur = n0
    for t in (1, 255, 256):
        pk.append(run.cfg, run.index, torch.from_numpy(np.ascontiguousarray(K[:, :, n_cur:n_cur + t])).cuda(),
                  n_cur)
        n_cur += t
    assert n_cur == n0 + extra
    Q = np.stack([np.concatenate([workloads.drift_query(wc.seed, s_, h, extra, total, g) for h in range(hkv)])
                  for s_ in range(b)])
    C = -(-n_cur // 16)
    budget = pk.Budget(C, 2 * C, wc.top_k)
    run.Q = torch.from_numpy(Q).cuda()
    run.budget, run.n = budget, n_cur
    o_gpu = run.retrieve_attend(torch.from_numpy(K).cuda(), torch.from_numpy(V).cuda())
    inter = run.intermediates()
    gids, grec, gcnt = run.host_index()
    cand = inter["cand"][:, :, :C]
    assert np.all(np.diff(cand, axis=-1) > 0) and cand.min() >= 0 and cand.max() < n_cur
    assert np.all(np.diff(inter["idx"], axis=-1) > 0)
    assert np.all(gcnt.reshape(b, hkv, 16, 256).sum(axis=-1) == n_cur)
    for s_, h in ((0, 2), (3, 7)):
        print(f"case drift full width oracle group ({s_}, {h})", flush=True)
        orc = oracle_group(K[s_, h, :n_cur], signs)
        check_index(gids[s_, h], grec[s_, h], gcnt[s_, h], orc)
        for gg in range(g):
            hq = h * g + gg
            check_head(inter, s_, h, gg, g, Q[s_, hq], orc, signs, budget, n_cur)
            check_attention(o_gpu[s_, hq], Q[s_, hq], K[s_, h, :n_cur], V[s_, h, :n_cur], inter["idx"][s_, hq],
                            SCALE)


def test_host_mapped_attention_matches_hbm():
    cfg = workloads.CONFIGS["layer32k"]
    wc, K, V, Q, _, signs = _inputs(cfg, n=8192)
    print("case host-mapped", flush=True)
    budget = pk.Budget(1024, 2048, 256)
    run = GpuRun(K, V, Q, signs, wc.q_per_kv, budget, SCALE).retrieve()
    o_hbm = run.attend()
    o_host = run.attend(host_mapped=True)
    np.testing.assert_array_equal(o_hbm, o_host)
    idx = run.out_idx.cpu().numpy()
    for hq in (0, 13, 31):
        check_attention(o_host[0, hq], Q[0, hq], K[0, hq // 4], V[0, hq // 4], idx[0, hq], SCALE)


@pytest.mark.timeout(400)
def test_batch8_128k_sampled_at_full_size():
    # The bench workload in its launch configuration: every output that the
    # oracle can recompute in seconds is checked (two whole (sequence, KV head)
    # groups with their 8 query heads, plus encode of 4096 sampled keys from
    # every group), the rest through properties that hold at any size.
    # The call is pariskv_retrieve_attend, the one the benchmark times (top-k with the
    # attention fused into it, 8 estimates per thread); retrieve + sparse_attend must give
    # the same bits for every head.
    cfg = workloads.CONFIGS["batch8_128k"]
    wc, K, V, Q, needles, signs = _inputs(cfg)
    print("case batch8_128k", flush=True)
    budget = pk.Budget(cfg.n_cand, cfg.n_collide, cfg.top_k)
    run = GpuRun(K, V, Q, signs, wc.q_per_kv, budget, SCALE)
    o_gpu = run.retrieve_attend()
    inter = run.intermediates()
    sep_idx, sep_score, _ = pk.retrieve(run.cfg, run.index, run.Q, wc.n, budget,
                                        out_score=torch.empty_like(run.out_score))
    sep_o = pk.sparse_attend(run.cfg, run.Q, run.K, run.V, sep_idx, SCALE)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(sep_idx.cpu().numpy(), inter["idx"])
    np.testing.assert_array_equal(sep_score.cpu().numpy().view(np.uint32), inter["score"].view(np.uint32))
    np.testing.assert_array_equal(sep_o.cpu().numpy().view(np.uint32), o_gpu.view(np.uint32))
    del sep_idx, sep_score, sep_o
    rng = np.random.default_rng(0)
    # encode, sampled keys of every group
    for s in range(wc.batch):
        for h in range(wc.n_kv_heads):
            rows = np.sort(rng.choice(wc.n, size=512, replace=False))
            gids = SLOT[run.index.ids[s, h, rows].cpu().numpy()]
            grec = run.index.rec[s, h, rows].cpu().numpy()
            from oracle import encode as oenc
            from parity import A, TAU
            ids, codes, W = oenc.encode(K[s, h, rows], signs, TAU, A, 16)
            np.testing.assert_array_equal(gids, ids)
            gc, gW = decode_rec(grec)
            np.testing.assert_array_equal(gc, codes)
            np.testing.assert_array_equal(gW.view(np.uint32), W.view(np.uint32))
    # properties of every head: counts sum, candidate count, sortedness, scores
    cnt = run.index.counts.cpu().numpy()
    assert np.all(cnt.sum(axis=-1) == wc.n)
    C, k = budget.n_cand, budget.top_k
    cand = inter["cand"][:, :, :C]
    assert np.all(np.diff(cand, axis=-1) > 0) and cand.min() >= 0 and cand.max() < wc.n
    S = inter["S"][:, :, :wc.n]
    th = inter["thresh"]
    # every head's threshold comes from the floored histogram, none from the recount
    print(f"histogram floors {np.unique(th[..., 4]).tolist()}, recounts {int(th[..., 5].sum())}", flush=True)
    assert np.all(th[..., 5] == 0) and np.all(th[..., 4] > 1)
    for s in range(wc.batch):
        for hq in range(wc.n_q_heads):
            assert np.sum(S[s, hq] >= th[s, hq, 4]) >= C
            sel = S[s, hq, cand[s, hq]]
            assert sel.min() >= th[s, hq, 0]
            assert np.sum(S[s, hq] > th[s, hq, 0]) == th[s, hq, 1]
    assert np.all(np.diff(inter["idx"], axis=-1) > 0)
    # three whole groups through the oracle
    for s, h in ((0, 0), (5, 3), (7, 7)):
        orc = oracle_group(K[s, h], signs)
        check_index(SLOT[run.index.ids[s, h].cpu().numpy()], run.index.rec[s, h].cpu().numpy(),
                    cnt[s, h].view(np.uint32), orc)
        for g in range(wc.q_per_kv):
            hq = h * wc.q_per_kv + g
            check_head(inter, s, h, g, wc.q_per_kv, Q[s, hq], orc, signs, budget, wc.n)
            check_attention(o_gpu[s, hq], Q[s, hq], K[s, h], V[s, h], inter["idx"][s, hq], SCALE)
    hits = np.mean([needles[s, hq] in set(inter["idx"][s, hq].tolist())
                    for s in range(wc.batch) for hq in range(wc.n_q_heads)])
    print(f"needle hit rate {hits:.3f}", flush=True)
    assert hits > 0.9


def test_host1m_sampled_at_full_size():
    # The 1M-key workload in its launch configuration, K/V in pinned host memory read
    # over the host link: one whole (KV head, 4 query heads) group through the oracle,
    # properties of every head, sampled encode of every group.
    # The call is pariskv_retrieve_attend with host-mapped K/V, as the benchmark runs it.
    cfg = workloads.CONFIGS["host1m"]
    wc, K, V, Q, needles, signs = _inputs(cfg)
    print("case host1m", flush=True)
    budget = pk.Budget(cfg.n_cand, cfg.n_collide, cfg.top_k)
    run = GpuRun(K, None, Q, signs, wc.q_per_kv, budget, SCALE)
    Kh = torch.from_numpy(K).pin_memory()
    Vh = torch.from_numpy(V).pin_memory()
    o_gpu = run.retrieve_attend(Kh, Vh, host_mapped=True)
    inter = run.intermediates()
    rng = np.random.default_rng(1)
    from oracle import encode as oenc
    from parity import A, TAU
    for h in range(wc.n_kv_heads):
        rows = np.sort(rng.choice(wc.n, size=512, replace=False))
        ids, codes, W = oenc.encode(K[0, h, rows], signs, TAU, A, 16)
        np.testing.assert_array_equal(SLOT[run.index.ids[0, h, rows].cpu().numpy()], ids)
        gc, gW = decode_rec(run.index.rec[0, h, rows].cpu().numpy())
        np.testing.assert_array_equal(gc, codes)
        np.testing.assert_array_equal(gW.view(np.uint32), W.view(np.uint32))
    cnt = run.index.counts.cpu().numpy()
    assert np.all(cnt.sum(axis=-1) == wc.n)
    C = budget.n_cand
    cand = inter["cand"][:, :, :C]
    assert np.all(np.diff(cand, axis=-1) > 0) and cand.min() >= 0 and cand.max() < wc.n
    S = inter["S"][:, :, :wc.n]
    th = inter["thresh"]
    for hq in range(wc.n_q_heads):
        assert S[0, hq, cand[0, hq]].min() >= th[0, hq, 0]
        assert np.sum(S[0, hq] > th[0, hq, 0]) == th[0, hq, 1]
    assert np.all(np.diff(inter["idx"], axis=-1) > 0)
    h = 6
    print("case host1m oracle group", flush=True)
    orc = oracle_group(K[0, h], signs)
    check_index(SLOT[run.index.ids[0, h].cpu().numpy()], run.index.rec[0, h].cpu().numpy(),
                cnt[0, h].view(np.uint32), orc)
    for g in range(wc.q_per_kv):
        hq = h * wc.q_per_kv + g
        check_head(inter, 0, h, g, wc.q_per_kv, Q[0, hq], orc, signs, budget, wc.n)
        check_attention(o_gpu[0, hq], Q[0, hq], K[0, h], V[0, h], inter["idx"][0, hq], SCALE)
    # At 1M keys with C = n/32 the planted needles are found less often (a quality figure
    # of the method on these keys, not a parity property): reported, not asserted.
    hits = np.mean([needles[0, hq] in set(inter["idx"][0, hq].tolist()) for hq in range(wc.n_q_heads)])
    print(f"needle hit rate {hits:.3f}", flush=True)


@pytest.mark.parametrize("n,G,bud,host", [
    (4096, 8, (512, 1024, 64), False),       # top-k staging 4 per thread, fused
    (20000, 4, (8192, 16384, 512), False),   # 8 per thread, fused (the bench shape per head)
    (40000, 2, (10000, 20000, 300), False),  # 16 per thread, fused
    (40000, 2, (20000, 30000, 1000), False), # 32 per thread, fused
    (70000, 1, (40000, 60000, 2048), False), # two-pass top-k, attention in the final pass
    (0, 4, (64, 128, 16), False),            # empty cache: padding and zero outputs
    (9000, 4, (700, 1500, 100), True),       # K/V in pinned host memory
], ids=["C512", "C8192", "C10000", "C20000", "C40000", "n0", "host"])
def test_retrieve_attend_equals_separate_calls(n, G, bud, host):
    # The fused call must give the same bits as retrieve followed by sparse_attend.
    wc = workloads.Config("fused", batch=2, n_kv_heads=2, q_per_kv=G, n=max(n, 1), n_cand=bud[0],
                          n_collide=bud[1], top_k=bud[2], seed=88)
    K, V = workloads.layer_kv(wc)
    Q, _ = workloads.layer_queries(wc, K)
    signs = workloads.rotation_signs(wc.seed)
    print(f"case fused n={n} G={G} budget={bud} host={host}", flush=True)
    cfg = pk.Config(2, G, max(n, 1), signs)
    budget = pk.Budget(*bud)
    Kd = torch.from_numpy(K).cuda()
    Vd = torch.from_numpy(V).cuda()
    Qd = torch.from_numpy(Q).cuda()
    index = pk.Index.empty(cfg, 2)
    pk.encode(cfg, index, Kd[:, :, :n].contiguous())
    Ka, Va = (Kd.cpu().pin_memory(), Vd.cpu().pin_memory()) if host else (Kd, Vd)
    hq = cfg.n_q_heads
    s1 = torch.empty((2, hq, bud[2]), dtype=torch.float32, device="cuda")
    i1, _, _ = pk.retrieve(cfg, index, Qd, n, budget, out_score=s1)
    o1 = pk.sparse_attend(cfg, Qd, Ka, Va, i1, SCALE, kv_host_mapped=host)
    s2 = torch.empty_like(s1)
    i2, _, o2, _ = pk.retrieve_attend(cfg, index, Qd, n, budget, Ka, Va, SCALE, out_score=s2,
                                      kv_host_mapped=host)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(i1.cpu().numpy(), i2.cpu().numpy())
    np.testing.assert_array_equal(s1.cpu().numpy().view(np.uint32), s2.cpu().numpy().view(np.uint32))
    np.testing.assert_array_equal(o1.cpu().numpy().view(np.uint32), o2.cpu().numpy().view(np.uint32))
    if n == 0:
        assert np.all(i2.cpu().numpy() == -1) and np.all(o2.cpu().numpy() == 0)
