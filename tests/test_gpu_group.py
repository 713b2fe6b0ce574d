"""GPU parity of the GQA-group attention (each distinct K/V row fetched once per KV head):
every head's output against the float64 oracle over that head's own list, and the number
of rows fetched against the union computed on the host."""

import numpy as np
import pytest
import torch

import paper_2602_07721_amd as pk
import workloads
from parity import check_attention

pytestmark = pytest.mark.gpu

SCALE = 1.0 / np.sqrt(128.0)


def _lists(b, hkv, g, k, cap, overlap, seed):
    """Ascending per-head lists with -1 padding at the end; heads of a KV head share a pool
    of rows (overlap = share of each list drawn from the pool)."""
    r = np.random.default_rng(seed)
    idx = np.full((b, hkv * g, k), -1, dtype=np.int32)
    for s in range(b):
        for h in range(hkv):
            pool = r.choice(cap, size=k, replace=False)
            for j in range(g):
                valid = int(r.integers(k // 2, k + 1))
                shared = r.choice(pool, size=int(overlap * valid), replace=False)
                rest = np.setdiff1d(np.arange(cap), shared)
                own = r.choice(rest, size=valid - shared.size, replace=False)
                idx[s, h * g + j, :valid] = np.sort(np.concatenate([shared, own]))
    return idx


@pytest.mark.parametrize("g,k,overlap,host,cap", [
    (4, 256, 0.6, False, 5000), (4, 1024, 0.3, False, 5000), (1, 512, 0.0, False, 5000),
    (3, 300, 0.9, False, 5000), (6, 128, 0.5, False, 5000), (4, 256, 0.6, True, 5000),
    (4, 512, 0.5, True, 70000), (6, 200, 0.7, False, 70000)],
    ids=["g4", "g4_k1024", "g1", "g3_odd_k", "g6_two_quads", "g4_host", "g4_host_merge", "g6_merge"])
def test_group_attend_matches_the_oracle_per_head(g, k, overlap, host, cap):
    # Over at most 65536 cache rows the union is built as a key bitmap, above that by
    # merging the sorted lists (the *_merge cases).
    b, hkv = 2, 2
    print(f"[group_attend] g {g} k {k} overlap {overlap} host {host} cap {cap}", flush=True)
    K = np.stack([np.stack([workloads.head_keys(51, s, h, cap) for h in range(hkv)]) for s in range(b)])
    V = np.stack([np.stack([workloads.head_values(51, s, h, cap) for h in range(hkv)]) for s in range(b)])
    Q = np.stack([np.concatenate([workloads.needle_queries(K[s, h], 51, s, h, g)[0] for h in range(hkv)])
                  for s in range(b)])
    idx = _lists(b, hkv, g, k, cap, overlap, seed=g * 1000 + k)
    cfg = pk.Config(hkv, g, cap, workloads.rotation_signs(51))
    Kt, Vt = torch.from_numpy(K), torch.from_numpy(V)
    Kt, Vt = (Kt.pin_memory(), Vt.pin_memory()) if host else (Kt.cuda(), Vt.cuda())
    quads = (g + 3) // 4
    un = torch.zeros((b, hkv, quads), dtype=torch.int32, device="cuda")
    out = pk.group_attend(cfg, torch.from_numpy(Q).cuda(), Kt, Vt, torch.from_numpy(idx).cuda(), SCALE,
                          union_rows=un, kv_host_mapped=host)
    out, un = out.cpu().numpy(), un.cpu().numpy()
    for s in range(b):
        for h in range(hkv):
            for qd in range(quads):
                heads = range(h * g + 4 * qd, h * g + min(g, 4 * qd + 4))
                rows = set()
                for hq in heads:
                    rows |= set(int(x) for x in idx[s, hq] if x >= 0)
                assert un[s, h, qd] == len(rows), (s, h, qd)
            for j in range(g):
                hq = h * g + j
                check_attention(out[s, hq], Q[s, hq], K[s, h], V[s, h], idx[s, hq], SCALE)


def test_group_attend_on_retrieval_output_and_empty_lists():
    wc = workloads.Config("grp", batch=1, n_kv_heads=2, q_per_kv=4, n=6000, n_cand=512, n_collide=1024,
                          top_k=128, seed=52)
    K, V = workloads.layer_kv(wc)
    Q, _ = workloads.layer_queries(wc, K)
    cfg = pk.Config(2, 4, wc.n, workloads.rotation_signs(52))
    Kd, Vd, Qd = (torch.from_numpy(x).cuda() for x in (K, V, Q))
    index = pk.Index.empty(cfg, 1)
    pk.encode(cfg, index, Kd)
    idx, _, _ = pk.retrieve(cfg, index, Qd, wc.n, pk.Budget(512, 1024, 128))
    # head 5's list emptied: it must come out as zeros
    idx[0, 5] = -1
    out = pk.group_attend(cfg, Qd, Kd, Vd, idx, SCALE).cpu().numpy()
    ref = pk.sparse_attend(cfg, Qd, Kd, Vd, idx, SCALE).cpu().numpy()
    ih = idx.cpu().numpy()
    for hq in range(8):
        check_attention(out[0, hq], Q[0, hq], K[0, hq // 4], V[0, hq // 4], ih[0, hq], SCALE)
    assert not out[0, 5].any() and not ref[0, 5].any()
    np.testing.assert_allclose(out, ref, rtol=0, atol=1e-5 * np.abs(ref).max())


@pytest.mark.parametrize("g,n,bud,host,splits", [
    (4, 9000, (700, 1500, 100), True, 1), (6, 5000, (400, 800, 64), False, 1),
    (4, 40000, (10000, 20000, 512), True, 8), (6, 12000, (1500, 3000, 256), False, 4),
    (4, 0, (64, 128, 16), False, 1), (4, 0, (600, 1200, 512), False, 8),
    (4, 140000, (4096, 8192, 64), True, 3), (3, 9000, (700, 1500, 300), True, 3),
    (1, 9000, (700, 1500, 300), False, 1)],
    ids=["g4_host", "g6_two_quads", "g4_two_pass_host_split8", "g6_two_quads_split4", "n0", "n0_split8",
         "g4_three_key_ranges_host", "g3_host_split3", "g1"])
def test_retrieve_attend_with_group_fetch(g, n, bud, host, splits):
    # PARISKV_GROUP_FETCH: the winners are those of the plain call bit for bit, each head's
    # attention matches the float64 oracle over its own winners, and the rows fetched per
    # quad are the union of the quad's winner lists.  With splits > 1 each quad's winners
    # are shared by that many blocks by key range (at most 65536 keys each, so 140000
    # keys take 3 even where the block count alone would ask for 1) and their states
    # merged by a second kernel.
    b, hkv = 2, 2
    wc = workloads.Config("gfetch", batch=b, n_kv_heads=hkv, q_per_kv=g, n=max(n, 1), n_cand=bud[0],
                          n_collide=bud[1], top_k=bud[2], seed=53)
    print(f"[group fetch] g {g} n {n} budget {bud} host {host} splits {splits}", flush=True)
    K, V = workloads.layer_kv(wc)
    Q, _ = workloads.layer_queries(wc, K)
    cfg = pk.Config(hkv, g, max(n, 1), workloads.rotation_signs(53))
    Kd, Qd = torch.from_numpy(K).cuda(), torch.from_numpy(Q).cuda()
    index = pk.Index.empty(cfg, b)
    pk.encode(cfg, index, Kd[:, :, :n].contiguous())
    Ka, Va = torch.from_numpy(K), torch.from_numpy(V)
    Ka, Va = (Ka.pin_memory(), Va.pin_memory()) if host else (Ka.cuda(), Va.cuda())
    plain = pk.Budget(*bud)
    grouped = pk.Budget(*bud, flags=pk.GROUP_FETCH)
    s1 = torch.empty((b, hkv * g, bud[2]), dtype=torch.float32, device="cuda")
    i1, _, o1, _ = pk.retrieve_attend(cfg, index, Qd, n, plain, Ka, Va, SCALE, out_score=s1, kv_host_mapped=host)
    s2 = torch.empty_like(s1)
    i2, _, o2, ws = pk.retrieve_attend(cfg, index, Qd, n, grouped, Ka, Va, SCALE, out_score=s2,
                                       kv_host_mapped=host)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(i1.cpu().numpy(), i2.cpu().numpy())
    np.testing.assert_array_equal(s1.cpu().numpy().view(np.uint32), s2.cpu().numpy().view(np.uint32))
    idx, out = i2.cpu().numpy(), o2.cpu().numpy()
    lay = pk.workspace_layout(cfg, b, n, grouped)
    assert lay["group_splits"] == splits
    quads = (g + 3) // 4
    from parity import ws_array
    un = ws_array(ws, lay["group_rows"], np.int32, (b, hkv, quads))
    for s in range(b):
        for h in range(hkv):
            for qd in range(quads):
                rows = set()
                for hq in range(h * g + 4 * qd, h * g + min(g, 4 * qd + 4)):
                    rows |= set(int(x) for x in idx[s, hq] if x >= 0)
                assert un[s, h, qd] == len(rows), (s, h, qd)
            for j in range(g):
                hq = h * g + j
                if n == 0:
                    assert not out[s, hq].any()
                else:
                    check_attention(out[s, hq], Q[s, hq], K[s, h], V[s, h], idx[s, hq], SCALE)
    np.testing.assert_allclose(out, o1.cpu().numpy(), rtol=0, atol=1e-5 * max(np.abs(out).max(), 1e-30))


def test_group_fetch_over_more_than_16_key_ranges():
    # 1.1M keys: 17 key ranges of at most 65536 per quad, so the combine kernel takes its
    # form for more than 16 shares.  One KV head, K/V in pinned host memory.
    b, hkv, g, n = 1, 1, 4, 1100000
    wc = workloads.Config("gfetch17", batch=b, n_kv_heads=hkv, q_per_kv=g, n=n, n_cand=4096, n_collide=8192,
                          top_k=64, seed=54)
    print("[group fetch] 17 key ranges", flush=True)
    K, V = workloads.layer_kv(wc, threads=16)
    Q, _ = workloads.layer_queries(wc, K)
    cfg = pk.Config(hkv, g, n, workloads.rotation_signs(54))
    index = pk.Index.empty(cfg, b)
    pk.encode(cfg, index, torch.from_numpy(K).cuda())
    Kh, Vh = torch.from_numpy(K).pin_memory(), torch.from_numpy(V).pin_memory()
    Qd = torch.from_numpy(Q).cuda()
    grouped = pk.Budget(4096, 8192, 64, flags=pk.GROUP_FETCH)
    lay = pk.workspace_layout(cfg, b, n, grouped)
    assert lay["group_splits"] == 17
    i1, _, o1, _ = pk.retrieve_attend(cfg, index, Qd, n, pk.Budget(4096, 8192, 64), Kh, Vh, SCALE,
                                      kv_host_mapped=True)
    i2, _, o2, ws = pk.retrieve_attend(cfg, index, Qd, n, grouped, Kh, Vh, SCALE, kv_host_mapped=True)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(i1.cpu().numpy(), i2.cpu().numpy())
    idx, out = i2.cpu().numpy(), o2.cpu().numpy()
    from parity import ws_array
    un = ws_array(ws, lay["group_rows"], np.int32, (b, hkv, 1))
    assert un[0, 0, 0] == len(set(int(x) for x in idx[0].ravel() if x >= 0))
    for hq in range(g):
        check_attention(out[0, hq], Q[0, hq], K[0, 0], V[0, 0], idx[0, hq], SCALE)
    np.testing.assert_allclose(out, o1.cpu().numpy(), rtol=0, atol=1e-5 * np.abs(out).max())


@pytest.mark.parametrize("tiered,host,splits_hint,n", [(True, True, "one share", 9000), (True, True, "shares", 9000),
                                                       (False, False, "shares", 9000), (True, True, "shares", 0)],
                         ids=["tiered_host", "tiered_host_shares", "window_hbm_shares", "tiered_n0_dense_only"])
def test_window_and_tiered_calls_with_group_fetch(tiered, host, splits_hint, n):
    # The window's dense rows (Sink, Local / Update Buffer) are attended by every head of
    # a quad, once per quad: retrieve_tiered_attend (dense rows from the GPU window ring,
    # retrieval rows from host memory) and retrieve_window_attend (dense rows in the main
    # cache) with PARISKV_GROUP_FETCH against the oracle's window attention per head, and
    # the winners bit for bit those of the plain call.
    from oracle import window as owin
    from test_gpu_window import _cache, _close, _dense, _index_over, _queries, _window_cache
    b, hkv, g = 1, 2, 4
    k = 64 if splits_hint == "one share" else 512
    sink, local, buf = 128, 512, 60
    cap = sink + n + local + buf
    win = pk.Window(sink, sink, sink + n, cap)
    wcap = sink + local + 2 * 256
    print(f"[group fetch window] tiered {tiered} host {host} k {k}", flush=True)
    K, V = _cache(b, hkv, cap, seed=29)
    Q = _queries(K, g, seed=29)
    cfg = pk.Config(hkv, g, max(n, 1), workloads.rotation_signs(29))
    Kd, Vd, Qd = (torch.from_numpy(x).cuda() for x in (K, V, Q))
    index = _index_over(cfg, Kd, sink, n)
    Kr, Vr = (torch.from_numpy(x) for x in (K, V))
    Kr, Vr = (Kr.pin_memory(), Vr.pin_memory()) if host else (Kd, Vd)
    plain, grouped = pk.Budget(1024, 2048, k), pk.Budget(1024, 2048, k, flags=pk.GROUP_FETCH)
    splits = pk.workspace_layout(cfg, b, n, grouped)["group_splits"]
    assert (splits == 1) == (splits_hint == "one share")
    if tiered:
        Kw, Vw = (torch.from_numpy(x).cuda() for x in _window_cache(K, V, win, wcap))
        call = lambda bud: pk.retrieve_tiered_attend(cfg, index, Qd, n, bud, Kw, Vw, Kr, Vr, win, SCALE,
                                                     kv_host_mapped=host)
    else:
        call = lambda bud: pk.retrieve_window_attend(cfg, index, Qd, n, bud, Kr, Vr, win, SCALE,
                                                     kv_host_mapped=host)
    i1, _, o1, _ = call(plain)
    i2, _, o2, _ = call(grouped)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(i1.cpu().numpy(), i2.cpu().numpy())
    idx, out = i2.cpu().numpy(), o2.cpu().numpy()
    for hq in range(hkv * g):
        retrieved = [sink + int(j) for j in idx[0, hq] if j >= 0]
        want = owin.window_attention(Q[0, hq], K[0, hq // g], V[0, hq // g], _dense(win), retrieved, SCALE)
        _close(out[0, hq], want, hq)
    np.testing.assert_allclose(out, o1.cpu().numpy(), rtol=0, atol=1e-5 * np.abs(out).max())
