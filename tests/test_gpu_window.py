"""GPU parity of the decode-time KV regions (Sec. "Buffer Update"): attention over Sink +
retrieved keys + Local/Update Buffer, the fused retrieve + window attention, encoding
evicted rows straight from the key cache, and a decode loop with batched buffer updates,
all checked against the CPU oracle (or, for the fused/split and cache/copy pairs, against
each other bit for bit)."""

import numpy as np
import pytest
import torch

import paper_2602_07721_amd as pk
import workloads
from oracle import attention as oatt
from oracle import window as owin
from parity import RTOL_ATT, check_head, check_index, oracle_group

pytestmark = pytest.mark.gpu

SCALE = 1.0 / np.sqrt(128.0)


def _cache(batch, hkv, n, seed):
    K = np.stack([np.stack([workloads.head_keys(seed, s, h, n) for h in range(hkv)]) for s in range(batch)])
    V = np.stack([np.stack([workloads.head_values(seed, s, h, n) for h in range(hkv)]) for s in range(batch)])
    return K, V


def _queries(K, g, seed, step=0, upto=None):
    b, hkv, n, D = K.shape
    upto = n if upto is None else upto
    Q = np.empty((b, hkv * g, D), dtype=np.float16)
    for s in range(b):
        for h in range(hkv):
            Q[s, h * g:(h + 1) * g] = workloads.needle_queries(K[s, h, :upto], seed, s, h, g, step)[0]
    return Q


def _close(o_gpu, o_ref, what):
    d = np.abs(o_gpu.astype(np.float64) - o_ref)
    mx = np.max(np.abs(o_ref))
    assert d.max() <= RTOL_ATT * mx + 1e-30, (what, d.max(), mx)
    assert np.linalg.norm(d) <= RTOL_ATT * np.linalg.norm(o_ref) + 1e-30, what


def _dense(w):
    return list(range(w.sink_len)) + list(range(w.dense_begin, w.dense_end))


@pytest.mark.parametrize("win", [pk.Window(128, 128, 5000, 5600), pk.Window(0, 300, 300, 300),
                                 pk.Window(128, 128, 5600, 5600), pk.Window(0, 0, 4000, 6000),
                                 pk.Window(1, 1, 5999, 6000)],
                         ids=["sink_local", "offset_only", "sink_only", "dense_2000", "one_each"])
def test_window_attend_matches_the_oracle(win):
    b, hkv, g, cap, k = 2, 2, 4, 6000, 256
    print(f"[window_attend] window {win} k {k}", flush=True)
    K, V = _cache(b, hkv, cap, seed=21)
    Q = _queries(K, g, seed=21)
    cfg = pk.Config(hkv, g, cap, workloads.rotation_signs(21))
    r = np.random.default_rng(5)
    n_retr = max(1, win.dense_begin - win.retr_begin)
    idx = np.full((b, hkv * g, k), -1, dtype=np.int32)
    for s in range(b):
        for hq in range(hkv * g):
            take = min(k - 7, n_retr)
            idx[s, hq, :take] = r.choice(n_retr, size=take, replace=False)
            r.shuffle(idx[s, hq])
    Kd, Vd, Qd = (torch.from_numpy(x).cuda() for x in (K, V, Q))
    out = pk.window_attend(cfg, Qd, Kd, Vd, torch.from_numpy(idx).cuda(), win, SCALE)
    out = out.cpu().numpy()
    for s in range(b):
        for hq in range(hkv * g):
            h = hq // g
            retrieved = [win.retr_begin + int(j) for j in idx[s, hq] if j >= 0]
            ref = owin.window_attention(Q[s, hq], K[s, h], V[s, h], _dense(win), retrieved, SCALE)
            _close(out[s, hq], ref, (s, hq))


def test_zero_window_is_sparse_attention_bit_for_bit():
    b, hkv, g, cap, k = 1, 2, 4, 3000, 300
    K, V = _cache(b, hkv, cap, seed=22)
    Q = _queries(K, g, seed=22)
    cfg = pk.Config(hkv, g, cap, workloads.rotation_signs(22))
    idx = np.random.default_rng(1).integers(-1, cap, size=(b, hkv * g, k)).astype(np.int32)
    Kd, Vd, Qd, Id = (torch.from_numpy(x).cuda() for x in (K, V, Q, idx))
    a = pk.sparse_attend(cfg, Qd, Kd, Vd, Id, SCALE).cpu().numpy()
    w = pk.window_attend(cfg, Qd, Kd, Vd, Id, pk.Window(), SCALE).cpu().numpy()
    np.testing.assert_array_equal(a.view(np.uint32), w.view(np.uint32))


def _index_over(cfg, Kd, row_begin, n):
    index = pk.Index.empty(cfg, int(Kd.shape[0]))
    if n > 0:
        pk.append_rows(cfg, index, Kd, row_begin, n, 0)
    return index


@pytest.mark.parametrize("n_cand,n,k", [(512, 6000, 64), (4096, 6000, 256), (10000, 20000, 512),
                                        (34000, 36000, 512), (512, 0, 64)],
                         ids=["C512", "C4096", "C10000", "C34000_two_pass", "n0"])
def test_fused_window_equals_retrieve_then_window_attend(n_cand, n, k):
    b, hkv, g = 1, 2, 4
    sink, local, buf = 128, 512, 40
    cap = sink + n + local + buf
    win = pk.Window(sink, sink, sink + n, cap)
    print(f"[retrieve_window_attend] C {n_cand} n {n} k {k}", flush=True)
    K, V = _cache(b, hkv, cap, seed=23)
    Q = _queries(K, g, seed=23)
    cfg = pk.Config(hkv, g, max(n, 1), workloads.rotation_signs(23))
    budget = pk.Budget(n_cand, 2 * n_cand, k)
    Kd, Vd, Qd = (torch.from_numpy(x).cuda() for x in (K, V, Q))
    index = _index_over(cfg, Kd, sink, n)
    sc1 = torch.empty((b, hkv * g, k), dtype=torch.float32, device="cuda")
    i1, _, o1, _ = pk.retrieve_window_attend(cfg, index, Qd, n, budget, Kd, Vd, win, SCALE, out_score=sc1)
    sc2 = torch.empty_like(sc1)
    i2, _, _ = pk.retrieve(cfg, index, Qd, n, budget, out_score=sc2)
    o2 = pk.window_attend(cfg, Qd, Kd, Vd, i2, win, SCALE)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(i1.cpu().numpy(), i2.cpu().numpy())
    np.testing.assert_array_equal(sc1.cpu().numpy().view(np.uint32), sc2.cpu().numpy().view(np.uint32))
    np.testing.assert_array_equal(o1.cpu().numpy().view(np.uint32), o2.cpu().numpy().view(np.uint32))


def test_append_rows_equals_append_of_copied_rows():
    b, hkv, cap = 2, 3, 2048
    K, _ = _cache(b, hkv, cap, seed=24)
    cfg = pk.Config(hkv, 4, 1024, workloads.rotation_signs(24))
    Kd = torch.from_numpy(K).cuda()
    one, two = pk.Index.empty(cfg, b), pk.Index.empty(cfg, b)
    for index in (one, two):
        pk.encode(cfg, index, Kd[:, :, :50].contiguous())
    pk.append_rows(cfg, one, Kd, 700, 300, 50)
    pk.append(cfg, two, Kd[:, :, 700:1000].contiguous(), 50)
    pk.append_rows(cfg, one, Kd, 1500, 1, 350)   # a single row, the per-step case
    pk.append(cfg, two, Kd[:, :, 1500:1501].contiguous(), 350)
    torch.cuda.synchronize()
    for a, c in ((one.ids, two.ids), (one.rec, two.rec)):
        np.testing.assert_array_equal(a[:, :, :351].cpu().numpy(), c[:, :, :351].cpu().numpy())
    np.testing.assert_array_equal(one.counts.cpu().numpy(), two.counts.cpu().numpy())
    # and the appended rows are the oracle's codes of those keys
    ids, rec, cnt = (one.ids[:, :, :351].cpu().numpy(), one.rec[:, :, :351].cpu().numpy(),
                     one.counts.cpu().numpy().view(np.uint32))
    from parity import SLOT
    rows = list(range(50)) + list(range(700, 1000)) + [1500]
    for s in range(b):
        for h in range(hkv):
            check_index(SLOT[ids[s, h]], rec[s, h], cnt[s, h],
                        oracle_group(K[s, h, rows], workloads.rotation_signs(24)))


def test_window_covering_every_retrieval_row_is_full_attention():
    b, hkv, g = 1, 2, 4
    sink, n, local = 64, 900, 300
    cap = sink + n + local
    win = pk.Window(sink, sink, sink + n, cap)
    K, V = _cache(b, hkv, cap, seed=25)
    Q = _queries(K, g, seed=25)
    cfg = pk.Config(hkv, g, n, workloads.rotation_signs(25))
    budget = pk.Budget(n, n, n)   # C = k = n: every retrieval key is attended
    Kd, Vd, Qd = (torch.from_numpy(x).cuda() for x in (K, V, Q))
    index = _index_over(cfg, Kd, sink, n)
    idx, _, out, _ = pk.retrieve_window_attend(cfg, index, Qd, n, budget, Kd, Vd, win, SCALE)
    idx, out = idx.cpu().numpy(), out.cpu().numpy()
    for hq in range(hkv * g):
        np.testing.assert_array_equal(idx[0, hq], np.arange(n))
        _close(out[0, hq], oatt.full_attention(Q[0, hq], K[0, hq // g], V[0, hq // g], SCALE), hq)


def test_decode_loop_with_buffer_updates_matches_the_oracle():
    """Prompt of P tokens, then decode steps: every m steps the oldest Local rows are encoded
    from the cache into the retrieval index; each step retrieves over Retrieval and attends
    over Sink + winners + Local/Buffer.  Checked against the oracle's replay at several steps."""
    b, hkv, g = 1, 2, 4
    P, steps, sink, local, m = 3000, 200, 128, 512, 64
    cap = P + steps
    K, V = _cache(b, hkv, cap, seed=26)
    signs = workloads.rotation_signs(26)
    cfg = pk.Config(hkv, g, cap, signs)
    budget = pk.Budget(256, 512, 64)
    Kd, Vd = (torch.from_numpy(x).cuda() for x in (K, V))
    index = pk.Index.empty(cfg, b)
    R = owin.after_prefill(P, sink, local, m)
    n_idx = 0
    check_at = {0, 1, 63, 64, 65, 128, 199}
    for t in range(steps):
        if t > 0:
            owin.decode_step(R)
        win, n_retr = pk.window_regions(P, t, sink, local, m)
        assert n_retr == len(R.retrieval) and _dense(win) == owin.dense_rows(R)
        if n_retr > n_idx:   # the rows that entered Retrieval since the last step
            pk.append_rows(cfg, index, Kd, win.retr_begin + n_idx, n_retr - n_idx, n_idx)
            n_idx = n_retr
        T = P + t
        Q = _queries(K, g, seed=26, step=t, upto=T)
        Qd = torch.from_numpy(Q).cuda()
        sc = torch.empty((b, hkv * g, budget.top_k), dtype=torch.float32, device="cuda")
        idx, _, out, ws = pk.retrieve_window_attend(cfg, index, Qd, n_idx, budget, Kd, Vd, win, SCALE,
                                                    out_score=sc)
        if t not in check_at:
            continue
        print(f"[decode loop] checking step {t}: n_retr {n_idx}, dense {win.dense_rows}", flush=True)
        torch.cuda.synchronize()
        lay = pk.workspace_layout(cfg, b, n_idx, budget)
        from parity import SLOT, ws_array
        inter = dict(
            zq=ws_array(ws, lay["zq"], np.float32, (b, hkv * g, 128)),
            lut=ws_array(ws, lay["lut"], np.uint32, (b, hkv, lay["quads"], 16, 256)),
            S=ws_array(ws, lay["score8"], np.uint8, (b, hkv * g, lay["n_pad"])),
            thresh=ws_array(ws, lay["thresh"], np.int32, (b, hkv * g, 8)),
            cand=ws_array(ws, lay["cand"], np.int32, (b, hkv * g, budget.n_cand)),
            cand_score=ws_array(ws, lay["cand_score"], np.float32, (b, hkv * g, budget.n_cand)),
            idx=idx.cpu().numpy(), score=sc.cpu().numpy())
        o = out.cpu().numpy()
        ids = SLOT[index.ids[:, :, :n_idx].cpu().numpy()]
        rec = index.rec[:, :, :n_idx].cpu().numpy()
        cnt = index.counts.cpu().numpy().view(np.uint32)
        for h in range(hkv):
            Kr = K[0, h, R.retrieval]
            orc = oracle_group(Kr, signs)
            check_index(ids[0, h], rec[0, h], cnt[0, h], orc)
            for gg in range(g):
                hq = h * g + gg
                check_head(inter, 0, h, gg, g, Q[0, hq], orc, signs, budget, n_idx)
                retrieved = [win.retr_begin + int(j) for j in inter["idx"][0, hq] if j >= 0]
                ref = owin.window_attention(Q[0, hq], K[0, h], V[0, h], owin.dense_rows(R), retrieved, SCALE)
                _close(o[0, hq], ref, (t, hq))


def _window_cache(K, V, win, wcap):
    """The dense rows of `win` placed at their slots of a window cache of wcap rows."""
    b, hkv, _, D = K.shape
    Kw = np.zeros((b, hkv, wcap, D), np.float16)
    Vw = np.zeros_like(Kw)
    for r in _dense(win):
        s = pk.window_slot(r, win.sink_len, wcap)
        Kw[:, :, s] = K[:, :, r]
        Vw[:, :, s] = V[:, :, r]
    return Kw, Vw


@pytest.mark.parametrize("host", [False, True], ids=["retrieval_in_hbm", "retrieval_in_host_memory"])
def test_tiered_attend_equals_window_attend_bit_for_bit(host):
    b, hkv, g, cap, k = 1, 2, 4, 6000, 256
    win = pk.Window(128, 128, 5000, 5700)      # 700 Local/Buffer rows
    wcap = 128 + 720                           # a ring of 720 slots: rows 5000..5699 wrap around it
    K, V = _cache(b, hkv, cap, seed=27)
    Q = _queries(K, g, seed=27)
    cfg = pk.Config(hkv, g, cap, workloads.rotation_signs(27))
    idx = np.random.default_rng(2).integers(-1, 4872, size=(b, hkv * g, k)).astype(np.int32)
    Qd, Id = torch.from_numpy(Q).cuda(), torch.from_numpy(idx).cuda()
    ref = pk.window_attend(cfg, Qd, torch.from_numpy(K).cuda(), torch.from_numpy(V).cuda(), Id, win, SCALE)
    Kw, Vw = _window_cache(K, V, win, wcap)
    # the main cache's copies of the dense rows are wrong on purpose: they must be read from the window cache
    Kr, Vr = K.copy(), V.copy()
    Kr[:, :, :128] = 7.0
    Vr[:, :, 5000:5700] = -3.0
    Kr_t, Vr_t = torch.from_numpy(Kr), torch.from_numpy(Vr)
    if host:
        Kr_t, Vr_t = Kr_t.pin_memory(), Vr_t.pin_memory()
    else:
        Kr_t, Vr_t = Kr_t.cuda(), Vr_t.cuda()
    out = pk.tiered_attend(cfg, Qd, torch.from_numpy(Kw).cuda(), torch.from_numpy(Vw).cuda(), Kr_t, Vr_t, Id,
                           win, SCALE, kv_host_mapped=host)
    torch.cuda.synchronize()
    o = out.cpu().numpy()
    np.testing.assert_array_equal(o.view(np.uint32), ref.cpu().numpy().view(np.uint32))
    # and against the oracle over the true rows: Sink + Local/Buffer + retrieved
    for hq in range(hkv * g):
        retrieved = [win.retr_begin + int(j) for j in idx[0, hq] if j >= 0]
        want = owin.window_attention(Q[0, hq], K[0, hq // g], V[0, hq // g], _dense(win), retrieved, SCALE)
        _close(o[0, hq], want, hq)


@pytest.mark.parametrize("n_cand,host", [(512, True), (4096, False), (34000, True)],
                         ids=["C512_host", "C4096_hbm", "C34000_two_pass_host"])
def test_fused_tiered_equals_separate_and_window_paths(n_cand, host):
    b, hkv, g, k = 1, 2, 4, 128
    sink, local, buf = 128, 512, 60
    n = max(6000, n_cand + 100)
    cap = sink + n + local + buf
    win = pk.Window(sink, sink, sink + n, cap)
    wcap = sink + local + 2 * 256
    print(f"[tiered] C {n_cand} n {n} host {host}", flush=True)
    K, V = _cache(b, hkv, cap, seed=28)
    Q = _queries(K, g, seed=28)
    cfg = pk.Config(hkv, g, n, workloads.rotation_signs(28))
    budget = pk.Budget(n_cand, 2 * n_cand, k)
    Kd, Vd, Qd = (torch.from_numpy(x).cuda() for x in (K, V, Q))
    index = _index_over(cfg, Kd, sink, n)
    Kw, Vw = (torch.from_numpy(x).cuda() for x in _window_cache(K, V, win, wcap))
    Kr, Vr = (torch.from_numpy(x) for x in (K, V))
    Kr, Vr = (Kr.pin_memory(), Vr.pin_memory()) if host else (Kd, Vd)
    sc1 = torch.empty((b, hkv * g, k), dtype=torch.float32, device="cuda")
    i1, _, o1, ws = pk.retrieve_tiered_attend(cfg, index, Qd, n, budget, Kw, Vw, Kr, Vr, win, SCALE,
                                              out_score=sc1, kv_host_mapped=host)
    torch.cuda.synchronize()
    # the fused call against the oracle: retrieval over the Retrieval rows, then attention
    # over Sink + winners + Local/Buffer
    from parity import SLOT, ws_array
    lay = pk.workspace_layout(cfg, b, n, budget)
    inter = dict(
        zq=ws_array(ws, lay["zq"], np.float32, (b, hkv * g, 128)),
        lut=ws_array(ws, lay["lut"], np.uint32, (b, hkv, lay["quads"], 16, 256)),
        S=ws_array(ws, lay["score8"], np.uint8, (b, hkv * g, lay["n_pad"])),
        thresh=ws_array(ws, lay["thresh"], np.int32, (b, hkv * g, 8)),
        cand=ws_array(ws, lay["cand"], np.int32, (b, hkv * g, budget.n_cand)),
        cand_score=ws_array(ws, lay["cand_score"], np.float32, (b, hkv * g, budget.n_cand)),
        idx=i1.cpu().numpy(), score=sc1.cpu().numpy())
    o1h = o1.cpu().numpy()
    signs = workloads.rotation_signs(28)
    for h in range(hkv):
        orc = oracle_group(K[0, h, sink:sink + n], signs)
        for gg in range(g):
            hq = h * g + gg
            check_head(inter, 0, h, gg, g, Q[0, hq], orc, signs, budget, n)
            retrieved = [sink + int(j) for j in inter["idx"][0, hq] if j >= 0]
            _close(o1h[0, hq], owin.window_attention(Q[0, hq], K[0, h], V[0, h], _dense(win), retrieved, SCALE),
                   (h, gg))
    i2, _, _ = pk.retrieve(cfg, index, Qd, n, budget)
    o2 = pk.tiered_attend(cfg, Qd, Kw, Vw, Kr, Vr, i2, win, SCALE, kv_host_mapped=host)
    _, _, o3, _ = pk.retrieve_window_attend(cfg, index, Qd, n, budget, Kd, Vd, win, SCALE)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(i1.cpu().numpy(), i2.cpu().numpy())
    for o in (o2, o3):
        np.testing.assert_array_equal(o1h.view(np.uint32), o.cpu().numpy().view(np.uint32))


@pytest.mark.parametrize("to_host", [True, False], ids=["to_pinned_host", "device_to_device"])
def test_offload_rows_copies_exactly(to_host):
    b, hkv, D = 2, 3, 128
    r = np.random.default_rng(3)
    Ks = torch.from_numpy(r.standard_normal((b, hkv, 300, D)).astype(np.float16)).cuda()
    Vs = torch.from_numpy(r.standard_normal((b, hkv, 300, D)).astype(np.float16)).cuda()
    Kd = torch.zeros((b, hkv, 1000, D), dtype=torch.float16)
    Vd = torch.zeros_like(Kd)
    Kd, Vd = (Kd.pin_memory(), Vd.pin_memory()) if to_host else (Kd.cuda(), Vd.cuda())
    side = torch.cuda.Stream()   # default priority
    with torch.cuda.stream(side):
        pk.offload_rows(Ks, Vs, 40, Kd, Vd, 700, 100)
        pk.offload_rows(Ks, Vs, 250, Kd, Vd, 0, 50)   # a second segment, as a wrapped ring range needs
    side.synchronize()
    Kh, Vh, Ksh, Vsh = (x.cpu().numpy() for x in (Kd, Vd, Ks, Vs))
    np.testing.assert_array_equal(Kh[:, :, 700:800], Ksh[:, :, 40:140])
    np.testing.assert_array_equal(Vh[:, :, 700:800], Vsh[:, :, 40:140])
    np.testing.assert_array_equal(Kh[:, :, 0:50], Ksh[:, :, 250:300])
    np.testing.assert_array_equal(Vh[:, :, 0:50], Vsh[:, :, 250:300])
    untouched = np.ones(1000, bool)
    untouched[700:800] = False
    untouched[0:50] = False
    assert not Kh[:, :, untouched].any() and not Vh[:, :, untouched].any()
