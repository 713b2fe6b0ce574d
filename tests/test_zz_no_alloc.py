"""pariskv_retrieve_attend_noalloc (intermediates in the library's static per-device
scratch array) against pariskv_retrieve_attend (caller workspace): the same outputs bit
for bit, on two calls in a row that share the array, the second with smaller shapes, and
one group of each call against the CPU oracle."""

import numpy as np
import pytest
import torch

import paper_2602_07721_amd as pk
import workloads
from parity import check_attention, check_head, check_index, oracle_group, GpuRun, SLOT

pytestmark = pytest.mark.gpu
SCALE = 1.0 / np.sqrt(128.0)

CASES = [
    # name, batch, hkv, G, n, (C, C_rho, k)
    ("larger", 2, 4, 4, 20000, (2048, 4096, 256)),
    ("smaller", 1, 2, 6, 5003, (512, 1024, 64)),
]


def _setup(name, batch, hkv, G, n, bud):
    wc = workloads.Config(name, batch=batch, n_kv_heads=hkv, q_per_kv=G, n=n, n_cand=bud[0],
                          n_collide=bud[1], top_k=bud[2], seed=300 + len(name))
    K, V = workloads.layer_kv(wc)
    Q, _ = workloads.layer_queries(wc, K)
    signs = workloads.rotation_signs(wc.seed)
    run = GpuRun(K, V, Q, signs, G, pk.Budget(*bud), SCALE)
    return wc, K, V, Q, signs, run


def test_noalloc_matches_the_workspace_entry_point_on_two_calls_in_a_row():
    runs = [_setup(*c) for c in CASES]
    torch.cuda.synchronize()
    # the two no-alloc calls back to back: the second reuses the array the first left behind
    outs = []
    for (wc, K, V, Q, signs, run), case in zip(runs, CASES):
        print(f"case noalloc {case}", flush=True)
        b, hq, k = wc.batch, run.cfg.n_q_heads, run.budget.top_k
        oi = torch.full((b, hq, k), -7, dtype=torch.int32, device="cuda")
        osc = torch.full((b, hq, k), 7.0, dtype=torch.float32, device="cuda")
        oo = torch.full((b, hq, 128), 7.0, dtype=torch.float32, device="cuda")
        pk.retrieve_attend_noalloc(run.cfg, run.index, run.Q, wc.n, run.budget, run.K, run.V, SCALE,
                                   out_idx=oi, out=oo, out_score=osc)
        outs.append((oi, osc, oo))
    torch.cuda.synchronize()
    for (wc, K, V, Q, signs, run), (oi, osc, oo), case in zip(runs, outs, CASES):
        print(f"case reference {case}", flush=True)
        o_ref = run.retrieve_attend()
        inter = run.intermediates()
        np.testing.assert_array_equal(oi.cpu().numpy(), inter["idx"])
        np.testing.assert_array_equal(osc.cpu().numpy().view(np.uint32), inter["score"].view(np.uint32))
        np.testing.assert_array_equal(oo.cpu().numpy().view(np.uint32), o_ref.view(np.uint32))
        # one (sequence, KV head) group of the call through the oracle as well
        s, h = wc.batch - 1, wc.n_kv_heads - 1
        gids, grec, gcnt = run.host_index()
        orc = oracle_group(K[s, h], signs)
        check_index(gids[s, h], grec[s, h], gcnt[s, h], orc)
        for g in range(wc.q_per_kv):
            hq = h * wc.q_per_kv + g
            check_head(inter, s, h, g, wc.q_per_kv, Q[s, hq], orc, signs, run.budget, wc.n)
            check_attention(oo.cpu().numpy()[s, hq], Q[s, hq], K[s, h], V[s, h], inter["idx"][s, hq], SCALE)
