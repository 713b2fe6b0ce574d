"""GPU parity of the ablation variants (Sec. "Ablation Studies"): an index encoded without
the rotation and/or without the alpha-correction, and binary (0/1) collision scores.  Codes,
weights, counts, bonus tables, scores and candidates bit for bit against the oracle's
variant; estimates, top-k and attention within the usual tolerances."""

import numpy as np
import pytest
import torch

import paper_2602_07721_amd as pk
import workloads
from parity import GpuRun, SLOT, check_attention, check_head, check_index, oracle_group

pytestmark = pytest.mark.gpu

VARIANTS = {
    "no_rotation": (pk.NO_ROTATION, 0),
    "no_alpha": (pk.NO_ALPHA_CORRECTION, 0),
    "binary": (0, pk.BINARY_COLLISIONS),
    "all_three": (pk.NO_ROTATION | pk.NO_ALPHA_CORRECTION, pk.BINARY_COLLISIONS),
}


@pytest.mark.parametrize("name", list(VARIANTS))
def test_variant_matches_the_oracle(name):
    cfg_flags, bud_flags = VARIANTS[name]
    rotate = not (cfg_flags & pk.NO_ROTATION)
    alpha = not (cfg_flags & pk.NO_ALPHA_CORRECTION)
    wc = workloads.Config("abl", batch=1, n_kv_heads=2, q_per_kv=4, n=6000, n_cand=512, n_collide=1024,
                          top_k=64, seed=41)
    print(f"[ablation] {name}: config flags {cfg_flags}, budget flags {bud_flags}", flush=True)
    K, V = workloads.layer_kv(wc)
    Q, _ = workloads.layer_queries(wc, K)
    signs = workloads.rotation_signs(wc.seed)
    budget = pk.Budget(wc.n_cand, wc.n_collide, wc.top_k, flags=bud_flags)
    scale = 1.0 / np.sqrt(128.0)
    run = GpuRun(K, V, Q, signs, wc.q_per_kv, budget, scale, encode=False)
    run.cfg = pk.Config(wc.n_kv_heads, wc.q_per_kv, wc.n, signs, flags=cfg_flags)
    run.index = pk.Index.empty(run.cfg, 1)
    pk.encode(run.cfg, run.index, run.K)
    run.retrieve()
    inter = run.intermediates()
    o = run.attend()
    ids, rec, cnt = run.host_index()
    for h in range(wc.n_kv_heads):
        orc = oracle_group(K[0, h], signs, rotate, alpha)
        check_index(ids[0, h], rec[0, h], cnt[0, h], orc)
        for g in range(wc.q_per_kv):
            hq = h * wc.q_per_kv + g
            r = check_head(inter, 0, h, g, wc.q_per_kv, Q[0, hq], orc, signs, budget, wc.n, rotate)
            if bud_flags & pk.BINARY_COLLISIONS:
                assert r["S"].max() <= 16
            check_attention(o[0, hq], Q[0, hq], K[0, h], V[0, h], inter["idx"][0, hq], scale)


def test_variants_leave_the_published_path_unchanged():
    # flags 0 through the new fields = the published method, bit for bit with a second encode
    wc = workloads.Config("abl0", batch=1, n_kv_heads=1, q_per_kv=4, n=3000, n_cand=256, n_collide=512,
                          top_k=32, seed=42)
    K, V = workloads.layer_kv(wc)
    Q, _ = workloads.layer_queries(wc, K)
    signs = workloads.rotation_signs(wc.seed)
    outs = []
    for flags in (0, pk.NO_ROTATION, 0):
        cfg = pk.Config(1, 4, wc.n, signs, flags=flags)
        index = pk.Index.empty(cfg, 1)
        pk.encode(cfg, index, torch.from_numpy(K).cuda())
        idx, _, _ = pk.retrieve(cfg, index, torch.from_numpy(Q).cuda(), wc.n, pk.Budget(256, 512, 32))
        outs.append((index.rec.cpu().numpy(), idx.cpu().numpy()))
    np.testing.assert_array_equal(outs[0][0], outs[2][0])
    np.testing.assert_array_equal(outs[0][1], outs[2][1])
    assert not np.array_equal(outs[0][0], outs[1][0])
