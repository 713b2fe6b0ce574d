"""Helpers shared by the GPU parity tests: run the HIP path through the C ABI,
read back every intermediate from the documented workspace layout, and
compare with the CPU oracle on the same seeded inputs.

Tolerances (floating point; every integer, byte and index result is compared
bit for bit):
  * RSQ-IP estimates: |s_gpu - s_oracle| <= 1e-4 * sum_b |term_b|, the sum of
    the absolute per-subspace terms of the oracle's estimate, so that scores
    near zero are judged against the size of what was summed;
  * top-k: every index in the symmetric difference of the GPU and oracle sets
    has an oracle estimate within that tolerance of the oracle's k-th score;
  * attention over the GPU's index set: max |do| <= 2e-3 max |o| and
    ||do||_2 <= 2e-3 ||o||_2 against float64.
"""

import numpy as np
import torch

import paper_2602_07721_amd as pk
from oracle import attention as oatt
from oracle import encode as oenc
from oracle import quantizer as oq
from oracle import retrieve as oret

TAU, A, _ = oq.lloyd_max(8)


def _slot(c):
    """Stored form of centroid id c, as documented for pariskv_index.ids."""
    return c ^ (0x07 if c & 32 else 0) ^ (0x19 if c & 64 else 0) ^ (0x0E if c & 128 else 0)


# slot is an involution, so the same table maps stored bytes back to ids.
SLOT = np.array([_slot(c) for c in range(256)], dtype=np.uint8)
RTOL_SCORE = 1e-4
RTOL_ATT = 2e-3


def decode_rec(rec):
    """Record bytes [..., 128] -> (codes uint8 [N, 128], W float32 [N, 16])."""
    words = np.ascontiguousarray(rec).reshape(-1, 128).view(np.uint32).reshape(-1, 8, 4)
    code_words = words[:, :, :2].reshape(-1, 16)
    W = np.ascontiguousarray(words[:, :, 2:]).reshape(-1, 16).view(np.float32)
    codes = np.stack([(code_words >> (4 * j)) & 15 for j in range(8)], axis=-1)
    return codes.reshape(-1, 128).astype(np.uint8), W


def ws_array(ws, off, dtype, shape):
    n = int(np.prod(shape)) * np.dtype(dtype).itemsize
    return ws[off:off + n].cpu().numpy().view(dtype).reshape(shape)


class GpuRun:
    """Encode K, retrieve for Q and attend, all on cuda:0; keeps host copies."""

    def __init__(self, K, V, Q, signs, q_per_kv, budget, scale, capacity=None, encode=True):
        b, hkv, n, D = K.shape
        self.n = n
        self.cfg = pk.Config(hkv, q_per_kv, capacity or max(n, 1), signs)
        self.budget = budget
        self.K = torch.from_numpy(np.ascontiguousarray(K)).cuda()
        self.V = torch.from_numpy(np.ascontiguousarray(V)).cuda() if V is not None else None
        self.Q = torch.from_numpy(np.ascontiguousarray(Q)).cuda()
        self.index = pk.Index.empty(self.cfg, b)
        self.scale = scale
        if encode:
            pk.encode(self.cfg, self.index, self.K)

    def retrieve(self, n=None):
        n = self.n if n is None else n
        b = self.Q.shape[0]
        self.out_score = torch.empty((b, self.cfg.n_q_heads, self.budget.top_k), dtype=torch.float32,
                                     device="cuda")
        self.out_idx, _, self.ws = pk.retrieve(self.cfg, self.index, self.Q, n, self.budget,
                                               out_score=self.out_score)
        self.layout = pk.workspace_layout(self.cfg, b, n, self.budget)
        return self

    def retrieve_attend(self, K=None, V=None, host_mapped=False):
        """pariskv_retrieve_attend (retrieval with the attention fused into its top-k), the
        call the benchmark times; returns the attention output on the host."""
        b = self.Q.shape[0]
        K = self.K if K is None else K
        V = self.V if V is None else V
        self.out_score = torch.empty((b, self.cfg.n_q_heads, self.budget.top_k), dtype=torch.float32,
                                     device="cuda")
        self.out_idx, _, self.out, self.ws = pk.retrieve_attend(
            self.cfg, self.index, self.Q, self.n, self.budget, K, V, self.scale, out_score=self.out_score,
            kv_host_mapped=host_mapped)
        self.layout = pk.workspace_layout(self.cfg, b, self.n, self.budget)
        torch.cuda.synchronize()
        return self.out.cpu().numpy()

    def attend(self, idx=None, host_mapped=False):
        idx = self.out_idx if idx is None else idx
        K, V = self.K, self.V
        if host_mapped:
            K = K.cpu().pin_memory()
            V = V.cpu().pin_memory()
        self.out = pk.sparse_attend(self.cfg, self.Q, K, V, idx, self.scale, kv_host_mapped=host_mapped)
        torch.cuda.synchronize()
        return self.out.cpu().numpy()

    # ---- read-back of the index and the workspace intermediates
    def host_index(self, n=None):
        n = self.n if n is None else n
        torch.cuda.synchronize()
        ids = SLOT[self.index.ids[:, :, :n].cpu().numpy()]
        rec = self.index.rec[:, :, :n].cpu().numpy()
        counts = self.index.counts.cpu().numpy().view(np.uint32)
        return ids, rec, counts

    def intermediates(self):
        torch.cuda.synchronize()
        L, ws = self.layout, self.ws
        b, hq, hkv = self.Q.shape[0], self.cfg.n_q_heads, self.cfg.n_kv_heads
        out = dict(
            zq=ws_array(ws, L["zq"], np.float32, (b, hq, 128)),
            lut=ws_array(ws, L["lut"], np.uint32, (b, hkv, L["quads"], 16, 256)),
            S=ws_array(ws, L["score8"], np.uint8, (b, hq, L["n_pad"])),
            thresh=ws_array(ws, L["thresh"], np.int32, (b, hq, 8)),
            cand=ws_array(ws, L["cand"], np.int32, (b, hq, self.budget.n_cand)),
            cand_score=ws_array(ws, L["cand_score"], np.float32, (b, hq, self.budget.n_cand)),
            idx=self.out_idx.cpu().numpy(),
            score=self.out_score.cpu().numpy(),
        )
        return out


def lut_for_head(lut, seq, kvh, g):
    """Unpack the packed bonus table of query head g (within its KV group) -> [16][256],
    indexed by centroid id (the table itself is indexed by slot)."""
    words = lut[seq, kvh, g // 4][:, SLOT]
    return ((words >> (8 * (g % 4))) & 0xFF).astype(np.int64)


def oracle_group(K_group, signs, rotate=True, alpha_correction=True):
    ids, codes, W = oenc.encode(K_group, signs, TAU, A, 16, rotate, alpha_correction)
    return ids, codes, W, oenc.cluster_counts(ids, 8)


def abs_terms(q, codes, W, signs, rotate=True):
    """sum_b |W_b <v_b, z_b>| / D per key, via the oracle estimator one subspace at a time."""
    W = np.asarray(W, dtype=np.float64)
    tot = np.zeros(W.shape[0])
    for b in range(16):
        Wb = np.zeros_like(W)
        Wb[:, b] = W[:, b]
        tot += np.abs(oret.rsqip_scores(q, codes, Wb, signs, A, 16, rotate))
    return tot


def check_index(gpu_ids, gpu_rec, gpu_counts, oracle):
    ids, codes, W, cnt = oracle
    np.testing.assert_array_equal(gpu_ids, ids)
    gcodes, gW = decode_rec(gpu_rec)
    np.testing.assert_array_equal(gcodes, codes)
    np.testing.assert_array_equal(gW.view(np.uint32), W.view(np.uint32))
    np.testing.assert_array_equal(gpu_counts.astype(np.int64), cnt)


def check_head(inter, seq, kvh, g, q_per_kv, q, oracle, signs, budget, n, rotate=True):
    """Bit-exact Stage I, toleranced Stage II for one query head; returns oracle result dict.
    rotate / budget.flags select the ablation variants the index and call used."""
    ids, codes, W, cnt = oracle
    hq = kvh * q_per_kv + g
    r = oret.retrieve_head(q, ids, codes, W, cnt, signs, A, 16, budget.n_cand, budget.n_collide,
                           budget.top_k, rotate=rotate, binary=bool(budget.flags & pk.BINARY_COLLISIONS))
    # query transform: z / D rounded to float
    np.testing.assert_array_equal(inter["zq"][seq, hq], (r["z"] / 128.0).astype(np.float32))
    np.testing.assert_array_equal(lut_for_head(inter["lut"], seq, kvh, g), r["lut"])
    np.testing.assert_array_equal(inter["S"][seq, hq, :n].astype(np.int64), r["S"])
    C = min(budget.n_cand, n)
    theta, gt, quota = oret.selection_threshold(r["S"], budget.n_cand)
    np.testing.assert_array_equal(inter["thresh"][seq, hq, :4], [theta, gt, quota, C])
    # the histogram floor the scan used, and whether the threshold came from the recount:
    # the recount runs exactly when the floor overshoots #{S >= floor} >= C
    floor, recount = int(inter["thresh"][seq, hq, 4]), int(inter["thresh"][seq, hq, 5])
    assert 1 <= floor <= 97 and recount == int(floor > 1 and np.sum(r["S"] >= floor) < C)
    if budget.flags & pk.EXACT_RECOUNT:
        assert floor == 97 and recount == 1
    np.testing.assert_array_equal(inter["cand"][seq, hq, :C], r["cand"])
    # RSQ-IP estimates
    at = abs_terms(q, codes[r["cand"]], W[r["cand"]], signs, rotate)
    gs = inter["cand_score"][seq, hq, :C].astype(np.float64)
    err = np.abs(gs - r["cand_scores"])
    bad = err > RTOL_SCORE * at + 1e-30
    assert not bad.any(), f"rerank off at {np.flatnonzero(bad)[:5]}: {err[bad][:5]} vs {at[bad][:5]}"
    # final top-k
    k = budget.top_k
    kk = min(k, C)
    gi = inter["idx"][seq, hq]
    gsc = inter["score"][seq, hq]
    assert np.all(gi[kk:] == -1) and np.all(np.isneginf(gsc[kk:]))
    gi, gsc = gi[:kk], gsc[:kk].astype(np.float64)
    assert len(set(gi.tolist())) == kk
    pos = {int(c): i for i, c in enumerate(r["cand"])}
    assert all(int(i) in pos for i in gi)
    o_sc = r["cand_scores"]
    tol = RTOL_SCORE * at
    kth = r["scores"][kk - 1]
    kth_tol = tol[pos[int(r["idx"][kk - 1])]]
    for i in set(gi.tolist()) ^ set(int(x) for x in r["idx"][:kk]):
        p = pos[i]
        assert abs(o_sc[p] - kth) <= tol[p] + kth_tol, (i, o_sc[p], kth)
    # the winners are listed in ascending key index
    assert np.all(np.diff(gi) > 0)
    # and are exactly the top kk of the GPU's own float32 estimates (ties: lower index)
    gcs = inter["cand_score"][seq, hq, :C]
    own = np.sort(r["cand"][np.lexsort((r["cand"], -gcs.astype(np.float64)))[:kk]])
    np.testing.assert_array_equal(gi, own)
    np.testing.assert_array_equal(gsc.astype(np.float32), gcs[[pos[int(i)] for i in gi]])
    g_at = np.array([tol[pos[int(i)]] for i in gi])
    g_ref = np.array([o_sc[pos[int(i)]] for i in gi])
    assert np.all(np.abs(gsc - g_ref) <= g_at + 1e-30)
    return r


def check_attention(o_gpu, q, Kg, Vg, idx, scale):
    o_ref = oatt.sparse_attention(q, Kg, Vg, idx, scale=scale)
    d = np.abs(o_gpu.astype(np.float64) - o_ref)
    mx = np.max(np.abs(o_ref))
    assert d.max() <= RTOL_ATT * mx + 1e-30, (d.max(), mx)
    assert np.linalg.norm(d) <= RTOL_ATT * np.linalg.norm(o_ref) + 1e-30
    return o_ref
