#!/usr/bin/env python3
"""Decode-step benchmark of the ParisKV retrieval path on one MI355X.

Workload (default): one Llama-3-8B-shaped layer at 128K context in the
throughput regime -- 8 independent sequences x 8 KV heads x 4 query heads,
N = 131072 keys per sequence, D = 128, candidate budget C = 8192, collision
budget C_rho = 16384, top-k = 512, synthetic keys (outlier-channel Gaussian,
see workloads/) and fresh planted-needle queries at every step.

One step = the whole hot path for the whole batch: pariskv_retrieve_attend
(query transform + bonus tables, collision scan, selection, RSQ-IP rerank,
top-k with the attention over the selected K/V rows fused into it), or with
--separate pariskv_retrieve followed by pariskv_sparse_attend.  Keys are
encoded once before timing (reported separately).  K, V, the index and all
queries are resident in HBM before the timed region starts.

Between timed steps the 256 MB Infinity Cache and the L2s are flushed by
reading a 1 GiB buffer (outside the step's events): in a real model the other
layers' weights evict this layer's codes between two of its steps.  The
flush reads rather than writes so that no dirty lines are left for the timed
step to write back.
The per-step time is the HIP-event interval around each step on the launch
stream; per-kernel times come from the library's own event profiler on the
same stream during the same timed steps.

Prints one JSON line (see the roofline and cpu_baseline fields).
"""

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0  # MI355X HBM3E, vendor figure


def parse():
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=64)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default="batch8_128k")
    ap.add_argument("--no-flush", action="store_true", help="keep caches warm between steps")
    ap.add_argument("--no-profile", action="store_true", help="no per-kernel events in the timed steps")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-groups", type=int, default=64,
                    help="(sequence, KV head) groups the oracle baseline samples, at most one per host core")
    ap.add_argument("--cpu-steps", type=int, default=4)
    ap.add_argument("--separate", action="store_true",
                    help="run the step as pariskv_retrieve + pariskv_sparse_attend instead of the fused "
                         "pariskv_retrieve_attend")
    ap.add_argument("--kv-host", action="store_true",
                    help="keep K/V in pinned host memory and attend through host-mapped pointers")
    ap.add_argument("--extras", action="store_true",
                    help="also measure the drift workload (append + retrieve + attend per step), the "
                         "same decode with Sink/Local/Update Buffer regions (buffer updates every 256 "
                         "steps and every step), the recall of the ablation variants, the candidate ratio "
                         "needed at each KV length, GQA-group "
                         "de-duplication of the host-link fetch, and attention over K/V in pinned host memory")
    ap.add_argument("--drift-steps", type=int, default=4096,
                    help="decode steps of the drift measurement (the full workload runs 32768)")
    ap.add_argument("--offload-steps", type=int, default=0,
                    help="also run the 1M-token offload setting (GPU window ring, Retrieval K/V in pinned "
                         "host memory, buffer updates offloaded on a second stream) for this many steps")
    ap.add_argument("--no-warm", action="store_true", help="skip the warm-cache loop")
    ap.add_argument("--group-fetch", action="store_true",
                    help="PARISKV_GROUP_FETCH: each quad of query heads fetches every distinct K/V row once")
    ap.add_argument("--group-share", type=int, default=0,
                    help="query heads per KV group planted on one shared needle (overlapping winner lists)")
    return ap.parse_args()


def algorithmic_bytes(wc, c_eff, parts=1):
    """Bytes each kernel must move per launch (whole batch), by its definition.  With a
    two-pass top-k (parts > 1 slices per row) the final pass reads the slices' winners."""
    b, hkv, G, n, k = wc.batch, wc.n_kv_heads, wc.q_per_kv, wc.n, wc.top_k
    hq = hkv * G
    quads = (G + 3) // 4
    n_chunks = (n + 4095) // 4096
    C = c_eff
    S = parts * k if parts > 1 else C  # entries the (final) top-k pass selects from
    return {
        # query heads (fp16) + counts read, bonus tables and z/D written
        "query_lut": b * hq * 128 * 2 + b * hkv * 16 * 256 * 4 + b * hkv * quads * 16 * 256 * 4
                     + b * hq * 128 * 4,
        # 16 id bytes per key and KV head (once per quad of query heads) + 1 score byte per key
        # and query head written (the per-chunk suffix histograms are 0.1% on top)
        "collide": b * hkv * quads * n * 16 + b * hq * n,
        # per-chunk suffix histograms read
        "threshold": b * hq * n_chunks * 98 * 4,
        # score bytes read, candidate index written, then per candidate the 128-byte record
        # gathered and its 4-byte estimate written
        "compact_rerank": b * hq * n + b * hq * C * (4 + 128 + 4),
        # first pass of a two-pass top-k: C estimates + C indices read, k winners (index +
        # estimate) written per 4096-candidate slice
        "topk_part": b * hq * (C * 8 + parts * k * 8),
        # S estimates + S indices read, k indices + k scores written
        "topk": b * hq * (S * 8 + k * 8),
        # 256-byte K row + 256-byte V row + 4-byte index per selected key
        "attend": b * hq * k * (512 + 4),
        # the fused top-k + attention: both, minus the index re-read
        "topk_attend": b * hq * (S * 8 + k * 8) + b * hq * k * 512,
    }


def source_digest():
    """SHA-256 of the kernel sources: HBM counter figures are valid only for this digest."""
    import hashlib
    h = hashlib.sha256()
    src = os.path.join(ROOT, "paper_2602_07721_amd", "csrc")
    for name in sorted(os.listdir(src)):
        with open(os.path.join(src, name), "rb") as f:
            h.update(name.encode() + b"\0" + f.read())
    return h.hexdigest()


def measured_traffic(workload):
    """HBM bytes per launch from the committed rocprofv3 FETCH_SIZE / WRITE_SIZE summary,
    or {} when it is missing or was taken from other kernel sources."""
    path = os.path.join(ROOT, "profiles", f"hbm_traffic_{workload}.md")
    if not os.path.exists(path):
        return {}
    for line in open(path):
        if line.startswith("<!-- traffic-json:"):
            data = json.loads(line[len("<!-- traffic-json:"):].rsplit("-->", 1)[0])
            if data.get("source_sha256") == source_digest():
                return data.get("bytes_per_launch", {})
    return {}


def _oracle_worker(wname, seq, kvh, steps, start, results):
    """Child process (spawned: no torch, no GPU): regenerate one (sequence, KV head)
    group of a workload from its seeds, encode it with the oracle (prefill, untimed),
    wait for the other workers, then time the oracle's retrieve + attend of the group's
    query heads over `steps` decode steps, single-threaded."""
    import numpy as np
    from threadpoolctl import threadpool_limits

    import workloads
    from oracle import attention as oatt
    from oracle import encode as oenc
    from oracle import quantizer as oq
    from oracle import retrieve as oret

    wc = workloads.CONFIGS[wname]
    signs = workloads.rotation_signs(wc.seed)
    tau, a, _ = oq.lloyd_max(8)
    K = workloads.head_keys(wc.seed, seq, kvh, wc.n)
    V = workloads.head_values(wc.seed, seq, kvh, wc.n)
    Qs = [workloads.needle_queries(K, wc.seed, seq, kvh, wc.q_per_kv, st)[0] for st in range(steps)]
    scale = 1.0 / np.sqrt(wc.head_dim)
    with threadpool_limits(limits=1):
        ids, codes, W = oenc.encode(K, signs, tau, a, 16)
        cnt = oenc.cluster_counts(ids, 8)
        start.wait()
        t0 = time.perf_counter()
        for st in range(steps):
            for g in range(wc.q_per_kv):
                q = Qs[st][g]
                r = oret.retrieve_head(q, ids, codes, W, cnt, signs, a, 16, wc.n_cand, wc.n_collide, wc.top_k)
                oatt.sparse_attention(q, K, V, r["idx"], scale=scale)
        results.put(time.perf_counter() - t0)


def cpu_baseline(wname, groups, steps):
    """The oracle's retrieve + attend timed on the host cores: one spawned process per
    sampled (sequence, KV head) group, all timed together after a common start, each
    single-threaded.  Returns the whole-layer step time the cores sustain."""
    import multiprocessing as mp

    import workloads

    wc = workloads.CONFIGS[wname]
    cores = len(os.sched_getaffinity(0))
    total = wc.batch * wc.n_kv_heads
    groups = max(1, min(groups, cores, total))
    picks = [((g * 3) % wc.batch, (g * 5) % wc.n_kv_heads) if total > groups else (g // wc.n_kv_heads,
             g % wc.n_kv_heads) for g in range(groups)]
    ctx = mp.get_context("spawn")
    start = ctx.Barrier(groups)
    results = ctx.Queue()
    procs = [ctx.Process(target=_oracle_worker, args=(wname, s, h, steps, start, results)) for s, h in picks]
    for p in procs:
        p.start()
    el = [results.get() for _ in procs]
    for p in procs:
        p.join()
    per_group_step = float(sum(el)) / (groups * steps)  # seconds, one core busy
    # `groups` cores work in parallel; a layer step is `total` group-steps.
    value = per_group_step * total / groups * 1e6
    return {
        "value": round(value, 1),
        "unit": "us/step/layer",
        "cores": groups,
        "kind": "oracle",
        "sample": (f"{wname}: {groups} of {total} (sequence, KV head) groups, one per core, each "
                   f"single-threaded NumPy float64 retrieve+attend for its {wc.q_per_kv} query heads x "
                   f"{steps} steps ({sum(el):.1f} s of CPU work, {max(el):.1f} s wall), scaled to all "
                   f"{total} groups of a step on {groups} cores; host has {cores} cores"),
    }


def drift_run(pk, torch, np, workloads, dev, steps):
    """The drift workload: 32K-key prefill, then per step one appended key per
    (sequence, KV head), retrieval with C = ceil(n/16), C_rho = 2C and attention.
    Returns per-step time and recall@k against exact top-k every 256 steps."""
    wc = workloads.CONFIGS["drift"]
    signs = workloads.rotation_signs(wc.seed)
    total = steps
    cap = wc.n + total
    K0, V0 = workloads.layer_kv(wc, threads=16)
    Kall = np.zeros((wc.batch, wc.n_kv_heads, cap, wc.head_dim), np.float16)
    Vall = np.zeros_like(Kall)
    Kall[:, :, :wc.n] = K0
    Vall[:, :, :wc.n] = V0
    rng = np.random.default_rng(wc.seed)
    for s in range(wc.batch):
        for h in range(wc.n_kv_heads):
            Kall[s, h, wc.n:] = workloads.drift_keys(wc.seed, s, h, 0, total, total)
            Vall[s, h, wc.n:] = rng.standard_normal((total, wc.head_dim)).astype(np.float16)
    Kd = torch.from_numpy(Kall).to(dev)
    Vd = torch.from_numpy(Vall).to(dev)
    cfg = pk.Config(wc.n_kv_heads, wc.q_per_kv, cap, signs)
    index = pk.Index.empty(cfg, wc.batch, dev)
    pk.encode(cfg, index, Kd[:, :, :wc.n].contiguous())
    hq = cfg.n_q_heads
    c_max = -(-cap // 16)
    ws = torch.empty(pk.retrieve_workspace_size(cfg, wc.batch, cap, pk.Budget(c_max, 2 * c_max, wc.top_k)),
                     dtype=torch.uint8, device=dev)
    out_idx = torch.empty((wc.batch, hq, wc.top_k), dtype=torch.int32, device=dev)
    out = torch.empty((wc.batch, hq, wc.head_dim), dtype=torch.float32, device=dev)
    # Queries of step t: fresh draws from the current key law, one per query head.
    evals = set(range(0, total, 256)) | {total - 1}
    Qs = np.stack([np.stack([workloads.drift_queries(wc.seed, s, h, total, wc.q_per_kv)
                             for h in range(wc.n_kv_heads)], axis=1)
                   for s in range(wc.batch)], axis=1).reshape(total, wc.batch, hq, wc.head_dim)
    Qd = torch.from_numpy(Qs).to(dev)
    newk = Kd[:, :, wc.n:].permute(2, 0, 1, 3).contiguous()  # [t][b][Hkv][D]
    scale = 1.0 / np.sqrt(wc.head_dim)
    recalls = []
    block_us = []  # per-step GPU time of each block of steps between evaluations
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    t_block = 0
    for t in range(total):
        n = wc.n + t + 1
        C = -(-n // 16)
        bud = pk.Budget(C, 2 * C, wc.top_k)
        pk.append(cfg, index, newk[t].unsqueeze(2), wc.n + t)
        pk.retrieve(cfg, index, Qd[t], n, bud, out_idx=out_idx, workspace=ws)
        pk.sparse_attend(cfg, Qd[t], Kd, Vd, out_idx, scale, out=out)
        t_block += 1
        if t in evals:
            e1.record()
            torch.cuda.synchronize()
            block_us.append((t, e0.elapsed_time(e1) * 1e3 / t_block))
            # exact top-k by float32 inner products over the n cached keys (reference only)
            kf = Kd[:, :, :n].float()
            q = Qd[t].float().reshape(wc.batch, wc.n_kv_heads, wc.q_per_kv, wc.head_dim)
            sc = torch.matmul(q, kf.transpose(2, 3).contiguous())
            ex = torch.topk(sc, wc.top_k, dim=-1).indices.reshape(wc.batch, hq, wc.top_k)
            got = out_idx.long()
            hit = (got.unsqueeze(-1) == ex.unsqueeze(-2)).any(-1).float().mean().item()
            recalls.append((t, hit))
            del kf, sc
            torch.cuda.synchronize()
            t_block = 0
            e0.record()
    torch.cuda.synchronize()
    steps_w = [b for b in block_us[1:]]  # the first block (step 0 alone) carries warm-up
    us = float(np.mean([u for _, u in steps_w])) if steps_w else block_us[0][1]
    r = np.array([h for _, h in recalls])
    return {
        "workload": (f"drift: {wc.batch} seqs x {wc.n_kv_heads} KV heads x {wc.q_per_kv} query heads, "
                     f"{wc.n}-key prefill + {total} decode steps (1 appended key per KV head per step, "
                     f"mean drifting 2 sigma), C = ceil(n/16), C_rho = 2C, k = {wc.top_k}"),
        "us_per_step_append_retrieve_attend": round(us, 2),
        "us_per_step_first_block": round(block_us[1][1], 2) if len(block_us) > 1 else None,
        "us_per_step_last_block": round(block_us[-1][1], 2),
        "timing": "HIP events around each block of 256 steps (host launch included), between recall checks",
        "recall_at_k_vs_exact": {"first": round(float(r[0]), 4), "last": round(float(r[-1]), 4),
                                 "min": round(float(r.min()), 4), "mean": round(float(r.mean()), 4),
                                 "every": 256, "points": len(r)},
        "note": "exact top-k by float32 inner products on the GPU (a quality figure, parity unpinned)",
    }


def window_run(pk, torch, np, workloads, dev, steps, sink=128, local=512, updates=(256, 1)):
    """Decode with the four KV regions (Sec. "Buffer Update") on the drift workload's keys:
    Sink 128 and Local 512 attended densely, the Retrieval region indexed; every m steps the
    rows leaving Local are encoded straight from the key cache (pariskv_append_rows), and each
    step runs pariskv_retrieve_window_attend (retrieval over Retrieval with C = ceil(n/16),
    C_rho = 2C, then attention over Sink + winners + Local + Update Buffer).  Runs the same
    decode once per update interval m; per-step GPU time from HIP events around every step."""
    wc = workloads.CONFIGS["drift"]
    signs = workloads.rotation_signs(wc.seed)
    P = wc.n
    cap = P + steps
    K0, V0 = workloads.layer_kv(wc, threads=16)
    Kall = np.zeros((wc.batch, wc.n_kv_heads, cap, wc.head_dim), np.float16)
    Vall = np.zeros_like(Kall)
    Kall[:, :, :P] = K0
    Vall[:, :, :P] = V0
    rng = np.random.default_rng(wc.seed)
    for s in range(wc.batch):
        for h in range(wc.n_kv_heads):
            Kall[s, h, P:] = workloads.drift_keys(wc.seed, s, h, 0, steps, steps)
            Vall[s, h, P:] = rng.standard_normal((steps, wc.head_dim)).astype(np.float16)
    Kd = torch.from_numpy(Kall).to(dev)
    Vd = torch.from_numpy(Vall).to(dev)
    hq = wc.n_kv_heads * wc.q_per_kv
    Qs = np.stack([np.stack([workloads.drift_queries(wc.seed, s, h, steps, wc.q_per_kv)
                             for h in range(wc.n_kv_heads)], axis=1)
                   for s in range(wc.batch)], axis=1).reshape(steps, wc.batch, hq, wc.head_dim)
    Qd = torch.from_numpy(Qs).to(dev)
    scale = 1.0 / np.sqrt(wc.head_dim)
    cfg = pk.Config(wc.n_kv_heads, wc.q_per_kv, cap, signs)
    c_max = -(-cap // 16)
    ws = torch.empty(pk.retrieve_workspace_size(cfg, wc.batch, cap, pk.Budget(c_max, 2 * c_max, wc.top_k)),
                     dtype=torch.uint8, device=dev)
    out_idx = torch.empty((wc.batch, hq, wc.top_k), dtype=torch.int32, device=dev)
    out = torch.empty((wc.batch, hq, wc.head_dim), dtype=torch.float32, device=dev)
    evals = set(range(0, steps, 512)) | {steps - 1}
    res = {}
    for m in updates:
        index = pk.Index.empty(cfg, wc.batch, dev)
        win0, n_idx = pk.window_regions(P, 0, sink, local, m)
        pk.append_rows(cfg, index, Kd, win0.retr_begin, n_idx, 0)  # the prompt's Retrieval region
        starts = [torch.cuda.Event(enable_timing=True) for _ in range(steps)]
        ends = [torch.cuda.Event(enable_timing=True) for _ in range(steps)]
        upd = np.zeros(steps, bool)
        recalls = []
        torch.cuda.synchronize()
        for t in range(steps):
            win, n_retr = pk.window_regions(P, t, sink, local, m)
            starts[t].record()
            if n_retr > n_idx:
                pk.append_rows(cfg, index, Kd, win.retr_begin + n_idx, n_retr - n_idx, n_idx)
                n_idx = n_retr
                upd[t] = True
            C = -(-n_retr // 16)
            pk.retrieve_window_attend(cfg, index, Qd[t], n_retr, pk.Budget(C, 2 * C, wc.top_k), Kd, Vd, win,
                                      scale, out_idx=out_idx, out=out, workspace=ws)
            ends[t].record()
            if t in evals:
                # recall of the exact top-k over all P + t tokens by the attended rows
                # (Sink + Local/Buffer + the retrieved winners); a quality figure
                T = P + t
                kf = Kd[:, :, :T].float()
                q = Qd[t].float().reshape(wc.batch, wc.n_kv_heads, wc.q_per_kv, wc.head_dim)
                sc = torch.matmul(q, kf.transpose(2, 3).contiguous())
                ex = torch.topk(sc, wc.top_k, dim=-1).indices.reshape(wc.batch, hq, wc.top_k)
                dense = (ex < win.sink_len) | ((ex >= win.dense_begin) & (ex < win.dense_end))
                got = out_idx.long() + win.retr_begin
                got = torch.where(out_idx >= 0, got, torch.full_like(got, -1))
                hit = dense | (ex.unsqueeze(-1) == got.unsqueeze(-2)).any(-1)
                recalls.append(float(hit.float().mean().item()))
                del kf, sc
        torch.cuda.synchronize()
        us = np.array([starts[t].elapsed_time(ends[t]) * 1e3 for t in range(steps)])
        body = us[8:]
        ub = upd[8:]
        res[f"m{m}"] = {
            "update_every": m,
            "us_per_step": round(float(body.mean()), 2),
            "us_per_update_step": round(float(body[ub].mean()), 2) if ub.any() else None,
            "us_per_other_step": round(float(body[~ub].mean()), 2) if (~ub).any() else None,
            "updates": int(upd.sum()),
            "retrieval_keys_last": int(n_idx),
            "recall_at_k_vs_exact_all_tokens": {"first": round(recalls[0], 4), "last": round(recalls[-1], 4),
                                                "mean": round(float(np.mean(recalls)), 4)},
        }
    return {
        "workload": (f"drift keys: {wc.batch} seqs x {wc.n_kv_heads} KV heads x {wc.q_per_kv} query heads, "
                     f"{P}-token prompt + {steps} decode steps; Sink {sink}, Local {local}, Retrieval indexed "
                     f"(C = ceil(n/16), C_rho = 2C, k = {wc.top_k}); buffer update every m steps"),
        "timing": ("HIP events around each step's calls (GPU time incl. launch gaps); steps 0-7 left out; "
                   "the prompt's Retrieval region is encoded before timing"),
        **res,
    }


def ablation_run(pk, torch, np, workloads, dev, drift_steps, n_queries=8):
    """Recall of the ablation variants (Sec. "Ablation Studies") on the drift workload's keys
    after `drift_steps` drifting decode keys: per variant, the coarse-stage recall (exact
    top-k keys that reach the candidate set) and the final recall@k (exact top-k keys among
    the k winners), averaged over all query heads and `n_queries` query draws from the last
    step's key law; plus a candidate-ratio (beta) sweep of the published method."""
    wc = workloads.CONFIGS["drift"]
    signs = workloads.rotation_signs(wc.seed)
    n = wc.n + drift_steps
    K0, _ = workloads.layer_kv(wc, values=False, threads=16)
    Kall = np.zeros((wc.batch, wc.n_kv_heads, n, wc.head_dim), np.float16)
    Kall[:, :, :wc.n] = K0
    for s in range(wc.batch):
        for h in range(wc.n_kv_heads):
            Kall[s, h, wc.n:] = workloads.drift_keys(wc.seed, s, h, 0, drift_steps, drift_steps)
    Kd = torch.from_numpy(Kall).to(dev)
    hq = wc.n_kv_heads * wc.q_per_kv
    # queries from the key law of the last drift step
    Qs = np.stack([np.stack([workloads.drift_queries(wc.seed, s, h, drift_steps, wc.q_per_kv)[-n_queries:]
                             for h in range(wc.n_kv_heads)], axis=1)
                   for s in range(wc.batch)], axis=1)  # [n_queries][b][Hkv][G][D]
    Qd = torch.from_numpy(Qs.reshape(n_queries, wc.batch, hq, wc.head_dim)).to(dev)
    k = wc.top_k
    exact = []
    for i in range(n_queries):
        q = Qd[i].float().reshape(wc.batch, wc.n_kv_heads, wc.q_per_kv, wc.head_dim)
        sc = torch.matmul(q, Kd.float().transpose(2, 3).contiguous())
        exact.append(torch.topk(sc, k, dim=-1).indices.reshape(wc.batch, hq, k))
        del sc
    C16 = -(-n // 16)
    runs = [("published (rotation + alpha-correction + 6 tiers)", 0, 0, C16),
            ("binary 0/1 collisions", 0, pk.BINARY_COLLISIONS, C16),
            ("no alpha-correction", pk.NO_ALPHA_CORRECTION, 0, C16),
            ("no rotation", pk.NO_ROTATION, 0, C16),
            ("no rotation, no alpha, binary", pk.NO_ROTATION | pk.NO_ALPHA_CORRECTION, pk.BINARY_COLLISIONS, C16),
            ("published, beta = 1/32", 0, 0, -(-n // 32)),
            ("published, beta = 1/8", 0, 0, -(-n // 8))]
    out = []
    indexes = {}
    for name, cfl, bfl, C in runs:
        cfg = pk.Config(wc.n_kv_heads, wc.q_per_kv, n, signs, flags=cfl)
        if cfl not in indexes:
            index = pk.Index.empty(cfg, wc.batch, dev)
            pk.encode(cfg, index, Kd)
            indexes[cfl] = index
        index = indexes[cfl]
        bud = pk.Budget(C, 2 * C, k, flags=bfl)
        lay = pk.workspace_layout(cfg, wc.batch, n, bud)
        ws = torch.empty(lay["total"], dtype=torch.uint8, device=dev)
        coarse, final = [], []
        for i in range(n_queries):
            idx, _, _ = pk.retrieve(cfg, index, Qd[i], n, bud, workspace=ws)
            cand = ws[lay["cand"]: lay["cand"] + wc.batch * hq * C * 4].view(torch.int32)
            cand = cand.reshape(wc.batch, hq, C).long()
            ex = exact[i]
            # the candidate list is ascending: membership by binary search
            pos = torch.searchsorted(cand, ex).clamp(max=C - 1)
            coarse.append((cand.gather(-1, pos) == ex).float().mean().item())
            final.append((ex.unsqueeze(-1) == idx.long().unsqueeze(-2)).any(-1).float().mean().item())
        out.append({"variant": name, "C": int(C), "coarse_recall": round(float(np.mean(coarse)), 4),
                    "recall_at_k": round(float(np.mean(final)), 4)})
    return {
        "workload": (f"drift keys: {wc.batch} seqs x {wc.n_kv_heads} KV heads x {wc.q_per_kv} query heads, "
                     f"{wc.n}-key prefill + {drift_steps} drifted keys (n = {n}); {n_queries} query draws per "
                     f"head from the last step's key law; C_rho = 2C, k = {k}; exact top-k by float32 "
                     "inner products"),
        "note": "quality figures on synthetic keys (the paper's recall is on real model keys): parity unpinned",
        "variants": out,
    }


def beta_length_run(pk, torch, np, workloads, dev, lengths=(4096, 16384, 65536, 131072),
                    betas=(1 / 64, 1 / 32, 3 / 64, 1 / 16, 3 / 32, 1 / 8, 3 / 16, 1 / 4), k=100, n_queries=8,
                    target=0.9):
    """Candidate ratio needed at each KV length (Sec. "Top-beta selection"; the paper reads that
    with k fixed, short caches need a larger beta and long ones allow a smaller one): the keys
    of 2 sequences x 8 KV heads (the prefill law of the drift workload, no drift), prefixes of
    each length, `n_queries` draws per query head from the key law; recall@k of the published
    method against exact top-k, for each beta (C = max(ceil(beta n), k), C_rho = 2C)."""
    wc = workloads.CONFIGS["drift"]
    batch = 2
    signs = workloads.rotation_signs(wc.seed)
    nmax = max(lengths)
    K = np.stack([np.stack([workloads.head_keys(wc.seed, s, h, nmax) for h in range(wc.n_kv_heads)])
                  for s in range(batch)])
    Kfull = torch.from_numpy(K).to(dev)
    hq = wc.n_kv_heads * wc.q_per_kv
    Q = np.stack([np.stack([workloads.drift_query(wc.seed, s, h, 0, 1, n_queries * wc.q_per_kv)
                            .reshape(n_queries, wc.q_per_kv, wc.head_dim) for h in range(wc.n_kv_heads)], axis=1)
                  for s in range(batch)], axis=1)  # [n_queries][b][Hkv][G][D]
    Qd = torch.from_numpy(Q.reshape(n_queries, batch, hq, wc.head_dim)).to(dev)
    rows = []
    for n in lengths:
        Kd = Kfull[:, :, :n].contiguous()
        exact = []
        for i in range(n_queries):
            q = Qd[i].float().reshape(batch, wc.n_kv_heads, wc.q_per_kv, wc.head_dim)
            sc = torch.matmul(q, Kd.float().transpose(2, 3).contiguous())
            exact.append(torch.topk(sc, k, dim=-1).indices.reshape(batch, hq, k))
            del sc
        cfg = pk.Config(wc.n_kv_heads, wc.q_per_kv, n, signs)
        index = pk.Index.empty(cfg, batch, dev)
        pk.encode(cfg, index, Kd)
        rec = {}
        for beta in betas:
            C = min(max(-(-n * beta // 1), k), n)
            C = int(C)
            bud = pk.Budget(C, min(2 * C, n), k)
            ws = torch.empty(pk.retrieve_workspace_size(cfg, batch, n, bud), dtype=torch.uint8, device=dev)
            hits = []
            for i in range(n_queries):
                idx, _, _ = pk.retrieve(cfg, index, Qd[i], n, bud, workspace=ws)
                hits.append((exact[i].unsqueeze(-1) == idx.long().unsqueeze(-2)).any(-1).float().mean().item())
            rec[f"{beta:.4f}"] = {"C": C, "recall_at_k": round(float(np.mean(hits)), 4)}
        ok = [b for b in betas if rec[f"{b:.4f}"]["recall_at_k"] >= target]
        rows.append({"n": n, "recall_by_beta": rec,
                     f"smallest_beta_for_recall_{target}": round(min(ok), 4) if ok else None})
        del Kd, index
        torch.cuda.empty_cache()
    return {
        "workload": (f"{batch} seqs x {wc.n_kv_heads} KV heads x {wc.q_per_kv} query heads, prefill-law keys "
                     f"(prefixes of {nmax}), {n_queries} query draws per head from the key law; k = {k}, "
                     "C = max(ceil(beta n), k), C_rho = 2C; exact top-k by float32 inner products"),
        "note": "quality figures on synthetic keys (the paper's figure is on real model keys): parity unpinned",
        "lengths": rows,
    }


def offload_run(pk, torch, np, workloads, dev, steps, sink=128, local=512, m=256, group_fetch=False, share=0):
    """The offload setting at 1M tokens (Sec. "Buffer Update" with GPU->CPU offload; Sec.
    "On-Demand UVA Fetch"): Sink and Local + Update Buffer K/V in a GPU window ring, the
    Retrieval region's K/V in pinned host memory.  Each decode step writes the new token into
    the ring and runs pariskv_retrieve_tiered_attend (retrieved rows read over the host link);
    every m steps the rows leaving Local are encoded from the ring (pariskv_append_rows) and
    copied to host memory by pariskv_offload_rows on a second stream, which the step's
    retrieval waits for only before it starts."""
    wc = workloads.CONFIGS["host1m"]
    signs = workloads.rotation_signs(wc.seed)
    P = wc.n
    total = P + steps
    K, V = workloads.layer_kv(wc, n=total, threads=16)
    Q = np.stack([workloads.layer_queries(wc, K[:, :, :P], step=t, shared=share)[0] for t in range(steps)])
    Kh = torch.from_numpy(K).pin_memory()   # the offloaded cache (rows of Retrieval)
    Vh = torch.from_numpy(V).pin_memory()
    hq = wc.n_kv_heads * wc.q_per_kv
    wcap = sink + local + 2 * m
    # decode tokens' K/V staged on the GPU (the model would produce them step by step)
    Knew = torch.from_numpy(K[:, :, P:]).to(dev)
    Vnew = torch.from_numpy(V[:, :, P:]).to(dev)
    Kw = torch.zeros((wc.batch, wc.n_kv_heads, wcap, wc.head_dim), dtype=torch.float16, device=dev)
    Vw = torch.zeros_like(Kw)
    win0, n_idx = pk.window_regions(P, 0, sink, local, m)
    for r in list(range(win0.sink_len)) + list(range(win0.dense_begin, win0.dense_end)):
        slot = pk.window_slot(r, sink, wcap)
        Kw[:, :, slot] = torch.from_numpy(K[:, :, r]).to(dev)
        Vw[:, :, slot] = torch.from_numpy(V[:, :, r]).to(dev)
    cfg = pk.Config(wc.n_kv_heads, wc.q_per_kv, total, signs)
    index = pk.Index.empty(cfg, wc.batch, dev)
    Kd = torch.from_numpy(K[:, :, :P]).to(dev)   # prefill: encode the prompt's Retrieval region
    pk.append_rows(cfg, index, Kd, win0.retr_begin, n_idx, 0)
    torch.cuda.synchronize()
    del Kd
    torch.cuda.empty_cache()
    Qd = torch.from_numpy(Q).to(dev)
    budget = pk.Budget(wc.n_cand, wc.n_collide, wc.top_k, flags=pk.GROUP_FETCH if group_fetch else 0)
    scale = 1.0 / np.sqrt(wc.head_dim)
    ws = torch.empty(pk.retrieve_workspace_size(cfg, wc.batch, total, budget), dtype=torch.uint8, device=dev)
    out_idx = torch.empty((wc.batch, hq, wc.top_k), dtype=torch.int32, device=dev)
    out = torch.empty((wc.batch, hq, wc.head_dim), dtype=torch.float32, device=dev)
    main = torch.cuda.current_stream()
    side = torch.cuda.Stream()  # default priority
    starts = [torch.cuda.Event(enable_timing=True) for _ in range(steps)]
    ends = [torch.cuda.Event(enable_timing=True) for _ in range(steps)]
    copies = []
    upd = np.zeros(steps, bool)

    def ring_ranges(r0, cnt):
        """[(slot, row, count)] contiguous slot runs of Local/Buffer rows [r0, r0 + cnt)."""
        runs, r = [], r0
        while r < r0 + cnt:
            slot = pk.window_slot(r, sink, wcap)
            c = min(r0 + cnt - r, wcap - slot)
            runs.append((slot, r, c))
            r += c
        return runs

    pk.profile_reset()
    pk.profile_enable(True)
    torch.cuda.synchronize()
    for t in range(1, steps + 1):
        i = t - 1
        starts[i].record()
        slot = pk.window_slot(P + t - 1, sink, wcap)   # the new token enters the Update Buffer
        Kw[:, :, slot].copy_(Knew[:, :, t - 1])
        Vw[:, :, slot].copy_(Vnew[:, :, t - 1])
        win, n_retr = pk.window_regions(P, t, sink, local, m)
        if n_retr > n_idx:
            upd[i] = True
            r0, cnt = win.retr_begin + n_idx, n_retr - n_idx
            side.wait_stream(main)
            c0, c1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            with torch.cuda.stream(side):
                c0.record()
                for sl, row, c in ring_ranges(r0, cnt):
                    pk.offload_rows(Kw, Vw, sl, Kh, Vh, row, c)
                c1.record()
            copies.append((c0, c1, cnt))
            done = n_idx
            for sl, row, c in ring_ranges(r0, cnt):
                pk.append_rows(cfg, index, Kw, sl, c, done)
                done += c
            n_idx = n_retr
            main.wait_event(c1)   # the retrieval may now pick the evicted rows from host memory
        pk.retrieve_tiered_attend(cfg, index, Qd[i], n_idx, budget, Kw, Vw, Kh, Vh, win, scale,
                                  out_idx=out_idx, out=out, workspace=ws, kv_host_mapped=True)
        ends[i].record()
    torch.cuda.synchronize()
    pk.profile_enable(False)
    prof = pk.profile_read()
    us = np.array([starts[i].elapsed_time(ends[i]) * 1e3 for i in range(steps)])
    body, ub = us[8:], upd[8:]
    copy_bytes = [2 * wc.batch * wc.n_kv_heads * c * wc.head_dim * 2 for _, _, c in copies]
    copy_us = [a.elapsed_time(b) * 1e3 for a, b, _ in copies]
    fetch_bytes = wc.batch * hq * wc.top_k * 2 * wc.head_dim * 2
    ta = prof.get("topk_attend")
    ta_us = ta[1] * 1e3 / ta[0] if ta else None
    return {
        "workload": (f"host1m: {wc.batch} seq x {wc.n_kv_heads} KV heads x {wc.q_per_kv} query heads, "
                     f"{P}-token prompt + {steps} decode steps; Sink {sink} + Local {local} + Update Buffer "
                     f"in a GPU window ring of {wcap} rows, Retrieval K/V in pinned host memory; "
                     f"C = {wc.n_cand}, C_rho = {wc.n_collide}, k = {wc.top_k}; buffer update every {m} steps"),
        "us_per_step": round(float(body.mean()), 1),
        "us_per_update_step": round(float(body[ub].mean()), 1) if ub.any() else None,
        "us_per_other_step": round(float(body[~ub].mean()), 1),
        "updates": int(upd.sum()),
        "offload_d2h": {"bytes_per_update": int(copy_bytes[0]) if copy_bytes else 0,
                        "us_per_update": round(float(np.mean(copy_us)), 1) if copy_us else None,
                        "GBps": (round(float(np.sum(copy_bytes) / (np.sum(copy_us) * 1e-6) / 1e9), 2)
                                 if copy_us else None)},
        "fetch_h2d": {"bytes_per_step": int(fetch_bytes),
                      "topk_attend_us": round(ta_us, 1) if ta_us else None,
                      "GBps_of_topk_attend": round(fetch_bytes / (ta_us * 1e-6) / 1e9, 2) if ta_us else None},
        "kernels_avg_us": {k: round(v[1] * 1e3 / max(1, v[0]), 1) for k, v in prof.items()},
        "group_fetch": group_fetch,
        "query_heads_per_needle": max(share, 1),
        "timing": ("HIP events on the main stream around each step (steps 1-8 left out); the offload "
                   "copies timed on their own stream"),
    }


def group_run(pk, torch, np, workloads, dev, drift_steps, reps=8):
    """GQA-group de-duplication of the fetch over the host link: the drift workload's keys
    (K/V in pinned host memory), top-256 retrieved per query head, then attention per head
    (pariskv_sparse_attend) and per KV head over the union of its heads' lists
    (pariskv_group_attend), for planted-needle queries (a different needle per head) and for
    queries drawn from the key law (the heads of a group ask similar questions); and the
    whole retrieve + attend step with and without PARISKV_GROUP_FETCH."""
    wc = workloads.CONFIGS["drift"]
    signs = workloads.rotation_signs(wc.seed)
    n = wc.n + drift_steps
    K0, V0 = workloads.layer_kv(wc, threads=16)
    K = np.zeros((wc.batch, wc.n_kv_heads, n, wc.head_dim), np.float16)
    V = np.zeros_like(K)
    K[:, :, :wc.n], V[:, :, :wc.n] = K0, V0
    rng = np.random.default_rng(wc.seed)
    for s in range(wc.batch):
        for h in range(wc.n_kv_heads):
            K[s, h, wc.n:] = workloads.drift_keys(wc.seed, s, h, 0, drift_steps, drift_steps)
            V[s, h, wc.n:] = rng.standard_normal((drift_steps, wc.head_dim)).astype(np.float16)
    Kd = torch.from_numpy(K).to(dev)
    Kh, Vh = torch.from_numpy(K).pin_memory(), torch.from_numpy(V).pin_memory()
    hq = wc.n_kv_heads * wc.q_per_kv
    cfg = pk.Config(wc.n_kv_heads, wc.q_per_kv, n, signs)
    index = pk.Index.empty(cfg, wc.batch, dev)
    pk.encode(cfg, index, Kd)
    C = -(-n // 16)
    bud = pk.Budget(C, 2 * C, wc.top_k)
    scale = 1.0 / np.sqrt(wc.head_dim)
    queries = {
        "needle queries (one needle per head)": workloads.layer_queries(wc, K)[0],
        "queries from the key law": np.stack([np.stack([workloads.drift_queries(wc.seed, s, h, drift_steps,
                                                                                wc.q_per_kv)[-1]
                                                        for h in range(wc.n_kv_heads)])
                                              for s in range(wc.batch)]).reshape(wc.batch, hq, wc.head_dim),
    }
    out = torch.empty((wc.batch, hq, wc.head_dim), dtype=torch.float32, device=dev)
    un = torch.zeros((wc.batch, wc.n_kv_heads, 1), dtype=torch.int32, device=dev)
    res = {}
    for name, Q in queries.items():
        Qd = torch.from_numpy(Q).to(dev)
        idx, _, _ = pk.retrieve(cfg, index, Qd, n, bud)
        rows = int((idx >= 0).sum().item())
        times = {}
        for label, fn in (("per_head", lambda: pk.sparse_attend(cfg, Qd, Kh, Vh, idx, scale, out=out,
                                                               kv_host_mapped=True)),
                          ("group", lambda: pk.group_attend(cfg, Qd, Kh, Vh, idx, scale, out=out, union_rows=un,
                                                            kv_host_mapped=True))):
            fn()
            torch.cuda.synchronize()
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record()
            for _ in range(reps):
                fn()
            e1.record()
            torch.cuda.synchronize()
            times[label] = e0.elapsed_time(e1) * 1e3 / reps
        urows = int(un.sum().item())
        row_b = 2 * wc.head_dim * 2
        # The whole step (pariskv_retrieve_attend) with the attention fused into the
        # top-k, and with PARISKV_GROUP_FETCH (top-k, then the split group attention).
        gbud = pk.Budget(C, 2 * C, wc.top_k, flags=pk.GROUP_FETCH)
        for label, b_ in (("step_per_head", bud), ("step_group_fetch", gbud)):
            ws = torch.empty(pk.retrieve_workspace_size(cfg, wc.batch, n, b_), dtype=torch.uint8, device=dev)
            oi = torch.empty((wc.batch, hq, wc.top_k), dtype=torch.int32, device=dev)

            def call():
                pk.retrieve_attend(cfg, index, Qd, n, b_, Kh, Vh, scale, out_idx=oi, out=out, workspace=ws,
                                   kv_host_mapped=True)
            call()
            torch.cuda.synchronize()
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record()
            for _ in range(reps):
                call()
            e1.record()
            torch.cuda.synchronize()
            times[label] = e0.elapsed_time(e1) * 1e3 / reps
        res[name] = {"rows_per_head_lists": rows, "rows_fetched_by_group": urows,
                     "fetch_ratio": round(urows / rows, 4),
                     "us_per_head_attend": round(times["per_head"], 1),
                     "us_group_attend": round(times["group"], 1),
                     "host_link_GBps_per_head": round(rows * row_b / (times["per_head"] * 1e-6) / 1e9, 2),
                     "host_link_GBps_group": round(urows * row_b / (times["group"] * 1e-6) / 1e9, 2),
                     "us_step_retrieve_attend": round(times["step_per_head"], 1),
                     "us_step_retrieve_attend_group_fetch": round(times["step_group_fetch"], 1),
                     "us_saved_per_step": round(times["step_per_head"] - times["step_group_fetch"], 1)}
    return {"workload": (f"drift keys ({wc.batch} seqs x {wc.n_kv_heads} KV heads x {wc.q_per_kv} query heads, "
                         f"n = {n}), K/V in pinned host memory, top-{wc.top_k} per head from C = {C}"),
            **res}


def host_link_run(pk, torch, np, cfg, K, V, Qd, idx_list, scale, dev, reps=8):
    """Sparse attention with K/V in pinned host memory, read through host-mapped pointers."""
    Kh = torch.from_numpy(K).pin_memory()
    Vh = torch.from_numpy(V).pin_memory()
    out = torch.empty((Qd.shape[1], cfg.n_q_heads, 128), dtype=torch.float32, device=dev)
    pk.sparse_attend(cfg, Qd[0], Kh, Vh, idx_list[0], scale, out=out, kv_host_mapped=True)
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for r in range(reps):
        i = r % len(idx_list)
        pk.sparse_attend(cfg, Qd[i], Kh, Vh, idx_list[i], scale, out=out, kv_host_mapped=True)
    e1.record()
    torch.cuda.synchronize()
    us = e0.elapsed_time(e1) * 1e3 / reps
    k = idx_list[0].shape[-1]
    rows = idx_list[0].numel()
    row_bytes = rows * 2 * 128 * 2
    return {"us_per_attend": round(us, 1), "kv_bytes": row_bytes,
            "host_link_GBps": round(row_bytes / (us * 1e-6) / 1e9, 2),
            "note": f"{rows} K and V rows of 256 B ({k} per query head) gathered over the host link per call"}


def main():
    args = parse()
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print(f"bench.py measures one GPU only (asked for --gpus {args.gpus}, WORLD_SIZE {world}): "
              f"the retrieval path shards by (sequence, KV head) with no exchange, so each GPU "
              f"of a larger run would repeat the one-GPU figure.", file=sys.stderr)
        sys.exit(2)

    # The oracle baselines run first, in spawned child processes, before this process
    # touches the GPU.
    cpu = cpu32 = None
    if not args.no_cpu_baseline:
        cpu = cpu_baseline(args.workload, args.cpu_groups, args.cpu_steps)
        if args.workload == "batch8_128k":
            cpu32 = cpu_baseline("layer32k", 8, args.cpu_steps)
        print(f"[bench] oracle baselines done", file=sys.stderr, flush=True)

    import numpy as np
    import torch

    import paper_2602_07721_amd as pk
    import workloads

    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(1)
    pk.lib()
    wc = workloads.CONFIGS[args.workload]
    signs = workloads.rotation_signs(wc.seed)
    budget = pk.Budget(wc.n_cand, wc.n_collide, wc.top_k, flags=pk.GROUP_FETCH if args.group_fetch else 0)
    scale = 1.0 / np.sqrt(wc.head_dim)
    total_steps = args.warmup + args.steps

    t_gen = time.perf_counter()
    K, V = workloads.layer_kv(wc, threads=16)
    Qs = [workloads.layer_queries(wc, K, step=s, shared=args.group_share)[0] for s in range(total_steps)]
    print(f"[bench] generated {wc.name} inputs in {time.perf_counter() - t_gen:.1f} s", file=sys.stderr,
          flush=True)

    dev = torch.device("cuda:0")
    if args.kv_host:
        Kd = torch.from_numpy(K).pin_memory()
        Vd = torch.from_numpy(V).pin_memory()
    else:
        Kd = torch.from_numpy(K).to(dev)
        Vd = torch.from_numpy(V).to(dev)
    Qd = torch.from_numpy(np.stack(Qs)).to(dev)
    cfg = pk.Config(wc.n_kv_heads, wc.q_per_kv, wc.n, signs)
    index = pk.Index.empty(cfg, wc.batch, dev)
    hq = cfg.n_q_heads
    out_idx = torch.empty((wc.batch, hq, wc.top_k), dtype=torch.int32, device=dev)
    out_score = torch.empty((wc.batch, hq, wc.top_k), dtype=torch.float32, device=dev)
    out = torch.empty((wc.batch, hq, wc.head_dim), dtype=torch.float32, device=dev)
    lay = pk.workspace_layout(cfg, wc.batch, wc.n, budget)
    ws = torch.empty(lay["total"], dtype=torch.uint8, device=dev)
    flush = torch.zeros((1 << 30) // 4, dtype=torch.int32, device=dev)
    flush_sink = torch.zeros((), dtype=torch.int32, device=dev)

    # Prefill encode, timed on its own.  The first call also loads the code objects,
    # so the timed call is the second (encode rewrites the index and its counts).
    Kenc = Kd.to(dev) if args.kv_host else Kd  # encode reads keys from device memory
    pk.encode(cfg, index, Kenc)
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    pk.encode(cfg, index, Kenc)
    e1.record()
    torch.cuda.synchronize()
    enc_ms = e0.elapsed_time(e1)
    n_keys = wc.batch * wc.n_kv_heads * wc.n

    def step(s):
        if args.separate:
            pk.retrieve(cfg, index, Qd[s], wc.n, budget, out_idx=out_idx, out_score=out_score, workspace=ws)
            pk.sparse_attend(cfg, Qd[s], Kd, Vd, out_idx, scale, out=out, kv_host_mapped=args.kv_host)
        else:
            pk.retrieve_attend(cfg, index, Qd[s], wc.n, budget, Kd, Vd, scale, out_idx=out_idx,
                               out_score=out_score, out=out, workspace=ws, kv_host_mapped=args.kv_host)

    for s in range(args.warmup):
        if not args.no_flush:
            flush_sink.copy_(flush.amax())
        step(s)
    torch.cuda.synchronize()

    def timed_loop(profile):
        starts = [torch.cuda.Event(enable_timing=True) for _ in range(args.steps)]
        ends = [torch.cuda.Event(enable_timing=True) for _ in range(args.steps)]
        pk.profile_reset()
        pk.profile_enable(profile)
        torch.cuda.synchronize()
        w0 = time.perf_counter()
        for i in range(args.steps):
            if not args.no_flush:
                flush_sink.copy_(flush.amax())
            starts[i].record()
            step(args.warmup + i)
            ends[i].record()
        torch.cuda.synchronize()
        wall = time.perf_counter() - w0
        pk.profile_enable(False)
        prof = pk.profile_read() if profile else {}
        return np.array([starts[i].elapsed_time(ends[i]) for i in range(args.steps)]), wall, prof

    # The step time comes from a clean loop; per-kernel durations from a second,
    # identical loop with an event pair around every kernel launch (the events
    # themselves lengthen that loop's steps, so it does not set the value).
    step_ms, wall, _ = timed_loop(False)
    prof_step_ms, _, prof = timed_loop(not args.no_profile) if not args.no_profile else (None, None, {})
    warm_ms = None
    if not args.no_warm and not args.no_flush:
        # The same steps back to back without the flush: the index and K/V rows that the
        # previous step touched may still sit in the 256 MB Infinity Cache and the L2s.
        flag = args.no_flush
        args.no_flush = True
        warm_ms, _, _ = timed_loop(False)
        args.no_flush = flag

    # Needle hit rate on the last step (a sanity figure, not a parity check).
    _, needles = workloads.layer_queries(wc, K, step=total_steps - 1)
    idx_h = out_idx.cpu().numpy()
    hits = float(np.mean([needles[s, h] in set(idx_h[s, h].tolist())
                          for s in range(wc.batch) for h in range(hq)]))

    # Achievable ceilings on this GPU: the library's reference streaming copy of 1 GiB
    # (read + write) and streaming read of 1 GiB, best of 5 each.
    def best_of(fn, reps=5):
        best = None
        for _ in range(reps):
            c0, c1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            c0.record()
            fn()
            c1.record()
            torch.cuda.synchronize()
            t = c0.elapsed_time(c1) * 1e-3
            best = t if best is None else min(best, t)
        return best

    src = torch.empty(1 << 30, dtype=torch.uint8, device=dev)
    dst = torch.empty_like(src)
    src.fill_(1)
    torch.cuda.synchronize()
    copy_gbs = 2 * src.numel() / best_of(lambda: pk.stream_copy(dst, src)) / 1e9
    del src, dst
    read_gbs = flush.numel() * 4 / best_of(lambda: pk.stream_read(flush, flush_sink)) / 1e9

    c_eff = min(wc.n_cand, wc.n)
    algo = algorithmic_bytes(wc, c_eff, lay["topk_parts"])
    fetch = None
    if args.group_fetch:
        # rows the last step's attention fetched, against the heads' own lists
        quads = (wc.q_per_kv + 3) // 4
        grows = int(ws[lay["group_rows"]:lay["group_rows"] + wc.batch * wc.n_kv_heads * quads * 4]
                    .view(torch.int32).sum().item())
        lists = int((out_idx >= 0).sum().item())
        algo["group_attend"] = grows * 512 + wc.batch * hq * wc.top_k * 4
        fetch = {"rows_fetched": grows, "rows_in_head_lists": lists, "fetch_ratio": round(grows / max(lists, 1), 4)}
    kernels = {}
    for name, (launches, ms) in prof.items():
        avg_ms = ms / max(1, launches)
        row = {"launches": int(launches), "avg_us": avg_ms * 1e3}
        if name in algo:
            row["bytes_per_launch"] = algo[name]
            row["GBps"] = algo[name] / (avg_ms * 1e-3) / 1e9
            row["frac_hbm_peak"] = row["GBps"] / HBM_PEAK_GBS
        kernels[name] = row
    # The dominant kernel: the longest one among those with an algorithmic byte count.
    dominant = max((k for k in kernels if k in algo), key=lambda k: kernels[k]["avg_us"], default=None)
    traffic = measured_traffic(wc.name)
    roofline = None
    if dominant:
        kr = kernels[dominant]
        tr = traffic.get(dominant)
        roofline = {"bound": "hbm", "kernel": dominant, "achieved": round(kr["GBps"], 1),
                    "peak": HBM_PEAK_GBS, "unit": "GB/s", "frac": round(kr["frac_hbm_peak"], 4),
                    "traffic": tr,
                    "algorithmic_bytes": algo[dominant],
                    # the same kernel against the copy ceiling measured in this run, and its
                    # measured HBM bytes (counters) per launch over the same duration
                    "frac_copy_ceiling": round(kr["GBps"] / copy_gbs, 4),
                    "traffic_frac_hbm_peak": (round(tr / (kr["avg_us"] * 1e-6) / 1e9 / HBM_PEAK_GBS, 4)
                                              if tr else None)}
    for name, row in kernels.items():
        if "GBps" in row:
            row["frac_copy_ceiling"] = row["GBps"] / copy_gbs
        if name in traffic:
            row["hbm_traffic_bytes"] = traffic[name]
            row["traffic_frac_hbm_peak"] = traffic[name] / (row["avg_us"] * 1e-6) / 1e9 / HBM_PEAK_GBS
    collide_gbs = kernels.get("collide", {}).get("GBps")


    extras = {}
    if args.extras:
        if not args.kv_host:
            # index sets of the last few timed steps, for host-mapped attention
            idx_list = []
            for i in range(4):
                st = args.warmup + args.steps - 1 - i
                oi = torch.empty_like(out_idx)
                pk.retrieve(cfg, index, Qd[st], wc.n, budget, out_idx=oi, workspace=ws)
                idx_list.append(oi)
            torch.cuda.synchronize()
            extras["host_link"] = host_link_run(pk, torch, np, cfg, K, V, Qd[-4:].flip(0), idx_list, scale, dev)
            extras["host_link"]["workload"] = f"{wc.name}, K/V in pinned host memory"
        del Kd, Vd
        torch.cuda.empty_cache()
        extras["drift"] = drift_run(pk, torch, np, workloads, dev, args.drift_steps)
        torch.cuda.empty_cache()
        extras["window"] = window_run(pk, torch, np, workloads, dev, args.drift_steps)
        torch.cuda.empty_cache()
        extras["ablation"] = ablation_run(pk, torch, np, workloads, dev, args.drift_steps)
        torch.cuda.empty_cache()
        extras["beta_vs_length"] = beta_length_run(pk, torch, np, workloads, dev)
        torch.cuda.empty_cache()
        extras["group_dedup"] = group_run(pk, torch, np, workloads, dev, args.drift_steps)
    if args.offload_steps > 0:
        torch.cuda.empty_cache()
        extras["offload"] = offload_run(pk, torch, np, workloads, dev, args.offload_steps,
                                        group_fetch=args.group_fetch, share=args.group_share)


    mean_us = float(step_ms.mean() * 1e3)
    result = {
        "metric": "retrieve+attend us/step/layer at 128K ctx; code-scan HBM GB/s vs peak",
        "path": "pariskv_retrieve + pariskv_sparse_attend" if args.separate else "pariskv_retrieve_attend",
        "value": round(mean_us, 2),
        "unit": "us/step/layer",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(float(step_ms.mean()), 5),
        "higher_is_better": False,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic",
        "config": {
            "workload": (f"{wc.name}: {wc.batch} seqs x {wc.n_kv_heads} KV heads x {wc.q_per_kv} query "
                         f"heads, N={wc.n}, D={wc.head_dim}, B=16, C={wc.n_cand}, C_rho={wc.n_collide}, "
                         f"k={wc.top_k}, float16 K/V/Q, "
                         + ("K/V in pinned host memory read through host-mapped pointers, Q and index "
                            "in HBM" if args.kv_host else "all in HBM")),
            "caches": "flushed between steps" if not args.no_flush else "warm",
            **({"group_share": args.group_share} if args.group_share > 1 else {}),
            **({"group_fetch": True} if args.group_fetch else {}),
        },
        "p10_us": round(float(np.percentile(step_ms, 10) * 1e3), 2),
        "p50_us": round(float(np.percentile(step_ms, 50) * 1e3), 2),
        "p90_us": round(float(np.percentile(step_ms, 90) * 1e3), 2),
        "wall_ms_per_step_incl_flush": round(wall / args.steps * 1e3, 4),
        "profiled_loop_us_per_step": (round(float(prof_step_ms.mean() * 1e3), 2)
                                      if prof_step_ms is not None else None),
        "warm_us": round(float(warm_ms.mean() * 1e3), 2) if warm_ms is not None else None,
        "warm_p10_us": round(float(np.percentile(warm_ms, 10) * 1e3), 2) if warm_ms is not None else None,
        "warm_p90_us": round(float(np.percentile(warm_ms, 90) * 1e3), 2) if warm_ms is not None else None,
        "code_scan_GBps": round(collide_gbs, 1) if collide_gbs else None,
        "code_scan_frac_hbm_peak": round(collide_gbs / HBM_PEAK_GBS, 4) if collide_gbs else None,
        "code_scan_frac_copy_ceiling": round(collide_gbs / copy_gbs, 4) if collide_gbs else None,
        "roofline": roofline,
        "kernels": {k: {kk: (round(vv, 3) if isinstance(vv, float) else vv) for kk, vv in v.items()}
                    for k, v in sorted(kernels.items())},
        "encode": {"ms": round(enc_ms, 3), "keys_per_s": round(n_keys / (enc_ms * 1e-3), 1),
                   "GBps": round(n_keys * (256 + 144) / (enc_ms * 1e-3) / 1e9, 1)},
        "needle_hit_rate": round(hits, 4),
        "copy_GBps": round(copy_gbs, 1),
        "read_GBps": round(read_gbs, 1),
        "group_fetch": fetch,
        "cpu_baseline": cpu,
        "cpu_baseline_layer32k": cpu32,
    }
    result.update(extras)
    print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()
