"""Seeded synthetic inputs shaped like LLM decode-time K/V/Q.

This module only draws random numbers; it holds none of the retrieval
method's arithmetic.  Both the HIP library's tests and the CPU oracle take
their inputs from here, so the two sides see the same arrays.

Recipe (per sequence and KV head), standing in for the real Llama-3-8B /
Qwen3-8B keys the paper measures on (LongBench-v2 prompts truncated to 128K;
the prompts, model weights and baselines are not available here):
  * a mean offset mu ~ N(0, 0.5^2) per channel;
  * per-channel scale 1, except 4 seeded "outlier" channels with scale 8;
  * keys k = mu + scale (.) eps, eps ~ N(0, I); values v ~ N(0, I);
  * a needle query for query head h is q = k_needle + 0.1 N(0, I) with the
    needle index drawn uniformly from [0, n);
  * everything is rounded to float16 (the model's storage type).
The SRHT sign vector s in {+1,-1}^D is also drawn here (Rademacher), because
random numbers the method draws are an input to it.

Seeds: numpy.random.SeedSequence([tag, config seed, sequence, kv head, ...])
feeding PCG64, so every (sequence, head) slice can be regenerated alone.
"""

from dataclasses import dataclass, field

import numpy as np

D_DEFAULT = 128
N_OUTLIERS = 4
OUTLIER_SCALE = 8.0
MEAN_STD = 0.5
NEEDLE_NOISE = 0.1

_TAG_SIGNS = 11
_TAG_KEYS = 23
_TAG_VALUES = 37
_TAG_QUERY = 41
_TAG_DRIFT = 53


def _rng(*words):
    return np.random.Generator(np.random.PCG64(np.random.SeedSequence(list(words))))


def rotation_signs(seed, D=D_DEFAULT):
    """Rademacher signs s_j in {+1, -1} (int8) for the SRHT diagonal."""
    bits = _rng(_TAG_SIGNS, seed).integers(0, 2, size=D)
    return np.where(bits == 1, -1, 1).astype(np.int8)


@dataclass
class HeadLaw:
    """Distribution of the keys of one (sequence, KV head)."""
    mu: np.ndarray          # [D] float64 mean offset
    scale: np.ndarray       # [D] float64 per-channel std
    outliers: np.ndarray    # [N_OUTLIERS] channel indices


def head_law(seed, seq, kvh, D=D_DEFAULT):
    r = _rng(_TAG_KEYS, seed, seq, kvh, 0)
    mu = r.normal(0.0, MEAN_STD, size=D)
    outliers = r.choice(D, size=N_OUTLIERS, replace=False)
    scale = np.ones(D)
    scale[outliers] = OUTLIER_SCALE
    return HeadLaw(mu=mu, scale=scale, outliers=np.sort(outliers))


def head_keys(seed, seq, kvh, n, D=D_DEFAULT):
    """Keys [n, D] float16 of one (sequence, KV head)."""
    law = head_law(seed, seq, kvh, D)
    r = _rng(_TAG_KEYS, seed, seq, kvh, 1)
    eps = r.standard_normal(size=(n, D), dtype=np.float32)
    eps *= law.scale.astype(np.float32)[None, :]
    eps += law.mu.astype(np.float32)[None, :]
    return eps.astype(np.float16)


def head_values(seed, seq, kvh, n, D=D_DEFAULT):
    """Values [n, D] float16 of one (sequence, KV head)."""
    r = _rng(_TAG_VALUES, seed, seq, kvh)
    return r.standard_normal(size=(n, D), dtype=np.float32).astype(np.float16)


def needle_queries(keys, seed, seq, kvh, n_queries, step=0, shared=0):
    """(q [n_queries, D] float16, needle index [n_queries]) planted on the given keys.
    shared > 1: the first `shared` queries share the first query's needle (each with its
    own noise), as query heads of one KV group that attend to the same key."""
    keys = np.asarray(keys)
    n, D = keys.shape
    r = _rng(_TAG_QUERY, seed, seq, kvh, step)
    needles = r.integers(0, n, size=n_queries)
    if shared > 1:
        needles[:shared] = needles[0]
    noise = r.standard_normal(size=(n_queries, D))
    q = keys[needles].astype(np.float64) + NEEDLE_NOISE * noise
    return q.astype(np.float16), needles


def drift_keys(seed, seq, kvh, t0, t, total_steps, D=D_DEFAULT):
    """Decode keys for steps [t0, t0+t) whose mean moves linearly away from the prefill mean.

    Reading of "the mean offset rotates linearly away (total shift 2 sigma)":
    mu_t = mu_0 + (t / total_steps) * 2 * scale (.) delta with delta a fixed
    Rademacher direction per (sequence, head).
    """
    law = head_law(seed, seq, kvh, D)
    delta = np.where(_rng(_TAG_DRIFT, seed, seq, kvh).integers(0, 2, size=D) == 1, -1.0, 1.0)
    steps = np.arange(t0, t0 + t, dtype=np.float64)
    mu = law.mu[None, :] + (steps / total_steps)[:, None] * 2.0 * (law.scale * delta)[None, :]
    r = _rng(_TAG_KEYS, seed, seq, kvh, 2, t0)
    eps = r.standard_normal(size=(t, D))
    return (mu + law.scale[None, :] * eps).astype(np.float16)


def drift_query(seed, seq, kvh, step, total_steps, n_queries, D=D_DEFAULT):
    """Fresh queries drawn from the current (drifted) key distribution."""
    law = head_law(seed, seq, kvh, D)
    delta = np.where(_rng(_TAG_DRIFT, seed, seq, kvh).integers(0, 2, size=D) == 1, -1.0, 1.0)
    mu = law.mu + (step / total_steps) * 2.0 * law.scale * delta
    r = _rng(_TAG_QUERY, seed, seq, kvh, 1_000_000 + step)
    eps = r.standard_normal(size=(n_queries, D))
    return (mu[None, :] + law.scale[None, :] * eps).astype(np.float16)


def drift_queries(seed, seq, kvh, total_steps, n_queries, D=D_DEFAULT):
    """Queries of every step t in [0, total_steps) at once, [t][n_queries][D]: draws
    from the key law of step t (as drift_query), one random stream per head."""
    law = head_law(seed, seq, kvh, D)
    delta = np.where(_rng(_TAG_DRIFT, seed, seq, kvh).integers(0, 2, size=D) == 1, -1.0, 1.0)
    steps = np.arange(total_steps, dtype=np.float64)
    mu = law.mu[None, :] + (steps / total_steps)[:, None] * 2.0 * (law.scale * delta)[None, :]
    r = _rng(_TAG_QUERY, seed, seq, kvh, 2_000_000)
    eps = r.standard_normal(size=(total_steps, n_queries, D))
    return (mu[:, None, :] + law.scale[None, None, :] * eps).astype(np.float16)


@dataclass
class Config:
    """Shapes and budgets of one workload."""
    name: str
    batch: int
    n_kv_heads: int
    q_per_kv: int
    n: int
    n_cand: int
    n_collide: int
    top_k: int
    head_dim: int = D_DEFAULT
    n_subspaces: int = 16
    seed: int = 0
    note: str = ""
    extra: dict = field(default_factory=dict)

    @property
    def n_q_heads(self):
        return self.n_kv_heads * self.q_per_kv


CONFIGS = {
    # One KV head, 8 planted-needle queries (as 8 query heads) over 4096 keys.
    "tiny": Config("tiny", batch=1, n_kv_heads=1, q_per_kv=8, n=4096,
                   n_cand=512, n_collide=1024, top_k=64, seed=1),
    # One Llama-3-8B-shaped layer (8 KV heads x 4 query heads), 32K keys.
    "layer32k": Config("layer32k", batch=1, n_kv_heads=8, q_per_kv=4, n=32768,
                       n_cand=2048, n_collide=4096, top_k=256, seed=2),
    # Throughput regime: 8 sequences x 8 KV heads x 4 query heads, 128K keys.
    "batch8_128k": Config("batch8_128k", batch=8, n_kv_heads=8, q_per_kv=4, n=131072,
                          n_cand=8192, n_collide=16384, top_k=512, seed=3),
    # Long-generation drift: 4 sequences, 32K prefill then per-step appends.
    "drift": Config("drift", batch=4, n_kv_heads=8, q_per_kv=4, n=32768,
                    n_cand=2048, n_collide=4096, top_k=256, seed=4,
                    extra=dict(decode_steps=32768)),
    # Million-token context with K/V in pinned host memory.
    "host1m": Config("host1m", batch=1, n_kv_heads=8, q_per_kv=4, n=1 << 20,
                     n_cand=32768, n_collide=65536, top_k=1024, seed=5),
}


def layer_kv(cfg, seqs=None, heads=None, n=None, values=True, threads=8):
    """K, V float16 arrays [len(seqs)][len(heads)][n][D] for a config (V None if not values)."""
    from concurrent.futures import ThreadPoolExecutor

    seqs = list(range(cfg.batch) if seqs is None else seqs)
    heads = list(range(cfg.n_kv_heads) if heads is None else heads)
    n = cfg.n if n is None else n
    D = cfg.head_dim
    K = np.empty((len(seqs), len(heads), n, D), dtype=np.float16)
    V = np.empty((len(seqs), len(heads), n, D), dtype=np.float16) if values else None

    def fill(job):
        i, j = job
        K[i, j] = head_keys(cfg.seed, seqs[i], heads[j], n, D)
        if values:
            V[i, j] = head_values(cfg.seed, seqs[i], heads[j], n, D)

    jobs = [(i, j) for i in range(len(seqs)) for j in range(len(heads))]
    with ThreadPoolExecutor(max(1, threads)) as ex:
        list(ex.map(fill, jobs))
    return K, V


def layer_queries(cfg, K, step=0, shared=0):
    """Needle queries Q [b][Hq][D] float16 and needle indices [b][Hq] for keys K [b][Hkv][n][D]
    (shared: query heads per KV group sharing one needle, see needle_queries)."""
    b, hkv, n, D = K.shape
    Q = np.empty((b, hkv * cfg.q_per_kv, D), dtype=np.float16)
    needles = np.empty((b, hkv * cfg.q_per_kv), dtype=np.int64)
    for s in range(b):
        for h in range(hkv):
            q, nd = needle_queries(K[s, h], cfg.seed, s, h, cfg.q_per_kv, step, shared)
            Q[s, h * cfg.q_per_kv:(h + 1) * cfg.q_per_kv] = q
            needles[s, h * cfg.q_per_kv:(h + 1) * cfg.q_per_kv] = nd
    return Q, needles
