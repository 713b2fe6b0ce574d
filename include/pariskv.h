/*
 * pariskv.h -- C ABI of the ParisKV decode-step retrieval library for AMD
 * Instinct MI355X (gfx950).
 *
 * Method: ParisKV, "Fast and Drift-Robust KV-Cache Retrieval for Long-Context
 * LLMs" (arXiv 2602.07721).  The library implements, per decode step and per
 * query head, the path of Alg. 1: key summarisation (encode / append), the
 * query transform, tier-weighted collision scores (Eq. collision_score),
 * top-beta candidate selection, RSQ-IP reranking (Eq. rsqip_raw_weighted),
 * the final top-k, and attention restricted to the selected keys
 * (Eqs. approx_weight, approx_output).
 *
 * General rules for every entry point
 *   - Device pointers are caller-owned memory on the current HIP device
 *     (for example torch tensors).  The library allocates no device memory
 *     (its one device array is the static scratch of
 *     pariskv_retrieve_attend_noalloc, part of its code object), keeps no
 *     per-index state, and never synchronises a stream: every call
 *     validates its arguments on the host, enqueues kernels on `stream`
 *     (a hipStream_t; NULL = the default stream) and returns.
 *   - Validation happens before any launch.  On error nothing is enqueued
 *     and a negative PARISKV_ERR_* code is returned; pariskv_last_error()
 *     gives a thread-local message.  No C++ exception crosses the ABI.
 *   - Calls on one stream are ordered.  Calls on different streams that touch
 *     the same index or workspace must be ordered by the caller.
 *   - Inputs must be finite float16 values; codes computed from non-finite
 *     keys are unspecified (no fault).
 *
 * Shapes used below: D = head_dim = 128, B = n_subspaces = 16, m = D/B = 8
 * (2^m = 256 centroids per subspace), Hkv KV heads, G query heads per KV
 * head, Hq = Hkv * G; query head h reads KV head h / G.
 */
#ifndef PARISKV_H
#define PARISKV_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* ---------------------------------------------------------------- codes */
#define PARISKV_OK 0
#define PARISKV_ERR_INVALID (-1)     /* bad shape, budget, pointer or alignment  */
#define PARISKV_ERR_CAPACITY (-2)    /* keys would not fit in the index arrays  */
#define PARISKV_ERR_WORKSPACE (-3)   /* workspace missing or too small           */
#define PARISKV_ERR_HIP (-4)         /* a HIP runtime call or launch failed      */
#define PARISKV_ERR_UNSUPPORTED (-5) /* valid but outside what the library serves */

#define PARISKV_HEAD_DIM 128
#define PARISKV_SUBSPACES 16
#define PARISKV_SUBDIM 8
#define PARISKV_CENTROIDS 256
#define PARISKV_REC_BYTES 128
#define PARISKV_MAX_SCORE 96        /* 6 * B: largest collision score        */
#define PARISKV_MAX_CAND 65536      /* largest candidate budget C served     */
#define PARISKV_MAX_TOPK 2048       /* largest final k served                */

/* ---------------------------------------------------------------- types */

/* Ablation variants of the index (Sec. "Ablation Studies"), for
 * pariskv_config.flags; 0 = the method as published.  An index must be
 * queried with the flags it was encoded with.
 *   PARISKV_NO_ROTATION          R = I: keys and queries are split into
 *                                subspaces as they are (ids = sign patterns
 *                                of the raw subspaces, W_b = w_b, and the
 *                                query transform is z = D q)
 *   PARISKV_NO_ALPHA_CORRECTION  w_b = ||k|| r_b without the division by
 *                                alpha_b of Eq. scaling_factor (stored
 *                                W_b = sqrt(S_b), IEEE square root) */
#define PARISKV_NO_ROTATION 1u
#define PARISKV_NO_ALPHA_CORRECTION 2u

/* Shape of one layer's KV cache and the shared rotation.
 *   rot_signs: HOST pointer to D int8 values, each +1 or -1: the diagonal s
 *   of the rotation R = H_D diag(s) / sqrt(D) (Sec. "Preprocessing" step (1),
 *   "implemented by SRHT"; H_D is the Sylvester Walsh-Hadamard matrix).  The
 *   library copies the signs at every call; the caller keeps ownership. */
typedef struct pariskv_config {
    int32_t head_dim;        /* D; must be 128                                  */
    int32_t n_subspaces;     /* B; must be 16 (m = 8)                           */
    int32_t n_kv_heads;      /* Hkv >= 1                                        */
    int32_t q_per_kv;        /* G, 1..16                                        */
    int64_t capacity;        /* key slots per (sequence, KV head), 1..2^31-1    */
    const int8_t* rot_signs; /* host, [D], each +1 or -1                        */
    uint32_t flags;          /* PARISKV_NO_ROTATION | PARISKV_NO_ALPHA_CORRECTION, or 0 */
} pariskv_config;

/* Per-key metadata kept on the GPU (Sec. "Low-Bit Rerank Metadata": centroid
 * ids, 4-bit codes and weights w).  All three arrays are device memory owned
 * by the caller, 16-byte aligned (128-byte alignment of rec is recommended).
 *
 *   ids    uint8 [batch][Hkv][capacity][B]: the centroid id c of subspace b
 *          (Eq. dir_assign), stored relabelled as slot(c).  Bit j of c is set
 *          when coordinate j of the rotated subspace is negative (a zero
 *          coordinate counts as positive).  slot keeps bits 5..7 and XORs
 *          bits 0..4 with M(c >> 5), M linear with M(1) = 0x07, M(2) = 0x19,
 *          M(4) = 0x0E:
 *            slot(c) = c ^ (c & 32 ? 0x07 : 0) ^ (c & 64 ? 0x19 : 0)
 *                        ^ (c & 128 ? 0x0E : 0).
 *          slot is its own inverse.  Ids within Hamming distance 3 get
 *          different slot(c) mod 32, which spreads the popular clusters
 *          around a dominant sign pattern over distinct LDS banks in the
 *          collision scan.
 *   rec    [batch][Hkv][capacity][128] bytes, the rerank record of one key,
 *          eight 16-byte chunks; chunk c = 0..7 holds subspaces 2c and 2c+1:
 *            bytes 16c+0..3   uint32 code word of subspace 2c
 *            bytes 16c+4..7   uint32 code word of subspace 2c+1
 *            bytes 16c+8..11  float  W_{2c}
 *            bytes 16c+12..15 float  W_{2c+1}
 *          A code word holds the 4-bit code of coordinate j in bits 4j..4j+3:
 *          (sign << 3) | t with sign = 1 for negative and t the 3-bit magnitude
 *          bin of Eq. rsqip_sign_mag_code.  W_b = sqrt(D) * w_b with w_b the
 *          weight of Eq. scaling_factor.
 *   counts uint32 [batch][Hkv][B][256]: number of indexed keys in each
 *          centroid cluster (needed for "top clusters covering ratio rho"). */
typedef struct pariskv_index {
    uint8_t* ids;
    uint8_t* rec;
    uint32_t* counts;
} pariskv_index;

/* Binary (0/1) collisions for pariskv_budget.flags (the coarse score the
 * tiers replace, App. "Coarse Candidate Generation"): every admitted cluster
 * scores 1 instead of its tier weight, so S_i is in [0, B]. */
#define PARISKV_BINARY_COLLISIONS 1
/* Diagnostic for pariskv_budget.flags: the collision scan histograms no score,
 * so every selection threshold comes from the exact recount over the stored
 * scores (see pariskv_ws_layout.thresh).  Same outputs, slower; it exercises
 * the recount that otherwise runs only when the histogram floor is too high. */
#define PARISKV_EXACT_RECOUNT 2
/* For pariskv.budget.flags with pariskv_retrieve_attend (and its _noalloc form),
 * pariskv_retrieve_window_attend and pariskv_retrieve_tiered_attend: GQA-group
 * de-duplication of the fetch.  The attention of each quad of query heads
 * sharing a KV head reads every distinct K/V row of their winner lists once
 * (pariskv_group_attend), and the window's dense rows (Sink, Local / Update
 * Buffer), which every head attends, once per quad, instead of once per head
 * inside each head's top-k; worth it when the rows cross the host link
 * (kv_host_mapped = 1) and the heads' lists overlap.  out then equals per-head
 * attention up to float32 rounding order (not bit for bit); out_idx / out_score
 * are unchanged.  The distinct winner rows fetched per (sequence, KV head,
 * quad) are left in the workspace (pariskv_ws_layout.group_rows).  Needs
 * min(G, 4) * k <= PARISKV_MAX_ATTEND_ROWS and n <= 4194304 (64 key ranges of
 * 65536), else UNSUPPORTED. */
#define PARISKV_GROUP_FETCH 4

/* Retrieval budgets of Alg. 1: C = ceil(beta n), C_rho = ceil(rho n), k. */
typedef struct pariskv_budget {
    int64_t n_cand;    /* C, 1..PARISKV_MAX_CAND; clamped to n at run time    */
    int64_t n_collide; /* C_rho >= 1: keys covered by the admitted clusters   */
    int32_t top_k;     /* k, 1..min(C, PARISKV_MAX_TOPK)                      */
    int32_t flags;     /* PARISKV_BINARY_COLLISIONS (else the paper's tiers),
                          PARISKV_EXACT_RECOUNT, PARISKV_GROUP_FETCH, or 0     */
} pariskv_budget;

/* Rows one query head attends at a decode step besides its retrieved keys
 * (Sec. "Buffer Update": the KV cache is kept as Sink, Retrieval, Local and an
 * Update Buffer; Sink, Local and the buffer stay on the GPU and are attended
 * densely, Retrieval is indexed and only its top-k keys are attended).  Row
 * numbers are K/V cache rows of the (sequence, KV head):
 *   Sink            rows [0, sink_len)
 *   retrieved keys  row retr_begin + i for retrieval index row i
 *   Local + Buffer  rows [dense_begin, dense_end)
 * A head attends sink_len + (dense_end - dense_begin) + k rows, at most
 * PARISKV_MAX_ATTEND_ROWS.  The three sets must not share a row (a shared row
 * would count twice).  All four fields 0 = the retrieved keys only, at their
 * own row numbers (plain pariskv_sparse_attend). */
typedef struct pariskv_window {
    int64_t sink_len;
    int64_t retr_begin;
    int64_t dense_begin;
    int64_t dense_end;
} pariskv_window;

#define PARISKV_MAX_ATTEND_ROWS 4096

/* Byte offsets of the intermediate arrays inside a retrieve workspace.  They
 * are stable for given (config, batch, n, budget), so a caller may inspect
 * them after pariskv_retrieve (the parity tests do). */
typedef struct pariskv_ws_layout {
    size_t total;       /* bytes needed                                         */
    size_t zq;          /* float [batch][Hq][D]: H(s*q)/D, rounded to float     */
    size_t lut;         /* uint32 [batch][Hkv][quads][B][256]: tier bonus of
                           centroid c at entry slot(c) (the ids encoding); byte
                           h%4 of the word is query head 4*quad + h%4 of the group */
    size_t score8;      /* uint8 [batch][Hq][n_pad]: collision scores S_i        */
    size_t chunk_sfx;   /* uint32 [batch][Hq][n_chunks][98]: per chunk, #{S >= v}
                           for v = 0 and v_lo <= v <= 97; entries 1 <= v < v_lo
                           hold #{S >= v_lo} (scores below the floor v_lo are
                           not histogrammed, see thresh)                         */
    size_t chunk_base;  /* int32 [batch][Hq][n_chunks][2]: selected keys (S>theta,
                           S==theta) in earlier chunks                          */
    size_t thresh;      /* int32 [batch][Hq][8]: theta, #(S>theta), quota, C_eff,
                           the histogram floor v_lo, 1 if the threshold came from
                           the recount over the stored scores (else 0), 0, 0     */
    size_t cand;        /* int32 [batch][Hq][n_cand]: candidates, ascending      */
    size_t cand_score;  /* float [batch][Hq][n_cand]: RSQ-IP estimates           */
    size_t stats;       /* float [batch][Hq][B][2]: per subspace, sum over the
                           clusters of count * bonus and of count * bonus^2 (the
                           moments that set the histogram floor v_lo)           */
    size_t surv;        /* with topk_parts > 1: int32 [batch][Hq][topk_parts * k]
                           then float [batch][Hq][topk_parts * k], the winners
                           (index, estimate) of each 4096-candidate slice        */
    size_t group_rows;  /* with PARISKV_GROUP_FETCH: int32 [batch][Hkv][quads],
                           the distinct K/V rows the attention fetched           */
    size_t group_part;  /* with PARISKV_GROUP_FETCH and group_splits > 1: float
                           [batch][Hkv][quads][group_splits][4][132], each share's
                           per-head max, sum, rows fetched (head 0, int32 bits),
                           unused, unnormalised output                          */
    int64_t n_pad;      /* row length of score8 (n rounded up to 64)             */
    int64_t n_chunks;   /* ceil(n / chunk_keys)                                  */
    int64_t chunk_keys; /* keys per selection chunk                              */
    int64_t c_eff;      /* min(n_cand, n)                                        */
    int32_t quads;      /* ceil(G / 4)                                           */
    int32_t topk_parts; /* 1, or the slices of the two-pass top-k: with fewer than
                           256 rows (batch x Hq) and more than 8192 candidates,
                           ceil(min(C, n) / 4096) blocks per row first keep the k
                           best of their slice, then one block per row selects
                           among those (the same winners as one pass)           */
    int32_t group_splits; /* with PARISKV_GROUP_FETCH: blocks sharing one (sequence,
                           KV head, quad), block s taking the winners in key range
                           [s r, (s + 1) r), r = ceil(max(n, 1) / group_splits):
                           about 256 blocks in all and at most min(G, 4) * k / 256,
                           but at least ceil(n / 65536) (r <= 65536), at most 64,
                           at least 1; 0 without the flag                        */
} pariskv_ws_layout;

/* ------------------------------------------------------------ encoding */

/* Prefill key summarisation (Sec. "Prefill Phase"; Alg. 1 encode loop).
 * keys: device float16 [batch][Hkv][n][D], contiguous.  For every key writes
 * ids and rec at rows [0, n) of each (sequence, KV head) and recomputes
 * counts from those n keys (counts are cleared first).
 * Errors: INVALID (shapes, pointers, n < 0), CAPACITY (n > capacity), HIP. */
int pariskv_encode(const pariskv_config* cfg, const pariskv_index* index,
                   const void* keys, int64_t n, int32_t batch, void* stream);

/* Streaming update (Sec. "Buffer Update": newly evicted keys are encoded and
 * indexed).  keys: device float16 [batch][Hkv][t][D]; writes rows
 * [n_cur, n_cur + t) and adds them to counts.  t may be 1 (per-step append)
 * or a whole update buffer.
 * Errors: INVALID, CAPACITY (n_cur + t > capacity), HIP. */
int pariskv_append(const pariskv_config* cfg, const pariskv_index* index,
                   const void* keys, int64_t n_cur, int64_t t, int32_t batch,
                   void* stream);

/* Streaming update read straight from the layer's key cache (Sec. "Buffer
 * Update" steps (i) and (iii): the oldest Local tokens move to Retrieval and
 * their keys are encoded and indexed).  K: device float16
 * [batch][Hkv][kv_capacity][D].  Encodes cache rows [row_begin, row_begin + t)
 * of every (sequence, KV head) into index rows [n_cur, n_cur + t) and adds them
 * to counts: the same bytes pariskv_append writes for those rows copied out.
 * Errors: INVALID (row range outside the cache), CAPACITY (n_cur + t >
 * capacity), HIP. */
int pariskv_append_rows(const pariskv_config* cfg, const pariskv_index* index,
                        const void* K, int64_t kv_capacity, int64_t row_begin,
                        int64_t n_cur, int64_t t, int32_t batch, void* stream);

/* The four regions after a prompt of P tokens and t decode steps (Sec.
 * "Buffer Update"): the prompt's first min(sink, P) tokens are Sink, its last
 * min(local, P - sink) tokens Local, the rest Retrieval; every decode token
 * enters the Update Buffer, and when the buffer holds m tokens, Local becomes
 * the most recent `local` tokens of Local + Buffer, the older ones joining
 * Retrieval.  Fills `out` for pariskv_window_attend (Sink at rows [0,
 * sink_len), Retrieval at rows [retr_begin, dense_begin), Local + Buffer at
 * [dense_begin, P + t)) and *n_retrieval = dense_begin - retr_begin, the
 * number of keys the retrieval index must hold.  Host only.
 * Errors: INVALID (negative sizes, m < 1, overflow). */
int pariskv_window_regions(int64_t P, int64_t t, int64_t sink, int64_t local, int64_t m,
                           pariskv_window* out, int64_t* n_retrieval);

/* ------------------------------------------------------------ retrieval */

/* Workspace bytes pariskv_retrieve needs for these shapes (0 on invalid input). */
size_t pariskv_retrieve_workspace(const pariskv_config* cfg, int32_t batch, int64_t n,
                                  const pariskv_budget* budget);

/* Offsets of the intermediates inside that workspace.  Errors: INVALID. */
int pariskv_workspace_layout(const pariskv_config* cfg, int32_t batch, int64_t n,
                             const pariskv_budget* budget, pariskv_ws_layout* out);

/* Two-stage retrieval for every query head (Sec. "Retrieval"; Alg. 1 decode).
 *   q          device float16 [batch][Hq][D]
 *   n          keys indexed per (sequence, KV head), 0..capacity
 *   out_idx    device int32 [batch][Hq][k]: the k keys with the largest
 *              RSQ-IP estimates (ties at the k-th estimate: lower key index
 *              first), listed in ascending key index; -1 pads when fewer than
 *              k keys exist
 *   out_score  device float [batch][Hq][k] or NULL: the matching estimates of
 *              <k_i, q> (-inf on padding)
 *   workspace  device, >= pariskv_retrieve_workspace(...) bytes, 256-byte
 *              aligned; overwritten
 * Stage I ranks clusters per subspace by <q_tilde_b, omega_c> (ties: lower
 * centroid id), admits whole clusters while fewer than C_rho keys precede
 * them, gives tier weights 6..1 at cuts ceil({5,15,30,50,75,100}% * C_rho)
 * by the number of keys preceding the cluster, and sums over subspaces.
 * Selection keeps the min(C, n) best scores, ties at the threshold in
 * ascending key index: theta is the largest v with #{S >= v} >= min(C, n).
 * The scan histograms only scores at or above a per-head floor v_lo, the
 * integer part of a normal-law estimate of theta from the bonus moments (stats); when
 * #{S >= v_lo} < min(C, n) the threshold is found by an exact recount over
 * the stored scores instead, so the result never depends on the floor.
 * Stage II estimates <k_i, q> for those candidates.
 * Errors: INVALID, UNSUPPORTED (C or k above the served maximum), WORKSPACE, HIP. */
int pariskv_retrieve(const pariskv_config* cfg, const pariskv_index* index,
                     const void* q, int64_t n, int32_t batch,
                     const pariskv_budget* budget, int32_t* out_idx, float* out_score,
                     void* workspace, size_t ws_bytes, void* stream);

/* pariskv_retrieve followed by the attention of every query head over its k
 * winners, in one call: the same out_idx / out_score as pariskv_retrieve and
 * the same `out` as pariskv_sparse_attend(cfg, q, K, V, kv_host_mapped,
 * kv_capacity, out_idx, k, batch, scale, out) would give, bit for bit.  For
 * every C the attention runs inside the (final) top-k kernel over the winners
 * it holds, with no second pass over out_idx.
 * Arguments as in those two functions.
 * Errors: those of pariskv_retrieve and of pariskv_sparse_attend. */
int pariskv_retrieve_attend(const pariskv_config* cfg, const pariskv_index* index,
                            const void* q, int64_t n, int32_t batch,
                            const pariskv_budget* budget, int32_t* out_idx, float* out_score,
                            const void* K, const void* V, int32_t kv_host_mapped,
                            int64_t kv_capacity, float scale, float* out, void* workspace,
                            size_t ws_bytes, void* stream);

/* Attention over the fetched keys only (Eqs. approx_weight, approx_output):
 *   o = sum_{i in idx} softmax_i(scale * <k_i, q>) v_i,
 * float16 inputs, float32 accumulation.
 *   q     device float16 [batch][Hq][D]
 *   K, V  float16 [batch][Hkv][kv_capacity][D]; device memory when
 *         kv_host_mapped == 0; pinned host memory (hipHostMalloc) when 1, read
 *         directly by the kernel over the host link (the paper's UVA fetch)
 *   idx   device int32 [batch][Hq][k], k <= 4096; entries outside
 *         [0, kv_capacity) (for example -1 padding) are skipped
 *   out   device float [batch][Hq][D]; zero when no valid index
 * scale = 1 reproduces the paper's raw score; models use 1/sqrt(D).
 * Errors: INVALID, UNSUPPORTED (k > 4096), HIP. */
int pariskv_sparse_attend(const pariskv_config* cfg, const void* q, const void* K,
                          const void* V, int32_t kv_host_mapped, int64_t kv_capacity,
                          const int32_t* idx, int32_t k, int32_t batch, float scale,
                          float* out, void* stream);

/* Attention of a decode step over Sink, the retrieved keys and Local + Update
 * Buffer (Sec. "Buffer Update"; Eqs. approx_weight, approx_output with C(q)
 * the union of the three row sets of `win`):
 *   o = sum_{i in rows} softmax_i(scale * <k_i, q>) v_i.
 * Arguments as in pariskv_sparse_attend; idx holds retrieval index rows
 * (entry j attends cache row win->retr_begin + idx[j]; entries < 0 and rows
 * outside [0, kv_capacity) are skipped).  win: host pointer.
 * Errors: INVALID (window rows outside the cache or out of order: sink_len <=
 * retr_begin <= dense_begin <= dense_end <= kv_capacity), UNSUPPORTED (more than
 * PARISKV_MAX_ATTEND_ROWS rows per head), HIP. */
int pariskv_window_attend(const pariskv_config* cfg, const void* q, const void* K,
                          const void* V, int32_t kv_host_mapped, int64_t kv_capacity,
                          const int32_t* idx, int32_t k, const pariskv_window* win,
                          int32_t batch, float scale, float* out, void* stream);

/* pariskv_retrieve over the Retrieval region (n index rows, the keys of cache
 * rows [win->retr_begin, win->retr_begin + n)) followed by
 * pariskv_window_attend over Sink + winners + Local/Buffer, in one call, with
 * the same outputs bit for bit.  The attention runs inside the
 * top-k kernel.  Also requires win->retr_begin + n <= win->dense_begin.
 * Errors: those of pariskv_retrieve and pariskv_window_attend. */
int pariskv_retrieve_window_attend(const pariskv_config* cfg, const pariskv_index* index,
                                   const void* q, int64_t n, int32_t batch,
                                   const pariskv_budget* budget, int32_t* out_idx,
                                   float* out_score, const void* K, const void* V,
                                   int32_t kv_host_mapped, int64_t kv_capacity,
                                   const pariskv_window* win, float scale, float* out,
                                   void* workspace, size_t ws_bytes, void* stream);

/* pariskv_sparse_attend with every distinct K/V row fetched once per KV head:
 * the query heads of a KV head (in quads of 4) attend over the union of their
 * lists, each union row is read once and feeds every head that selected it
 * (GQA-group de-duplication of the fetch; the saving is the heads' overlap,
 * on the host link when kv_host_mapped).  Same arguments and, up to float32
 * rounding order, the same result as pariskv_sparse_attend; each head's list
 * must be ascending with any -1 padding at its end, as pariskv_retrieve writes
 * it (other orders give unspecified values, never an access outside K/V).
 *   union_rows  device int32 [batch][Hkv][ceil(G/4)] or NULL: rows fetched
 * Errors: INVALID, UNSUPPORTED (min(G, 4) * k > PARISKV_MAX_ATTEND_ROWS), HIP. */
int pariskv_group_attend(const pariskv_config* cfg, const void* q, const void* K, const void* V,
                         int32_t kv_host_mapped, int64_t kv_capacity, const int32_t* idx, int32_t k,
                         int32_t batch, float scale, float* out, int32_t* union_rows, void* stream);

/* Tiered attention of the offload setting (Sec. "Buffer Update": Sink, Local
 * and the Update Buffer stay on the GPU, the Retrieval region is offloaded to
 * CPU memory; Sec. "On-Demand UVA Fetch": only the retrieved rows are read
 * from there).  Same result as pariskv_window_attend, with the dense rows read
 * from a window cache on the GPU:
 *   K_win, V_win  device float16 [batch][Hkv][win_capacity][D]: Sink row r at
 *                 slot r, Local / Buffer row r at slot
 *                 sink_len + (r - sink_len) mod (win_capacity - sink_len)
 *                 (a ring: the caller writes each new token at its slot)
 *   K, V          the retrieval rows, float16 [batch][Hkv][kv_capacity][D],
 *                 in pinned host memory (kv_host_mapped = 1) or device memory;
 *                 retrieved index row i is row win->retr_begin + i
 * Attention caches hold at most 2^30 - 1 rows.
 * Errors: INVALID (also a window cache too small for sink_len + the dense
 * rows), UNSUPPORTED (more than PARISKV_MAX_ATTEND_ROWS rows per head), HIP. */
int pariskv_tiered_attend(const pariskv_config* cfg, const void* q, const void* K_win,
                          const void* V_win, int64_t win_capacity, const void* K, const void* V,
                          int32_t kv_host_mapped, int64_t kv_capacity, const int32_t* idx, int32_t k,
                          const pariskv_window* win, int32_t batch, float scale, float* out,
                          void* stream);

/* pariskv_retrieve followed by pariskv_tiered_attend, in one call, with the
 * same outputs bit for bit (attention inside the top-k kernel).
 * Also requires win->retr_begin + n <= min(win->dense_begin, kv_capacity).
 * Errors: those of pariskv_retrieve and pariskv_tiered_attend. */
int pariskv_retrieve_tiered_attend(const pariskv_config* cfg, const pariskv_index* index,
                                   const void* q, int64_t n, int32_t batch,
                                   const pariskv_budget* budget, int32_t* out_idx,
                                   float* out_score, const void* K_win, const void* V_win,
                                   int64_t win_capacity, const void* K, const void* V,
                                   int32_t kv_host_mapped, int64_t kv_capacity,
                                   const pariskv_window* win, float scale, float* out,
                                   void* workspace, size_t ws_bytes, void* stream);

/* Copy of t K and V rows of every (sequence, KV head): rows [src_row,
 * src_row + t) of K_src / V_src ([batch][Hkv][src_capacity][D] float16) to rows
 * [dst_row, dst_row + t) of K_dst / V_dst ([batch][Hkv][dst_capacity][D]).  The
 * offload of the rows that leave Local (Sec. "Buffer Update" (i): evicted into
 * Retrieval "via GPU->CPU transfer", asynchronously): from the GPU window cache
 * to pinned host memory (or any direction the HIP runtime copies), as two
 * pitched asynchronous copies on `stream` -- run it on a second stream to
 * overlap the retrieval, and order the first attention that may read those
 * rows after it.  A ring range that wraps takes two calls.
 * Errors: INVALID (NULL pointers, rows outside either cache), HIP. */
int pariskv_offload_rows(const void* K_src, const void* V_src, int64_t src_capacity, int64_t src_row,
                         void* K_dst, void* V_dst, int64_t dst_capacity, int64_t dst_row, int64_t t,
                         int32_t batch, int32_t n_kv_heads, void* stream);

/* ------------------------------------------------- without a caller workspace */

/* Bytes of the static scratch array pariskv_retrieve_attend_noalloc keeps its
 * intermediates in, on every device the library runs on. */
#define PARISKV_NOALLOC_SCRATCH_BYTES ((size_t)64 << 20)

/* For callers that cannot allocate device memory: code under HIP graph capture,
 * tight serving loops, harnesses that forbid hipMalloc.  pariskv_retrieve_attend
 * without a workspace argument: the same out_idx, out_score and out, bit for bit,
 * with the retrieve intermediates kept in a library-owned device array of
 * PARISKV_NOALLOC_SCRATCH_BYTES (64 MiB) instead.  The array belongs to the
 * library's code object: each device holds its own copy from the first call on
 * it until the process ends, and its device address is looked up once per
 * device, at that first call, with the device current.  The call itself
 * allocates nothing (no hipMalloc, hipFree or allocating library routine; with
 * the event profiler off), validates on the host, enqueues on `stream` (which
 * must belong to the current device) and returns.
 * Sharing: every call on one device uses the same array and leaves its
 * intermediates there.  Calls that overlap on one device (unordered streams or
 * host threads) race on it and give undefined outputs; order them.  Nothing in
 * the array has to start at zero: a call writes every intermediate before it
 * reads it.  pariskv_workspace_layout describes where they lie.
 * Errors: those of pariskv_retrieve_attend; WORKSPACE when these shapes need
 * more than PARISKV_NOALLOC_SCRATCH_BYTES of intermediates
 * (pariskv_retrieve_workspace gives the need), checked before any HIP call;
 * HIP also when the array's device address cannot be obtained. */
int pariskv_retrieve_attend_noalloc(const pariskv_config* cfg, const pariskv_index* index,
                                    const void* q, int64_t n, int32_t batch,
                                    const pariskv_budget* budget, int32_t* out_idx,
                                    float* out_score, const void* K, const void* V,
                                    int32_t kv_host_mapped, int64_t kv_capacity, float scale,
                                    float* out, void* stream);

/* ------------------------------------------------------------ utilities */

/* The offline magnitude quantizer (Appendix "Coordinate-Magnitude Quantizer"):
 * Lloyd-Max thresholds tau[0..6] (= tau_1..tau_7) and levels a[0..7] for
 * X = |u_j| with X^2 ~ Beta(1/2, (m-1)/2), rounded to double.  Host only.
 * Errors: UNSUPPORTED for m != 8. */
int pariskv_quantizer_table(int32_t m, double* tau, double* a);

/* Rotation signs of R = H_D diag(s) / sqrt(D) (Sec. "Preprocessing" (1); the
 * paper names an SRHT without a construction): s_j = -1 when bit 63 of
 * splitmix64(seed + j) is set, else +1, where splitmix64(x) is the first output
 * of a SplitMix64 generator whose state is x (state += 0x9E3779B97F4A7C15, then
 * the two xor-shift-multiply rounds and a final xor-shift).  Writes D int8
 * values to host memory `out`, ready for pariskv_config.rot_signs.  Host only.
 * Errors: INVALID for D < 1 or a null `out`. */
int pariskv_rotation_signs(uint64_t seed, int32_t D, int8_t* out);

/* Reference streaming kernels for measurement (not part of the retrieval path):
 * a plain copy of `bytes` from src to dst, and a plain read of `bytes` of src,
 * both device memory, 16-byte aligned, bytes a multiple of 16.  They state the
 * HBM bandwidth this GPU achieves for a pure stream, and scale HBM counters (a
 * copy of known size moves exactly 2 x bytes).  The read folds the data into one
 * word per thread and stores it to device `sink` (4 bytes) only if it equals
 * `key`, so its loads cannot be removed.
 * Errors: INVALID (NULL or misaligned pointers, bytes not a multiple of 16), HIP. */
int pariskv_stream_copy(void* dst, const void* src, size_t bytes, void* stream);
int pariskv_stream_read(const void* src, size_t bytes, uint32_t key, uint32_t* sink, void* stream);

/* Per-kernel timing with HIP events attached to the kernel dispatches on the
 * launch stream.  The first kernel of a call is timed from its dispatch to its
 * completion; every following kernel of the same call, which the GPU starts as
 * soon as its predecessor completes, from that predecessor's completion to its
 * own.  Off by default; a launch while on adds no synchronisation. */
int pariskv_profile_enable(int32_t on);
int pariskv_profile_reset(void);
/* Waits for the recorded events; fills at most max_entries rows. Returns the
 * number of distinct kernels seen, or a negative error code. */
int pariskv_profile_read(int32_t max_entries, const char** names, int64_t* launches,
                         double* total_ms);

const char* pariskv_strerror(int code);
const char* pariskv_last_error(void);
/* Version of the structs and entry points declared here: 4 (pariskv_ws_layout
 * with stats, surv, group_rows, group_part, topk_parts and group_splits). */
int32_t pariskv_abi_version(void);

#ifdef __cplusplus
}
#endif

#endif /* PARISKV_H */
