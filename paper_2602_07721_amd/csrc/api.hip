// Host side of the C ABI declared in include/pariskv.h: argument validation,
// workspace layout, kernel sequencing and per-kernel event timing.  No
// device memory is allocated here; every HIP call happens after validation.

#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <map>
#include <mutex>
#include <string>
#include <vector>

#include "../../include/pariskv.h"
#include "internal.hpp"

namespace pariskv {

namespace {

thread_local std::string t_last_error;

int fail(int code, const char* fmt, ...) {
    char buf[512];
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(buf, sizeof buf, fmt, ap);
    va_end(ap);
    t_last_error = buf;
    return code;
}

int hip_fail(hipError_t e, const char* where) {
    return fail(PARISKV_ERR_HIP, "%s: %s", where, hipGetErrorString(e));
}

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

constexpr int64_t kMaxGridY = 65535;

// Multiply non-negative int64 values, false on overflow past 2^62.
bool mul_ok(int64_t a, int64_t b, int64_t* out) {
    if (a < 0 || b < 0) return false;
    if (a != 0 && b > (int64_t(1) << 62) / a) return false;
    *out = a * b;
    return true;
}

int check_config(const pariskv_config* cfg, int32_t batch) {
    if (!cfg) return fail(PARISKV_ERR_INVALID, "config is NULL");
    const int32_t D = cfg->head_dim, B = cfg->n_subspaces;
    if (D <= 0 || (D & (D - 1)) != 0)
        return fail(PARISKV_ERR_INVALID, "head_dim %d is not a positive power of two", D);
    if (B <= 0 || D % B != 0)
        return fail(PARISKV_ERR_INVALID, "n_subspaces %d does not divide head_dim %d", B, D);
    if (D != kD || B != kB)
        return fail(PARISKV_ERR_UNSUPPORTED, "only head_dim 128 with 16 subspaces (m = 8) is built");
    if (cfg->n_kv_heads < 1) return fail(PARISKV_ERR_INVALID, "n_kv_heads %d < 1", cfg->n_kv_heads);
    if (cfg->q_per_kv < 1 || cfg->q_per_kv > 16)
        return fail(PARISKV_ERR_INVALID, "q_per_kv %d outside 1..16", cfg->q_per_kv);
    if (cfg->capacity < 1 || cfg->capacity > INT32_MAX)
        return fail(PARISKV_ERR_INVALID, "capacity %lld outside 1..2^31-1", (long long)cfg->capacity);
    if (!cfg->rot_signs) return fail(PARISKV_ERR_INVALID, "rot_signs is NULL");
    if (cfg->flags & ~(PARISKV_NO_ROTATION | PARISKV_NO_ALPHA_CORRECTION))
        return fail(PARISKV_ERR_INVALID, "unknown config flags 0x%x", cfg->flags);
    for (int j = 0; j < D; ++j)
        if (cfg->rot_signs[j] != 1 && cfg->rot_signs[j] != -1)
            return fail(PARISKV_ERR_INVALID, "rot_signs[%d] = %d is not +1 or -1", j, cfg->rot_signs[j]);
    if (batch < 1) return fail(PARISKV_ERR_INVALID, "batch %d < 1", batch);
    int64_t t;
    if (!mul_ok((int64_t)batch * cfg->n_kv_heads, cfg->capacity, &t) || !mul_ok(t, kRec, &t))
        return fail(PARISKV_ERR_INVALID, "batch * n_kv_heads * capacity overflows");
    if ((int64_t)batch * cfg->n_kv_heads * cfg->q_per_kv > kMaxGridY)
        return fail(PARISKV_ERR_UNSUPPORTED, "batch * query heads above %lld", (long long)kMaxGridY);
    return PARISKV_OK;
}

int check_index(const pariskv_index* ix) {
    if (!ix) return fail(PARISKV_ERR_INVALID, "index is NULL");
    if (!ix->ids || !ix->rec || !ix->counts)
        return fail(PARISKV_ERR_INVALID, "index arrays must be non-NULL");
    if (!aligned16(ix->ids) || !aligned16(ix->rec) || !aligned16(ix->counts))
        return fail(PARISKV_ERR_INVALID, "index arrays must be 16-byte aligned");
    return PARISKV_OK;
}

SignBits pack_signs(const int8_t* s) {
    SignBits b{};
    for (int j = 0; j < kD; ++j)
        if (s[j] < 0) b.w[j >> 5] |= 1u << (j & 31);
    return b;
}

const QuantConsts& quant_consts() {
    static QuantConsts qc;
    static std::once_flag once;
    std::call_once(once, [] {
        double tau[7], a[8];
        quantizer_table_m8(tau, a);
        for (int t = 0; t < 8; ++t) {
            qc.a[t] = a[t];
            qc.a32[t] = (float)a[t];
        }
        for (int t = 0; t < 7; ++t) qc.tau2[t] = tau[t] * tau[t];
    });
    return qc;
}

int layout(const pariskv_config* cfg, int32_t batch, int64_t n, const pariskv_budget* bud,
           pariskv_ws_layout* L) {
    int rc = check_config(cfg, batch);
    if (rc) return rc;
    if (!bud) return fail(PARISKV_ERR_INVALID, "budget is NULL");
    if (n < 0) return fail(PARISKV_ERR_INVALID, "n %lld < 0", (long long)n);
    if (n > cfg->capacity)
        return fail(PARISKV_ERR_INVALID, "n %lld exceeds capacity %lld", (long long)n,
                    (long long)cfg->capacity);
    if (bud->n_cand < 1) return fail(PARISKV_ERR_INVALID, "n_cand %lld < 1", (long long)bud->n_cand);
    if (bud->n_cand > PARISKV_MAX_CAND)
        return fail(PARISKV_ERR_UNSUPPORTED, "n_cand %lld above %d", (long long)bud->n_cand,
                    PARISKV_MAX_CAND);
    if (bud->n_collide < 1)
        return fail(PARISKV_ERR_INVALID, "n_collide %lld < 1", (long long)bud->n_collide);
    if (bud->top_k < 1 || bud->top_k > bud->n_cand)
        return fail(PARISKV_ERR_INVALID, "top_k %d outside 1..n_cand", bud->top_k);
    if (bud->top_k > PARISKV_MAX_TOPK)
        return fail(PARISKV_ERR_UNSUPPORTED, "top_k %d above %d", bud->top_k, PARISKV_MAX_TOPK);
    if (bud->flags & ~(PARISKV_BINARY_COLLISIONS | PARISKV_EXACT_RECOUNT | PARISKV_GROUP_FETCH))
        return fail(PARISKV_ERR_INVALID, "unknown budget flags 0x%x", bud->flags);

    const int64_t hkv = cfg->n_kv_heads, g = cfg->q_per_kv, hq = hkv * g;
    const int64_t quads = (g + 3) / 4;
    const int64_t rows = (int64_t)batch * hq;
    std::memset(L, 0, sizeof *L);
    L->n_pad = ((n > 0 ? n : 1) + 63) / 64 * 64;
    L->chunk_keys = kChunk;
    L->n_chunks = (n + kChunk - 1) / kChunk;
    L->c_eff = bud->n_cand < n ? bud->n_cand : n;
    L->quads = (int32_t)quads;
    size_t off = 0;
    auto take = [&](size_t bytes) {
        const size_t at = off;
        off += (bytes + 255) / 256 * 256;
        return at;
    };
    L->zq = take((size_t)rows * kD * 4);
    L->lut = take((size_t)batch * hkv * quads * kB * kCentroids * 4);
    L->score8 = take((size_t)rows * L->n_pad);
    L->chunk_sfx = take((size_t)rows * L->n_chunks * kSfx * 4);
    L->chunk_base = take((size_t)rows * L->n_chunks * 2 * 4);
    L->thresh = take((size_t)rows * 8 * 4);
    L->cand = take((size_t)rows * bud->n_cand * 4);
    L->cand_score = take((size_t)rows * bud->n_cand * 4);
    L->stats = take((size_t)rows * kB * 2 * 4);
    L->topk_parts = topk_parts(rows, L->c_eff, bud->top_k);
    L->surv = take(L->topk_parts > 1 ? (size_t)rows * L->topk_parts * bud->top_k * 8 : 0);
    const bool group_fetch = (bud->flags & PARISKV_GROUP_FETCH) != 0;
    L->group_rows = take(group_fetch ? (size_t)batch * hkv * quads * 4 : 0);
    L->group_splits = group_fetch ? group_splits((int64_t)batch * hkv * quads, (g < 4 ? g : 4) * (int64_t)bud->top_k, n) : 0;
    L->group_part = take(group_fetch ? group_part_bytes((int64_t)batch * hkv * quads, L->group_splits) : 0);
    L->total = off;
    return PARISKV_OK;
}

// ---------------------------------------------------------------- profiler

struct Pending {
    std::string name;
    hipEvent_t start, stop;
    bool own_start;  // false: start is the previous launch's stop event
};
struct Acc {
    int64_t launches = 0;
    double ms = 0.0;
};

std::mutex g_prof_mu;
bool g_prof_on = false;
std::vector<Pending> g_pending;
std::vector<hipEvent_t> g_pool;
std::map<std::string, Acc> g_acc;

hipEvent_t pool_get() {
    if (!g_pool.empty()) {
        hipEvent_t e = g_pool.back();
        g_pool.pop_back();
        return e;
    }
    // Timing-only events: without the system-scope fence the recording does not
    // write back and invalidate the caches, which would delay and slow the next kernel.
    hipEvent_t e = nullptr;
    if (hipEventCreateWithFlags(&e, hipEventDisableSystemFence) != hipSuccess) return nullptr;
    return e;
}

int collect_locked() {
    for (auto& p : g_pending) {
        float ms = 0.f;
        if (hipEventSynchronize(p.stop) != hipSuccess) return hip_fail(hipGetLastError(), "hipEventSynchronize");
        if (hipEventElapsedTime(&ms, p.start, p.stop) == hipSuccess) {
            Acc& a = g_acc[p.name];
            a.launches += 1;
            a.ms += ms;
        }
        if (p.own_start) g_pool.push_back(p.start);
        g_pool.push_back(p.stop);
    }
    g_pending.clear();
    return PARISKV_OK;
}

}  // namespace

// Completion event of the previous profiled launch in the current API call.
thread_local hipEvent_t t_chain = nullptr;

void prof_chain_start() { t_chain = nullptr; }

ProfEvents prof_begin(const char* name) {
    std::lock_guard<std::mutex> lk(g_prof_mu);
    if (!g_prof_on) return {};
    hipEvent_t stop = pool_get();
    if (!stop) return {};
    if (t_chain) {
        // Launched right behind another kernel of the same call: timed from that
        // kernel's completion to this one's.
        g_pending.push_back(Pending{name, t_chain, stop, false});
        t_chain = stop;
        return {nullptr, stop};
    }
    hipEvent_t start = pool_get();
    if (!start) {
        g_pool.push_back(stop);
        return {};
    }
    g_pending.push_back(Pending{name, start, stop, true});
    t_chain = stop;
    return {start, stop};
}

// ---- pariskv_retrieve_attend_noalloc: intermediates in a static device array

// One copy per device, loaded with the code object and kept until the process ends.
// In host code `scratch` names a host-side stand-in, never the device array: only the
// address hipGetSymbolAddress returns for the current device is passed to kernels.
static __device__ __align__(256) unsigned char scratch[PARISKV_NOALLOC_SCRATCH_BYTES];

constexpr int kMaxScratchDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxScratchDevices] = {};

// Device address of the current device's scratch array, looked up on its first use.
int scratch_ptr(void** out) {
    int dev = -1;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return hip_fail(e, "hipGetDevice");
    if (dev < 0 || dev >= kMaxScratchDevices)
        return fail(PARISKV_ERR_UNSUPPORTED, "device %d above the %d devices served", dev, kMaxScratchDevices);
    std::lock_guard<std::mutex> lk(g_scratch_mu);
    if (!g_scratch_ptr[dev]) {
        void* p = nullptr;
        e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess) return hip_fail(e, "hipGetSymbolAddress(scratch)");
        if (!p || (reinterpret_cast<uintptr_t>(p) & 255u) != 0)
            return fail(PARISKV_ERR_HIP, "scratch array at %p is not 256-byte aligned", p);
        g_scratch_ptr[dev] = p;
    }
    *out = g_scratch_ptr[dev];
    return PARISKV_OK;
}

}  // namespace pariskv

using namespace pariskv;

extern "C" {

int32_t pariskv_abi_version(void) { return 4; }

const char* pariskv_strerror(int code) {
    switch (code) {
        case PARISKV_OK: return "ok";
        case PARISKV_ERR_INVALID: return "invalid argument";
        case PARISKV_ERR_CAPACITY: return "index capacity exceeded";
        case PARISKV_ERR_WORKSPACE: return "workspace missing or too small";
        case PARISKV_ERR_HIP: return "HIP runtime error";
        case PARISKV_ERR_UNSUPPORTED: return "unsupported configuration";
        default: return "unknown error";
    }
}

const char* pariskv_last_error(void) { return t_last_error.c_str(); }

int pariskv_rotation_signs(uint64_t seed, int32_t D, int8_t* out) {
    if (D < 1) return fail(PARISKV_ERR_INVALID, "D = %d < 1", D);
    if (!out) return fail(PARISKV_ERR_INVALID, "out is null");
    for (int32_t j = 0; j < D; ++j) {
        uint64_t z = seed + (uint64_t)j + 0x9E3779B97F4A7C15ull;
        z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
        z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
        z ^= z >> 31;
        out[j] = (z >> 63) ? int8_t(-1) : int8_t(1);
    }
    return PARISKV_OK;
}

int pariskv_quantizer_table(int32_t m, double* tau, double* a) {
    if (!tau || !a) return fail(PARISKV_ERR_INVALID, "NULL output");
    if (m != kM) return fail(PARISKV_ERR_UNSUPPORTED, "only m = 8 is built");
    quantizer_table_m8(tau, a);
    return PARISKV_OK;
}

static int encode_common(const pariskv_config* cfg, const pariskv_index* index, const void* keys,
                         int64_t src_stride, int64_t row0, int64_t t, int32_t batch, bool reset_counts,
                         void* stream) {
    prof_chain_start();
    int rc = check_config(cfg, batch);
    if (rc) return rc;
    rc = check_index(index);
    if (rc) return rc;
    if (row0 < 0 || t < 0) return fail(PARISKV_ERR_INVALID, "negative key range");
    if (t > 0 && (!keys || !aligned16(keys)))
        return fail(PARISKV_ERR_INVALID, "keys must be non-NULL and 16-byte aligned");
    if (row0 + t > cfg->capacity)
        return fail(PARISKV_ERR_CAPACITY, "rows [%lld, %lld) exceed capacity %lld", (long long)row0,
                    (long long)(row0 + t), (long long)cfg->capacity);
    hipStream_t s = static_cast<hipStream_t>(stream);
    const int64_t groups = (int64_t)batch * cfg->n_kv_heads;
    hipError_t e;
    if (reset_counts) {
        e = launch_zero_u32(index->counts, groups * kB * kCentroids, s);
        if (e != hipSuccess) return hip_fail(e, "zero counts");
    }
    e = launch_encode(keys, t, src_stride < 0 ? t : src_stride, groups, row0, cfg->capacity, index->ids,
                      index->rec, index->counts, pack_signs(cfg->rot_signs), quant_consts(),
                      ((cfg->flags & PARISKV_NO_ROTATION) ? kFlagNoRotation : 0u) |
                          ((cfg->flags & PARISKV_NO_ALPHA_CORRECTION) ? kFlagNoAlpha : 0u),
                      s);
    if (e != hipSuccess) return hip_fail(e, "encode launch");
    return PARISKV_OK;
}

int pariskv_encode(const pariskv_config* cfg, const pariskv_index* index, const void* keys,
                   int64_t n, int32_t batch, void* stream) {
    if (n < 0) return fail(PARISKV_ERR_INVALID, "n %lld < 0", (long long)n);
    return encode_common(cfg, index, keys, -1, 0, n, batch, true, stream);
}

int pariskv_append(const pariskv_config* cfg, const pariskv_index* index, const void* keys,
                   int64_t n_cur, int64_t t, int32_t batch, void* stream) {
    return encode_common(cfg, index, keys, -1, n_cur, t, batch, false, stream);
}

int pariskv_append_rows(const pariskv_config* cfg, const pariskv_index* index, const void* K,
                        int64_t kv_capacity, int64_t row_begin, int64_t n_cur, int64_t t,
                        int32_t batch, void* stream) {
    if (kv_capacity < 1 || kv_capacity > INT32_MAX)
        return fail(PARISKV_ERR_INVALID, "kv_capacity %lld outside 1..2^31-1", (long long)kv_capacity);
    if (row_begin < 0 || t < 0 || row_begin > kv_capacity - t)
        return fail(PARISKV_ERR_INVALID, "cache rows [%lld, %lld + %lld) outside [0, %lld)",
                    (long long)row_begin, (long long)row_begin, (long long)t, (long long)kv_capacity);
    const void* src = K ? static_cast<const void*>(static_cast<const char*>(K) + row_begin * kD * 2) : nullptr;
    return encode_common(cfg, index, src, kv_capacity, n_cur, t, batch, false, stream);
}

int pariskv_window_regions(int64_t P, int64_t t, int64_t sink, int64_t local, int64_t m,
                           pariskv_window* out, int64_t* n_retrieval) {
    if (!out || !n_retrieval) return fail(PARISKV_ERR_INVALID, "NULL output");
    if (P < 0 || t < 0 || sink < 0 || local < 0 || m < 1)
        return fail(PARISKV_ERR_INVALID, "negative size or m < 1");
    if (P > (int64_t(1) << 40) || t > (int64_t(1) << 40))
        return fail(PARISKV_ERR_INVALID, "P or t above 2^40");
    // After the prompt: Sink = first min(sink, P) tokens, Local = last min(local,
    // rest) tokens, Retrieval in between.  After u = t / m buffer updates Local
    // holds min(local, l0 + u m) tokens ending at P + u m; the buffer holds the
    // t - u m newest tokens.
    const int64_t s_len = sink < P ? sink : P;
    const int64_t l0 = local < P - s_len ? local : P - s_len;
    const int64_t u = t / m;
    const int64_t grown = l0 + u * m;
    const int64_t l_u = local < grown ? local : grown;
    const int64_t local_end = P + u * m;
    out->sink_len = s_len;
    out->retr_begin = s_len;
    out->dense_begin = local_end - l_u;
    out->dense_end = P + t;
    *n_retrieval = out->dense_begin - s_len;
    return PARISKV_OK;
}

size_t pariskv_retrieve_workspace(const pariskv_config* cfg, int32_t batch, int64_t n,
                                  const pariskv_budget* budget) {
    pariskv_ws_layout L;
    if (layout(cfg, batch, n, budget, &L) != PARISKV_OK) return 0;
    return L.total;
}

int pariskv_workspace_layout(const pariskv_config* cfg, int32_t batch, int64_t n,
                             const pariskv_budget* budget, pariskv_ws_layout* out) {
    if (!out) return fail(PARISKV_ERR_INVALID, "layout output is NULL");
    return layout(cfg, batch, n, budget, out);
}

// Attention arguments of the retrieve + attend entry points.
struct AttendReq {
    const void* K;
    const void* V;
    int32_t kv_host_mapped;
    int64_t kv_capacity;
    float scale;
    float* out;
    AttendWindow win;
    const void* Kw = nullptr;  // window cache (device), win.win_capacity > 0
    const void* Vw = nullptr;
};

// Window rows in order; dense rows inside the main cache, or inside the window
// cache's ring when win_capacity > 0; with k retrieved rows per head the list
// fits one attention block.  n >= 0: the retrieval index holds n keys, whose
// rows [retr_begin, retr_begin + n) must end before the dense rows (and, with a
// window cache, inside the main cache).
static int check_window(const pariskv_window* w, int64_t kv_capacity, int64_t k, int64_t n,
                        int64_t win_capacity, AttendWindow* out) {
    *out = AttendWindow{};
    if (!w) return PARISKV_OK;
    const int64_t dense_cap = win_capacity > 0 ? INT64_MAX : kv_capacity;
    if (w->sink_len < 0 || w->retr_begin < w->sink_len || w->dense_begin < w->retr_begin ||
        w->dense_end < w->dense_begin || w->dense_end > dense_cap)
        return fail(PARISKV_ERR_INVALID,
                    "window needs 0 <= sink_len (%lld) <= retr_begin (%lld) <= dense_begin (%lld) <= "
                    "dense_end (%lld) <= kv_capacity (%lld)",
                    (long long)w->sink_len, (long long)w->retr_begin, (long long)w->dense_begin,
                    (long long)w->dense_end, (long long)kv_capacity);
    if (n >= 0 && w->retr_begin + n > w->dense_begin)
        return fail(PARISKV_ERR_INVALID, "retrieval rows [%lld, %lld) overlap the dense rows from %lld",
                    (long long)w->retr_begin, (long long)(w->retr_begin + n), (long long)w->dense_begin);
    if (win_capacity > 0) {
        if (win_capacity > kMaxKvRows)
            return fail(PARISKV_ERR_INVALID, "win_capacity %lld above 2^30-1", (long long)win_capacity);
        if (w->sink_len > win_capacity ||
            w->dense_end - w->dense_begin > win_capacity - w->sink_len)
            return fail(PARISKV_ERR_INVALID,
                        "window cache of %lld rows holds neither %lld Sink rows and a ring for %lld "
                        "Local / Buffer rows", (long long)win_capacity, (long long)w->sink_len,
                        (long long)(w->dense_end - w->dense_begin));
        if (n >= 0 && w->retr_begin + n > kv_capacity)
            return fail(PARISKV_ERR_INVALID, "retrieval rows end at %lld, past kv_capacity %lld",
                        (long long)(w->retr_begin + n), (long long)kv_capacity);
    }
    const int64_t rows = w->sink_len + (w->dense_end - w->dense_begin) + k;
    if (rows > kMaxAttendRows)
        return fail(PARISKV_ERR_UNSUPPORTED, "%lld attended rows per head, above %d", (long long)rows,
                    kMaxAttendRows);
    out->sink = w->sink_len;
    out->retr_begin = w->retr_begin;
    out->dense_begin = w->dense_begin;
    out->dense_end = w->dense_end;
    out->win_capacity = win_capacity > 0 ? win_capacity : 0;
    return PARISKV_OK;
}

static int check_window_cache(const void* Kw, const void* Vw, int64_t win_capacity) {
    if (win_capacity < 1) return fail(PARISKV_ERR_INVALID, "win_capacity %lld < 1", (long long)win_capacity);
    if (!Kw || !Vw || !aligned16(Kw) || !aligned16(Vw))
        return fail(PARISKV_ERR_INVALID, "K_win and V_win must be non-NULL and 16-byte aligned");
    return PARISKV_OK;
}

static int check_attend_args(const AttendReq& r) {
    if (!r.K || !r.V || !r.out) return fail(PARISKV_ERR_INVALID, "K, V and out must be non-NULL");
    if (!aligned16(r.K) || !aligned16(r.V) || !aligned16(r.out))
        return fail(PARISKV_ERR_INVALID, "K, V and out must be 16-byte aligned");
    if (r.kv_capacity < 1 || r.kv_capacity > kMaxKvRows)
        return fail(PARISKV_ERR_INVALID, "kv_capacity %lld outside 1..2^30-1", (long long)r.kv_capacity);
    if (r.kv_host_mapped != 0 && r.kv_host_mapped != 1)
        return fail(PARISKV_ERR_INVALID, "kv_host_mapped must be 0 or 1");
    if (!std::isfinite(r.scale)) return fail(PARISKV_ERR_INVALID, "scale is not finite");
    return PARISKV_OK;
}

// Device-usable K and V (host-mapped memory goes through its device pointer).
static int device_kv(const AttendReq& r, const void** Kd, const void** Vd) {
    *Kd = r.K;
    *Vd = r.V;
    if (r.kv_host_mapped) {
        void* p = nullptr;
        hipError_t e = hipHostGetDevicePointer(&p, const_cast<void*>(r.K), 0);
        if (e != hipSuccess) return hip_fail(e, "hipHostGetDevicePointer(K)");
        *Kd = p;
        e = hipHostGetDevicePointer(&p, const_cast<void*>(r.V), 0);
        if (e != hipSuccess) return hip_fail(e, "hipHostGetDevicePointer(V)");
        *Vd = p;
    }
    return PARISKV_OK;
}

static int retrieve_impl(const pariskv_config* cfg, const pariskv_index* index, const void* q,
                         int64_t n, int32_t batch, const pariskv_budget* budget, int32_t* out_idx,
                         float* out_score, void* workspace, size_t ws_bytes, void* stream,
                         const AttendReq* att) {
    prof_chain_start();
    pariskv_ws_layout L;
    int rc = layout(cfg, batch, n, budget, &L);
    if (rc) return rc;
    rc = check_index(index);
    if (rc) return rc;
    if (!q || !aligned16(q)) return fail(PARISKV_ERR_INVALID, "q must be non-NULL and 16-byte aligned");
    if (!out_idx || !aligned16(out_idx))
        return fail(PARISKV_ERR_INVALID, "out_idx must be non-NULL and 16-byte aligned");
    if (out_score && !aligned16(out_score))
        return fail(PARISKV_ERR_INVALID, "out_score must be 16-byte aligned");
    if (!workspace || (reinterpret_cast<uintptr_t>(workspace) & 255u) != 0)
        return fail(PARISKV_ERR_WORKSPACE, "workspace must be non-NULL and 256-byte aligned");
    if (ws_bytes < L.total)
        return fail(PARISKV_ERR_WORKSPACE, "workspace has %zu bytes, needs %zu", ws_bytes, L.total);
    const void* Kd = nullptr;
    const void* Vd = nullptr;
    if (att) {
        if ((rc = check_attend_args(*att)) != PARISKV_OK) return rc;
        if (budget->flags & PARISKV_GROUP_FETCH) {
            const int64_t per = (int64_t)(cfg->q_per_kv < 4 ? cfg->q_per_kv : 4) * budget->top_k;
            if (per > kMaxAttendRows)
                return fail(PARISKV_ERR_UNSUPPORTED, "PARISKV_GROUP_FETCH: min(G, 4) * k = %lld above %d",
                            (long long)per, kMaxAttendRows);
            if (n > kGaMaxSplits * kGaRangeKeys)
                return fail(PARISKV_ERR_UNSUPPORTED, "PARISKV_GROUP_FETCH: n = %lld above %lld keys", (long long)n,
                            (long long)(kGaMaxSplits * kGaRangeKeys));
        }
        if ((rc = device_kv(*att, &Kd, &Vd)) != PARISKV_OK) return rc;
    }

    RetrieveArgs a{};
    a.batch = batch;
    a.hkv = cfg->n_kv_heads;
    a.g = cfg->q_per_kv;
    a.quads = L.quads;
    a.hq = a.hkv * a.g;
    a.n = n;
    a.n_pad = L.n_pad;
    a.n_chunks = L.n_chunks;
    a.capacity = cfg->capacity;
    a.n_cand = budget->n_cand;
    a.c_eff = L.c_eff;
    a.top_k = budget->top_k;
    a.flags = ((cfg->flags & PARISKV_NO_ROTATION) ? kFlagNoRotation : 0u) |
              ((budget->flags & PARISKV_BINARY_COLLISIONS) ? kFlagBinary : 0u) |
              ((budget->flags & PARISKV_EXACT_RECOUNT) ? kFlagRecount : 0u);
    for (int l = 0; l < kTierCount; ++l) {
        static const int64_t pct[kTierCount] = {5, 15, 30, 50, 75, 100};
        // ceil(pct * C_rho / 100) in integers; start ranks never exceed 2^31.
        const int64_t c = budget->n_collide > (int64_t(1) << 40)
                              ? (int64_t(1) << 40)
                              : (pct[l] * budget->n_collide + 99) / 100;
        a.cuts[l] = c > 0xffffffffLL ? 0xffffffffu : (uint32_t)c;
    }
    a.q = q;
    a.ids = index->ids;
    a.rec = index->rec;
    a.counts = index->counts;
    char* ws = static_cast<char*>(workspace);
    a.zq = reinterpret_cast<float*>(ws + L.zq);
    a.lut = reinterpret_cast<uint32_t*>(ws + L.lut);
    a.score8 = reinterpret_cast<uint8_t*>(ws + L.score8);
    a.chunk_sfx = reinterpret_cast<uint32_t*>(ws + L.chunk_sfx);
    a.chunk_base = reinterpret_cast<int32_t*>(ws + L.chunk_base);
    a.thresh = reinterpret_cast<int32_t*>(ws + L.thresh);
    a.cand = reinterpret_cast<int32_t*>(ws + L.cand);
    a.cand_score = reinterpret_cast<float*>(ws + L.cand_score);
    a.stats = reinterpret_cast<float*>(ws + L.stats);
    a.topk_parts = L.topk_parts;
    a.surv_idx = reinterpret_cast<int32_t*>(ws + L.surv);
    a.surv_score = reinterpret_cast<float*>(ws + L.surv + (size_t)a.batch * a.hq * L.topk_parts * a.top_k * 4);
    a.out_idx = out_idx;
    a.out_score = out_score;
    a.sb = pack_signs(cfg->rot_signs);
    a.qc = quant_consts();
    if (att) {
        a.K = Kd;
        a.V = Vd;
        a.kv_capacity = att->kv_capacity;
        a.Kw = att->Kw;
        a.Vw = att->Vw;
        a.scale = att->scale;
        a.attn_out = att->out;
        a.win = att->win;
    }

    hipStream_t s = static_cast<hipStream_t>(stream);
    hipError_t e;
    // Attention by its own kernel over out_idx (when the top-k did not fuse it).
    auto attend_separately = [&]() -> int {
        const hipError_t ea = launch_attend(q, Kd, Vd, att->kv_capacity, att->Kw, att->Vw, out_idx,
                                            budget->top_k, batch, a.hkv, a.g, att->scale, att->out,
                                            att->win, s);
        return ea == hipSuccess ? PARISKV_OK : hip_fail(ea, "attend launch");
    };
    const bool group_fetch = att && (budget->flags & PARISKV_GROUP_FETCH);
    // Attention per quad of heads over the union of their winner lists, share s of a
    // quad taking the rows in [s * group_range, (s + 1) * group_range).
    const int64_t group_range = group_fetch ? ((n > 0 ? n : 1) + L.group_splits - 1) / L.group_splits : 0;
    auto attend_groups = [&]() -> int {
        const hipError_t eg = launch_group_attend(q, Kd, Vd, att->kv_capacity, out_idx, budget->top_k, batch,
                                                  a.hkv, a.g, att->scale, att->out,
                                                  reinterpret_cast<int32_t*>(ws + L.group_rows), L.group_splits,
                                                  group_range, reinterpret_cast<float*>(ws + L.group_part),
                                                  att->win, att->Kw, att->Vw, att->kv_host_mapped != 0, s);
        return eg == hipSuccess ? PARISKV_OK : hip_fail(eg, "group_attend launch");
    };
    if (n == 0) {
        e = launch_pad_outputs(a, s);
        if (e != hipSuccess) return hip_fail(e, "pad outputs");
        return !att ? PARISKV_OK : group_fetch ? attend_groups() : attend_separately();
    }
    if ((e = launch_query_lut(a, s)) != hipSuccess) return hip_fail(e, "query_lut launch");
    if ((e = launch_collide(a, s)) != hipSuccess) return hip_fail(e, "collide launch");
    if ((e = launch_threshold(a, s)) != hipSuccess) return hip_fail(e, "threshold launch");
    if ((e = launch_compact_rerank(a, s)) != hipSuccess) return hip_fail(e, "compact_rerank launch");
    if (group_fetch) {
        if ((e = launch_topk(a, s, false)) != hipSuccess) return hip_fail(e, "topk launch");
        return attend_groups();
    }
    bool fused = false;
    if ((e = launch_topk(a, s, att != nullptr, &fused)) != hipSuccess) return hip_fail(e, "topk launch");
    if (att && !fused) return attend_separately();
    return PARISKV_OK;
}

int pariskv_retrieve(const pariskv_config* cfg, const pariskv_index* index, const void* q,
                     int64_t n, int32_t batch, const pariskv_budget* budget, int32_t* out_idx,
                     float* out_score, void* workspace, size_t ws_bytes, void* stream) {
    return retrieve_impl(cfg, index, q, n, batch, budget, out_idx, out_score, workspace, ws_bytes,
                         stream, nullptr);
}

int pariskv_retrieve_attend(const pariskv_config* cfg, const pariskv_index* index, const void* q,
                            int64_t n, int32_t batch, const pariskv_budget* budget, int32_t* out_idx,
                            float* out_score, const void* K, const void* V, int32_t kv_host_mapped,
                            int64_t kv_capacity, float scale, float* out, void* workspace,
                            size_t ws_bytes, void* stream) {
    const AttendReq att{K, V, kv_host_mapped, kv_capacity, scale, out, AttendWindow{}};
    return retrieve_impl(cfg, index, q, n, batch, budget, out_idx, out_score, workspace, ws_bytes,
                         stream, &att);
}

int pariskv_retrieve_attend_noalloc(const pariskv_config* cfg, const pariskv_index* index,
                                    const void* q, int64_t n, int32_t batch,
                                    const pariskv_budget* budget, int32_t* out_idx, float* out_score,
                                    const void* K, const void* V, int32_t kv_host_mapped,
                                    int64_t kv_capacity, float scale, float* out, void* stream) {
    prof_chain_start();
    pariskv_ws_layout L;
    int rc = layout(cfg, batch, n, budget, &L);
    if (rc) return rc;
    if (L.total > PARISKV_NOALLOC_SCRATCH_BYTES)
        return fail(PARISKV_ERR_WORKSPACE,
                    "these shapes need %zu bytes of intermediates, above the %zu-byte static scratch; "
                    "call pariskv_retrieve_attend with a workspace",
                    L.total, (size_t)PARISKV_NOALLOC_SCRATCH_BYTES);
    void* ws = nullptr;
    if ((rc = scratch_ptr(&ws)) != PARISKV_OK) return rc;
    const AttendReq att{K, V, kv_host_mapped, kv_capacity, scale, out, AttendWindow{}};
    return retrieve_impl(cfg, index, q, n, batch, budget, out_idx, out_score, ws,
                         PARISKV_NOALLOC_SCRATCH_BYTES, stream, &att);
}

int pariskv_retrieve_window_attend(const pariskv_config* cfg, const pariskv_index* index,
                                   const void* q, int64_t n, int32_t batch,
                                   const pariskv_budget* budget, int32_t* out_idx, float* out_score,
                                   const void* K, const void* V, int32_t kv_host_mapped,
                                   int64_t kv_capacity, const pariskv_window* win, float scale,
                                   float* out, void* workspace, size_t ws_bytes, void* stream) {
    prof_chain_start();
    if (!win) return fail(PARISKV_ERR_INVALID, "win must be non-NULL");
    if (!budget) return fail(PARISKV_ERR_INVALID, "budget must be non-NULL");
    AttendReq att{K, V, kv_host_mapped, kv_capacity, scale, out, AttendWindow{}};
    int rc = check_window(win, kv_capacity, budget->top_k, n < 0 ? 0 : n, 0, &att.win);
    if (rc) return rc;
    return retrieve_impl(cfg, index, q, n, batch, budget, out_idx, out_score, workspace, ws_bytes,
                         stream, &att);
}

int pariskv_retrieve_tiered_attend(const pariskv_config* cfg, const pariskv_index* index,
                                   const void* q, int64_t n, int32_t batch,
                                   const pariskv_budget* budget, int32_t* out_idx, float* out_score,
                                   const void* K_win, const void* V_win, int64_t win_capacity,
                                   const void* K, const void* V, int32_t kv_host_mapped,
                                   int64_t kv_capacity, const pariskv_window* win, float scale,
                                   float* out, void* workspace, size_t ws_bytes, void* stream) {
    prof_chain_start();
    if (!win) return fail(PARISKV_ERR_INVALID, "win must be non-NULL");
    if (!budget) return fail(PARISKV_ERR_INVALID, "budget must be non-NULL");
    int rc = check_window_cache(K_win, V_win, win_capacity);
    if (rc) return rc;
    AttendReq att{K, V, kv_host_mapped, kv_capacity, scale, out, AttendWindow{}, K_win, V_win};
    if ((rc = check_window(win, kv_capacity, budget->top_k, n < 0 ? 0 : n, win_capacity, &att.win)))
        return rc;
    return retrieve_impl(cfg, index, q, n, batch, budget, out_idx, out_score, workspace, ws_bytes,
                         stream, &att);
}

static int attend_impl(const pariskv_config* cfg, const void* q, const void* K, const void* V,
                       int32_t kv_host_mapped, int64_t kv_capacity, const int32_t* idx, int32_t k,
                       const pariskv_window* win, int32_t batch, float scale, float* out,
                       void* stream, const void* Kw = nullptr, const void* Vw = nullptr,
                       int64_t win_capacity = 0) {
    prof_chain_start();
    int rc = check_config(cfg, batch);
    if (rc) return rc;
    if (!q || !K || !V || !idx || !out)
        return fail(PARISKV_ERR_INVALID, "q, K, V, idx and out must be non-NULL");
    if (!aligned16(q) || !aligned16(K) || !aligned16(V) || !aligned16(out) ||
        (reinterpret_cast<uintptr_t>(idx) & 3u) != 0)
        return fail(PARISKV_ERR_INVALID, "q, K, V, out must be 16-byte aligned, idx 4-byte aligned");
    if (k < 1) return fail(PARISKV_ERR_INVALID, "k %d < 1", k);
    if (k > kMaxAttendRows) return fail(PARISKV_ERR_UNSUPPORTED, "k %d above %d", k, kMaxAttendRows);
    if (kv_capacity < 1 || kv_capacity > kMaxKvRows)
        return fail(PARISKV_ERR_INVALID, "kv_capacity %lld outside 1..2^30-1", (long long)kv_capacity);
    if (kv_host_mapped != 0 && kv_host_mapped != 1)
        return fail(PARISKV_ERR_INVALID, "kv_host_mapped must be 0 or 1");
    if (!std::isfinite(scale)) return fail(PARISKV_ERR_INVALID, "scale is not finite");
    AttendWindow aw;
    if ((rc = check_window(win, kv_capacity, k, -1, win_capacity, &aw)) != PARISKV_OK) return rc;
    const void* Kd = K;
    const void* Vd = V;
    if (kv_host_mapped) {
        void* p = nullptr;
        hipError_t e = hipHostGetDevicePointer(&p, const_cast<void*>(K), 0);
        if (e != hipSuccess) return hip_fail(e, "hipHostGetDevicePointer(K)");
        Kd = p;
        e = hipHostGetDevicePointer(&p, const_cast<void*>(V), 0);
        if (e != hipSuccess) return hip_fail(e, "hipHostGetDevicePointer(V)");
        Vd = p;
    }
    hipError_t e = launch_attend(q, Kd, Vd, kv_capacity, Kw, Vw, idx, k, batch, cfg->n_kv_heads,
                                 cfg->q_per_kv, scale, out, aw, static_cast<hipStream_t>(stream));
    if (e != hipSuccess) return hip_fail(e, "attend launch");
    return PARISKV_OK;
}

int pariskv_sparse_attend(const pariskv_config* cfg, const void* q, const void* K, const void* V,
                          int32_t kv_host_mapped, int64_t kv_capacity, const int32_t* idx, int32_t k,
                          int32_t batch, float scale, float* out, void* stream) {
    return attend_impl(cfg, q, K, V, kv_host_mapped, kv_capacity, idx, k, nullptr, batch, scale, out,
                       stream);
}

int pariskv_window_attend(const pariskv_config* cfg, const void* q, const void* K, const void* V,
                          int32_t kv_host_mapped, int64_t kv_capacity, const int32_t* idx, int32_t k,
                          const pariskv_window* win, int32_t batch, float scale, float* out,
                          void* stream) {
    if (!win) return fail(PARISKV_ERR_INVALID, "win must be non-NULL");
    return attend_impl(cfg, q, K, V, kv_host_mapped, kv_capacity, idx, k, win, batch, scale, out,
                       stream);
}

int pariskv_group_attend(const pariskv_config* cfg, const void* q, const void* K, const void* V,
                         int32_t kv_host_mapped, int64_t kv_capacity, const int32_t* idx, int32_t k,
                         int32_t batch, float scale, float* out, int32_t* union_rows, void* stream) {
    prof_chain_start();
    int rc = check_config(cfg, batch);
    if (rc) return rc;
    if (!q || !K || !V || !idx || !out)
        return fail(PARISKV_ERR_INVALID, "q, K, V, idx and out must be non-NULL");
    if (!aligned16(q) || !aligned16(K) || !aligned16(V) || !aligned16(out) ||
        (reinterpret_cast<uintptr_t>(idx) & 3u) != 0 || (reinterpret_cast<uintptr_t>(union_rows) & 3u) != 0)
        return fail(PARISKV_ERR_INVALID, "q, K, V, out must be 16-byte aligned, idx and union_rows 4-byte");
    if (k < 1) return fail(PARISKV_ERR_INVALID, "k %d < 1", k);
    const int64_t per = (int64_t)(cfg->q_per_kv < 4 ? cfg->q_per_kv : 4) * k;
    if (per > kMaxAttendRows)
        return fail(PARISKV_ERR_UNSUPPORTED, "min(G, 4) * k = %lld above %d", (long long)per, kMaxAttendRows);
    if (kv_capacity < 1 || kv_capacity > kMaxKvRows)
        return fail(PARISKV_ERR_INVALID, "kv_capacity %lld outside 1..2^30-1", (long long)kv_capacity);
    if (kv_host_mapped != 0 && kv_host_mapped != 1)
        return fail(PARISKV_ERR_INVALID, "kv_host_mapped must be 0 or 1");
    if (!std::isfinite(scale)) return fail(PARISKV_ERR_INVALID, "scale is not finite");
    const void* Kd = K;
    const void* Vd = V;
    if (kv_host_mapped) {
        void* p = nullptr;
        hipError_t e = hipHostGetDevicePointer(&p, const_cast<void*>(K), 0);
        if (e != hipSuccess) return hip_fail(e, "hipHostGetDevicePointer(K)");
        Kd = p;
        e = hipHostGetDevicePointer(&p, const_cast<void*>(V), 0);
        if (e != hipSuccess) return hip_fail(e, "hipHostGetDevicePointer(V)");
        Vd = p;
    }
    // One share per quad: the union by key bitmap over the whole cache when it spans at
    // most kGaRangeKeys rows, else by merging the lists.
    hipError_t e = launch_group_attend(q, Kd, Vd, kv_capacity, idx, k, batch, cfg->n_kv_heads,
                                       cfg->q_per_kv, scale, out, union_rows, 1,
                                       kv_capacity <= kGaRangeKeys ? kv_capacity : 0, nullptr, AttendWindow{},
                                       nullptr, nullptr, kv_host_mapped != 0, static_cast<hipStream_t>(stream));
    if (e != hipSuccess) return hip_fail(e, "group_attend launch");
    return PARISKV_OK;
}

int pariskv_tiered_attend(const pariskv_config* cfg, const void* q, const void* K_win,
                          const void* V_win, int64_t win_capacity, const void* K, const void* V,
                          int32_t kv_host_mapped, int64_t kv_capacity, const int32_t* idx, int32_t k,
                          const pariskv_window* win, int32_t batch, float scale, float* out,
                          void* stream) {
    if (!win) return fail(PARISKV_ERR_INVALID, "win must be non-NULL");
    int rc = check_window_cache(K_win, V_win, win_capacity);
    if (rc) return rc;
    return attend_impl(cfg, q, K, V, kv_host_mapped, kv_capacity, idx, k, win, batch, scale, out,
                       stream, K_win, V_win, win_capacity);
}

int pariskv_offload_rows(const void* K_src, const void* V_src, int64_t src_capacity, int64_t src_row,
                         void* K_dst, void* V_dst, int64_t dst_capacity, int64_t dst_row, int64_t t,
                         int32_t batch, int32_t n_kv_heads, void* stream) {
    prof_chain_start();
    if (!K_src || !V_src || !K_dst || !V_dst)
        return fail(PARISKV_ERR_INVALID, "K/V source and destination must be non-NULL");
    if (batch < 1 || n_kv_heads < 1) return fail(PARISKV_ERR_INVALID, "batch and n_kv_heads must be >= 1");
    if (src_capacity < 1 || dst_capacity < 1) return fail(PARISKV_ERR_INVALID, "capacities must be >= 1");
    if (t < 0 || src_row < 0 || dst_row < 0 || src_row > src_capacity - t || dst_row > dst_capacity - t)
        return fail(PARISKV_ERR_INVALID, "rows [%lld, +%lld) -> [%lld, +%lld) outside the caches",
                    (long long)src_row, (long long)t, (long long)dst_row, (long long)t);
    if (t == 0) return PARISKV_OK;
    // One pitched copy per tensor: height = the (sequence, KV head) groups, width = t rows.
    const size_t row_bytes = (size_t)kD * 2;
    const size_t groups = (size_t)batch * (size_t)n_kv_heads;
    hipStream_t s = static_cast<hipStream_t>(stream);
    const void* src[2] = {K_src, V_src};
    void* dst[2] = {K_dst, V_dst};
    for (int i = 0; i < 2; ++i) {
        const hipError_t e = hipMemcpy2DAsync(
            static_cast<char*>(dst[i]) + (size_t)dst_row * row_bytes, (size_t)dst_capacity * row_bytes,
            static_cast<const char*>(src[i]) + (size_t)src_row * row_bytes, (size_t)src_capacity * row_bytes,
            (size_t)t * row_bytes, groups, hipMemcpyDefault, s);
        if (e != hipSuccess) return hip_fail(e, "hipMemcpy2DAsync");
    }
    return PARISKV_OK;
}

int pariskv_stream_copy(void* dst, const void* src, size_t bytes, void* stream) {
    prof_chain_start();
    if (!dst || !src || !aligned16(dst) || !aligned16(src) || bytes % 16 != 0)
        return fail(PARISKV_ERR_INVALID, "stream copy needs 16-byte aligned pointers and a multiple of 16 bytes");
    const hipError_t e = launch_stream_copy(dst, src, bytes, static_cast<hipStream_t>(stream));
    return e == hipSuccess ? PARISKV_OK : hip_fail(e, "stream_copy launch");
}

int pariskv_stream_read(const void* src, size_t bytes, uint32_t key, uint32_t* sink, void* stream) {
    prof_chain_start();
    if (!src || !sink || !aligned16(src) || (reinterpret_cast<uintptr_t>(sink) & 3u) != 0 || bytes % 16 != 0)
        return fail(PARISKV_ERR_INVALID, "stream read needs aligned pointers and a multiple of 16 bytes");
    const hipError_t e = launch_stream_read(src, bytes, key, sink, static_cast<hipStream_t>(stream));
    return e == hipSuccess ? PARISKV_OK : hip_fail(e, "stream_read launch");
}

int pariskv_profile_enable(int32_t on) {
    std::lock_guard<std::mutex> lk(g_prof_mu);
    g_prof_on = on != 0;
    return PARISKV_OK;
}

int pariskv_profile_reset(void) {
    std::lock_guard<std::mutex> lk(g_prof_mu);
    int rc = collect_locked();
    g_acc.clear();
    return rc;
}

int pariskv_profile_read(int32_t max_entries, const char** names, int64_t* launches,
                         double* total_ms) {
    std::lock_guard<std::mutex> lk(g_prof_mu);
    int rc = collect_locked();
    if (rc) return rc;
    int i = 0;
    for (auto& kv : g_acc) {
        if (i < max_entries) {
            if (names) names[i] = kv.first.c_str();
            if (launches) launches[i] = kv.second.launches;
            if (total_ms) total_ms[i] = kv.second.ms;
        }
        ++i;
    }
    return i;
}

}  // extern "C"
