// Library-internal declarations shared by the host API and the kernel files.
#pragma once

#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>

#include <cstddef>
#include <cstdint>

#include "pariskv.h"

namespace pariskv {

constexpr int kD = 128;           // head dimension
constexpr int kB = 16;            // subspaces
constexpr int kM = 8;             // coordinates per subspace
constexpr int kCentroids = 256;   // 2^m
constexpr int kRec = 128;         // bytes per rerank record
constexpr int kMaxScore = 96;     // 6 * B
constexpr int kBins = kMaxScore + 1;
constexpr int kSfx = kBins + 1;   // suffix histogram entries v = 0..97 (entry 97 is 0)
constexpr int kChunk = 4096;      // keys per collision / selection chunk
constexpr int kThreshRow = 8;     // int32 per query head in the thresh array
constexpr int kTopkPart = 4096;   // candidates per block in the first of two top-k passes

// Slices per row of the two-pass top-k: a first pass takes the top k of every
// 4096-candidate slice in its own block, and the final pass selects among the slices'
// winners (at most 16 slices x 2048 = 32768, which one block holds in LDS).  Used for
// more than 32768 candidates per row, and for more than 8192 when fewer than 256 rows
// (query heads x sequences) would leave most CUs idle; otherwise 1 (one pass, one
// block per row).
__host__ __device__ inline int32_t topk_parts(int64_t rows, int64_t c_eff, int32_t k) {
    (void)k;
    if (c_eff <= 8192 || (rows >= 256 && c_eff <= 32768)) return 1;
    return (int32_t)((c_eff + kTopkPart - 1) / kTopkPart);
}
constexpr int kTierCount = 6;

// Stored form of a centroid id (the ids array holds slot(c)): bits 5..7 kept,
// bits 0..4 XORed with a linear function of bits 5..7 whose kernel code has
// minimum distance 4, so ids within Hamming distance 3 differ modulo 32 (the
// LDS bank of the collision scan's lookup).  An involution.
__host__ __device__ __forceinline__ uint32_t id_slot(uint32_t c) {
    return c ^ ((c >> 5) & 1u) * 0x07u ^ ((c >> 6) & 1u) * 0x19u ^ ((c >> 7) & 1u) * 0x0Eu;
}

// mask[lane] ? if1 : if0, with the mask in an SGPR pair.
__device__ __forceinline__ uint32_t select_mask(uint64_t mask, uint32_t if1, uint32_t if0) {
    uint32_t r;
    asm("v_cndmask_b32 %0, %1, %2, %3" : "=v"(r) : "v"(if0), "v"(if1), "s"(mask));
    return r;
}

// The value of lane ^ lm (lm a power of two below 64, known after unrolling).
__device__ __forceinline__ uint32_t lane_xor(uint32_t v, int lm, int lane) {
    switch (lm) {
        case 1: return (uint32_t)__builtin_amdgcn_mov_dpp((int)v, 0xB1, 0xF, 0xF, false);
        case 2: return (uint32_t)__builtin_amdgcn_mov_dpp((int)v, 0x4E, 0xF, 0xF, false);
        case 4: return (uint32_t)__builtin_amdgcn_ds_swizzle((int)v, 0x1F | (4 << 10));
        case 8: return (uint32_t)__builtin_amdgcn_ds_swizzle((int)v, 0x1F | (8 << 10));
        case 16: return (uint32_t)__builtin_amdgcn_ds_swizzle((int)v, 0x1F | (16 << 10));
        default: return (uint32_t)__builtin_amdgcn_ds_bpermute((lane ^ 32) << 2, (int)v);
    }
}

// Inclusive sum over the 64 lanes of a wave through DPP moves, without LDS: shifts
// of 1, 2, 4 and 8 lanes inside each row of 16 lanes, then the total of row 0 into
// row 1 and of row 2 into row 3 (row_bcast:15), then lane 31's running total into
// rows 2 and 3 (row_bcast:31).  Lanes a move cannot reach add 0.  Every lane of the
// wave must be active.
__device__ __forceinline__ uint32_t wave_incl_sum(uint32_t v) {
    v += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x111, 0xF, 0xF, false);  // row_shr:1
    v += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x112, 0xF, 0xF, false);  // row_shr:2
    v += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x114, 0xF, 0xF, false);  // row_shr:4
    v += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x118, 0xF, 0xF, false);  // row_shr:8
    v += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x142, 0xA, 0xF, false);  // row_bcast:15
    v += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x143, 0xC, 0xF, false);  // row_bcast:31
    return v;
}

// Sum of x over the 64 lanes of the wave, the same value in every lane, through
// DPP adds inside each row of 16 lanes (quad partners, then the mirrored lane in
// the half row and in the row) and the four row sums read out by readlane, added
// in row order.  Every lane of the wave must be active.
__device__ __forceinline__ float wave_sum_f32(float x) {
    x += __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(x), 0xB1, 0xF, 0xF, false));   // quad_perm 1,0,3,2
    x += __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(x), 0x4E, 0xF, 0xF, false));   // quad_perm 2,3,0,1
    x += __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(x), 0x141, 0xF, 0xF, false));  // row_half_mirror
    x += __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(x), 0x140, 0xF, 0xF, false));  // row_mirror
    const float r0 = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(x), 0));
    const float r1 = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(x), 16));
    const float r2 = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(x), 32));
    const float r3 = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(x), 48));
    return ((r0 + r1) + r2) + r3;
}

// Minimum and maximum of x over the 64 lanes of the wave (same DPP pattern).
__device__ __forceinline__ uint32_t wave_min_u32(uint32_t x) {
    x = min(x, (uint32_t)__builtin_amdgcn_mov_dpp((int)x, 0xB1, 0xF, 0xF, false));
    x = min(x, (uint32_t)__builtin_amdgcn_mov_dpp((int)x, 0x4E, 0xF, 0xF, false));
    x = min(x, (uint32_t)__builtin_amdgcn_mov_dpp((int)x, 0x141, 0xF, 0xF, false));
    x = min(x, (uint32_t)__builtin_amdgcn_mov_dpp((int)x, 0x140, 0xF, 0xF, false));
    const uint32_t a = min((uint32_t)__builtin_amdgcn_readlane((int)x, 0), (uint32_t)__builtin_amdgcn_readlane((int)x, 16));
    const uint32_t b = min((uint32_t)__builtin_amdgcn_readlane((int)x, 32), (uint32_t)__builtin_amdgcn_readlane((int)x, 48));
    return min(a, b);
}
__device__ __forceinline__ uint32_t wave_max_u32(uint32_t x) {
    x = max(x, (uint32_t)__builtin_amdgcn_mov_dpp((int)x, 0xB1, 0xF, 0xF, false));
    x = max(x, (uint32_t)__builtin_amdgcn_mov_dpp((int)x, 0x4E, 0xF, 0xF, false));
    x = max(x, (uint32_t)__builtin_amdgcn_mov_dpp((int)x, 0x141, 0xF, 0xF, false));
    x = max(x, (uint32_t)__builtin_amdgcn_mov_dpp((int)x, 0x140, 0xF, 0xF, false));
    const uint32_t a = max((uint32_t)__builtin_amdgcn_readlane((int)x, 0), (uint32_t)__builtin_amdgcn_readlane((int)x, 16));
    const uint32_t b = max((uint32_t)__builtin_amdgcn_readlane((int)x, 32), (uint32_t)__builtin_amdgcn_readlane((int)x, 48));
    return max(a, b);
}

// Byte k of x shifted left (right) by 2 in one SDWA instruction: the byte
// offset of table entry byte_k(x) (byte_k(x) >> 4) for 4-byte entries.
template <int K>
__device__ __forceinline__ uint32_t byte_shl2(uint32_t x, uint32_t two) {
    uint32_t r;
    if constexpr (K == 0)
        asm("v_lshlrev_b32_sdwa %0, %1, %2 dst_sel:DWORD dst_unused:UNUSED_PAD src0_sel:DWORD src1_sel:BYTE_0" : "=v"(r) : "v"(two), "v"(x));
    else if constexpr (K == 1)
        asm("v_lshlrev_b32_sdwa %0, %1, %2 dst_sel:DWORD dst_unused:UNUSED_PAD src0_sel:DWORD src1_sel:BYTE_1" : "=v"(r) : "v"(two), "v"(x));
    else if constexpr (K == 2)
        asm("v_lshlrev_b32_sdwa %0, %1, %2 dst_sel:DWORD dst_unused:UNUSED_PAD src0_sel:DWORD src1_sel:BYTE_2" : "=v"(r) : "v"(two), "v"(x));
    else
        asm("v_lshlrev_b32_sdwa %0, %1, %2 dst_sel:DWORD dst_unused:UNUSED_PAD src0_sel:DWORD src1_sel:BYTE_3" : "=v"(r) : "v"(two), "v"(x));
    return r;
}
template <int K>
__device__ __forceinline__ uint32_t byte_shr2(uint32_t x, uint32_t two) {
    uint32_t r;
    if constexpr (K == 0)
        asm("v_lshrrev_b32_sdwa %0, %1, %2 dst_sel:DWORD dst_unused:UNUSED_PAD src0_sel:DWORD src1_sel:BYTE_0" : "=v"(r) : "v"(two), "v"(x));
    else if constexpr (K == 1)
        asm("v_lshrrev_b32_sdwa %0, %1, %2 dst_sel:DWORD dst_unused:UNUSED_PAD src0_sel:DWORD src1_sel:BYTE_1" : "=v"(r) : "v"(two), "v"(x));
    else if constexpr (K == 2)
        asm("v_lshrrev_b32_sdwa %0, %1, %2 dst_sel:DWORD dst_unused:UNUSED_PAD src0_sel:DWORD src1_sel:BYTE_2" : "=v"(r) : "v"(two), "v"(x));
    else
        asm("v_lshrrev_b32_sdwa %0, %1, %2 dst_sel:DWORD dst_unused:UNUSED_PAD src0_sel:DWORD src1_sel:BYTE_3" : "=v"(r) : "v"(two), "v"(x));
    return r;
}

// 128 rotation signs packed as bits: bit j of word j/32 set <=> s_j = -1.
struct SignBits {
    uint32_t w[4];
};

// Offline quantizer constants as the kernels consume them.
struct QuantConsts {
    double a[8];    // reconstruction levels a[0..7]
    double tau2[7]; // fl(tau_t * tau_t), t = 1..7
    float a32[8];   // a rounded to float, for the float32 rerank
};

bool quantizer_table_m8(double* tau, double* a);

// ---- launchers (each lives next to its kernel) --------------------------

hipError_t launch_zero_u32(uint32_t* p, int64_t count, hipStream_t s);

// Encode the first n_src rows of keys [groups][src_stride][D] into rows
// [row0, row0 + n_src) of each group (src_stride = n_src for a packed batch of
// keys, the cache capacity when the rows are read straight from a K cache).
// flags: the index variant (kFlagNoRotation, kFlagNoAlpha).
hipError_t launch_encode(const void* keys, int64_t n_src, int64_t src_stride, int64_t groups,
                         int64_t row0, int64_t capacity, uint8_t* ids, uint8_t* rec,
                         uint32_t* counts, const SignBits& sb, const QuantConsts& qc, uint32_t flags,
                         hipStream_t s);

// Variant bits carried to the kernels (the config's and the budget's flags).
constexpr uint32_t kFlagNoRotation = 1u;     // R = I (encode and query transform)
constexpr uint32_t kFlagNoAlpha = 2u;        // W_b = sqrt(S_b) (encode)
constexpr uint32_t kFlagBinary = 1u << 8;    // admitted clusters score 1 (bonus tables)
constexpr uint32_t kFlagRecount = 1u << 9;   // no score histogrammed: threshold by recount

// List-entry flag of the attention body: the entry names a row of the window
// cache (Sink + Local / Update Buffer kept on the GPU), not of the main cache.
constexpr int32_t kWinRow = 1 << 30;
// Largest cache row an attention list can name (rows stay below the flag bit).
constexpr int64_t kMaxKvRows = (int64_t)kWinRow - 1;

// Rows one query head attends (Sec. "Buffer Update": Sink and Local + Update
// Buffer densely, the retrieved keys sparsely).  The head's list is
//   [0, sink) ++ [dense_begin, dense_end) ++ (retr_begin + idx_j for idx_j >= 0),
// in that order (idx_j < 0 stays an empty slot).  All zero = the retrieved keys
// only, at their own row numbers.  With win_capacity > 0 the dense rows are read
// from the window cache instead of the main cache: Sink row r at slot r, Local /
// Buffer row r at slot sink + (r - sink) mod (win_capacity - sink).
struct AttendWindow {
    int64_t sink = 0;
    int64_t retr_begin = 0;
    int64_t dense_begin = 0;
    int64_t dense_end = 0;
    int64_t win_capacity = 0;
    __host__ __device__ int64_t dense_rows() const { return sink + (dense_end - dense_begin); }
    // List entry of dense position r (0 <= r < dense_rows()).
    __host__ __device__ int32_t dense_entry(int64_t r) const {
        const int64_t row = r < sink ? r : dense_begin + (r - sink);
        if (win_capacity <= 0) return (int32_t)row;
        const int64_t slot = row < sink ? row : sink + (row - sink) % (win_capacity - sink);
        return kWinRow | (int32_t)slot;
    }
};

struct RetrieveArgs {
    // shapes
    int32_t batch, hkv, g, quads, hq;
    int64_t n, n_pad, n_chunks, capacity;
    int64_t n_cand, c_eff;   // row stride of cand / cand_score, and min(C, n)
    int32_t top_k;
    uint32_t flags;  // kFlagNoRotation, kFlagBinary, kFlagRecount
    uint32_t cuts[kTierCount];
    // inputs
    const void* q;
    const uint8_t* ids;
    const uint8_t* rec;
    const uint32_t* counts;
    // workspace
    float* zq;
    uint32_t* lut;
    uint8_t* score8;
    uint32_t* chunk_sfx;
    int32_t* chunk_base;
    int32_t* thresh;
    int32_t* cand;
    float* cand_score;
    float* stats;      // [rows][B][2] bonus moments (the histogram floor)
    int32_t* surv_idx;  // [rows][topk_parts * top_k] survivors of the partial top-k pass
    float* surv_score;
    int32_t topk_parts; // 1, or the slices of a row the first of two top-k passes splits it into
    // The list a top-k launch selects from (set by launch_topk): block b takes part
    // b % tk_parts of row b / tk_parts, entries [p * tk_part_len, min((p + 1) *
    // tk_part_len, tk_c)) of that row of tk_score / tk_idx (row stride tk_stride), and
    // writes top_k entries at tk_out_idx / tk_out_score + b * top_k.
    const float* tk_score;
    const int32_t* tk_idx;
    int64_t tk_stride, tk_c;
    int32_t tk_parts, tk_part_len;
    int32_t* tk_out_idx;
    float* tk_out_score;
    // outputs
    int32_t* out_idx;
    float* out_score;
    SignBits sb;
    QuantConsts qc;
    // attention over the winners, when fused with the top-k (device-usable K/V)
    const void* K;
    const void* V;
    int64_t kv_capacity;
    const void* Kw;    // window cache (win.win_capacity > 0)
    const void* Vw;
    float scale;
    float* attn_out;
    AttendWindow win;  // dense rows attended next to the winners
};

hipError_t launch_query_lut(const RetrieveArgs& a, hipStream_t s);
hipError_t launch_collide(const RetrieveArgs& a, hipStream_t s);
hipError_t launch_threshold(const RetrieveArgs& a, hipStream_t s);
hipError_t launch_compact_rerank(const RetrieveArgs& a, hipStream_t s);
// With `attend`, the top-k kernel also runs the attention over its winners
// (a.K, a.V, a.kv_capacity, a.scale -> a.attn_out) when C fits the LDS variant;
// returns false in `fused` when it did not (the caller then launches attention).
hipError_t launch_topk(const RetrieveArgs& a, hipStream_t s, bool attend = false, bool* fused = nullptr);
hipError_t launch_pad_outputs(const RetrieveArgs& a, hipStream_t s);

// Kw, Vw: the window cache [batch][Hkv][win.win_capacity][D] when
// win.win_capacity > 0 (ignored otherwise).
hipError_t launch_attend(const void* q, const void* K, const void* V, int64_t kv_capacity,
                         const void* Kw, const void* Vw, const int32_t* idx, int32_t k, int32_t batch,
                         int32_t hkv, int32_t g, float scale, float* out, const AttendWindow& win,
                         hipStream_t s);

// Largest list (dense rows + retrieved rows) one attention block stages in LDS.
constexpr int kMaxAttendRows = 4096;

// Attention of each quad of query heads sharing a KV head over the union of
// their (ascending) lists, every distinct row fetched once; min(G, 4) * k must
// not exceed kMaxAttendRows.  union_rows (nullable): [batch][Hkv][quads] sizes.
// With 1 <= range <= kGaRangeKeys, share s of `splits` per quad takes the rows
// in [s * range, (s + 1) * range) (rows past splits * range are dropped); with
// splits > 1 a second kernel merges the shares' states (group_part_bytes of
// `part`).  range = 0: one share per quad, the union by merging the lists.
constexpr int kGaMaxSplits = 64;
constexpr int64_t kGaRangeKeys = 65536;
// win: the dense rows every head also attends and the retrieval rows' offset
// (list entry v is cache row win.retr_begin + v), with the window cache Kw, Vw
// when win.win_capacity > 0, as for launch_attend.  host_kv: K and V are
// host-mapped (the fetch then keeps fewer rows in flight).
hipError_t launch_group_attend(const void* q, const void* K, const void* V, int64_t kv_capacity,
                               const int32_t* idx, int32_t k, int32_t batch, int32_t hkv, int32_t g,
                               float scale, float* out, int32_t* union_rows, int32_t splits, int64_t range,
                               float* part, const AttendWindow& win, const void* Kw, const void* Vw,
                               bool host_kv, hipStream_t s);
// Shares per quad for `groups` (sequence, KV head, quad) triples with at most
// `per` = min(G, 4) * k entries each over n keys: enough for ~256 blocks, no
// more than per / 256, at least ceil(n / kGaRangeKeys), at most kGaMaxSplits.
int32_t group_splits(int64_t groups, int64_t per, int64_t n);
size_t group_part_bytes(int64_t groups, int32_t splits);

// Reference streaming kernels (measurement only): a copy and a read of `bytes`.
hipError_t launch_stream_copy(void* dst, const void* src, size_t bytes, hipStream_t s);
hipError_t launch_stream_read(const void* src, size_t bytes, uint32_t key, uint32_t* sink, hipStream_t s);

// Kernel-level profiling hooks (no-ops unless enabled).
// Event pair for one kernel launch when profiling is on (nulls otherwise), to be
// passed to hipExtLaunchKernelGGL so the timestamps are the dispatch's own.
struct ProfEvents {
    hipEvent_t start = nullptr;
    hipEvent_t stop = nullptr;
};
ProfEvents prof_begin(const char* name);
// Starts a new chain of back-to-back launches (called at every API entry).
void prof_chain_start();

}  // namespace pariskv
