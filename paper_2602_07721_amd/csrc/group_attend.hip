// Attention of the query heads that share a KV head over their retrieved keys,
// with every distinct K/V row fetched once (GQA-group de-duplication of the
// sparse attention of Eqs. approx_weight / approx_output; Sec. "On-Demand UVA
// Fetch": the fetched rows are what crosses the host link).
//
//   o_h = sum_{i in idx_h} softmax_i(scale <k_i, q_h>) v_i   for each head h,
//   float16 in, float32 math -- the same value as the per-head attention.
//
// One block of 512 threads per (sequence, KV head, quad of query heads):
//   1. the quad's lists (each ascending with -1 padding at its end, as the
//      retrieval writes them) are staged in LDS, invalid entries as +inf;
//   2. merge by rank: an entry's place in the merged order is its index plus,
//      for every other list, the number of entries before it there (binary
//      search; ties ordered by head), so the merged rows are ascending and
//      equal rows adjacent.  Every place is below G * k whatever the input
//      order, so unsorted lists give an unspecified result, never a stray
//      access;
//   3. union: a block scan over "first of its row" flags numbers the distinct
//      rows; each head ORs its bit into its row's mask;
//   4. 32 slots of 16 lanes (lane l16 owns dims [8 l16, 8 l16 + 8)) walk the
//      union, 4 rows in flight per lane; each K and V row segment is read once
//      and feeds the online softmax of every head whose bit is set;
//   5. per head, the 32 slot states are merged in LDS.

#include "attend_row.hpp"

namespace pariskv {

namespace {

constexpr int kGaThreads = 512;  // 8 waves: room for 4 heads of state per lane
constexpr int kGaSlots = kGaThreads / 16;
constexpr int kGaUnroll = 4;
constexpr int kGaMaxEntries = 4096;  // G * k per quad staged in LDS
constexpr int32_t kGaInvalid = 0x7fffffff;

struct GroupScratch {
    int32_t list[kGaMaxEntries];   // staged lists, then the union's rows
    int32_t row[kGaMaxEntries];    // merged rows
    uint8_t head[kGaMaxEntries];   // head of each merged entry
    uint32_t mask[kGaMaxEntries];  // head mask of each union row
    uint32_t wsum[kGaThreads / 64];
    uint32_t nunion;
};

// Number of entries of the ascending list a[0, n) below v (lower) or not above v (upper).
__device__ __forceinline__ int rank_in(const int32_t* a, int n, int32_t v, bool upper) {
    int lo = 0, hi = n;
    while (lo < hi) {
        const int mid = (lo + hi) >> 1;
        const bool before = upper ? a[mid] <= v : a[mid] < v;
        if (before) lo = mid + 1;
        else hi = mid;
    }
    return lo;
}

__global__ __launch_bounds__(kGaThreads) void group_attend_kernel(
    const __half* __restrict__ q, const __half* __restrict__ K, const __half* __restrict__ V,
    int64_t kv_capacity, const int32_t* __restrict__ idx, int32_t k, int32_t hkv, int32_t g,
    int32_t quads, float scale, float* __restrict__ out, int32_t* __restrict__ union_rows) {
    __shared__ GroupScratch sg;
    __shared__ AttendScratch sa;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int64_t blk = blockIdx.x;  // (seq * hkv + kvh) * quads + quad
    const int quad = (int)(blk % quads);
    const int64_t grp = blk / quads;  // seq * hkv + kvh
    const int seq = (int)(grp / hkv), kvh = (int)(grp % hkv);
    const int nh = min(4, g - 4 * quad);
    const int64_t row0 = (int64_t)seq * hkv * g + (int64_t)kvh * g + 4 * quad;  // first query head row
    const int ne = nh * k;  // entries of the quad (host checked <= kGaMaxEntries)

    // 1. stage the lists; invalid entries sort last
    for (int r = tid; r < ne; r += kGaThreads) {
        const int32_t v = idx[(row0 + r / k) * k + r % k];
        sg.list[r] = (v >= 0 && v < kv_capacity) ? v : kGaInvalid;
        sg.row[r] = kGaInvalid;  // a place no entry lands on (unsorted input) stays empty
        sg.mask[r] = 0u;
    }
    __syncthreads();
    // 2. merge by rank
    for (int r = tid; r < ne; r += kGaThreads) {
        const int h = r / k, j = r % k;
        const int32_t v = sg.list[r];
        int pos = j;
        for (int o = 0; o < nh; ++o)
            if (o != h) pos += rank_in(sg.list + o * k, k, v, o < h);
        pos = min(pos, ne - 1);
        sg.row[pos] = v;
        sg.head[pos] = (uint8_t)h;
    }
    __syncthreads();
    // 3. union: thread t owns merged entries [8t, 8t + 8)
    constexpr int kPer = kGaMaxEntries / kGaThreads;
    uint32_t first[kPer];
    uint32_t cnt = 0;
#pragma unroll
    for (int e = 0; e < kPer; ++e) {
        const int p = kPer * tid + e;
        const int32_t v = p < ne ? sg.row[p] : kGaInvalid;
        first[e] = (v != kGaInvalid && (p == 0 || sg.row[p - 1] != v)) ? 1u : 0u;
        cnt += first[e];
    }
    const uint32_t incl = wave_incl_sum(cnt);
    if (lane == 63) sg.wsum[wave] = incl;
    __syncthreads();
    uint32_t before = incl - cnt;
    uint32_t total = 0;
#pragma unroll
    for (int w = 0; w < kGaThreads / 64; ++w) {
        if (w < wave) before += sg.wsum[w];
        total += sg.wsum[w];
    }
    // union row u keeps its row in list[u] (the staged lists are no longer read)
    uint32_t u = before;
#pragma unroll
    for (int e = 0; e < kPer; ++e) {
        const int p = kPer * tid + e;
        if (first[e]) sg.list[u] = sg.row[p];
        u += first[e];
        // a duplicate belongs to the union row of the last first at or before it
        if (p < ne && sg.row[p] != kGaInvalid) atomicOr(&sg.mask[u - 1], 1u << sg.head[p]);
    }
    if (tid == 0) {
        sg.nunion = total;
        if (union_rows) union_rows[blk] = (int32_t)total;
    }
    __syncthreads();
    const int U = (int)sg.nunion;

    // 4. attention over the union, every head of the quad at once
    const int slot = tid >> 4, l16 = tid & 15;
    const int64_t kvrow0 = grp * kv_capacity;
    float qf[4][8];
#pragma unroll
    for (int h = 0; h < 4; ++h) {
        const int hh = min(h, nh - 1);
        unpack8_half(reinterpret_cast<const uint4*>(q + (row0 + hh) * kD)[l16], qf[h]);
#pragma unroll
        for (int d = 0; d < 8; ++d) qf[h][d] *= scale;
    }
    float m[4], lsum[4], acc[4][8];
#pragma unroll
    for (int h = 0; h < 4; ++h) {
        m[h] = -__builtin_huge_valf();
        lsum[h] = 0.f;
#pragma unroll
        for (int d = 0; d < 8; ++d) acc[h][d] = 0.f;
    }
    for (int base = 0; base < U; base += kGaSlots * kGaUnroll) {
        uint32_t msk[kGaUnroll];
        uint4 kc[kGaUnroll], vc[kGaUnroll];
#pragma unroll
        for (int w = 0; w < kGaUnroll; ++w) {
            const int r = base + slot + kGaSlots * w;
            msk[w] = 0u;
            kc[w] = make_uint4(0, 0, 0, 0);
            vc[w] = make_uint4(0, 0, 0, 0);
            if (r < U) {
                msk[w] = sg.mask[r];
                const int64_t off = (kvrow0 + sg.list[r]) * kD;
                kc[w] = reinterpret_cast<const uint4*>(K + off)[l16];
                vc[w] = reinterpret_cast<const uint4*>(V + off)[l16];
            }
        }
#pragma unroll
        for (int w = 0; w < kGaUnroll; ++w) {
            float kf[8], vf[8];
            unpack8_half(kc[w], kf);
            unpack8_half(vc[w], vf);
#pragma unroll
            for (int h = 0; h < 4; ++h) {
                float dot = 0.f;
#pragma unroll
                for (int d = 0; d < 8; ++d) dot += qf[h][d] * kf[d];
#pragma unroll
                for (int st = 1; st < 16; st <<= 1) dot += __shfl_xor(dot, st, 64);
                if ((msk[w] >> h) & 1u) {
                    const float mn = fmaxf(m[h], dot);
                    const float corr = __expf(m[h] - mn);
                    const float p = __expf(dot - mn);
                    lsum[h] = lsum[h] * corr + p;
#pragma unroll
                    for (int d = 0; d < 8; ++d) acc[h][d] = acc[h][d] * corr + p * vf[d];
                    m[h] = mn;
                }
            }
        }
    }
    // 5. merge the 32 slot states of each head
    for (int h = 0; h < nh; ++h) {
        if (l16 == 0) {
            sa.m[slot] = m[h];
            sa.l[slot] = lsum[h];
        }
#pragma unroll
        for (int d = 0; d < 8; ++d) sa.acc[slot][8 * l16 + d] = acc[h][d];
        __syncthreads();
        if (tid < kD) {
            float M = -__builtin_huge_valf();
#pragma unroll
            for (int j = 0; j < kGaSlots; ++j) M = fmaxf(M, sa.m[j]);
            float L = 0.f, O = 0.f;
            if (M > -__builtin_huge_valf()) {
#pragma unroll
                for (int j = 0; j < kGaSlots; ++j) {
                    if (sa.l[j] > 0.f) {
                        const float c = __expf(sa.m[j] - M);
                        L += sa.l[j] * c;
                        O += sa.acc[j][tid] * c;
                    }
                }
            }
            out[(row0 + h) * kD + tid] = L > 0.f ? O / L : 0.f;
        }
        __syncthreads();
    }
}

}  // namespace

hipError_t launch_group_attend(const void* q, const void* K, const void* V, int64_t kv_capacity,
                               const int32_t* idx, int32_t k, int32_t batch, int32_t hkv, int32_t g,
                               float scale, float* out, int32_t* union_rows, hipStream_t s) {
    const int32_t quads = (g + 3) / 4;
    const ProfEvents pe = prof_begin("group_attend");
    hipExtLaunchKernelGGL(group_attend_kernel, dim3((unsigned)((int64_t)batch * hkv * quads)),
                          dim3(kGaThreads), 0, s, pe.start, pe.stop, 0, static_cast<const __half*>(q),
                          static_cast<const __half*>(K), static_cast<const __half*>(V), kv_capacity, idx, k,
                          hkv, g, quads, scale, out, union_rows);
    return hipGetLastError();
}

}  // namespace pariskv
