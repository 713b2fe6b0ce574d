// Attention of the query heads that share a KV head over their retrieved keys,
// with every distinct K/V row fetched once (GQA-group de-duplication of the
// sparse attention of Eqs. approx_weight / approx_output; Sec. "On-Demand UVA
// Fetch": the fetched rows are what crosses the host link).
//
//   o_h = sum_{i in idx_h} softmax_i(scale <k_i, q_h>) v_i   for each head h,
//   float16 in, float32 math -- the per-head attention's value up to the
//   order of the float32 sums.
//
// One block of 512 threads per (sequence, KV head, quad of query heads) and
// share of it:
//   1-3. the union of the quad's lists with each row's head mask, in one of two
//      ways.  Key ranges (the retrieval path, and stand-alone calls over at most
//      65536 cache rows): share s of `splits` takes the rows in
//      [s * range, (s + 1) * range), range <= 65536; each head sets its rows'
//      bits in a bitmap of the range, and a block scan over the OR of the four
//      bitmaps numbers the distinct rows in ascending order.  Merge (larger
//      stand-alone calls, one share): the lists (each ascending with -1 padding
//      at its end, as the retrieval writes them) are staged in LDS, merged by
//      rank (an entry's place is its index plus, for every other list, the
//      number of entries before it there; ties ordered by head), and a block
//      scan over "first of its row" flags numbers the distinct rows.  Unsorted
//      lists give an unspecified result there, never a stray access;
//   4. 32 slots of 16 lanes (lane l16 owns dims [8 l16, 8 l16 + 8)) walk the
//      share's union rows, then its share of the window's dense rows (Sink,
//      Local / Update Buffer: every head's list holds them, so they feed every
//      head; dense position j goes to share j mod splits, read from the window
//      cache or the main cache as the window says), 1 row in flight per lane
//      over the host link, 4 from HBM; each K and V row segment is read once
//      and feeds the online softmax of every head whose bit is set (one rescale
//      per head per batch of rows in flight);
//   5. the 32 slot states of every head are merged: the 4 of a wave by lane
//      exchanges, then the 8 wave states in LDS.
// With one share the block writes `out`; with several, each leaves its per-head
// state (running max, sum, unnormalised output) and its row count in `part`,
// and group_combine_kernel merges the shares of each head as step 5 merges
// slots.

#include "attend_row.hpp"

namespace pariskv {

namespace {

constexpr int kGaThreads = 512;  // 8 waves: room for 4 heads of state per lane
constexpr int kGaSlots = kGaThreads / 16;
constexpr int kGaWaves = kGaThreads / 64;  // slot states per head left after the in-wave merge
constexpr int kGaMaxEntries = 4096;  // G * k per quad staged in LDS
constexpr int32_t kGaInvalid = 0x7fffffff;
constexpr int kGaPart = 4 + kD;  // one head's share state: max, sum, row count (head 0), pad, output
constexpr int kGaRangeWords = kGaRangeKeys / 32;
static_assert(kGaThreads == 4 * kD, "the slot merge gives one thread to every (head, dim)");
static_assert(kGaRangeWords % kGaThreads == 0, "range words per thread");

struct GroupScratch {
    int32_t list[kGaMaxEntries];   // merge: staged lists; then the union's rows
    uint32_t mask[kGaMaxEntries];  // head mask of each union row
    union {
        struct {
            int32_t row[kGaMaxEntries];  // merged rows
            uint8_t head[kGaMaxEntries]; // head of each merged entry
        } m;
        uint32_t bits[4][kGaRangeWords];  // key ranges: each head's rows in the range
    } u;
    uint32_t wsum[kGaThreads / 64];
};

// LDS for the final merge of the wave states, every head of the quad at once.
struct GroupMerge {
    float m[4][kGaWaves];
    float l[4][kGaWaves];
    float acc[4][kGaWaves][kD];
};

// Block scan of per-thread counts: (exclusive prefix of this thread, block total).
__device__ __forceinline__ void block_count_scan(uint32_t cnt, uint32_t* wsum, uint32_t* before, uint32_t* total) {
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const uint32_t incl = wave_incl_sum(cnt);
    if (lane == 63) wsum[wave] = incl;
    __syncthreads();
    uint32_t b = incl - cnt, t = 0;
#pragma unroll
    for (int w = 0; w < kGaThreads / 64; ++w) {
        if (w < wave) b += wsum[w];
        t += wsum[w];
    }
    *before = b;
    *total = t;
}

// kUnroll: K/V rows in flight per lane.  Over the host link fewer requests in flight
// fetch faster (one row per lane, 4096 rows for 128 blocks; 8 per lane measured
// 10% slower); from HBM 4 per lane gathers fastest.
template <bool kRanges, int kUnroll>
__global__ __launch_bounds__(kGaThreads) void group_attend_kernel(
    const __half* __restrict__ q, const __half* __restrict__ K, const __half* __restrict__ V,
    int64_t kv_capacity, const int32_t* __restrict__ idx, int32_t k, int32_t hkv, int32_t g,
    int32_t quads, float scale, float* __restrict__ out, int32_t* __restrict__ union_rows, int32_t splits,
    int64_t range, float* __restrict__ part, AttendWindow win, const __half* __restrict__ Kw,
    const __half* __restrict__ Vw) {
    __shared__ GroupScratch sg;
    __shared__ GroupMerge gm;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int64_t blk = blockIdx.x / splits;  // (seq * hkv + kvh) * quads + quad
    const int split = (int)(blockIdx.x % splits);
    const int quad = (int)(blk % quads);
    const int64_t grp = blk / quads;  // seq * hkv + kvh
    const int seq = (int)(grp / hkv), kvh = (int)(grp % hkv);
    const int nh = min(4, g - 4 * quad);
    const int64_t row0 = (int64_t)seq * hkv * g + (int64_t)kvh * g + 4 * quad;  // first query head row
    const int ne = nh * k;  // entries of the quad (host checked <= kGaMaxEntries)
    // list entry v names cache row retr_begin + v; entries past the cache are skipped
    const int64_t v_end = kv_capacity - win.retr_begin;

    constexpr int kPer = kGaMaxEntries / kGaThreads;
    int U;  // union rows of this share, in sg.list / sg.mask [0, U)
    if constexpr (kRanges) {
        // 1. each head's rows in [r0, r0 + range) as bits
        const int64_t r0 = (int64_t)split * range;
        for (int i = tid; i < 4 * kGaRangeWords; i += kGaThreads) (&sg.u.bits[0][0])[i] = 0u;
        __syncthreads();
        for (int r = tid; r < ne; r += kGaThreads) {
            const int h = r / k;
            const int32_t v = idx[(row0 + h) * k + r % k];
            const int64_t d = (int64_t)v - r0;
            if (v >= 0 && v < v_end && d >= 0 && d < range)
                atomicOr(&sg.u.bits[h][d >> 5], 1u << (d & 31));
        }
        __syncthreads();
        // 2-3. thread t owns words [4t, 4t + 4) of the range; rows in ascending order
        constexpr int kWords = kGaRangeWords / kGaThreads;
        uint32_t uw[kWords];
        uint32_t cnt = 0;
#pragma unroll
        for (int e = 0; e < kWords; ++e) {
            const int w = kWords * tid + e;
            uw[e] = sg.u.bits[0][w] | sg.u.bits[1][w] | sg.u.bits[2][w] | sg.u.bits[3][w];
            cnt += (uint32_t)__popc(uw[e]);
        }
        uint32_t before, total;
        block_count_scan(cnt, sg.wsum, &before, &total);
        uint32_t u = before;
#pragma unroll
        for (int e = 0; e < kWords; ++e) {
            const int w = kWords * tid + e;
            for (uint32_t x = uw[e]; x; x &= x - 1u) {
                const int bit = __builtin_ctz(x);
                sg.list[u] = (int32_t)(r0 + 32 * w + bit);
                sg.mask[u] = ((sg.u.bits[0][w] >> bit) & 1u) | (((sg.u.bits[1][w] >> bit) & 1u) << 1) |
                             (((sg.u.bits[2][w] >> bit) & 1u) << 2) | (((sg.u.bits[3][w] >> bit) & 1u) << 3);
                ++u;
            }
        }
        U = (int)total;
    } else {
        // 1. stage the lists; invalid entries sort last
        for (int r = tid; r < ne; r += kGaThreads) {
            const int32_t v = idx[(row0 + r / k) * k + r % k];
            sg.list[r] = (v >= 0 && v < v_end) ? v : kGaInvalid;
            sg.u.m.row[r] = kGaInvalid;  // a place no entry lands on (unsorted input) stays empty
            sg.mask[r] = 0u;
        }
        __syncthreads();
        // 2. merge by rank.  Thread t places entries t + 512 e (e < kPer); the rank of an
        // entry in list o is found by binary lifting (the largest prefix of list o whose
        // entries come before it), the kPer searches of a thread interleaved step by step.
        {
            int32_t v[kPer];
            int hd[kPer], pos[kPer];
#pragma unroll
            for (int e = 0; e < kPer; ++e) {
                const int r = tid + kGaThreads * e;
                hd[e] = r < ne ? r / k : -1;
                v[e] = r < ne ? sg.list[r] : kGaInvalid;
                pos[e] = r < ne ? r % k : 0;
            }
            int top = 1;
            while (2 * top <= k) top *= 2;
            for (int o = 0; o < nh; ++o) {
                const int32_t* a = sg.list + o * k;
                int lo[kPer];
                bool upper[kPer];  // ties: entries of lower heads first
#pragma unroll
                for (int e = 0; e < kPer; ++e) {
                    lo[e] = 0;
                    upper[e] = o < hd[e];
                }
                // branch-free steps: all kPer reads issued before any compare
                for (int step = top; step > 0; step >>= 1) {
                    int32_t x[kPer];
#pragma unroll
                    for (int e = 0; e < kPer; ++e) x[e] = a[min(lo[e] + step, k) - 1];
#pragma unroll
                    for (int e = 0; e < kPer; ++e) {
                        const bool take = (lo[e] + step <= k) & ((x[e] < v[e]) | (upper[e] & (x[e] == v[e])));
                        lo[e] = take ? lo[e] + step : lo[e];
                    }
                }
#pragma unroll
                for (int e = 0; e < kPer; ++e) pos[e] += o != hd[e] ? lo[e] : 0;
            }
#pragma unroll
            for (int e = 0; e < kPer; ++e) {
                if (hd[e] >= 0) {
                    const int p = min(pos[e], ne - 1);
                    sg.u.m.row[p] = v[e];
                    sg.u.m.head[p] = (uint8_t)hd[e];
                }
            }
        }
        __syncthreads();
        // 3. union: thread t owns merged entries [8t, 8t + 8)
        uint32_t first[kPer];
        uint32_t cnt = 0;
#pragma unroll
        for (int e = 0; e < kPer; ++e) {
            const int p = kPer * tid + e;
            const int32_t v = p < ne ? sg.u.m.row[p] : kGaInvalid;
            first[e] = (v != kGaInvalid && (p == 0 || sg.u.m.row[p - 1] != v)) ? 1u : 0u;
            cnt += first[e];
        }
        uint32_t before, total;
        block_count_scan(cnt, sg.wsum, &before, &total);
        // union row u keeps its row in list[u] (the staged lists are no longer read)
        uint32_t u = before;
#pragma unroll
        for (int e = 0; e < kPer; ++e) {
            const int p = kPer * tid + e;
            if (first[e]) sg.list[u] = sg.u.m.row[p];
            u += first[e];
            // a duplicate belongs to the union row of the last first at or before it
            if (p < ne && sg.u.m.row[p] != kGaInvalid) atomicOr(&sg.mask[u - 1], 1u << sg.u.m.head[p]);
        }
        U = (int)total;
    }
    if (tid == 0) {
        if (splits == 1) {
            if (union_rows) union_rows[blk] = U;
        } else {
            part[((blk * splits + split) * 4) * kGaPart + 2] = __int_as_float(U);  // head 0's count slot
        }
    }
    __syncthreads();

    // 4. attention over the union, every head of the quad at once
    const int slot = tid >> 4, l16 = tid & 15;
    const int64_t kvrow0 = grp * kv_capacity;
    const int64_t wrow0 = grp * win.win_capacity;
    // After the share's U union rows come its dense rows (Sink, Local / Update Buffer),
    // attended by every head of the quad: dense position j = split + splits * i.
    const int64_t nd = win.dense_rows();
    const int Ut = U + (int)(nd > split ? (nd - split + splits - 1) / splits : 0);
    const uint32_t all_heads = (1u << nh) - 1u;
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
    for (int base = 0; base < Ut; base += kGaSlots * kUnroll) {
        uint32_t msk[kUnroll];
        uint4 kc[kUnroll], vc[kUnroll];
#pragma unroll
        for (int w = 0; w < kUnroll; ++w) {
            const int r = base + slot + kGaSlots * w;
            msk[w] = 0u;
            kc[w] = make_uint4(0, 0, 0, 0);
            vc[w] = make_uint4(0, 0, 0, 0);
            if (r < U) {
                msk[w] = sg.mask[r];
                const int64_t off = (kvrow0 + win.retr_begin + sg.list[r]) * kD;
                kc[w] = reinterpret_cast<const uint4*>(K + off)[l16];
                vc[w] = reinterpret_cast<const uint4*>(V + off)[l16];
            } else if (r < Ut) {
                msk[w] = all_heads;
                const int32_t e = win.dense_entry(split + (int64_t)splits * (r - U));
                const bool in_win = (e & kWinRow) != 0;
                const int64_t off = in_win ? (wrow0 + (e - kWinRow)) * kD : (kvrow0 + e) * kD;
                kc[w] = reinterpret_cast<const uint4*>((in_win ? Kw : K) + off)[l16];
                vc[w] = reinterpret_cast<const uint4*>((in_win ? Vw : V) + off)[l16];
            }
        }
        // scores of every row for every head of the quad
        float dot[4][kUnroll];
#pragma unroll
        for (int w = 0; w < kUnroll; ++w) {
            float kf[8];
            unpack8_half(kc[w], kf);
#pragma unroll
            for (int h = 0; h < 4; ++h) {
                float d0 = 0.f;
#pragma unroll
                for (int d = 0; d < 8; ++d) d0 += qf[h][d] * kf[d];
                dot[h][w] = sum16(d0);
            }
        }
        // one online-softmax update per head for the rows carrying its bit
#pragma unroll
        for (int h = 0; h < 4; ++h) {
            float mn = m[h];
#pragma unroll
            for (int w = 0; w < kUnroll; ++w)
                if ((msk[w] >> h) & 1u) mn = fmaxf(mn, dot[h][w]);
            if (mn > -__builtin_huge_valf()) {
                const float corr = __expf(m[h] - mn);
                lsum[h] *= corr;
#pragma unroll
                for (int d = 0; d < 8; ++d) acc[h][d] *= corr;
#pragma unroll
                for (int w = 0; w < kUnroll; ++w) {
                    if ((msk[w] >> h) & 1u) {
                        const float p = __expf(dot[h][w] - mn);
                        float vf[8];
                        unpack8_half(vc[w], vf);
                        lsum[h] += p;
#pragma unroll
                        for (int d = 0; d < 8; ++d) acc[h][d] += p * vf[d];
                    }
                }
                m[h] = mn;
            }
        }
    }
    // 5. merge the 32 slot states of each head: the 4 slots of a wave (its rows of 16
    // lanes hold the same dims) by two butterfly steps across rows (partners lane ^ 16,
    // then lane ^ 32), the 8 wave states in LDS behind one barrier, where thread
    // (h, d) = (tid / 128, tid % 128) folds dim d of head h.
#pragma unroll
    for (int step = 16; step <= 32; step <<= 1) {
#pragma unroll
        for (int h = 0; h < 4; ++h) {
            const float mp = __uint_as_float(lane_xor(__float_as_uint(m[h]), step, lane));
            const float lp = __uint_as_float(lane_xor(__float_as_uint(lsum[h]), step, lane));
            float ap[8];
#pragma unroll
            for (int d = 0; d < 8; ++d) ap[d] = __uint_as_float(lane_xor(__float_as_uint(acc[h][d]), step, lane));
            const float mn = fmaxf(m[h], mp);
            if (mn > -__builtin_huge_valf()) {
                const float c0 = __expf(m[h] - mn), c1 = __expf(mp - mn);
                lsum[h] = lsum[h] * c0 + lp * c1;
#pragma unroll
                for (int d = 0; d < 8; ++d) acc[h][d] = acc[h][d] * c0 + ap[d] * c1;
            }
            m[h] = mn;
        }
    }
    if (lane < 16) {
#pragma unroll
        for (int h = 0; h < 4; ++h) {
            if (l16 == 0) {
                gm.m[h][wave] = m[h];
                gm.l[h][wave] = lsum[h];
            }
#pragma unroll
            for (int d = 0; d < 8; ++d) gm.acc[h][wave][8 * l16 + d] = acc[h][d];
        }
    }
    __syncthreads();
    const int h = tid / kD, dd = tid % kD;
    if (h < nh) {
        float M = -__builtin_huge_valf();
#pragma unroll
        for (int j = 0; j < kGaWaves; ++j) M = fmaxf(M, gm.m[h][j]);
        float L = 0.f, O = 0.f;
        if (M > -__builtin_huge_valf()) {
            // An empty state (m = -inf, l = 0, acc = 0) is scaled by exp(-inf) = 0.
#pragma unroll
            for (int j = 0; j < kGaWaves; ++j) {
                const float c = __expf(gm.m[h][j] - M);
                L += gm.l[h][j] * c;
                O += gm.acc[h][j][dd] * c;
            }
        }
        if (splits == 1) {
            out[(row0 + h) * kD + dd] = L > 0.f ? O / L : 0.f;
        } else {
            float* ps = part + ((blk * splits + split) * 4 + h) * kGaPart;
            if (dd == 0) {
                ps[0] = M;
                ps[1] = L;
            }
            ps[4 + dd] = O;
        }
    }
}

// One block of kD threads per (group block, head): merges the `splits` share
// states of the head (thread d owns output dim d); kMaxShares >= splits sizes
// the registers that take every share's state at once.
template <int kMaxShares>
__global__ __launch_bounds__(kD) void group_combine_kernel(const float* __restrict__ part, int32_t splits,
                                                           int32_t hkv, int32_t g, int32_t quads,
                                                           float* __restrict__ out, int32_t* __restrict__ union_rows) {
    const int tid = threadIdx.x;
    const int64_t blk = blockIdx.x >> 2;  // (seq * hkv + kvh) * quads + quad
    const int h = (int)(blockIdx.x & 3);
    const int quad = (int)(blk % quads);
    if (h >= min(4, g - 4 * quad)) return;
    const int64_t grp = blk / quads;
    const int64_t row = (grp / hkv) * hkv * g + (grp % hkv) * g + 4 * quad + h;
    const float* ps = part + (blk * splits * 4 + h) * kGaPart;
    const int64_t stride = 4 * kGaPart;  // next share of the same head
    if (h == 0 && tid == 0 && union_rows) {
        int32_t rows = 0;
        for (int j = 0; j < splits; ++j) rows += __float_as_int(ps[j * stride + 2]);
        union_rows[blk] = rows;
    }
    // every share's state loaded at once (splits <= kMaxShares)
    float mj[kMaxShares], lj[kMaxShares], oj[kMaxShares];
#pragma unroll
    for (int j = 0; j < kMaxShares; ++j) {
        lj[j] = 0.f;
        mj[j] = oj[j] = 0.f;
        if (j < splits) {
            mj[j] = ps[j * stride];
            lj[j] = ps[j * stride + 1];
            oj[j] = ps[j * stride + 4 + tid];
        }
    }
    float M = -__builtin_huge_valf();
#pragma unroll
    for (int j = 0; j < kMaxShares; ++j)
        if (lj[j] > 0.f) M = fmaxf(M, mj[j]);
    float L = 0.f, O = 0.f;
#pragma unroll
    for (int j = 0; j < kMaxShares; ++j) {
        if (lj[j] > 0.f) {
            const float c = __expf(mj[j] - M);
            L += lj[j] * c;
            O += oj[j] * c;
        }
    }
    out[row * kD + tid] = L > 0.f ? O / L : 0.f;
}

}  // namespace

int32_t group_splits(int64_t groups, int64_t per, int64_t n) {
    int64_t s = groups >= 256 ? 1 : (256 + groups - 1) / groups;
    s = s < kGaMaxSplits ? s : kGaMaxSplits;
    const int64_t by_rows = per / 256;  // no more shares than 256-entry slices of the quad's lists
    s = s < by_rows ? s : by_rows;
    const int64_t need = (n + kGaRangeKeys - 1) / kGaRangeKeys;  // key ranges of at most kGaRangeKeys
    s = s > need ? s : need;
    s = s < kGaMaxSplits ? s : kGaMaxSplits;
    return (int32_t)(s < 1 ? 1 : s);
}

size_t group_part_bytes(int64_t groups, int32_t splits) {
    return splits > 1 ? (size_t)groups * splits * 4 * kGaPart * sizeof(float) : 0;
}

hipError_t launch_group_attend(const void* q, const void* K, const void* V, int64_t kv_capacity,
                               const int32_t* idx, int32_t k, int32_t batch, int32_t hkv, int32_t g,
                               float scale, float* out, int32_t* union_rows, int32_t splits, int64_t range,
                               float* part, const AttendWindow& win, const void* Kw, const void* Vw,
                               bool host_kv, hipStream_t s) {
    const int32_t quads = (g + 3) / 4;
    const int64_t groups = (int64_t)batch * hkv * quads;
    const bool ranges = range >= 1 && range <= kGaRangeKeys;
    if (splits < 1 || splits > kGaMaxSplits || (splits > 1 && (!part || !ranges))) return hipErrorInvalidValue;
    {
        const ProfEvents pe = prof_begin("group_attend");
        const dim3 grid((unsigned)(groups * splits)), block(kGaThreads);
        const __half *qh = static_cast<const __half*>(q), *Kh = static_cast<const __half*>(K),
                     *Vh = static_cast<const __half*>(V);
        const __half *Kwh = static_cast<const __half*>(Kw), *Vwh = static_cast<const __half*>(Vw);
#define PARISKV_GROUP_LAUNCH(RANGES, UNROLL)                                                              \
    hipExtLaunchKernelGGL((group_attend_kernel<RANGES, UNROLL>), grid, block, 0, s, pe.start, pe.stop, 0, qh, Kh, \
                          Vh, kv_capacity, idx, k, hkv, g, quads, scale, out, union_rows, splits, range, part,    \
                          win, Kwh, Vwh)
        if (ranges && host_kv)
            PARISKV_GROUP_LAUNCH(true, 1);
        else if (ranges)
            PARISKV_GROUP_LAUNCH(true, 4);
        else if (host_kv)
            PARISKV_GROUP_LAUNCH(false, 1);
        else
            PARISKV_GROUP_LAUNCH(false, 4);
#undef PARISKV_GROUP_LAUNCH
        const hipError_t e = hipGetLastError();
        if (e != hipSuccess || splits == 1) return e;
    }
    const ProfEvents pe = prof_begin("group_combine");
    const dim3 cgrid((unsigned)(groups * 4)), cblock(kD);
    const float* pc = part;
    if (splits <= 16)
        hipExtLaunchKernelGGL(group_combine_kernel<16>, cgrid, cblock, 0, s, pe.start, pe.stop, 0, pc, splits, hkv,
                              g, quads, out, union_rows);
    else
        hipExtLaunchKernelGGL(group_combine_kernel<kGaMaxSplits>, cgrid, cblock, 0, s, pe.start, pe.stop, 0, pc,
                              splits, hkv, g, quads, out, union_rows);
    return hipGetLastError();
}

}  // namespace pariskv
