// Step (1) of the tensor-relational EinSum (Sec. 5): the natural join of two
// relations on their shared promoted labels, and the GROUP BY keys.
//
//   stage 0  validate keys (optional), pack V's join key (join labels in V's
//            key order, most significant first) and radix-sort V by it when
//            V's key order does not start with the join labels; for every U
//            tuple binary-search the run of equal join keys in V, then an
//            exclusive scan of the run lengths gives each U tuple its first
//            pair index and the total pair count.  When W's key is V's key
//            prefix followed by the join labels (and U's key starts with
//            them), the roles turn: every V tuple searches its run of U
//            tuples and the pairs come out already grouped by W key.
//   stage 1  load-balanced expansion: a thread owns 8 consecutive pair
//            indices, finds the U tuple of the first by binary search over
//            the scanned counts and walks forward, so hub tuples with long
//            runs are spread over many threads; pairs come out in (u, v)
//            order.  Each pair gets its packed W key; a stable radix sort by
//            W key (skipped when W's keys are a prefix of U's) carrying the
//            packed (u, v) gives the canonical (w_key, u, v) order; run-length
//            encoding gives the output keys and segment offsets (by a scan
//            over the key space instead of the pairs when the W key space
//            is smaller than the pair count).
#include "tre_internal.h"

namespace tre {

namespace {

constexpr int kThreads = 256;
constexpr int kPairsPerThread = 8;  // pairs per thread of the expansion

struct KeyDesc {
    int32_t n;
    int32_t pos[26];
    int32_t bits[26];
};

struct WDesc {
    int32_t n;
    int32_t src[26];
    int32_t pos[26];
    int32_t bits[26];
};

struct Radix {
    int32_t r[26];
};

inline unsigned blocks_for(int64_t n) { return unsigned((n + kThreads - 1) / kThreads); }

__device__ inline uint64_t pack_row(const int32_t* row, const KeyDesc& d) {
    uint64_t k = 0;
    for (int i = 0; i < d.n; i++) k = (k << d.bits[i]) | uint64_t(uint32_t(row[d.pos[i]]));
    return k;
}

// (dn: the tuple count on the device, at most n; null: n)
// Key validation of up to kValJobs relations in one launch: job j's rows take
// blocks block0[j] .. block0[j + 1] - 1.  Per row: every attribute inside its
// radix (flag 4), and strictly above the previous row (1: below, 2: equal).
constexpr int kValJobs = 3;
struct ValSet {
    int32_t n_jobs;
    const int32_t* keys[kValJobs];
    int64_t n[kValJobs];
    int32_t r[kValJobs];
    int32_t* err[kValJobs];
    const int64_t* dn[kValJobs];  // optional device row count (n is then a bound)
    int64_t block0[kValJobs + 1];
    Radix rad[kValJobs];
};

__global__ void k_validate(ValSet vs) {
    const int64_t b = blockIdx.x;
    int j = 0;
    while (j + 1 < vs.n_jobs && b >= vs.block0[j + 1]) j++;
    const int64_t i = (b - vs.block0[j]) * blockDim.x + threadIdx.x;
    int64_t n = vs.n[j];
    if (vs.dn[j]) n = min(n, *vs.dn[j]);
    if (i >= n) return;
    const int r = vs.r[j];
    int flags = 0;
    const int32_t* row = vs.keys[j] + i * r;
    for (int a = 0; a < r; a++)
        if (row[a] < 0 || row[a] >= vs.rad[j].r[a]) flags |= 4;
    if (i > 0) {
        const int32_t* prev = row - r;
        int c = 0;
        for (int a = 0; a < r && c == 0; a++) c = (prev[a] < row[a]) ? -1 : (prev[a] > row[a] ? 1 : 0);
        if (c == 0) flags |= 2;
        if (c > 0) flags |= 1;
    }
    if (flags) atomicOr(vs.err[j], flags);
}

__global__ void k_pack_join(const int32_t* __restrict__ keys, int64_t n, int r, KeyDesc d, uint64_t* __restrict__ out,
                            uint32_t* __restrict__ perm) {
    const int64_t i = int64_t(blockIdx.x) * blockDim.x + threadIdx.x;
    if (i >= n) return;
    out[i] = pack_row(keys + i * r, d);
    if (perm) perm[i] = uint32_t(i);
}

// Run of V tuples whose join key equals U tuple u's: [lo, lo + cnt).
__global__ void k_count(const int32_t* __restrict__ ukeys, int64_t n_u, int ru, KeyDesc du,
                        const uint64_t* __restrict__ vjk, int64_t n_v, int has_join, int64_t* __restrict__ cnt,
                        int64_t* __restrict__ lo) {
    const int64_t u = int64_t(blockIdx.x) * blockDim.x + threadIdx.x;
    if (u > n_u) return;
    if (u == n_u) {
        cnt[u] = 0;
        return;
    }
    if (!has_join) {
        cnt[u] = n_v;
        lo[u] = 0;
        return;
    }
    const uint64_t key = pack_row(ukeys + u * ru, du);
    int64_t a = 0, b = n_v;
    while (a < b) {
        int64_t m = (a + b) >> 1;
        if (vjk[m] < key) a = m + 1; else b = m;
    }
    // end of the run: gallop from its start (runs are short), then bisect
    int64_t c = a;
    if (a < n_v && vjk[a] == key) {
        int64_t last = a, step = 1, probe = a + 1;
        while (probe < n_v && vjk[probe] == key) {
            last = probe;
            step <<= 1;
            probe = a + step;
        }
        int64_t x = last + 1, y = min(probe, n_v);
        while (x < y) {
            int64_t m = (x + y) >> 1;
            if (vjk[m] == key) x = m + 1; else y = m;
        }
        c = x;
    }
    lo[u] = a;
    cnt[u] = c - a;
}

// Same as k_count when the join labels are the first attributes of V's key
// (V is then sorted by them): the search compares those attributes of V's
// rows directly, so V's join keys need not be packed first.
__device__ inline int cmp_prefix(const int32_t* vrow, const int32_t* key, int n) {
    for (int i = 0; i < n; i++) {
        if (vrow[i] != key[i]) return vrow[i] < key[i] ? -1 : 1;
    }
    return 0;
}

__global__ void k_count_prefix(const int32_t* __restrict__ ukeys, int64_t n_u, int ru, KeyDesc du,
                               const int32_t* __restrict__ vkeys, int64_t n_v, int rv, int64_t* __restrict__ cnt,
                               int64_t* __restrict__ lo) {
    const int64_t u = int64_t(blockIdx.x) * blockDim.x + threadIdx.x;
    if (u > n_u) return;
    if (u == n_u) {
        cnt[u] = 0;
        return;
    }
    int32_t key[26];
    for (int i = 0; i < du.n; i++) key[i] = ukeys[u * ru + du.pos[i]];
    int64_t a = 0, b = n_v;
    while (a < b) {
        const int64_t m = (a + b) >> 1;
        if (cmp_prefix(vkeys + m * rv, key, du.n) < 0) a = m + 1; else b = m;
    }
    int64_t c = a;
    if (a < n_v && cmp_prefix(vkeys + a * rv, key, du.n) == 0) {
        int64_t last = a, step = 1, probe = a + 1;
        while (probe < n_v && cmp_prefix(vkeys + probe * rv, key, du.n) == 0) {
            last = probe;
            step <<= 1;
            probe = a + step;
        }
        int64_t x = last + 1, y = min(probe, n_v);
        while (x < y) {
            const int64_t m = (x + y) >> 1;
            if (cmp_prefix(vkeys + m * rv, key, du.n) == 0) x = m + 1; else y = m;
        }
        c = x;
    }
    lo[u] = a;
    cnt[u] = c - a;
}

__global__ void k_store_count(const int64_t* __restrict__ off, int64_t n_u, WsHeader* hdr) {
    hdr->n_pairs = off[n_u];
}

// The join driven by V when U's key is exactly the join labels: a V tuple
// meets at most one U tuple.  k_vmatch1 finds it (flag[v] = 1, uidx[v] = u)
// by a search over U's rows that starts, for a one-attribute key, at the
// position the key would have if U's keys were spread evenly over their
// range (exact when every key is present) and gallops from there; an
// exclusive scan of the flags gives every matched V tuple its pair index.
__device__ inline int64_t find_row(const int32_t* __restrict__ ukeys, int64_t n_u, int ru, const int32_t* key,
                                   int n, int32_t radix0) {
    int64_t a = 0, b = n_u;  // the lower bound of key lies in [a, b]
    if (ru == 1 && n == 1 && radix0 > 0 && n_u > 0) {
        const int32_t k = key[0];
        // clamped: keys outside [0, radix0) only come from unvalidated input
        const int64_t g = max<int64_t>(0, min<int64_t>(n_u - 1, int64_t(k) * n_u / radix0));
        if (ukeys[g] < k) {  // gallop right: the bound is in (prev, pos]
            int64_t prev = g, step = 1, pos = g + 1;
            while (pos < n_u && ukeys[pos] < k) {
                prev = pos;
                step <<= 1;
                pos = g + step;
            }
            a = prev + 1;
            b = min(pos, n_u);
        } else {  // gallop left: the bound is in (pos, hi]
            int64_t hi = g, step = 1, pos = g - 1;
            while (pos >= 0 && ukeys[pos] >= k) {
                hi = pos;
                step <<= 1;
                pos = g - step;
            }
            a = pos < 0 ? 0 : pos + 1;
            b = hi;
        }
    }
    while (a < b) {
        const int64_t m = (a + b) >> 1;
        if (cmp_prefix(ukeys + m * ru, key, n) < 0) a = m + 1; else b = m;
    }
    return (a < n_u && cmp_prefix(ukeys + a * ru, key, n) == 0) ? a : -1;
}

__global__ void k_vmatch1(const int32_t* __restrict__ vkeys, int64_t n_v, int rv, KeyDesc dv,
                          const int32_t* __restrict__ ukeys, int64_t n_u, int ru, int32_t radix0,
                          int32_t* __restrict__ flag, int32_t* __restrict__ uidx) {
    const int64_t v = int64_t(blockIdx.x) * blockDim.x + threadIdx.x;
    if (v > n_v) return;
    if (v == n_v) {
        flag[v] = 0;
        return;
    }
    int32_t key[26];
    for (int i = 0; i < dv.n; i++) key[i] = vkeys[v * rv + dv.pos[i]];
    const int64_t u = find_row(ukeys, n_u, ru, key, dv.n, radix0);
    flag[v] = u >= 0 ? 1 : 0;
    uidx[v] = int32_t(u);
}

__global__ void k_store_count32(const int32_t* __restrict__ pos, int64_t n, WsHeader* hdr) {
    hdr->n_pairs = pos[n];
}


__device__ inline uint64_t pack_w(const int32_t* urow, const int32_t* vrow, const WDesc& d) {
    uint64_t k = 0;
    for (int i = 0; i < d.n; i++) {
        int32_t f = d.src[i] == 0 ? urow[d.pos[i]] : vrow[d.pos[i]];
        k = (k << d.bits[i]) | uint64_t(uint32_t(f));
    }
    return k;
}

// Pairs [t*8, t*8 + 8) of the expansion.  Writes either the final (u, v)
// arrays (no group sort) or packed (u << 32 | v) payloads for the sort.  A
// workgroup's 2048 pairs are staged in LDS and written out by consecutive
// threads, so every store instruction covers consecutive pairs.
// KT: uint32 W keys when they fit in 32 bits (less traffic in the sort),
// else uint64.
// Expansion of the join into pairs: a workgroup writes the consecutive pairs
// [b0, b0 + kBlockPairs), thread t the pairs b0 + t + i * kThreads, so every
// load of V keys and every store is coalesced.  The U tuples whose pair runs
// meet the block are found by two binary searches over the run offsets; when
// there are at most kSpan of them their offsets are staged in LDS and each
// pair finds its U tuple there (the search starts from the thread's previous
// answer, pairs being visited in increasing order).
constexpr int kSpan = 4096;

// Largest u in [a, b] with off[u] <= x (off non-decreasing, off[a] <= x),
// found by the 64 lanes of one wavefront together: each round the lanes probe
// 64 evenly spaced positions of the interval and one ballot keeps the part
// between the last probe that passes and the next, so an interval of n
// positions takes about log64(n) dependent loads instead of log2(n).
__device__ inline int64_t wave_find_u(const int64_t* __restrict__ off, int64_t x, int64_t a, int64_t b) {
    const int lane = threadIdx.x & 63;
    while (a < b) {
        const int64_t len = b - a;
        const int64_t pos = a + ((int64_t(lane) + 1) * len + 63) / 64;  // in (a, b], non-decreasing in lane
        const uint64_t ok = __ballot(off[pos] <= x);
        const int L = __popcll(ok);  // the passing probes are the lowest L lanes
        const int64_t first = a + (len + 63) / 64;
        if (L == 0) {
            b = first - 1;
        } else {
            const int64_t lastok = a + ((int64_t(L) * len + 63) / 64);
            const int64_t next = L < 64 ? a + ((int64_t(L) + 1) * len + 63) / 64 : b + 1;
            a = lastok;
            b = next - 1;
        }
    }
    return a;
}

// The pair count comes from device memory (the scan's total in the
// header), clamped to the capacity `cap` the grid is sized for.
__device__ inline int64_t pair_count(const WsHeader* hdr, int64_t cap) { return min(hdr->n_pairs, cap); }

// VO: the outer relation (whose runs `off` / `lo` describe) is V and the
// runs index U (the join driven by V); otherwise the outer relation is U.
template <typename KT, bool VO>
__global__ __launch_bounds__(kThreads) void k_expand(const int64_t* __restrict__ off, const int64_t* __restrict__ lo,
                                                     int64_t n_u, const WsHeader* __restrict__ hdr, int64_t cap,
                                                     const uint32_t* __restrict__ vperm,
                                                     const int32_t* __restrict__ ukeys, int ru,
                                                     const int32_t* __restrict__ vkeys, int rv, WDesc wd,
                                                     int32_t* __restrict__ pu, int32_t* __restrict__ pv,
                                                     KT* __restrict__ wk, uint64_t* __restrict__ uv) {
    constexpr int kBlockPairs = kThreads * kPairsPerThread;
    __shared__ int32_t s_off[kSpan + 1];  // pair counts stay below 2^31
    __shared__ int64_t s_ends[2];
    const int64_t n_pairs = pair_count(hdr, cap);
    const int64_t b0 = int64_t(blockIdx.x) * kBlockPairs;
    if (b0 >= n_pairs) return;
    const int64_t b1 = min<int64_t>(b0 + kBlockPairs, n_pairs);
    // largest u with off[u] <= x
    auto find_u = [&](int64_t x, int64_t a, int64_t b) {
        while (a < b) {
            const int64_t m = (a + b + 1) >> 1;
            if (off[m] <= x) a = m;
            else b = m - 1;
        }
        return a;
    };
    if (threadIdx.x < 128) {
        const int64_t e = wave_find_u(off, threadIdx.x < 64 ? b0 : b1 - 1, 0, n_u - 1);
        if ((threadIdx.x & 63) == 0) s_ends[threadIdx.x >> 6] = e;
    }
    __syncthreads();
    const int64_t ua = s_ends[0], ub = s_ends[1];
    const int64_t span = ub - ua + 1;
    const bool staged = span <= kSpan;
    if (staged) {
        for (int64_t i = threadIdx.x; i <= span; i += kThreads) s_off[i] = int32_t(off[ua + i]);
        __syncthreads();
    }
    // the thread's pairs in three rounds, each issuing all of its loads
    // before using them: U tuple and run offset (LDS), then the run starts,
    // then the V keys
    int32_t u[kPairsPerThread], vv[kPairsPerThread];
    int32_t idx = 0;  // position of the current U tuple in [ua, ub]
#pragma unroll
    for (int i = 0; i < kPairsPerThread; i++) {
        const int64_t p = b0 + int64_t(i) * kThreads + threadIdx.x;
        u[i] = -1;
        if (p < b1) {
            if (staged) {
                int32_t a = idx, b = int32_t(span) - 1;
                while (a < b) {
                    const int32_t m = (a + b + 1) >> 1;
                    if (s_off[m] <= p) a = m;
                    else b = m - 1;
                }
                idx = a;
                vv[i] = int32_t(p - s_off[a]);
            } else {
                idx = int32_t(find_u(p, ua + idx, ub) - ua);
                vv[i] = int32_t(p - off[ua + idx]);
            }
            u[i] = int32_t(ua + idx);
        }
    }
#pragma unroll
    for (int i = 0; i < kPairsPerThread; i++)
        if (u[i] >= 0) vv[i] += int32_t(lo[u[i]]);
    if (vperm) {
#pragma unroll
        for (int i = 0; i < kPairsPerThread; i++)
            if (u[i] >= 0) vv[i] = int32_t(vperm[vv[i]]);
    }
#pragma unroll
    for (int i = 0; i < kPairsPerThread; i++) {
        if (u[i] < 0) continue;
        const int64_t p = b0 + int64_t(i) * kThreads + threadIdx.x;
        const int32_t iu = VO ? vv[i] : u[i], iv = VO ? u[i] : vv[i];  // (outer, run) -> (u, v)
        wk[p] = KT(pack_w(ukeys + int64_t(iu) * ru, vkeys + int64_t(iv) * rv, wd));
        if (uv) {
            uv[p] = (uint64_t(uint32_t(iu)) << 32) | uint64_t(uint32_t(iv));
        } else {
            pu[p] = iu;
            pv[p] = iv;
        }
    }
}

// A join where the searched relation holds every key of its key space and
// that key is exactly the join labels: sorted strictly increasing keys are
// then 0 .. n - 1 read as mixed-radix numbers, so every tuple of the driving
// ("outer") relation meets the one tuple whose index is its join key -- no
// search, no counts, no scan; pair o is the outer tuple o.  VO: the outer
// relation is V (a V-driven join, the pairs come out grouped by W key);
// otherwise U drives and V is the complete one.  Attributes outside their
// range (keys that fail validation, reported by the host) are clamped so
// nothing is read out of bounds.
struct Radices {
    int32_t n;
    int32_t r[26];
};

// With `uv` (the GROUP BY sort follows) the pass writes packed (u, v)
// payloads instead of the pair arrays.  With `first` (the key-space segment
// search, zeroed; only when no sort follows), it also marks every W key's
// first pair, as k_first_of_key would: first[k] = 1 + o.
template <typename KT, bool VO>
__global__ void k_dense(const int32_t* __restrict__ okeys, int64_t n_o, int ro, KeyDesc dout, Radices ir,
                        const int32_t* __restrict__ ukeys, int ru, const int32_t* __restrict__ vkeys, int rv, WDesc wd,
                        int32_t* __restrict__ pu, int32_t* __restrict__ pv, KT* __restrict__ wk,
                        uint64_t* __restrict__ uv, WsHeader* __restrict__ hdr, int32_t* __restrict__ first,
                        int64_t nk) {
    const int64_t o = int64_t(blockIdx.x) * blockDim.x + threadIdx.x;
    if (o >= n_o) return;
    if (o == 0) hdr->n_pairs = n_o;
    if (dout.n == 1 && wd.n == 1 && wd.src[0] == (VO ? 1 : 0)) {
        // one join label and W keyed by one label of the outer relation
        // (whose keys okeys are): the pair's join key, its W key and the
        // previous pair's W key are loaded at once (the general path below
        // waits for each in turn)
        const int32_t* row = okeys + o * ro;
        const int32_t jk = row[dout.pos[0]];
        const KT k = KT(uint32_t(row[wd.pos[0]]));
        const KT kp = o > 0 ? KT(uint32_t(row[wd.pos[0] - ro])) : k;
        const int64_t in = min(max(jk, 0), ir.r[0] - 1);
        const int64_t u = VO ? in : o, v = VO ? o : in;
        wk[o] = k;
        if (uv) {
            uv[o] = (uint64_t(uint32_t(u)) << 32) | uint64_t(uint32_t(v));
            return;
        }
        pu[o] = int32_t(u);
        pv[o] = int32_t(v);
        if (first && uint64_t(k) < uint64_t(nk) && (o == 0 || kp != k)) first[k] = int32_t(o + 1);
        return;
    }
    auto pair_of = [&](int64_t x, int64_t& u, int64_t& v) {
        const int32_t* row = okeys + x * ro;
        int64_t in = 0;
        for (int i = 0; i < dout.n; i++) in = in * ir.r[i] + min(max(row[dout.pos[i]], 0), ir.r[i] - 1);
        u = VO ? in : x;
        v = VO ? x : in;
    };
    int64_t u, v;
    pair_of(o, u, v);
    const KT k = KT(pack_w(ukeys + u * ru, vkeys + v * rv, wd));
    wk[o] = k;
    if (uv) {
        uv[o] = (uint64_t(uint32_t(u)) << 32) | uint64_t(uint32_t(v));
        return;
    }
    pu[o] = int32_t(u);
    pv[o] = int32_t(v);
    if (first && uint64_t(k) < uint64_t(nk)) {
        bool head = o == 0;
        if (!head) {
            int64_t u1, v1;
            pair_of(o - 1, u1, v1);
            head = KT(pack_w(ukeys + u1 * ru, vkeys + v1 * rv, wd)) != k;
        }
        if (head) first[k] = int32_t(o + 1);
    }
}

// Pairs of the join driven by V with at most one U tuple per V tuple:
// matched V tuple v writes pair pos[v] = (uidx[v], v) and its W key.  Pair
// indices follow V order, so consecutive threads write consecutive pairs.
template <typename KT>
__global__ void k_vwrite(const int32_t* __restrict__ pos, const int32_t* __restrict__ uidx, int64_t n_v,
                         const WsHeader* __restrict__ hdr, int64_t cap, const int32_t* __restrict__ ukeys, int ru,
                         const int32_t* __restrict__ vkeys, int rv, WDesc wd, int32_t* __restrict__ pu,
                         int32_t* __restrict__ pv, KT* __restrict__ wk) {
    const int64_t v = int64_t(blockIdx.x) * blockDim.x + threadIdx.x;
    if (v >= n_v) return;
    const int64_t p = pos[v];
    if (pos[v + 1] == p || p >= pair_count(hdr, cap)) return;
    const int32_t u = uidx[v];
    pu[p] = u;
    pv[p] = int32_t(v);
    wk[p] = KT(pack_w(ukeys + int64_t(u) * ru, vkeys + v * rv, wd));
}

// One workgroup for the whole join of a small input (at most kSmallMax outer
// tuples and kSmallMax pairs): the same steps as the multi-kernel path --
// every outer tuple finds its run of inner tuples by binary search on the
// inner relation's key prefix, an exclusive scan gives the pair offsets, the
// expansion lists the pairs in (outer, inner) order with their W keys, a
// sort by (W key, expansion index) puts them in the canonical (W key, u, v)
// order when the join order does not already group them, and head flags
// with a second scan give the segments -- all in LDS, in one launch.
constexpr int kSmallThreads = 1024;
constexpr int kSmallMax = 4096;
constexpr int kSmallPer = kSmallMax / kSmallThreads;
constexpr int kSmallIdxBits = 12;  // pair index bits of the sort key
static_assert((1 << kSmallIdxBits) == kSmallMax, "sort key layout");

__device__ inline int32_t small_scan(int32_t v, int32_t* wsum, int32_t* total) {
    return block_scan_excl<kSmallThreads>(v, wsum, total);
}

// VO: the outer relation is V (a V-driven join) and the inner one U.
template <bool VO>
__global__ __launch_bounds__(kSmallThreads) void k_join_small(
    const int32_t* __restrict__ okeys, int64_t n_o, int ro, KeyDesc dout, const int32_t* __restrict__ ikeys,
    int64_t n_i, int ri, const int32_t* __restrict__ ukeys, int ru, const int32_t* __restrict__ vkeys, int rv,
    WDesc wd, int sort, int64_t cap, int32_t* __restrict__ pu, int32_t* __restrict__ pv,
    int32_t* __restrict__ seg_start, uint64_t* __restrict__ seg_key, WsHeader* __restrict__ hdr) {
    __shared__ int32_t s_off[kSmallMax + 1];
    __shared__ int32_t s_lo[kSmallMax];
    __shared__ uint64_t s_key[kSmallMax];  // W key << kSmallIdxBits | expansion index
    __shared__ int32_t s_pu[kSmallMax], s_pv[kSmallMax];
    __shared__ uint64_t s_ikey[kSmallMax];  // the inner relation's packed join keys (non-decreasing)
    __shared__ int32_t s_wsum[kSmallThreads / 64];
    const int t = threadIdx.x;
    // join keys packed into one word (the caller checks that they fit): the
    // inner relation's are a prefix of its sorted key, staged in LDS
    auto pack_join = [&](const int32_t* row, bool outer) {
        uint64_t k = 0;
        for (int i = 0; i < dout.n; i++) k = (k << dout.bits[i]) | uint64_t(uint32_t(row[outer ? dout.pos[i] : i]));
        return k;
    };
    for (int64_t i = t; i < n_i; i += kSmallThreads) s_ikey[i] = pack_join(ikeys + i * ri, false);
    __syncthreads();
    // runs: outer tuple o meets inner tuples [s_lo[o], s_lo[o] + c); the
    // kSmallPer searches of a thread advance in lockstep (branch-free lower
    // and upper bounds, the same step count for every thread)
    int32_t c[kSmallPer];
    uint64_t kk[kSmallPer];
    int32_t lb[kSmallPer], ub[kSmallPer];
#pragma unroll
    for (int j = 0; j < kSmallPer; j++) {
        const int64_t o = int64_t(t) * kSmallPer + j;
        kk[j] = o < n_o ? pack_join(okeys + o * ro, true) : 0;
        lb[j] = 0;
        ub[j] = 0;
    }
    if (n_i > 0) {
        for (int32_t len = int32_t(n_i); len > 1;) {
            const int32_t half = len >> 1;
#pragma unroll
            for (int j = 0; j < kSmallPer; j++) {
                if (s_ikey[lb[j] + half] < kk[j]) lb[j] += half;
                if (s_ikey[ub[j] + half] <= kk[j]) ub[j] += half;
            }
            len -= half;
        }
#pragma unroll
        for (int j = 0; j < kSmallPer; j++) {
            lb[j] += s_ikey[lb[j]] < kk[j] ? 1 : 0;
            ub[j] += s_ikey[ub[j]] <= kk[j] ? 1 : 0;
        }
    }
    int32_t csum = 0;
#pragma unroll
    for (int j = 0; j < kSmallPer; j++) {
        const int64_t o = int64_t(t) * kSmallPer + j;
        c[j] = 0;
        if (o < n_o) {
            s_lo[o] = lb[j];
            c[j] = min(ub[j] - lb[j], kSmallMax);  // more cannot be listed (and the sums stay small)
        }
        csum += c[j];
    }
    int32_t total;
    int32_t run = small_scan(csum, s_wsum, &total);
#pragma unroll
    for (int j = 0; j < kSmallPer; j++) {
        const int64_t o = int64_t(t) * kSmallPer + j;
        if (o < n_o) s_off[o] = run;
        run += c[j];
    }
    if (t == 0) {
        s_off[n_o] = total;
        hdr->n_pairs = total;
    }
    __syncthreads();
    const int32_t n = int32_t(min<int64_t>(total, min<int64_t>(cap, kSmallMax)));
    // expansion: pair q belongs to the last outer tuple whose offset is <= q
#pragma unroll
    for (int j = 0; j < kSmallPer; j++) {
        const int32_t q = t * kSmallPer + j;
        if (q >= n) continue;
        int32_t a = 0, b = int32_t(n_o) - 1;
        while (a < b) {
            const int32_t m = (a + b + 1) >> 1;
            if (s_off[m] <= q) a = m; else b = m - 1;
        }
        const int32_t in = s_lo[a] + (q - s_off[a]);
        const int32_t u = VO ? in : a, v = VO ? a : in;
        s_pu[q] = u;
        s_pv[q] = v;
        s_key[q] = (pack_w(ukeys + int64_t(u) * ru, vkeys + int64_t(v) * rv, wd) << kSmallIdxBits) | uint64_t(q);
    }
    __syncthreads();
    if (sort) {
        // bitonic sort of the (W key, index) words, padded to a power of two
        int32_t m = 1;
        while (m < n) m <<= 1;
        for (int32_t q = n + t; q < m; q += kSmallThreads) s_key[q] = ~0ull;
        __syncthreads();
        for (int32_t k = 2; k <= m; k <<= 1) {
            for (int32_t jj = k >> 1; jj > 0; jj >>= 1) {
                for (int32_t i = t; i < m; i += kSmallThreads) {
                    const int32_t ixj = i ^ jj;
                    if (ixj > i) {
                        const uint64_t x = s_key[i], y = s_key[ixj];
                        if ((x > y) == ((i & k) == 0)) {
                            s_key[i] = y;
                            s_key[ixj] = x;
                        }
                    }
                }
                __syncthreads();
            }
        }
    }
    // pairs in order, segment heads, segments
    int32_t h[kSmallPer];
    int32_t hs = 0;
#pragma unroll
    for (int j = 0; j < kSmallPer; j++) {
        const int32_t q = t * kSmallPer + j;
        h[j] = 0;
        if (q < n) {
            const int32_t e = int32_t(s_key[q] & uint64_t(kSmallMax - 1));
            pu[q] = s_pu[e];
            pv[q] = s_pv[e];
            h[j] = (q == 0 || (s_key[q] >> kSmallIdxBits) != (s_key[q - 1] >> kSmallIdxBits)) ? 1 : 0;
        }
        hs += h[j];
    }
    int32_t n_seg;
    int32_t sr = small_scan(hs, s_wsum, &n_seg);
#pragma unroll
    for (int j = 0; j < kSmallPer; j++) {
        const int32_t q = t * kSmallPer + j;
        if (q < n && h[j]) {
            seg_start[sr] = q;
            seg_key[sr] = s_key[q] >> kSmallIdxBits;
            sr++;
        }
    }
    if (t == 0) {
        seg_start[n_seg] = n;
        hdr->n_w = n_seg;
    }
}

// Join with a keyless single-tuple V whose output is keyed by U's own key
// (e.g. T keyed k times a whole weight matrix): every U tuple is one pair and
// its own group, in U order, so the pair list and the segments are written
// directly and the counts are known on the host.
// (n_dev: U's tuple count on the device, at most n_u; null: n_u)
__global__ void k_keyed_by_u(const int32_t* __restrict__ ukeys, int64_t n_u, int ru, WDesc wd,
                             int32_t* __restrict__ pu, int32_t* __restrict__ pv, int32_t* __restrict__ seg_start,
                             uint64_t* __restrict__ seg_key, WsHeader* __restrict__ hdr,
                             const int64_t* __restrict__ n_dev) {
    const int64_t u = int64_t(blockIdx.x) * blockDim.x + threadIdx.x;
    if (n_dev) n_u = max<int64_t>(0, min(n_u, *n_dev));
    if (u > n_u) return;
    seg_start[u] = int32_t(u);
    if (u == n_u) {
        hdr->n_pairs = n_u;
        hdr->n_w = n_u;
        return;
    }
    pu[u] = int32_t(u);
    pv[u] = 0;
    seg_key[u] = pack_w(ukeys + u * ru, ukeys + u * ru, wd);
}

// Segments over a small key space (2^bits <= pairs): first[k] = 1 + the
// index of key k's first pair (0: absent), then the present keys are
// compacted in key order by a scan over the key space instead of over the
// pairs.
// (keys outside the key space come only from keys that fail validation,
// which the host reports; they are skipped so nothing is written out of
// bounds)
template <typename KT>
__global__ void k_first_of_key(const KT* __restrict__ wk, const WsHeader* __restrict__ hdr, int64_t cap,
                               int64_t nk, int32_t* __restrict__ first) {
    const int64_t p = int64_t(blockIdx.x) * blockDim.x + threadIdx.x;
    if (p >= pair_count(hdr, cap)) return;
    const KT k = wk[p];
    if ((p == 0 || k != wk[p - 1]) && uint64_t(k) < uint64_t(nk)) first[k] = int32_t(p + 1);
}

__global__ void k_key_flags(const int32_t* __restrict__ first, int64_t nk, int32_t* __restrict__ flags) {
    const int64_t q = int64_t(blockIdx.x) * blockDim.x + threadIdx.x;
    if (q > nk) return;
    flags[q] = (q < nk && first[q] != 0) ? 1 : 0;
}

__global__ void k_key_compact(const int32_t* __restrict__ first, int64_t nk, const int32_t* __restrict__ seg_of,
                              int64_t cap, int32_t* __restrict__ seg_start, uint64_t* __restrict__ seg_key,
                              WsHeader* hdr) {
    const int64_t q = int64_t(blockIdx.x) * blockDim.x + threadIdx.x;
    if (q > nk) return;
    if (q == nk) {
        seg_start[seg_of[nk]] = int32_t(pair_count(hdr, cap));
        hdr->n_w = seg_of[nk];
        return;
    }
    const int32_t f = first[q];
    if (f != 0) {
        seg_start[seg_of[q]] = f - 1;
        seg_key[seg_of[q]] = uint64_t(q);
    }
}

// The three steps above in one workgroup for a key space of at most
// kKeySmallMax keys: each wavefront owns a contiguous range of keys and reads
// it 64 keys at a time (all its loads issued at once), counts the present
// keys with ballots, a scan over the wavefront totals gives each wavefront
// its first segment, and the segments are written in key order (a lane's
// position within a batch from the ballot mask below it).
constexpr int kKeySmallThreads = 1024;
constexpr int kKeySmallWaves = kKeySmallThreads / 64;
constexpr int kKeySmallBatches = 32;  // batches of 64 keys per wavefront
constexpr int64_t kKeySmallMax = int64_t(kKeySmallWaves) * 64 * kKeySmallBatches;

__global__ __launch_bounds__(kKeySmallThreads) void k_key_segments_small(const int32_t* __restrict__ first,
                                                                           int64_t nk, int64_t cap,
                                                                           int32_t* __restrict__ seg_start,
                                                                           uint64_t* __restrict__ seg_key,
                                                                           WsHeader* hdr) {
    __shared__ int32_t wtot[kKeySmallWaves];
    const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
    const int32_t per = int32_t((nk + kKeySmallWaves * 64 - 1) / (kKeySmallWaves * 64)) * 64;  // keys per wavefront
    const int32_t q0 = w * per;
    const int32_t q1 = min(q0 + per, int32_t(nk));
    int32_t f[kKeySmallBatches];
#pragma unroll
    for (int b = 0; b < kKeySmallBatches; b++) {
        const int32_t q = q0 + b * 64 + lane;
        f[b] = q < q1 ? first[q] : 0;
    }
    int32_t c = 0;
#pragma unroll
    for (int b = 0; b < kKeySmallBatches; b++) c += __popcll(__ballot(f[b] != 0));
    if (lane == 0) wtot[w] = c;
    __syncthreads();
    int32_t base = 0, n_seg = 0;
#pragma unroll
    for (int i = 0; i < kKeySmallWaves; i++) {
        const int32_t x = wtot[i];
        if (i < w) base += x;
        n_seg += x;
    }
    const uint64_t below = (lane == 0) ? 0ull : (~0ull >> (64 - lane));
#pragma unroll
    for (int b = 0; b < kKeySmallBatches; b++) {
        const uint64_t m = __ballot(f[b] != 0);
        if (f[b] != 0) {
            const int32_t o = base + __popcll(m & below);
            seg_start[o] = f[b] - 1;
            seg_key[o] = uint64_t(q0 + b * 64 + lane);
        }
        base += __popcll(m);
    }
    if (threadIdx.x == 0) {
        seg_start[n_seg] = int32_t(pair_count(hdr, cap));
        hdr->n_w = n_seg;
    }
}

// flags over [0, cap] (zero from the pair count on, so the scan over the
// capacity counts the segments of the pairs only)
template <typename KT>
__global__ void k_heads(const KT* __restrict__ wk, const WsHeader* __restrict__ hdr, int64_t cap,
                        int32_t* __restrict__ flags) {
    const int64_t p = int64_t(blockIdx.x) * blockDim.x + threadIdx.x;
    if (p > cap) return;
    const int64_t n = pair_count(hdr, cap);
    flags[p] = (p < n && (p == 0 || wk[p] != wk[p - 1])) ? 1 : 0;
}

template <typename KT>
__global__ void k_compact(const KT* __restrict__ wk, int64_t cap, const int32_t* __restrict__ seg_of,
                          int32_t* __restrict__ seg_start, uint64_t* __restrict__ seg_key, WsHeader* hdr) {
    const int64_t p = int64_t(blockIdx.x) * blockDim.x + threadIdx.x;
    const int64_t n = pair_count(hdr, cap);
    if (p > n) return;
    if (p == n) {
        seg_start[seg_of[n]] = int32_t(n);
        hdr->n_w = seg_of[n];
        return;
    }
    if (p == 0 || wk[p] != wk[p - 1]) {
        const int32_t s = seg_of[p];
        seg_start[s] = int32_t(p);
        seg_key[s] = uint64_t(wk[p]);
    }
}

KeyDesc desc_u(const Plan& p) {
    KeyDesc d{};
    d.n = p.n_join;
    for (int i = 0; i < p.n_join; i++) {
        d.pos[i] = p.join_pos_u[i];
        d.bits[i] = p.join_bits[i];
    }
    return d;
}

KeyDesc desc_v(const Plan& p) {
    KeyDesc d{};
    d.n = p.n_join;
    for (int i = 0; i < p.n_join; i++) {
        d.pos[i] = p.join_pos_v[i];
        d.bits[i] = p.join_bits[i];
    }
    return d;
}

}  // namespace

hipError_t launch_validate(const ValJob* jobs, int n_jobs, hipStream_t s) {
    ValSet vs{};
    int64_t blocks = 0;
    for (int k = 0; k < n_jobs; k++) {
        const ValJob& jb = jobs[k];
        if (jb.n <= 0 || jb.r == 0) continue;  // r == 0: at most one tuple, checked on the host
        if (vs.n_jobs == kValJobs || jb.r > 26) return hipErrorInvalidValue;
        const int j = vs.n_jobs++;
        vs.keys[j] = jb.keys;
        vs.n[j] = jb.n;
        vs.r[j] = jb.r;
        vs.err[j] = jb.err;
        vs.dn[j] = jb.dn;
        for (int a = 0; a < jb.r; a++) vs.rad[j].r[a] = jb.radix[a];
        vs.block0[j] = blocks;
        blocks += blocks_for(jb.n);
    }
    if (vs.n_jobs == 0) return hipSuccess;
    vs.block0[vs.n_jobs] = blocks;
    if (blocks > int64_t(0x7fffffff)) return hipErrorInvalidConfiguration;
    k_validate<<<dim3(unsigned(blocks)), kThreads, 0, s>>>(vs);
    return hipGetLastError();
}

hipError_t launch_validate(const int32_t* keys, int64_t n, int r, const int32_t* radix, int32_t* err_flag,
                           hipStream_t s, const int64_t* dn) {
    const ValJob jb{keys, n, r, radix, err_flag, dn};
    return launch_validate(&jb, 1, s);
}

hipError_t launch_join(const Plan& p, const Layout& L, char* ws, const int32_t* u_keys, const int32_t* v_keys,
                       hipStream_t s, int stage) {
    if (stage != 0) return hipErrorInvalidValue;
    WsHeader* hdr = reinterpret_cast<WsHeader*>(ws + L.hdr);
    uint64_t* vjk = reinterpret_cast<uint64_t*>(ws + L.vjk);
    uint32_t* vperm = p.v_needs_sort ? reinterpret_cast<uint32_t*>(ws + L.vperm) : nullptr;
    // the sorted join keys end up in the alt buffer after an odd pass count
    const uint64_t* vjk_sorted =
        (p.v_needs_sort && radix_result_in_alt(L.n_v, p.join_total_bits)) ? reinterpret_cast<uint64_t*>(ws + L.vjk_alt)
                                                                           : vjk;
    int64_t* cnt = reinterpret_cast<int64_t*>(ws + L.ucnt);
    int64_t* lo = reinterpret_cast<int64_t*>(ws + L.ulo);
    int64_t* tmp = reinterpret_cast<int64_t*>(ws + L.scan_tmp);
    int32_t* hist = reinterpret_cast<int32_t*>(ws + L.hist);
    const int64_t n_u = L.n_u, n_v = L.n_v;
    hipError_t e = hipSuccess;
    // one pair per tuple of the driving relation, written by the GROUP BY stage
    if (v_dense(p, n_u) || u_dense(p, n_v)) return hipSuccess;
    if (p.v_outer && p.nk[0] == p.n_join) {
        // walk V: each V tuple meets at most one U tuple (U's key is the join labels)
        int32_t* pos = reinterpret_cast<int32_t*>(ws + L.ucnt);
        int32_t* uidx = reinterpret_cast<int32_t*>(ws + L.ulo);
        k_vmatch1<<<blocks_for(n_v + 1), kThreads, 0, s>>>(v_keys, n_v, p.nk[1], desc_v(p), u_keys, n_u, p.nk[0],
                                                            p.nk[0] == 1 ? p.radix[0][0] : 0, pos, uidx);
        if ((e = hipGetLastError()) != hipSuccess) return e;
        if ((e = scan_exclusive_i32(pos, pos, n_v + 1, reinterpret_cast<int32_t*>(tmp), s)) != hipSuccess) return e;
        k_store_count32<<<1, 1, 0, s>>>(pos, n_v, hdr);
        return hipGetLastError();
    }
    if (p.v_outer) {
        // walk V: each V tuple's run of U tuples, searched on U's key prefix
        k_count_prefix<<<blocks_for(n_v + 1), kThreads, 0, s>>>(v_keys, n_v, p.nk[1], desc_v(p), u_keys, n_u,
                                                                 p.nk[0], cnt, lo);
        if ((e = hipGetLastError()) != hipSuccess) return e;
        if ((e = scan_exclusive_i64(cnt, cnt, n_v + 1, tmp, s)) != hipSuccess) return e;
        k_store_count<<<1, 1, 0, s>>>(cnt, n_v, hdr);
        return hipGetLastError();
    }
    if (p.n_join > 0 && n_v > 0 && !p.v_needs_sort) {
        // the join labels lead V's key: search V's rows as they are
        k_count_prefix<<<blocks_for(n_u + 1), kThreads, 0, s>>>(u_keys, n_u, p.nk[0], desc_u(p), v_keys, n_v,
                                                                 p.nk[1], cnt, lo);
    } else {
        if (p.n_join > 0 && n_v > 0) {
            k_pack_join<<<blocks_for(n_v), kThreads, 0, s>>>(v_keys, n_v, p.nk[1], desc_v(p), vjk, vperm);
            if ((e = hipGetLastError()) != hipSuccess) return e;
            e = radix_sort_u64(vjk, vperm, reinterpret_cast<uint64_t*>(ws + L.vjk_alt),
                               reinterpret_cast<uint32_t*>(ws + L.vperm_alt), n_v, p.join_total_bits, hist,
                               reinterpret_cast<int32_t*>(tmp), s);
            if (e != hipSuccess) return e;
        }
        k_count<<<blocks_for(n_u + 1), kThreads, 0, s>>>(u_keys, n_u, p.nk[0], desc_u(p), vjk_sorted, n_v,
                                                          p.n_join > 0, cnt, lo);
    }
    if ((e = hipGetLastError()) != hipSuccess) return e;
    if ((e = scan_exclusive_i64(cnt, cnt, n_u + 1, tmp, s)) != hipSuccess) return e;
    k_store_count<<<1, 1, 0, s>>>(cnt, n_u, hdr);
    return hipGetLastError();
}

namespace {

template <typename KT>
hipError_t group_impl(const Plan& p, const Layout& L, char* ws, const int32_t* u_keys, const int32_t* v_keys,
                      int64_t cap, hipStream_t s) {
    // every grid below is sized for the capacity; the kernels read the
    // pair count itself from the header
    WsHeader* hdr = reinterpret_cast<WsHeader*>(ws + L.hdr);
    int64_t* off = reinterpret_cast<int64_t*>(ws + L.ucnt);
    int64_t* lo = reinterpret_cast<int64_t*>(ws + L.ulo);
    uint32_t* vperm = nullptr;
    if (p.v_needs_sort)
        vperm = reinterpret_cast<uint32_t*>(ws + (radix_result_in_alt(L.n_v, p.join_total_bits) ? L.vperm_alt : L.vperm));
    int32_t* pu = reinterpret_cast<int32_t*>(ws + L.pu);
    int32_t* pv = reinterpret_cast<int32_t*>(ws + L.pv);
    KT* wk = reinterpret_cast<KT*>(ws + L.wk);
    int32_t* tmp = reinterpret_cast<int32_t*>(ws + L.scan_tmp);
    int32_t* hist = reinterpret_cast<int32_t*>(ws + L.hist);
    int32_t* flags = reinterpret_cast<int32_t*>(ws + L.flags);
    int32_t* seg_start = reinterpret_cast<int32_t*>(ws + L.seg_start);
    uint64_t* seg_key = reinterpret_cast<uint64_t*>(ws + L.seg_key);
    WDesc wd{};
    wd.n = p.nk[2];
    for (int c = 0; c < p.nk[2]; c++) {
        wd.src[c] = p.w_src[c];
        wd.pos[c] = p.w_pos[c];
        wd.bits[c] = p.w_bits[c];
    }
    hipError_t e;
    const bool sort = p.group_needs_sort && cap > 1 && p.w_total_bits > 0;
    uint64_t* uv = sort ? reinterpret_cast<uint64_t*>(ws + L.pidx) : nullptr;
    const int64_t key_space = int64_t(1) << p.w_total_bits;
    const bool by_key = p.w_total_bits > 0 && p.w_total_bits <= 30 && key_space <= cap;
    int32_t* first = flags;  // key-space segment search: key_space + 1 <= cap + 1 entries
    bool first_done = false;
    if (cap > 0 && (v_dense(p, L.n_u) || u_dense(p, L.n_v))) {
        const bool vo = v_dense(p, L.n_u);
        const int in_op = vo ? 0 : 1;  // the complete relation, indexed by the join key
        Radices ir{};
        ir.n = p.nk[in_op];
        for (int i = 0; i < p.nk[in_op]; i++) ir.r[i] = p.radix[in_op][i];
        const bool mark = by_key && !sort;
        if (mark && (e = launch_fill_zero(first, sizeof(int32_t) * size_t(key_space), s)) != hipSuccess) return e;
        if (vo)
            k_dense<KT, true><<<blocks_for(L.n_v), kThreads, 0, s>>>(v_keys, L.n_v, p.nk[1], desc_v(p), ir, u_keys,
                                                                     p.nk[0], v_keys, p.nk[1], wd, pu, pv, wk, uv, hdr,
                                                                     mark ? first : nullptr, key_space);
        else
            k_dense<KT, false><<<blocks_for(L.n_u), kThreads, 0, s>>>(u_keys, L.n_u, p.nk[0], desc_u(p), ir, u_keys,
                                                                      p.nk[0], v_keys, p.nk[1], wd, pu, pv, wk, uv, hdr,
                                                                      mark ? first : nullptr, key_space);
        if ((e = hipGetLastError()) != hipSuccess) return e;
        first_done = mark;
    } else if (cap > 0 && p.v_outer && p.nk[0] == p.n_join) {
        k_vwrite<KT><<<blocks_for(L.n_v), kThreads, 0, s>>>(
            reinterpret_cast<const int32_t*>(ws + L.ucnt), reinterpret_cast<const int32_t*>(ws + L.ulo), L.n_v, hdr,
            cap, u_keys, p.nk[0], v_keys, p.nk[1], wd, pu, pv, wk);
        if ((e = hipGetLastError()) != hipSuccess) return e;
    } else if (cap > 0) {
        const int64_t threads = (cap + kPairsPerThread - 1) / kPairsPerThread;
        if (p.v_outer)
            k_expand<KT, true><<<blocks_for(threads), kThreads, 0, s>>>(off, lo, L.n_v, hdr, cap, nullptr, u_keys,
                                                                        p.nk[0], v_keys, p.nk[1], wd, pu, pv, wk, uv);
        else
            k_expand<KT, false><<<blocks_for(threads), kThreads, 0, s>>>(off, lo, L.n_u, hdr, cap, vperm, u_keys,
                                                                         p.nk[0], v_keys, p.nk[1], wd, pu, pv, wk, uv);
        if ((e = hipGetLastError()) != hipSuccess) return e;
    }
    if (sort) {
        // the last pass writes the sorted (u, v) straight into pu / pv
        KT* wk_alt = reinterpret_cast<KT*>(ws + L.wk_alt);
        uint64_t* uv_alt = reinterpret_cast<uint64_t*>(ws + L.pidx_alt);
        const int64_t* dn = &hdr->n_pairs;
        if constexpr (sizeof(KT) == 4)
            e = radix_sort_u32_pairs(wk, uv, wk_alt, uv_alt, cap, dn, p.w_total_bits, hist, tmp, pu, pv, s);
        else
            e = radix_sort_u64_pairs(wk, uv, wk_alt, uv_alt, cap, dn, p.w_total_bits, hist, tmp, pu, pv, s);
        if (e != hipSuccess) return e;
        if (radix_result_in_alt(cap, p.w_total_bits)) wk = wk_alt;
    }
    if (by_key) {
        // small key space: find the segments by key instead of by pair
        int32_t* kflags = reinterpret_cast<int32_t*>(ws + L.part_off);  // free until the work units are made
        if (!first_done) {
            if ((e = launch_fill_zero(first, sizeof(int32_t) * size_t(key_space), s)) != hipSuccess) return e;
            k_first_of_key<KT><<<blocks_for(cap), kThreads, 0, s>>>(wk, hdr, cap, key_space, first);
            if ((e = hipGetLastError()) != hipSuccess) return e;
        }
        if (key_space <= kKeySmallMax) {
            k_key_segments_small<<<1, kKeySmallThreads, 0, s>>>(first, key_space, cap, seg_start, seg_key, hdr);
            return hipGetLastError();
        }
        k_key_flags<<<blocks_for(key_space + 1), kThreads, 0, s>>>(first, key_space, kflags);
        if ((e = hipGetLastError()) != hipSuccess) return e;
        if ((e = scan_exclusive_i32(kflags, kflags, key_space + 1, tmp, s)) != hipSuccess) return e;
        k_key_compact<<<blocks_for(key_space + 1), kThreads, 0, s>>>(first, key_space, kflags, cap, seg_start,
                                                                      seg_key, hdr);
        return hipGetLastError();
    }
    k_heads<KT><<<blocks_for(cap + 1), kThreads, 0, s>>>(wk, hdr, cap, flags);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    if ((e = scan_exclusive_i32(flags, flags, cap + 1, tmp, s)) != hipSuccess) return e;
    k_compact<KT><<<blocks_for(cap + 1), kThreads, 0, s>>>(wk, cap, flags, seg_start, seg_key, hdr);
    return hipGetLastError();
}

}  // namespace

bool small_join_ok(const Plan& p, int64_t n_u, int64_t n_v, int64_t cap) {
    // joins whose pairs need the GROUP BY sort stay on the multi-kernel path:
    // sorting 4096 pairs on one CU (a bitonic sort, 78 barrier stages) took
    // longer than the device-wide radix sort it replaces (96 us against about
    // 90 us for the whole multi-kernel join of the 4096-vertex chain's E1)
    if (p.opt.small_join < 0 || p.v_needs_sort || p.group_needs_sort || keyed_by_u(p) || v_dense(p, n_u) ||
        p.w_total_bits > 32)
        return false;
    // the inner relation's join keys, packed into one word each, are staged in LDS
    int join_bits = 0;
    for (int i = 0; i < p.n_join; i++) join_bits += p.join_bits[i];
    const int64_t n_o = p.v_outer ? n_v : n_u, n_i = p.v_outer ? n_u : n_v;
    return join_bits <= 64 && n_i <= kSmallMax && n_o >= 1 && n_o <= kSmallMax && cap >= 1 && cap <= kSmallMax;
}

hipError_t launch_join_small(const Plan& p, const Layout& L, char* ws, const int32_t* u_keys, const int32_t* v_keys,
                             int64_t cap, hipStream_t s) {
    WDesc wd{};
    wd.n = p.nk[2];
    for (int c = 0; c < p.nk[2]; c++) {
        wd.src[c] = p.w_src[c];
        wd.pos[c] = p.w_pos[c];
        wd.bits[c] = p.w_bits[c];
    }
    int32_t* pu = reinterpret_cast<int32_t*>(ws + L.pu);
    int32_t* pv = reinterpret_cast<int32_t*>(ws + L.pv);
    int32_t* seg_start = reinterpret_cast<int32_t*>(ws + L.seg_start);
    uint64_t* seg_key = reinterpret_cast<uint64_t*>(ws + L.seg_key);
    WsHeader* hdr = reinterpret_cast<WsHeader*>(ws + L.hdr);
    const int sort = p.group_needs_sort ? 1 : 0;
    if (p.v_outer)
        k_join_small<true><<<1, kSmallThreads, 0, s>>>(v_keys, L.n_v, p.nk[1], desc_v(p), u_keys, L.n_u, p.nk[0],
                                                        u_keys, p.nk[0], v_keys, p.nk[1], wd, sort, cap, pu, pv,
                                                        seg_start, seg_key, hdr);
    else
        k_join_small<false><<<1, kSmallThreads, 0, s>>>(u_keys, L.n_u, p.nk[0], desc_u(p), v_keys, L.n_v, p.nk[1],
                                                         u_keys, p.nk[0], v_keys, p.nk[1], wd, sort, cap, pu, pv,
                                                         seg_start, seg_key, hdr);
    return hipGetLastError();
}

bool u_dense(const Plan& p, int64_t n_v) {
    if (p.v_outer || p.v_needs_sort || !(p.nk[1] == p.n_join && p.nk[1] > 0)) return false;
    int64_t space = 1;
    for (int i = 0; i < p.nk[1]; i++) {
        space *= p.radix[1][i];
        if (space > n_v) return false;
    }
    return space == n_v;
}

bool v_dense(const Plan& p, int64_t n_u) {
    if (!(p.nk[0] == p.n_join && p.nk[0] > 0) || (!p.v_outer && p.v_needs_sort)) return false;
    int64_t space = 1;
    for (int i = 0; i < p.nk[0]; i++) {
        space *= p.radix[0][i];
        if (space > n_u) return false;
    }
    return space == n_u;
}

bool keyed_by_u(const Plan& p) {
    if (p.nk[1] != 0 || p.nk[2] != p.nk[0]) return false;
    for (int c = 0; c < p.nk[2]; c++)
        if (p.w_src[c] != 0 || p.w_pos[c] != c) return false;
    return true;
}

hipError_t launch_keyed_by_u(const Plan& p, const Layout& L, char* ws, const int32_t* u_keys, hipStream_t s,
                             const int64_t* n_dev) {
    WDesc wd{};
    wd.n = p.nk[2];
    for (int c = 0; c < p.nk[2]; c++) {
        wd.src[c] = 0;
        wd.pos[c] = c;
        wd.bits[c] = p.w_bits[c];
    }
    k_keyed_by_u<<<blocks_for(L.n_u + 1), kThreads, 0, s>>>(
        u_keys, L.n_u, p.nk[0], wd, reinterpret_cast<int32_t*>(ws + L.pu), reinterpret_cast<int32_t*>(ws + L.pv),
        reinterpret_cast<int32_t*>(ws + L.seg_start), reinterpret_cast<uint64_t*>(ws + L.seg_key),
        reinterpret_cast<WsHeader*>(ws + L.hdr), n_dev);
    return hipGetLastError();
}

hipError_t launch_group(const Plan& p, const Layout& L, char* ws, const int32_t* u_keys, const int32_t* v_keys,
                        int64_t cap, hipStream_t s) {
    if (cap < 0 || cap > L.max_pairs) return hipErrorInvalidValue;
    return p.w_total_bits <= 32 ? group_impl<uint32_t>(p, L, ws, u_keys, v_keys, cap, s)
                                : group_impl<uint64_t>(p, L, ws, u_keys, v_keys, cap, s);
}

}  // namespace tre
