// Repartition of a tensor relation between two decompositions (Sec. 6: when
// the decomposition an EinSum produces differs from the one its consumer
// reads, the relation is decomposed on all labels promoted in either
// decomposition -- ALLINTS -- and re-composed with the STACK aggregate
// grouped by the consumer's promoted labels).
//
// On the device the two steps are fused: every source tile meets a small box
// of target tiles; the (target key, source tuple) pairs are listed, sorted by
// target key (stable LSD radix sort, so the target keys come out sorted and
// a target's sources in source order; skipped when the listing is already
// in target order, as when row blocks are stacked), run-length encoded into
// the target key set, and each pair copies the intersection of its source
// tile and its target tile (see k_rp_copy).  Target elements no source tile
// covers are zero.
#include "tre_internal.h"

#include <algorithm>
#include <cstring>

namespace tre {

namespace {

constexpr int kThreads = 256;

inline unsigned blocks_for(int64_t n) { return unsigned((n + kThreads - 1) / kThreads); }

constexpr int kRpMaxLabels = kMaxDims;  // labels of one tensor (kept in registers)

// Both decompositions of one tensor, per label position in the label string.
struct RpDesc {
    int32_t nl, rin, rout;
    int32_t pin[kRpMaxLabels], pout[kRpMaxLabels];  // promoted in the source / target
    int64_t ext[kRpMaxLabels], tin[kRpMaxLabels], tout[kRpMaxLabels];
    int64_t sin_[kRpMaxLabels], sout[kRpMaxLabels];  // row-major strides of the source / target tile
    int32_t bits[kRpMaxLabels];                      // bits of each target key attribute (target order)
    int32_t kshift[kRpMaxLabels], kbits[kRpMaxLabels];  // per label: place in the packed target key (0 bits: not promoted)
    int32_t key_bits;
    int64_t te_in, te_out;
    int64_t max_cover;              // target tiles one source tile can meet
    int32_t regroup;                // a source tile is one contiguous run of its target tile
};

struct RpHeader {
    int32_t err;
    int32_t unsorted;  // nonzero: listing the pairs by source leaves target keys out of order
    int64_t pairs;
    int64_t n_out;
    int64_t pad1[5];
};

__device__ inline void source_range(const RpDesc& d, const int32_t* key, int i, int ka, int64_t& lo, int64_t& hi) {
    lo = d.pin[i] ? int64_t(key[ka]) * d.tin[i] : 0;
    hi = lo + d.tin[i];
}

// Packed target key of the target tile holding the lower (upper = false) or
// upper corner of a source tile.
__device__ inline uint64_t corner_key(const RpDesc& d, const int32_t* key, bool upper) {
    uint64_t k = 0;
    int ka = 0, ko = 0;
#pragma unroll
    for (int i = 0; i < kRpMaxLabels; i++) {
        if (i >= d.nl) break;
        int64_t lo, hi;
        source_range(d, key, i, ka, lo, hi);
        ka += d.pin[i];
        if (d.pout[i]) {
            k = (k << d.bits[ko]) | uint64_t((upper ? hi - 1 : lo) / d.tout[i]);
            ko++;
        }
    }
    return k;
}

// Per source tuple: the number of target tiles it meets.  Also flags whether
// listing the pairs source by source (each source's targets in key order)
// already leaves the target keys sorted: it does when no source's first
// target precedes the previous source's last.
__global__ void k_rp_count(const int32_t* __restrict__ keys, int64_t n, RpDesc d, int64_t* __restrict__ cnt,
                           RpHeader* __restrict__ hdr) {
    const int64_t s = int64_t(blockIdx.x) * blockDim.x + threadIdx.x;
    if (s > n) return;
    if (s == n) {
        cnt[s] = 0;
        return;
    }
    const int32_t* key = keys + s * d.rin;
    int64_t c = 1;
    int ka = 0;
#pragma unroll
    for (int i = 0; i < kRpMaxLabels; i++) {
        if (i >= d.nl) break;
        int64_t lo, hi;
        source_range(d, key, i, ka, lo, hi);
        ka += d.pin[i];
        if (d.pout[i]) c *= (hi - 1) / d.tout[i] - lo / d.tout[i] + 1;
    }
    cnt[s] = c;
    if (s > 0 && corner_key(d, key, false) < corner_key(d, key - d.rin, true)) atomicOr(&hdr->unsorted, 1);
}

// List (target key, source) for every target tile source s meets, in target
// key order within s.
__global__ __launch_bounds__(kThreads) void k_rp_expand(const int32_t* __restrict__ keys, int64_t n, RpDesc d,
                                                        const int64_t* __restrict__ off, uint64_t* __restrict__ tk,
                                                        uint32_t* __restrict__ src) {
    const int64_t s = int64_t(blockIdx.x) * blockDim.x + threadIdx.x;
    if (s >= n) return;
    const int32_t* key = keys + s * d.rin;
    int64_t blo[kRpMaxLabels], bn[kRpMaxLabels];
    int ka = 0;
#pragma unroll
    for (int i = 0; i < kRpMaxLabels; i++) {
        blo[i] = 0;
        bn[i] = 1;
        if (i >= d.nl) continue;
        int64_t lo, hi;
        source_range(d, key, i, ka, lo, hi);
        ka += d.pin[i];
        blo[i] = lo / d.tout[i];
        bn[i] = (hi - 1) / d.tout[i] - blo[i] + 1;
    }
    const int64_t c = off[s + 1] - off[s];
    for (int64_t j = 0; j < c; j++) {
        // digits of j over the target-promoted labels, last label fastest
        int64_t rem = j, block[kRpMaxLabels];
#pragma unroll
        for (int i = kRpMaxLabels - 1; i >= 0; i--) {
            block[i] = blo[i];
            if (i >= d.nl || !d.pout[i]) continue;
            block[i] += rem % bn[i];
            rem /= bn[i];
        }
        uint64_t k = 0;
        int ko = 0;
#pragma unroll
        for (int i = 0; i < kRpMaxLabels; i++) {
            if (i >= d.nl || !d.pout[i]) continue;
            k = (k << d.bits[ko]) | uint64_t(block[i]);
            ko++;
        }
        tk[off[s] + j] = k;
        src[off[s] + j] = uint32_t(s);
    }
}

__global__ void k_rp_heads(const uint64_t* __restrict__ tk, int64_t m, int32_t* __restrict__ flags) {
    const int64_t p = int64_t(blockIdx.x) * blockDim.x + threadIdx.x;
    if (p > m) return;
    flags[p] = (p < m && (p == 0 || tk[p] != tk[p - 1])) ? 1 : 0;
}

__global__ void k_rp_compact(const uint64_t* __restrict__ tk, int64_t m, const int32_t* __restrict__ seg_of,
                             uint64_t* __restrict__ seg_key, RpHeader* hdr) {
    const int64_t p = int64_t(blockIdx.x) * blockDim.x + threadIdx.x;
    if (p > m) return;
    if (p == m) {
        hdr->n_out = seg_of[m];
        return;
    }
    if (p == 0 || tk[p] != tk[p - 1]) seg_key[seg_of[p]] = tk[p];
}

__global__ void k_rp_write_keys(const uint64_t* __restrict__ seg_key, int64_t n_out, RpDesc d,
                                int32_t* __restrict__ keys_out) {
    const int64_t q = int64_t(blockIdx.x) * blockDim.x + threadIdx.x;
    if (q >= n_out) return;
    uint64_t k = seg_key[q];
    for (int a = d.rout - 1; a >= 0; a--) {
        keys_out[q * d.rout + a] = int32_t(k & ((uint64_t(1) << d.bits[a]) - 1));
        k >>= d.bits[a];
    }
}

// The copy: a workgroup takes a run of up to kRpPairs consecutive pairs.
// One thread per pair works out the pair's intersection box and cuts it into
// runs that are contiguous in both tiles (the innermost labels, merged while
// the box spans them whole in both tiles); the runs are cut into 16-byte
// chunks when every run of every pair of the workgroup starts on a 16-byte
// boundary in both tiles, else into elements.  The chunks of the
// workgroup's pairs are numbered end to end and the threads stride over
// them with kRpUnroll loads in flight per thread; a chunk's pair is found by
// division when all pairs have the same chunk count, else by binary search
// of the chunk prefix in LDS.
constexpr int kRpPairs = kThreads;
constexpr int kRpUnroll = 4;

struct RpPair {
    int64_t so, to;           // element offset of the box in the source / target tile array
    int32_t run, runs, j;     // elements per contiguous run, runs, first merged label
    int32_t per_run;          // chunks per run
    int32_t n[kRpMaxLabels];  // box extent of the unmerged (outer) labels
};

// Copy the chunks [0, total) of the workgroup's pairs; V is one chunk.
template <typename E, typename V>
__device__ inline void rp_copy_chunks(const E* __restrict__ tin, E* __restrict__ tout, const RpDesc& d,
                                      const RpPair* pr, const int32_t* pre, int np, bool uni, int32_t cpp,
                                      int32_t total) {
    constexpr int kW = sizeof(V) / sizeof(E);  // elements per chunk
    for (int32_t c0 = threadIdx.x; c0 < total; c0 += kThreads * kRpUnroll) {
        V v[kRpUnroll];
        int64_t dst[kRpUnroll];
#pragma unroll
        for (int u = 0; u < kRpUnroll; u++) {
            // past the end: copy the last chunk again (the same bytes to the
            // same place), which keeps the loads and stores unconditional
            const int32_t c = min(c0 + u * kThreads, total - 1);
            int i;
            if (uni) {
                i = c / cpp;
            } else {
                int lo = 0, hi = np;  // pre[lo] <= c < pre[hi]
                while (hi - lo > 1) {
                    const int mid = (lo + hi) >> 1;
                    if (pre[mid] <= c) lo = mid;
                    else hi = mid;
                }
                i = lo;
            }
            const RpPair& P = pr[i];
            int32_t x = c - (uni ? i * cpp : pre[i]);
            int64_t os = P.so, ot = P.to;
            if (P.runs > 1) {
                int32_t r = x / P.per_run;
                x -= r * P.per_run;
#pragma unroll
                for (int k = kRpMaxLabels - 2; k >= 0; k--) {
                    if (k >= P.j) continue;
                    const int32_t cc = r % P.n[k];
                    r /= P.n[k];
                    os += cc * d.sin_[k];
                    ot += cc * d.sout[k];
                }
            }
            os += int64_t(x) * kW;
            ot += int64_t(x) * kW;
            v[u] = *reinterpret_cast<const V*>(tin + os);
            dst[u] = ot;
        }
#pragma unroll
        for (int u = 0; u < kRpUnroll; u++) *reinterpret_cast<V*>(tout + dst[u]) = v[u];
    }
}

template <typename E>
__global__ __launch_bounds__(kThreads) void k_rp_copy(const int32_t* __restrict__ keys, const E* __restrict__ tin,
                                                      const uint64_t* __restrict__ tk,
                                                      const uint32_t* __restrict__ src,
                                                      const int32_t* __restrict__ seg_of, int64_t m, int32_t per_wg,
                                                      RpDesc d, E* __restrict__ tout) {
    __shared__ RpPair pr[kRpPairs];
    __shared__ int32_t pre[kRpPairs + 1];
    __shared__ int32_t wsum[kThreads / 64];
    __shared__ int32_t uniform, allvec;
    constexpr int kV = 16 / sizeof(E);
    const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
    const bool aligned = ((reinterpret_cast<uintptr_t>(tin) | reinterpret_cast<uintptr_t>(tout)) % 16) == 0;
    const int64_t n_batches = (m + per_wg - 1) / per_wg;
    for (int64_t bt = blockIdx.x; bt < n_batches; bt += gridDim.x) {
        const int64_t p0 = bt * per_wg;
        const int np = int(min<int64_t>(per_wg, m - p0));
        if (tid == 0) {
            uniform = 1;
            allvec = aligned ? 1 : 0;
        }
        __syncthreads();
        if (tid < np) {
            const int64_t p = p0 + tid;
            // the pair's target tuple: segments are numbered by an exclusive
            // scan of the head flags, so pair p belongs to segment seg_of[p + 1] - 1
            const int64_t s = src[p], q = seg_of[p + 1] - 1;
            const int32_t* key = keys + s * d.rin;
            // target block of each target-promoted label, from the packed key
            const uint64_t k = tk[p];
            // intersection box: per label, start in source and target, and length
            int32_t n[kRpMaxLabels];
            int64_t so = s * d.te_in, to = q * d.te_out;
            int ka = 0;
#pragma unroll
            for (int i = 0; i < kRpMaxLabels; i++) {
                n[i] = 1;
                if (i >= d.nl) continue;
                int64_t slo, shi;
                source_range(d, key, i, ka, slo, shi);
                ka += d.pin[i];
                const int64_t block = int64_t((k >> d.kshift[i]) & ((uint64_t(1) << d.kbits[i]) - 1));
                const int64_t tlo = d.pout[i] ? block * d.tout[i] : 0, thi = tlo + d.tout[i];
                const int64_t a = max(slo, tlo);
                n[i] = int32_t(min(shi, thi) - a);
                so += (a - slo) * d.sin_[i];
                to += (a - tlo) * d.sout[i];
            }
            // merge labels, innermost first, into one contiguous run while
            // each next label steps exactly one run in both tiles
            int j = d.nl;
            int64_t run = 1;
            bool open = true;
#pragma unroll
            for (int i = kRpMaxLabels - 1; i >= 0; i--) {
                if (i >= d.nl || !open) continue;
                if (j == d.nl || (d.sin_[i] == run && d.sout[i] == run)) {
                    run *= n[i];
                    j = i;
                } else {
                    open = false;
                }
            }
            int32_t runs = 1;
            bool vec = run % kV == 0 && so % kV == 0 && to % kV == 0;
            RpPair& P = pr[tid];
#pragma unroll
            for (int i = 0; i < kRpMaxLabels; i++) {
                P.n[i] = 1;
                if (i >= j) continue;
                P.n[i] = n[i];
                runs *= n[i];
                if (n[i] > 1 && (d.sin_[i] % kV || d.sout[i] % kV)) vec = false;
            }
            P.so = so;
            P.to = to;
            P.run = int32_t(run);
            P.runs = runs;
            P.j = j;
            if (!vec) allvec = 0;
        }
        __syncthreads();
        // chunk counts (all pairs cut alike) and their exclusive scan
        const bool v16 = allvec != 0;
        int32_t chunks = 0;
        if (tid < np) {
            const int32_t per_run = v16 ? pr[tid].run / kV : pr[tid].run;
            pr[tid].per_run = per_run;
            chunks = pr[tid].runs * per_run;
        }
        int32_t incl = chunks;
#pragma unroll
        for (int o = 1; o < 64; o <<= 1) {
            const int32_t y = __shfl_up(incl, o);
            if (lane >= o) incl += y;
        }
        if (lane == 63) wsum[w] = incl;
        __syncthreads();
        int32_t excl = incl - chunks;
        for (int i = 0; i < w; i++) excl += wsum[i];
        if (tid < np) {
            pre[tid] = excl;
            if (tid == np - 1) pre[np] = excl + chunks;
            if (chunks != pr[0].runs * pr[0].per_run) uniform = 0;
        }
        __syncthreads();
        const int32_t total = pre[np];
        const int32_t cpp = pr[0].runs * pr[0].per_run;
        const bool uni = uniform != 0;
        if (v16) rp_copy_chunks<E, uint4>(tin, tout, d, pr, pre, np, uni, cpp, total);
        else rp_copy_chunks<E, E>(tin, tout, d, pr, pre, np, uni, cpp, total);
        __syncthreads();  // pr, pre and the flags are rewritten by the next batch
    }
}

tre_status dev_fail(hipError_t e, const char* where) {
    set_error(std::string("tre_repartition: ") + where + ": " + hipGetErrorString(e));
    return TRE_E_DEVICE;
}

int32_t bit_width(int64_t x) {
    int32_t b = 0;
    while (x > 0) {
        b++;
        x >>= 1;
    }
    return b;
}

tre_status make_desc(const char* labels, const char* up_in, const char* up_out, const int64_t* extent,
                     const int32_t* tile_in, const int32_t* tile_out, RpDesc& d) {
    std::memset(&d, 0, sizeof(d));
    if (!labels || !up_in || !up_out || !extent || !tile_in || !tile_out) {
        set_error("tre_repartition: null argument");
        return TRE_E_ARG;
    }
    bool seen[26] = {}, in_up[26] = {}, out_up[26] = {};
    int lab[26];
    for (const char* c = labels; *c; c++) {
        if (*c < 'a' || *c > 'z' || seen[*c - 'a']) {
            set_error("tre_repartition: labels must be distinct lower-case letters");
            return TRE_E_PARSE;
        }
        if (d.nl == kRpMaxLabels) {
            set_error("tre_repartition: at most 8 labels");
            return TRE_E_SHAPE;
        }
        seen[*c - 'a'] = true;
        lab[d.nl++] = *c - 'a';
    }
    for (int pass = 0; pass < 2; pass++) {
        for (const char* c = pass ? up_out : up_in; *c; c++) {
            if (*c < 'a' || *c > 'z' || !seen[*c - 'a']) {
                set_error("tre_repartition: a promoted label is not a label of the tensor");
                return TRE_E_SPLIT;
            }
            (pass ? out_up : in_up)[*c - 'a'] = true;
        }
    }
    d.te_in = d.te_out = 1;
    d.max_cover = 1;
    for (int i = 0; i < d.nl; i++) {
        const int l = lab[i];
        d.ext[i] = extent[l];
        d.pin[i] = in_up[l];
        d.pout[i] = out_up[l];
        d.tin[i] = in_up[l] ? tile_in[l] : extent[l];
        d.tout[i] = out_up[l] ? tile_out[l] : extent[l];
        if (d.ext[i] < 1 || d.tin[i] < 1 || d.tout[i] < 1 || d.ext[i] % d.tin[i] || d.ext[i] % d.tout[i]) {
            set_error("tre_repartition: every tile size must divide its label's extent");
            return TRE_E_SHAPE;
        }
        d.rin += d.pin[i];
        if (d.pout[i]) {
            d.bits[d.rout] = bit_width(d.ext[i] / d.tout[i] - 1);
            d.key_bits += d.bits[d.rout];
            d.rout++;
            // blocks of size tout met by an aligned run of length tin
            d.max_cover *= std::min<int64_t>(d.ext[i] / d.tout[i], (d.tin[i] - 1) / d.tout[i] + 2);
        }
        if (d.tin[i] > (int64_t(1) << 30) / d.te_in || d.tout[i] > (int64_t(1) << 30) / d.te_out) {
            set_error("tre_repartition: a tile holds more than 2^30 elements");
            return TRE_E_SHAPE;
        }
        d.te_in *= d.tin[i];
        d.te_out *= d.tout[i];
    }
    if (d.key_bits > 64) {
        set_error("tre_repartition: target key space exceeds 64 bits");
        return TRE_E_SHAPE;
    }
    // A source tile is one contiguous run of the target tile (row-major) when,
    // at the first label whose source tile is shorter than the target's, every
    // label before it has a source tile of 1 and every label after it the
    // target's tile.  Sources of one target then sit in source key order.
    d.regroup = 1;
    int first = 0;
    while (first < d.nl && d.tin[first] >= d.tout[first]) first++;
    for (int i = 0; i < d.nl; i++)
        if (i < first ? d.tin[i] != 1 : (i > first && d.tin[i] != d.tout[i])) d.regroup = 0;
    if (first == d.nl) {  // no source tile shorter than its target: the same tiles
        d.regroup = 1;
        for (int i = 0; i < d.nl; i++)
            if (d.tin[i] != d.tout[i]) d.regroup = 0;
    }
    int64_t si = 1, so = 1;
    for (int i = d.nl - 1, sh = 0, ko = d.rout - 1; i >= 0; i--) {
        if (d.pout[i]) {
            d.kbits[i] = d.bits[ko--];
            d.kshift[i] = sh;
            sh += d.kbits[i];
        }
        d.sin_[i] = si;
        d.sout[i] = so;
        si *= d.tin[i];
        so *= d.tout[i];
    }
    return TRE_OK;
}

struct RpLayout {
    size_t hdr, cnt, tmp, tk, tk_alt, src, src_alt, hist, seg_of, seg_key, total;
};

size_t align256(size_t x) { return (x + 255) / 256 * 256; }

RpLayout rp_layout(const RpDesc& d, int64_t n_in) {
    const int64_t m = std::max<int64_t>(n_in * d.max_cover, 1);
    RpLayout L{};
    size_t off = 0;
    auto take = [&](size_t b) {
        const size_t o = off;
        off += align256(std::max<size_t>(b, 1));
        return o;
    };
    L.hdr = take(sizeof(RpHeader));
    L.cnt = take(sizeof(int64_t) * size_t(n_in + 1));
    L.tmp = take(sizeof(int64_t) * scan_tmp_elems(std::max<int64_t>(n_in, m) + 1));
    L.tk = take(sizeof(uint64_t) * size_t(m));
    L.tk_alt = take(sizeof(uint64_t) * size_t(m));
    L.src = take(sizeof(uint32_t) * size_t(m));
    L.src_alt = take(sizeof(uint32_t) * size_t(m));
    L.hist = take(sizeof(int32_t) * size_t(radix_hist_elems(m)));
    L.seg_of = take(sizeof(int32_t) * size_t(m + 1));
    L.seg_key = take(sizeof(uint64_t) * size_t(m));
    L.total = off;
    return L;
}

}  // namespace

}  // namespace tre

using namespace tre;

extern "C" {

size_t tre_repartition_workspace_bytes(const char* labels, const char* upper_in, const char* upper_out,
                                       const int64_t extent[26], const int32_t tile_in[26],
                                       const int32_t tile_out[26], int64_t n_in) {
    RpDesc d;
    if (n_in < 0 || make_desc(labels, upper_in, upper_out, extent, tile_in, tile_out, d) != TRE_OK) return 0;
    return rp_layout(d, n_in).total;
}

tre_status tre_repartition(const char* labels, const char* upper_in, const char* upper_out,
                           const int64_t extent[26], const int32_t tile_in[26], const int32_t tile_out[26],
                           int32_t elem_bytes, const int32_t* keys_in, int64_t n_in, const void* tiles_in,
                           int32_t* keys_out, void* tiles_out, int64_t out_cap, int64_t* n_out, void* ws,
                           size_t ws_bytes, void* stream) {
    RpDesc d;
    tre_status st = make_desc(labels, upper_in, upper_out, extent, tile_in, tile_out, d);
    if (st != TRE_OK) return st;
    if (!n_out || n_in < 0 || out_cap < 0 || (elem_bytes != 2 && elem_bytes != 4)) {
        set_error("tre_repartition: null n_out, negative size or elem_bytes not 2 / 4");
        return TRE_E_ARG;
    }
    *n_out = 0;
    if (n_in == 0) return TRE_OK;
    if (d.rin == 0 && n_in > 1) {
        set_error("tre_repartition: a relation without promoted labels holds at most one tuple");
        return TRE_E_DUPKEY;
    }
    if ((d.rin > 0 && !keys_in) || !tiles_in || !ws || (reinterpret_cast<uintptr_t>(ws) & 255)) {
        set_error("tre_repartition: null keys / tiles / workspace, or workspace not 256-byte aligned");
        return TRE_E_ARG;
    }
    if (n_in * d.max_cover > int64_t(0xffffffffll) || n_in > int64_t(0x7fffffff)) {
        set_error("tre_repartition: too many tuples");
        return TRE_E_SHAPE;
    }
    const RpLayout L = rp_layout(d, n_in);
    if (ws_bytes < L.total) {
        set_error("tre_repartition: workspace too small");
        return TRE_E_WORKSPACE;
    }
    hipStream_t s = reinterpret_cast<hipStream_t>(stream);
    char* w = reinterpret_cast<char*>(ws);
    RpHeader* hdr = reinterpret_cast<RpHeader*>(w + L.hdr);
    int64_t* cnt = reinterpret_cast<int64_t*>(w + L.cnt);
    uint64_t* tk = reinterpret_cast<uint64_t*>(w + L.tk);
    uint32_t* src = reinterpret_cast<uint32_t*>(w + L.src);
    int32_t* seg_of = reinterpret_cast<int32_t*>(w + L.seg_of);
    uint64_t* seg_key = reinterpret_cast<uint64_t*>(w + L.seg_key);
    hipError_t e;
    // keys: sorted, unique and in range (the relation conventions)
    if ((e = launch_fill_zero(hdr, sizeof(RpHeader), s)) != hipSuccess) return dev_fail(e, "header");
    if (d.rin > 0) {
        int32_t radix[26];
        for (int i = 0, ka = 0; i < d.nl; i++)
            if (d.pin[i]) radix[ka++] = int32_t(d.ext[i] / d.tin[i]);
        if ((e = launch_validate(keys_in, n_in, d.rin, radix, &hdr->err, s)) != hipSuccess)
            return dev_fail(e, "validate");
    }
    k_rp_count<<<blocks_for(n_in + 1), kThreads, 0, s>>>(keys_in, n_in, d, cnt, hdr);
    if ((e = hipGetLastError()) != hipSuccess) return dev_fail(e, "count");
    if ((e = scan_exclusive_i64(cnt, cnt, n_in + 1, reinterpret_cast<int64_t*>(w + L.tmp), s)) != hipSuccess)
        return dev_fail(e, "scan");
    RpHeader h{};
    if ((e = hipMemcpyAsync(&h, hdr, sizeof(h), hipMemcpyDeviceToHost, s)) != hipSuccess ||
        (e = hipMemcpyAsync(&h.pairs, cnt + n_in, sizeof(int64_t), hipMemcpyDeviceToHost, s)) != hipSuccess ||
        (e = hipStreamSynchronize(s)) != hipSuccess)
        return dev_fail(e, "count read-back");
    if (h.err) {
        set_error("tre_repartition: source keys out of range, unsorted or repeated");
        return (h.err & 4) ? TRE_E_KEYRANGE : (h.err & 1) ? TRE_E_UNSORTED : TRE_E_DUPKEY;
    }
    const int64_t m = h.pairs;
    k_rp_expand<<<blocks_for(n_in), kThreads, 0, s>>>(keys_in, n_in, d, cnt, tk, src);
    if ((e = hipGetLastError()) != hipSuccess) return dev_fail(e, "expand");
    // the listing is in source order; sort it by target key unless that
    // order already has the target keys sorted (then the stable sort would
    // leave it as it is)
    if (h.unsorted) {
        if ((e = radix_sort_u64(tk, src, reinterpret_cast<uint64_t*>(w + L.tk_alt),
                                reinterpret_cast<uint32_t*>(w + L.src_alt), m, d.key_bits,
                                reinterpret_cast<int32_t*>(w + L.hist), reinterpret_cast<int32_t*>(w + L.tmp), s)) !=
            hipSuccess)
            return dev_fail(e, "sort");
        if (radix_result_in_alt(m, d.key_bits)) {
            tk = reinterpret_cast<uint64_t*>(w + L.tk_alt);
            src = reinterpret_cast<uint32_t*>(w + L.src_alt);
        }
    }
    k_rp_heads<<<blocks_for(m + 1), kThreads, 0, s>>>(tk, m, seg_of);
    if ((e = hipGetLastError()) != hipSuccess) return dev_fail(e, "heads");
    if ((e = scan_exclusive_i32(seg_of, seg_of, m + 1, reinterpret_cast<int32_t*>(w + L.tmp), s)) != hipSuccess)
        return dev_fail(e, "segments");
    k_rp_compact<<<blocks_for(m + 1), kThreads, 0, s>>>(tk, m, seg_of, seg_key, hdr);
    if ((e = hipGetLastError()) != hipSuccess) return dev_fail(e, "compact");
    if ((e = hipMemcpyAsync(&h, hdr, sizeof(h), hipMemcpyDeviceToHost, s)) != hipSuccess ||
        (e = hipStreamSynchronize(s)) != hipSuccess)
        return dev_fail(e, "target count read-back");
    *n_out = h.n_out;
    // in place: only a regrouping of whole source tiles, in source order,
    // with nothing missing, leaves the bytes where they are
    const bool in_place = tiles_out == tiles_in;
    if (in_place && !(d.regroup && !h.unsorted && m == n_in && n_in * d.te_in == h.n_out * d.te_out)) {
        set_error("tre_repartition: tiles_out == tiles_in needs every target tile to be its source tiles, "
                  "complete and in source order");
        return TRE_E_ARG;
    }
    if (h.n_out > out_cap) {
        set_error("tre_repartition: output capacity below the target tuple count");
        return TRE_E_CAPACITY;
    }
    if ((d.rout > 0 && !keys_out) || !tiles_out) {
        set_error("tre_repartition: null output buffers");
        return TRE_E_ARG;
    }
    if (in_place) {
        if (d.rout > 0) {
            k_rp_write_keys<<<blocks_for(h.n_out), kThreads, 0, s>>>(seg_key, h.n_out, d, keys_out);
            if ((e = hipGetLastError()) != hipSuccess) return dev_fail(e, "keys");
        }
        return TRE_OK;
    }
    // source tiles are disjoint, so they cover n_in x tile_elems_in target
    // positions; zero the targets only when that leaves some uncovered
    if (n_in * d.te_in < h.n_out * d.te_out &&
        (e = launch_fill_zero(tiles_out, size_t(h.n_out) * size_t(d.te_out) * size_t(elem_bytes), s)) != hipSuccess)
        return dev_fail(e, "zero fill");
    if (d.rout > 0) {
        k_rp_write_keys<<<blocks_for(h.n_out), kThreads, 0, s>>>(seg_key, h.n_out, d, keys_out);
        if ((e = hipGetLastError()) != hipSuccess) return dev_fail(e, "keys");
    }
    // pairs per workgroup: about 128 KB of chunks each (the boxes partition
    // the source tiles, so a pair averages n_in x tile_elems_in / m
    // elements), at most one pair per thread, chunk numbers within int32
    const int64_t avg_bytes = std::max<int64_t>(1, n_in * d.te_in * elem_bytes / m);
    int64_t per_wg = std::max<int64_t>(1, (int64_t(128) << 10) / avg_bytes);
    per_wg = std::min<int64_t>({per_wg, kRpPairs, std::max<int64_t>(1, (int64_t(1) << 30) / std::min(d.te_in, d.te_out))});
    const int64_t batches = (m + per_wg - 1) / per_wg;
    // 4096 workgroups fill 256 CUs twice over; the rest loop (k_rp_copy's batch loop)
    const unsigned grid = unsigned(std::min<int64_t>(batches, 4096));
    if (elem_bytes == 2)
        k_rp_copy<uint16_t><<<grid, kThreads, 0, s>>>(keys_in, reinterpret_cast<const uint16_t*>(tiles_in), tk, src,
                                                       seg_of, m, int32_t(per_wg), d,
                                                       reinterpret_cast<uint16_t*>(tiles_out));
    else
        k_rp_copy<uint32_t><<<grid, kThreads, 0, s>>>(keys_in, reinterpret_cast<const uint32_t*>(tiles_in), tk, src,
                                                       seg_of, m, int32_t(per_wg), d,
                                                       reinterpret_cast<uint32_t*>(tiles_out));
    if ((e = hipGetLastError()) != hipSuccess) return dev_fail(e, "copy");
    return TRE_OK;
}

}  // extern "C"
