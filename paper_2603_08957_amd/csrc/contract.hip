// Steps (2) and (3) of the tensor-relational EinSum (Sec. 5): the kernel K on
// every matched tile pair and the sum of the results per output key.
//
// Pairs arrive sorted by output key; a segment is the run of pairs of one
// key.  Segments are cut into work units of at most P pairs.  A workgroup
// owns one (unit, output block) and accumulates Sum_{pairs in unit} K(U, V)
// in registers, so no per-pair partial tile ever reaches memory.  A segment
// that fits one unit is written straight to W; the units of a longer segment
// write partial tiles that k_reduce sums in unit order (atomic-free, hence
// deterministic).
//
// K is the EinSum over the tile labels, W[b,m,n] += sum_k A[b,m,k] B[b,k,n];
// element offsets inside a tile come from per-role tables, so any label
// order / layout of the operand tiles is accepted.
//   KC_GEMM: 64x64 output block per 256-thread workgroup (2x2 waves of one
//            32x32 MFMA tile each), 32-deep K chunks staged in LDS, the next
//            two chunks' global loads in flight in registers;
//            fp32 -> v_mfma_f32_32x32x2_f32, bf16 -> v_mfma_f32_32x32x16_bf16.
//   KC_VEC : one output element per thread, fp32 FMA (scale, GEMV, dot).
#include "tre_internal.h"

#include <type_traits>

namespace tre {

namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef unsigned short u16x8 __attribute__((ext_vector_type(8)));
typedef float floatx16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

constexpr int kThreads = 256;

__device__ inline float ld_f(const float* p) { return *p; }
__device__ inline float ld_f(const uint16_t* p) { return __uint_as_float(uint32_t(*p) << 16); }

// ---------------------------------------------------------------- tables

// off[t] < 0: the plan's contraction kernel does not read table t (the
// GEMM class reads the A/B/W tables, the vector class the E/K ones, the
// 128x128 path none), so it is not written.
struct TableSet {
    Dims d[T_COUNT];
    int64_t off[T_COUNT];
};

__global__ void k_tables(TableSet ts, int32_t* __restrict__ out) {
    const int t = blockIdx.y;
    if (ts.off[t] < 0) return;
    const Dims& d = ts.d[t];
    int64_t cnt = 1;
    for (int i = 0; i < d.n; i++) cnt *= d.size[i];
    for (int64_t x = int64_t(blockIdx.x) * blockDim.x + threadIdx.x; x < cnt; x += int64_t(gridDim.x) * blockDim.x) {
        int64_t rem = x, o = 0;
        for (int i = d.n - 1; i >= 0; i--) {
            o += (rem % d.size[i]) * d.stride[i];
            rem /= d.size[i];
        }
        out[ts.off[t] + x] = int32_t(o);
    }
}

// ----------------------------------------------------------------- units

__global__ void k_seg_units(const int32_t* __restrict__ seg_start, int64_t n_w, int64_t p_unit,
                            int32_t* __restrict__ nunits, int32_t* __restrict__ nparts, int32_t* __restrict__ nsplit) {
    const int64_t s = int64_t(blockIdx.x) * blockDim.x + threadIdx.x;
    if (s > n_w) return;
    if (s == n_w) {
        nunits[s] = 0;
        nparts[s] = 0;
        nsplit[s] = 0;
        return;
    }
    const int64_t len = seg_start[s + 1] - seg_start[s];
    const int64_t u = (len + p_unit - 1) / p_unit;
    nunits[s] = int32_t(u);
    nparts[s] = u > 1 ? int32_t(u) : 0;
    nsplit[s] = u > 1 ? 1 : 0;
}

__global__ void k_fill_units(const int32_t* __restrict__ seg_start, int64_t n_w,
                             const int32_t* __restrict__ uoff, const int32_t* __restrict__ poff,
                             const int32_t* __restrict__ soff, Unit* __restrict__ units, int32_t* __restrict__ split,
                             WsHeader* hdr) {
    const int64_t s = int64_t(blockIdx.x) * blockDim.x + threadIdx.x;
    if (s > n_w) return;
    if (s == n_w) {
        hdr->n_units = uoff[n_w];
        hdr->n_parts = poff[n_w];
        hdr->n_split = soff[n_w];
        return;
    }
    const int32_t a = seg_start[s], b = seg_start[s + 1];
    const int32_t nu = uoff[s + 1] - uoff[s];
    // a split key is cut into nu units of equal length (within one pair)
    const int64_t len = int64_t(b) - a;
    for (int32_t j = 0; j < nu; j++) {
        Unit u;
        u.seg = int32_t(s);
        u.p0 = a + int32_t(len * j / nu);
        u.p1 = a + int32_t(len * (j + 1) / nu);
        u.slot = nu > 1 ? poff[s] + j : -1;
        units[uoff[s] + j] = u;
    }
    if (nu > 1) split[soff[s]] = int32_t(s);
}

// Longest units first: one workgroup reorders a unit table of at most
// kOrderMax entries by decreasing length (counting sort on the length, capped
// at kOrderBins - 1), so that the hardware's in-order dispatch of the
// contraction grid is a longest-processing-time-first schedule and the
// longest keys do not start in the last wave.  Each unit's sum does not depend
// on when it runs, so the order within a length class is left to the LDS
// atomics.
constexpr int kOrderMax = 4096, kOrderBins = 1024;

__global__ __launch_bounds__(kOrderBins) void k_order_units(Unit* __restrict__ units, const WsHeader* __restrict__ hdr) {
    __shared__ Unit buf[kOrderMax];
    __shared__ int32_t cnt[kOrderBins];
    const int32_t n = hdr->n_units;
    if (n < 2 || n > kOrderMax) return;
    const int t = threadIdx.x;
    auto bin = [](const Unit& u) { return kOrderBins - 1 - min(u.p1 - u.p0, kOrderBins - 1); };
    cnt[t] = 0;
    __syncthreads();
    for (int i = t; i < n; i += kOrderBins) {
        const Unit u = units[i];
        buf[i] = u;
        atomicAdd(&cnt[bin(u)], 1);
    }
    __syncthreads();
    const int32_t own = cnt[t];
    for (int off = 1; off < kOrderBins; off <<= 1) {
        const int32_t add = t >= off ? cnt[t - off] : 0;
        __syncthreads();
        cnt[t] += add;
        __syncthreads();
    }
    cnt[t] -= own;  // exclusive start of bin t
    __syncthreads();
    for (int i = t; i < n; i += kOrderBins) {
        const Unit u = buf[i];
        units[atomicAdd(&cnt[bin(u)], 1)] = u;
    }
}

// The unit table of at most kOrderMax keys in one workgroup: per key the
// unit count (keys longer than the cap cut into equal units), scans of the
// unit, partial-slot and split counts, the fill, and for the GEMM class the
// longest-first order (counting sort on the unit length, as k_order_units)
// -- one launch instead of up to six.  Each thread counts four consecutive
// keys; the fill then gives each thread whole units (a unit finds its key by
// binary search of the per-key unit offsets in LDS), so a cut key's units
// are written by many threads at once.  With `ts` non-null the workgroup also
// writes the tile offset tables first (small tables only, `tables`
// non-null), saving their launch.  With `dev_nw` the key count is the one the
// join wrote into the header (`n_w` is then an upper bound), so the launch
// needs no count from the host.
constexpr int kUnitsThreads = kOrderBins;
constexpr int kUnitsPer = kOrderMax / kUnitsThreads;
constexpr int64_t kUnitsTableMax = 16384;
static_assert(kUnitsTableMax < (1 << 16) && T_COUNT * kMaxDims <= kUnitsThreads, "table set-up in k_units_small");

// part_off[s]: the first partial slot of key s (n_w + 1 entries; k_reduce
// sums slots part_off[s] .. part_off[s + 1] - 1 of each split key).
__global__ __launch_bounds__(kUnitsThreads) void k_units_small(const int32_t* __restrict__ seg_start, int64_t n_w,
                                                                int64_t p_unit, int order, Unit* __restrict__ units,
                                                                int32_t* __restrict__ split,
                                                                int32_t* __restrict__ part_off,
                                                                WsHeader* __restrict__ hdr, TableSet ts,
                                                                int32_t* __restrict__ tables, int dev_nw) {
    __shared__ Unit buf[kOrderMax];
    __shared__ int32_t cnt[kOrderBins];
    __shared__ int32_t wsum[kUnitsThreads / 64];
    __shared__ int32_t key_uo[kOrderMax + 1], key_po[kOrderMax], key_a[kOrderMax + 1];
    const int t = threadIdx.x;
    if (dev_nw) n_w = min(n_w, hdr->n_w);  // n_w is then a bound; the key count is the join's
    if (tables) {
        // the table shapes through LDS: read from the kernel arguments with
        // dynamic indices they would be one dependent scalar load each
        constexpr int kWords = int(sizeof(TableSet) / sizeof(int32_t));
        static_assert(sizeof(TableSet) % sizeof(int64_t) == 0, "TableSet words");
        __shared__ int64_t s_ts_raw[sizeof(TableSet) / sizeof(int64_t)];
        __shared__ uint32_t s_magic[T_COUNT][kMaxDims];
        __shared__ int32_t s_first[T_COUNT + 1];
        for (int i = t; i < kWords; i += kUnitsThreads)
            reinterpret_cast<int32_t*>(s_ts_raw)[i] = reinterpret_cast<const int32_t*>(&ts)[i];
        __syncthreads();
        const TableSet& s_ts = *reinterpret_cast<const TableSet*>(s_ts_raw);
        // Every used table holds at most kUnitsTableMax < 2^16 entries, so
        // an index and every size are below 2^16, and x / d = umulhi(x, m)
        // with m = ceil(2^32 / d) exactly (x * (m d - 2^32) < 2^32); m = 0
        // stands for d <= 1.
        if (t < T_COUNT * kMaxDims) {
            const int k = t / kMaxDims, i = t % kMaxDims;
            const uint32_t d = i < s_ts.d[k].n ? uint32_t(s_ts.d[k].size[i]) : 1u;
            s_magic[k][i] = d > 1 ? 0xffffffffu / d + 1u : 0u;
        }
        if (t == 0) {
            // the used tables' entries, numbered one after another
            int32_t f = 0;
            for (int k = 0; k < T_COUNT; k++) {
                s_first[k] = f;
                if (s_ts.off[k] < 0) continue;
                int32_t c = 1;
                for (int i = 0; i < s_ts.d[k].n; i++) c *= s_ts.d[k].size[i];
                f += c;
            }
            s_first[T_COUNT] = f;
        }
        __syncthreads();
        const int32_t total = s_first[T_COUNT];
        for (int32_t x = t; x < total; x += kUnitsThreads) {
            int k = 0;
            while (x >= s_first[k + 1]) k++;
            const Dims& d = s_ts.d[k];
            const int32_t xi = x - s_first[k];
            uint32_t rem = uint32_t(xi);
            int32_t o = 0;
            for (int i = d.n - 1; i >= 0; i--) {
                const uint32_t m = s_magic[k][i];
                const uint32_t q = m ? __umulhi(rem, m) : rem;
                o += int32_t(rem - q * uint32_t(d.size[i])) * d.stride[i];
                rem = q;
            }
            tables[s_ts.off[k] + xi] = o;
        }
    }
    int32_t nu[kUnitsPer], a0[kUnitsPer], su = 0, sp = 0, ss = 0;
#pragma unroll
    for (int j = 0; j < kUnitsPer; j++) {
        const int64_t s = int64_t(t) * kUnitsPer + j;
        nu[j] = 0;
        a0[j] = 0;
        if (s < n_w) {
            a0[j] = seg_start[s];
            const int32_t len = seg_start[s + 1] - a0[j];
            nu[j] = len <= 0     ? 0
                    : p_unit >= len ? 1
                                    : int32_t((uint32_t(len) + uint32_t(p_unit) - 1) / uint32_t(p_unit));
        }
        su += nu[j];
        sp += nu[j] > 1 ? nu[j] : 0;
        ss += nu[j] > 1 ? 1 : 0;
    }
    int32_t n_units, n_parts, n_split;
    int32_t uo = block_scan_excl<kUnitsThreads>(su, wsum, &n_units);
    int32_t po = block_scan_excl<kUnitsThreads>(sp, wsum, &n_parts);
    int32_t so = block_scan_excl<kUnitsThreads>(ss, wsum, &n_split);
#pragma unroll
    for (int j = 0; j < kUnitsPer; j++) {
        const int64_t s = int64_t(t) * kUnitsPer + j;
        if (s >= n_w) continue;
        part_off[s] = po;
        key_uo[s] = uo;
        key_po[s] = po;
        key_a[s] = a0[j];
        if (nu[j] > 1) {
            split[so++] = int32_t(s);
            po += nu[j];
        }
        uo += nu[j];
    }
    if (t == 0) {
        key_uo[n_w] = n_units;
        key_a[n_w] = seg_start[n_w];
        part_off[n_w] = n_parts;
        hdr->n_units = n_units;
        hdr->n_parts = n_parts;
        hdr->n_split = n_split;
    }
    __syncthreads();
    const bool in_lds = order && n_units >= 2 && n_units <= kOrderMax;
    for (int32_t i = t; i < n_units; i += kUnitsThreads) {
        // the key of unit i: the last s with key_uo[s] <= i (keys without
        // pairs own no unit and are skipped by taking the last such s)
        int32_t lo = 0, hi = int32_t(n_w) - 1;
        while (lo < hi) {
            const int32_t m = (lo + hi + 1) >> 1;
            if (key_uo[m] <= i) lo = m; else hi = m - 1;
        }
        const int32_t k = key_uo[lo + 1] - key_uo[lo];
        const int32_t q = i - key_uo[lo];
        const int32_t a = key_a[lo];
        const uint32_t len = uint32_t(key_a[lo + 1] - a);
        Unit u;
        u.seg = lo;
        if (k == 1) {
            u.p0 = a;
            u.p1 = a + int32_t(len);
            u.slot = -1;
        } else {
            // a cut key: k units of equal length (within one pair)
            const uint64_t x0 = uint64_t(len) * uint32_t(q), x1 = x0 + len;
            u.p0 = a + int32_t(x1 >> 32 ? x0 / uint32_t(k) : uint32_t(x0) / uint32_t(k));
            u.p1 = a + int32_t(x1 >> 32 ? x1 / uint32_t(k) : uint32_t(x1) / uint32_t(k));
            u.slot = key_po[lo] + q;
        }
        if (in_lds) buf[i] = u;
        else units[i] = u;
    }
    if (!in_lds) return;
    // longest first (unit lengths capped at kOrderBins - 1; order within a
    // length class is free: a unit's sum does not depend on when it runs)
    // (units mostly share one or two lengths, and LDS atomics on one
    // address serialise: the lanes of a wavefront with the leading lane's
    // length take one atomic together, twice; any lanes left take one each)
    auto bin = [](const Unit& u) { return kOrderBins - 1 - min(u.p1 - u.p0, kOrderBins - 1); };
    const int lane = t & 63;
    const uint64_t below = (uint64_t(1) << lane) - 1;
    // counting pass (place false): adds the lane to its bin's count;
    // placing pass: returns the lane's slot from its bin's running start
    auto wave_rank = [&](bool valid, int b, bool place) {
        uint64_t todo = __ballot(valid);
        int32_t rank = 0;
        for (int round = 0; round < 2 && todo; round++) {
            const int leader = __ffsll((unsigned long long)todo) - 1;
            const int lb = __shfl(b, leader, 64);
            const uint64_t m = __ballot(valid && b == lb);
            int32_t base = 0;
            if (lane == leader) base = atomicAdd(&cnt[lb], __popcll(m));
            base = __shfl(base, leader, 64);
            if (valid && b == lb) rank = base + __popcll(m & below);
            todo &= ~m;
        }
        if ((todo >> lane) & 1) rank = atomicAdd(&cnt[b], 1);
        return place ? rank : 0;
    };
    cnt[t] = 0;
    __syncthreads();
    for (int i0 = t - lane; i0 < n_units; i0 += kUnitsThreads) {
        const int i = i0 + lane;
        (void)wave_rank(i < n_units, i < n_units ? bin(buf[i]) : 0, false);
    }
    __syncthreads();
    int32_t total;
    const int32_t start = block_scan_excl<kUnitsThreads>(cnt[t], wsum, &total);
    __syncthreads();
    cnt[t] = start;
    __syncthreads();
    for (int i0 = t - lane; i0 < n_units; i0 += kUnitsThreads) {
        const int i = i0 + lane;
        const bool valid = i < n_units;
        const Unit u = valid ? buf[i] : Unit{};
        const int32_t r = wave_rank(valid, valid ? bin(u) : 0, true);
        if (valid) units[r] = u;
    }
}

// U-range units (see launch_range_units): unit r * n_w + s covers the pairs of
// key s with U index in [r * n_u / R, (r + 1) * n_u / R); within a key the
// pairs are sorted by U index, so that is one contiguous run, found by binary
// search.  Dispatch order is range-major, so workgroups running together use
// the same slice of U.
__global__ void k_range_units(const int32_t* __restrict__ seg_start, const int32_t* __restrict__ pu, int64_t n_w,
                              int64_t n_u, int32_t R, Unit* __restrict__ units, int32_t* __restrict__ part_off,
                              int32_t* __restrict__ split, WsHeader* hdr) {
    const int64_t idx = int64_t(blockIdx.x) * blockDim.x + threadIdx.x;
    if (idx <= n_w) {
        part_off[idx] = int32_t(idx * R);
        if (idx < n_w) split[idx] = int32_t(idx);
    }
    if (idx == 0) {
        hdr->n_units = int64_t(R) * n_w;
        hdr->n_parts = int64_t(R) * n_w;
        hdr->n_split = n_w;
    }
    if (idx >= int64_t(R) * n_w) return;
    const int32_t r = int32_t(idx / n_w);
    const int32_t s = int32_t(idx % n_w);
    const int32_t lo = seg_start[s], hi = seg_start[s + 1];
    auto lower = [&](int64_t key) {
        int32_t a = lo, b = hi;
        while (a < b) {
            const int32_t m = (a + b) >> 1;
            if (pu[m] < key) a = m + 1; else b = m;
        }
        return a;
    };
    Unit u;
    u.seg = s;
    u.p0 = lower(int64_t(r) * n_u / R);
    u.p1 = r + 1 == R ? hi : lower(int64_t(r + 1) * n_u / R);
    u.slot = s * R + r;
    units[idx] = u;
}

// ------------------------------------------------------------------ GEMM

struct GemmArgs {
    const void* A;
    const void* B;
    const int32_t* pa;
    const int32_t* pb;
    int64_t a_elems, b_elems, w_elems;
    const int32_t *tAM, *tAK, *tBK, *tBN, *tWM, *tWN, *tAB, *tBB, *tWB;
    int32_t M, N, K, nB, mblocks, nblocks;
    int32_t vec_a, vec_b;
    const Unit* units;
    const WsHeader* hdr;
    float* W;
    float* partials;
};

constexpr int kBM = 64, kBN = 64, kBK = 32;

// LDS row pitches (elements).  fp32 [row][k] rows of 36 floats are 16-byte
// aligned and a 16-lane b128 read of 16 rows at one k offset hits 16
// distinct 4-bank groups; [k][row] rows are padded by one element.
template <typename T>
struct LdsPitch;
template <>
struct LdsPitch<float> {
    static constexpr int kfast = kBK + 4;   // [row][k]
    static constexpr int rfast = kBM + 1;   // [k][row]
};
template <>
struct LdsPitch<uint16_t> {
    static constexpr int kfast = kBK + 8;   // keeps 16-byte row alignment for 8-wide reads
    static constexpr int rfast = kBM + 2;
};

// 8 consecutive elements from a 16-byte aligned address.
__device__ inline void load8(float* v, const float* src) {
    const uint4 a = reinterpret_cast<const uint4*>(src)[0], b = reinterpret_cast<const uint4*>(src)[1];
    __builtin_memcpy(v, &a, 16);
    __builtin_memcpy(v + 4, &b, 16);
}
__device__ inline void load8(uint16_t* v, const uint16_t* src) {
    const uint4 a = *reinterpret_cast<const uint4*>(src);
    __builtin_memcpy(v, &a, 16);
}

// One thread's share (8 elements) of a 64 x 32 (rows x k) chunk of one
// operand, held in registers between its global load and its LDS store so
// the next chunk's loads overlap the current chunk's MFMAs.
//   KF: the operand's unit-stride dim is k (LDS [row][k]); else rows ([k][row]).
template <typename T, bool KF>
struct Staged {
    T v[8];
    // tR: element offsets of the block's rows (local index, rows < nr valid);
    // tK: offsets of the contracted index (both tables in LDS)
    __device__ void load(const T* __restrict__ base, const int32_t* tR, const int32_t* tK, int nr, int k0, int K,
                         bool vec) {
        const int t = threadIdx.x;
        if (KF) {
            const int lr = t >> 2, gk = k0 + (t & 3) * 8;
            if (vec && lr < nr && gk + 8 <= K) {
                load8(v, base + tR[lr] + tK[gk]);
            } else {
#pragma unroll
                for (int j = 0; j < 8; j++) v[j] = (lr < nr && gk + j < K) ? base[tR[lr] + tK[gk + j]] : T(0);
            }
        } else {
            const int gk = k0 + (t >> 3), lr = (t & 7) * 8;
            if (vec && gk < K && lr + 8 <= nr) {
                load8(v, base + tK[gk] + tR[lr]);
            } else {
#pragma unroll
                for (int j = 0; j < 8; j++) v[j] = (gk < K && lr + j < nr) ? base[tK[gk] + tR[lr + j]] : T(0);
            }
        }
    }
    __device__ void store(T* __restrict__ lds) const {
        const int t = threadIdx.x;
        if (KF) {
            T* d = lds + (t >> 2) * LdsPitch<T>::kfast + (t & 3) * 8;
            if constexpr (sizeof(T) == 4) {
                reinterpret_cast<f32x4*>(d)[0] = f32x4{v[0], v[1], v[2], v[3]};
                reinterpret_cast<f32x4*>(d)[1] = f32x4{v[4], v[5], v[6], v[7]};
            } else {
#pragma unroll
                for (int j = 0; j < 8; j++) d[j] = v[j];
            }
        } else {
            T* d = lds + (t >> 3) * LdsPitch<T>::rfast + (t & 7) * 8;
#pragma unroll
            for (int j = 0; j < 8; j++) d[j] = v[j];
        }
    }
};

template <bool KF>
__device__ inline bf16x8 frag_bf16(const uint16_t* lds, int row, int k) {
    u16x8 v;
    if (KF) {
        v = *reinterpret_cast<const u16x8*>(lds + row * LdsPitch<uint16_t>::kfast + k);
    } else {
#pragma unroll
        for (int j = 0; j < 8; j++) v[j] = lds[(k + j) * LdsPitch<uint16_t>::rfast + row];
    }
    return __builtin_bit_cast(bf16x8, v);
}

// fp32 operand values of 4 consecutive MFMA k-steps (k = k4 .. k4 + 3) for
// the lane's row: one 16-byte read from [row][k], four reads from [k][row].
template <bool KF>
__device__ inline f32x4 frag4_f32(const float* lds, int row, int k4) {
    if (KF) return *reinterpret_cast<const f32x4*>(lds + row * LdsPitch<float>::kfast + k4);
    f32x4 v;
#pragma unroll
    for (int j = 0; j < 4; j++) v[j] = lds[(k4 + j) * LdsPitch<float>::rfast + row];
    return v;
}

// PF: load two chunks ahead (worth it for long units; short units keep the
// registers and get more workgroups per CU instead).
template <typename T, bool AK, bool BK, bool PF>
__global__ __launch_bounds__(kThreads) void k_gemm(GemmArgs g) {
    const int64_t n_units = g.hdr->n_units;
    if (blockIdx.x >= n_units) return;
    int y = blockIdx.y;
    const int nblk = y % g.nblocks;
    y /= g.nblocks;
    const int mblk = y % g.mblocks;
    const int b = y / g.mblocks;
    const int m0 = mblk * kBM, n0 = nblk * kBN;

    constexpr int kAs = AK ? kBM * LdsPitch<T>::kfast : kBK * LdsPitch<T>::rfast;
    constexpr int kBs = BK ? kBN * LdsPitch<T>::kfast : kBK * LdsPitch<T>::rfast;
    __shared__ __attribute__((aligned(16))) T As[kAs];
    __shared__ __attribute__((aligned(16))) T Bs[kBs];

    const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
    const int wm = w >> 1, wn = w & 1;
    floatx16 acc;
#pragma unroll
    for (int r = 0; r < 16; r++) acc[r] = 0.f;

    // offset tables of this block's rows and of the contracted index, copied
    // to LDS once so the loads of the chunk loop depend on no global read
    extern __shared__ int32_t tabs[];  // [kBM rows of A][kBN rows of B][K of A][K of B]
    int32_t* sAM = tabs;
    int32_t* sBN = tabs + kBM;
    int32_t* sAK = tabs + kBM + kBN;
    int32_t* sBK = sAK + g.K;
    for (int i = threadIdx.x; i < kBM; i += kThreads) sAM[i] = m0 + i < g.M ? g.tAM[m0 + i] : 0;
    for (int i = threadIdx.x; i < kBN; i += kThreads) sBN[i] = n0 + i < g.N ? g.tBN[n0 + i] : 0;
    for (int i = threadIdx.x; i < g.K; i += kThreads) {
        sAK[i] = g.tAK[i];
        sBK[i] = g.tBK[i];
    }
    __syncthreads();
    const int nra = min(kBM, g.M - m0), nrb = min(kBN, g.N - n0);

    const T* Ag = reinterpret_cast<const T*>(g.A);
    const T* Bg = reinterpret_cast<const T*>(g.B);
    const int32_t offAB = g.tAB[b], offBB = g.tBB[b];
    // output offset of this lane's accumulator r (the block is fixed); short
    // units (no prefetch) keep them in registers across units
    const int n = n0 + wn * 32 + (lane & 31);
    auto w_offset = [&](int r) {
        const int m = m0 + wm * 32 + (r >> 2) * 8 + (lane >> 5) * 4 + (r & 3);
        return (m < g.M && n < g.N) ? g.tWB[b] + g.tWM[m] + g.tWN[n] : -1;
    };
    int32_t wofs[PF ? 1 : 16];
    if constexpr (!PF) {
#pragma unroll
        for (int r = 0; r < 16; r++) wofs[r] = w_offset(r);
    }
    const int kcn = (g.K + kBK - 1) / kBK;
    // without prefetch (short units) the grid may be smaller than the unit
    // count: a workgroup takes units blockIdx.x, blockIdx.x + gridDim.x, ...
    // (tables loaded once); with prefetch the grid covers every unit
    const int64_t unit_step = PF ? n_units : int64_t(gridDim.x);
    for (int64_t unit_id = blockIdx.x; unit_id < n_units; unit_id += unit_step) {
        const Unit un = g.units[unit_id];
#pragma unroll
        for (int r = 0; r < 16; r++) acc[r] = 0.f;
        // chunk c of the unit: pair p0 + c / kcn, k offset (c % kcn) * kBK; with
        // PF two chunks are loaded ahead into two register sets used alternately
        // (the LDS tile stays single, so many workgroups fit on a CU)
        const int total = (un.p1 - un.p0) * kcn;
        Staged<T, AK> sa[PF ? 2 : 1];
        Staged<T, BK> sb[PF ? 2 : 1];
        auto load = [&](int c, auto slot) {
            constexpr int q = decltype(slot)::value;
            const int p = un.p0 + c / kcn, k0 = (c % kcn) * kBK;
            sa[q].load(Ag + int64_t(g.pa[p]) * g.a_elems + offAB, sAM, sAK, nra, k0, g.K, g.vec_a);
            sb[q].load(Bg + int64_t(g.pb[p]) * g.b_elems + offBB, sBN, sBK, nrb, k0, g.K, g.vec_b);
        };
        const int row = lane & 31, half = lane >> 5;
        auto step = [&](int c, auto slot) {
            constexpr int q = decltype(slot)::value;
            if (!PF) load(c, slot);
            sa[q].store(As);
            sb[q].store(Bs);
            __syncthreads();
            if (PF && c + 2 < total) load(c + 2, slot);
            if constexpr (sizeof(T) == 4) {
                // k-steps are taken in the order k = 16 half + s (s = 0 .. 15) in
                // both operands, so a lane's k run is contiguous
#pragma unroll
                for (int s4 = 0; s4 < kBK / 2; s4 += 4) {
                    const f32x4 a = frag4_f32<AK>(As, wm * 32 + row, 16 * half + s4);
                    const f32x4 bb = frag4_f32<BK>(Bs, wn * 32 + row, 16 * half + s4);
#pragma unroll
                    for (int j = 0; j < 4; j++) acc = __builtin_amdgcn_mfma_f32_32x32x2f32(a[j], bb[j], acc, 0, 0, 0);
                }
            } else {
#pragma unroll
                for (int ks = 0; ks < kBK; ks += 16) {
                    bf16x8 a = frag_bf16<AK>(reinterpret_cast<const uint16_t*>(As), wm * 32 + row, ks + half * 8);
                    bf16x8 bb = frag_bf16<BK>(reinterpret_cast<const uint16_t*>(Bs), wn * 32 + row, ks + half * 8);
                    acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, bb, acc, 0, 0, 0);
                }
            }
            __syncthreads();
        };
        using S0 = std::integral_constant<int, 0>;
        using S1 = std::integral_constant<int, PF ? 1 : 0>;
        if (PF && total > 0) load(0, S0{});
        if (PF && total > 1) load(1, S1{});
        for (int c = 0; c < total; c += 2) {
            step(c, S0{});
            if (c + 1 < total) step(c + 1, S1{});
        }
        float* out = un.slot < 0 ? g.W + int64_t(un.seg) * g.w_elems : g.partials + int64_t(un.slot) * g.w_elems;
#pragma unroll
        for (int r = 0; r < 16; r++) {
            const int32_t o = PF ? w_offset(r) : wofs[r];
            if (o >= 0) out[o] = acc[r];
        }
    }
}

// ------------------------------------------------------------------- VEC
//
// Vector class (scale, batched GEMV, dot): W[e] += sum_k U[eu(e) + ku(k)] *
// V[ev(e) + kv(k)] per pair.  A thread owns EPT consecutive W elements, loaded
// as one 16-byte vector when the plan shows the U offsets (and V's, or V is
// the same scalar for the whole group) run contiguously in aligned groups; a
// unit needing fewer than 256 threads shares its workgroup with other units.
// The contracted-index tables sit in LDS; for K <= 2 the pair loop is unrolled
// by four so four tiles are in flight per thread.  A workgroup first copies
// the pair indices of its units' span into LDS (their pairs are consecutive;
// up to kVecSpan of them), so the tile loads of a group of pairs wait for no
// index load from memory; when a pair's V factor is one scalar (y_scalar),
// its value is staged too and only the U tiles are loaded per pair (the
// attention projections, one unit of about 38 pairs per workgroup: 0.131 ->
// 0.082 ms each).

struct VecArgs {
    const void* U;
    const void* V;
    const int32_t* pu;
    const int32_t* pv;
    int64_t u_elems, v_elems, w_elems;
    const int32_t *tEU, *tEV, *tKU, *tKV;
    int32_t K;
    int32_t tpu;  // threads per unit (power of two when several units share a block)
    int32_t upb;  // units per block
    const Unit* units;
    const WsHeader* hdr;
    float* W;  // bf16 bits when w_bf16 (partials stay fp32)
    float* partials;
    int32_t w_bf16;
    int32_t y_scalar;  // V broadcast, K = 1 and one-element V tiles: a pair's factor is V[pv]
};

constexpr int kVecMaxK = 2048;

template <typename T, int EPT>
__device__ inline void load_vec(const T* p, float (&x)[EPT]) {
    if constexpr (EPT == 1) {
        x[0] = ld_f(p);
    } else if constexpr (sizeof(T) == 4 && EPT == 4) {
        const float4 v = *reinterpret_cast<const float4*>(p);
        x[0] = v.x; x[1] = v.y; x[2] = v.z; x[3] = v.w;
    } else {
        static_assert(sizeof(T) == 2 && EPT == 8, "unsupported vector width");
        const uint4 v = *reinterpret_cast<const uint4*>(p);
        const uint32_t w[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
        for (int i = 0; i < 4; i++) {
            x[2 * i] = __uint_as_float(w[i] << 16);
            x[2 * i + 1] = __uint_as_float(w[i] & 0xffff0000u);
        }
    }
}

constexpr int kVecSpan = 512;

template <typename T, int EPT, bool VB, int PU>
__global__ __launch_bounds__(kThreads) void k_vec(VecArgs a) {
    __shared__ int32_t sKU[kVecMaxK], sKV[kVecMaxK];
    __shared__ int32_t sPU[kVecSpan], sPV[kVecSpan];
    __shared__ float sY[VB ? kVecSpan : 1];
    const bool lds_tables = a.K <= kVecMaxK;
    if (lds_tables) {
        for (int k = threadIdx.x; k < a.K; k += kThreads) {
            sKU[k] = a.tKU[k];
            sKV[k] = a.tKV[k];
        }
        __syncthreads();
    }
    const int64_t unit_id = int64_t(blockIdx.x) * a.upb + (a.upb > 1 ? threadIdx.x / a.tpu : 0);
    const int64_t ti = a.upb > 1 ? threadIdx.x % a.tpu : int64_t(blockIdx.y) * kThreads + threadIdx.x;
    const int64_t e0 = ti * EPT;
    const int64_t n_units = a.hdr->n_units;
    // the staged span of pairs (empty: none staged); every thread reaches
    // the barrier (the tests before it are uniform over the workgroup)
    const int64_t u0 = int64_t(blockIdx.x) * a.upb;
    if (u0 >= n_units) return;
    const int32_t s0 = a.units[u0].p0;
    int32_t s1 = a.units[min<int64_t>(u0 + a.upb, n_units) - 1].p1;
    if (s1 < s0 || s1 - s0 > kVecSpan) s1 = s0;
    for (int i = threadIdx.x; i < s1 - s0; i += kThreads) {
        const int32_t v = a.pv[s0 + i];
        sPU[i] = a.pu[s0 + i];
        sPV[i] = v;
        if constexpr (VB)
            if (a.y_scalar) sY[i] = ld_f(reinterpret_cast<const T*>(a.V) + v);
    }
    __syncthreads();
    if (unit_id >= n_units || e0 >= a.w_elems) return;
    const Unit un = a.units[unit_id];
    const T* U = reinterpret_cast<const T*>(a.U);
    const T* V = reinterpret_cast<const T*>(a.V);
    const int32_t eu = a.tEU[e0], ev = a.tEV[e0];
    const int32_t* kU = lds_tables ? sKU : a.tKU;
    const int32_t* kV = lds_tables ? sKV : a.tKV;
    float acc[EPT];
#pragma unroll
    for (int i = 0; i < EPT; i++) acc[i] = 0.f;
    auto pair_step = [&](const T* ub, const T* vb, int k) {
        float x[EPT];
        load_vec<T, EPT>(ub + kU[k], x);
        if constexpr (VB) {
            const float y = ld_f(vb + kV[k]);
#pragma unroll
            for (int i = 0; i < EPT; i++) acc[i] = fmaf(x[i], y, acc[i]);
        } else {
            float y[EPT];
            load_vec<T, EPT>(vb + kV[k], y);
#pragma unroll
            for (int i = 0; i < EPT; i++) acc[i] = fmaf(x[i], y[i], acc[i]);
        }
    };
    // the unit's pairs, their indices read through get_u / get_v
    auto run_pairs = [&](auto get_u, auto get_v) {
        int p = un.p0;
        if constexpr (PU > 1) {
            for (; p + PU <= un.p1; p += PU) {
                const T* ub[PU];
                const T* vb[PU];
#pragma unroll
                for (int j = 0; j < PU; j++) {
                    ub[j] = U + int64_t(get_u(p + j)) * a.u_elems + eu;
                    vb[j] = V + int64_t(get_v(p + j)) * a.v_elems + ev;
                }
                for (int k = 0; k < a.K; k++)
#pragma unroll
                    for (int j = 0; j < PU; j++) pair_step(ub[j], vb[j], k);
            }
        }
        for (; p < un.p1; p++) {
            const T* ub = U + int64_t(get_u(p)) * a.u_elems + eu;
            const T* vb = V + int64_t(get_v(p)) * a.v_elems + ev;
#pragma unroll 4
            for (int k = 0; k < a.K; k++) pair_step(ub, vb, k);
        }
    };
    const bool staged = un.p0 >= s0 && un.p1 <= s1;
    if (VB && staged && a.y_scalar) {
        // the staged factors: only the U tiles are loaded (same order of
        // the sums as pair_step's)
        const int32_t ku0 = kU[0];
        int p = un.p0;
        if constexpr (PU > 1) {
            for (; p + PU <= un.p1; p += PU) {
                float x[PU][EPT];
#pragma unroll
                for (int j = 0; j < PU; j++) load_vec<T, EPT>(U + int64_t(sPU[p + j - s0]) * a.u_elems + eu + ku0, x[j]);
#pragma unroll
                for (int j = 0; j < PU; j++) {
                    const float y = sY[p + j - s0];
#pragma unroll
                    for (int i = 0; i < EPT; i++) acc[i] = fmaf(x[j][i], y, acc[i]);
                }
            }
        }
        for (; p < un.p1; p++) {
            float x[EPT];
            load_vec<T, EPT>(U + int64_t(sPU[p - s0]) * a.u_elems + eu + ku0, x);
            const float y = sY[p - s0];
#pragma unroll
            for (int i = 0; i < EPT; i++) acc[i] = fmaf(x[i], y, acc[i]);
        }
    } else if (staged) {
        run_pairs([&](int q) { return sPU[q - s0]; }, [&](int q) { return sPV[q - s0]; });
    } else {
        run_pairs([&](int q) { return a.pu[q]; }, [&](int q) { return a.pv[q]; });
    }
    if (a.w_bf16 && un.slot < 0) {
        uint16_t* o = reinterpret_cast<uint16_t*>(a.W) + int64_t(un.seg) * a.w_elems + e0;
        if constexpr (EPT % 4 == 0) {
#pragma unroll
            for (int i = 0; i < EPT; i += 4) {
                ushort4 v;
                v.x = f32_to_bf16_rne(acc[i]);
                v.y = f32_to_bf16_rne(acc[i + 1]);
                v.z = f32_to_bf16_rne(acc[i + 2]);
                v.w = f32_to_bf16_rne(acc[i + 3]);
                *reinterpret_cast<ushort4*>(o + i) = v;
            }
        } else {
#pragma unroll
            for (int i = 0; i < EPT; i++) o[i] = f32_to_bf16_rne(acc[i]);
        }
        return;
    }
    float* out = un.slot < 0 ? a.W + int64_t(un.seg) * a.w_elems : a.partials + int64_t(un.slot) * a.w_elems;
    if constexpr (EPT == 1) {
        out[e0] = acc[0];
    } else {
#pragma unroll
        for (int i = 0; i < EPT; i += 4)
            *reinterpret_cast<float4*>(out + e0 + i) = make_float4(acc[i], acc[i + 1], acc[i + 2], acc[i + 3]);
    }
}

template <typename T, int EPT>
hipError_t vec_dispatch(const Plan& p, const VecArgs& a, dim3 grid, hipStream_t s) {
    const bool pu4 = p.nK <= 2;
    const dim3 block{unsigned(kThreads)};
    if (p.vec_vbcast) return pu4 ? launch_k(k_vec<T, EPT, true, 4>, grid, block, 0, s, a)
                                 : launch_k(k_vec<T, EPT, true, 1>, grid, block, 0, s, a);
    return pu4 ? launch_k(k_vec<T, EPT, false, 4>, grid, block, 0, s, a)
               : launch_k(k_vec<T, EPT, false, 1>, grid, block, 0, s, a);
}

// ---------------------------------------------------------------- reduce

constexpr int kReduceBatch = 8;

__global__ __launch_bounds__(kThreads) void k_reduce(const int32_t* __restrict__ split, const WsHeader* hdr,
                                                     const int32_t* __restrict__ poff, const float* __restrict__ parts,
                                                     float* __restrict__ W, int64_t w_elems, int32_t w_bf16) {
    const int64_t x = blockIdx.x;
    if (x >= hdr->n_split) return;
    const int32_t s = split[x];
    const int32_t first = poff[s], cnt = poff[s + 1] - poff[s];
    if (w_elems % 4 == 0) {
        // 16-byte lanes; partials are read once, so they bypass L2 retention
        // (a bf16 W takes the four sums of a lane as one 8-byte store)
        const int64_t q = w_elems / 4;
        for (int64_t e = int64_t(blockIdx.y) * kThreads + threadIdx.x; e < q; e += int64_t(gridDim.y) * kThreads) {
            const f32x4* src = reinterpret_cast<const f32x4*>(parts) + int64_t(first) * q + e;
            f32x4 acc = {0.f, 0.f, 0.f, 0.f};
            int j = 0;
            // eight partials in flight, added in slot order
            for (; j + kReduceBatch <= cnt; j += kReduceBatch) {
                f32x4 v[kReduceBatch];
#pragma unroll
                for (int i = 0; i < kReduceBatch; i++) v[i] = __builtin_nontemporal_load(src + int64_t(j + i) * q);
#pragma unroll
                for (int i = 0; i < kReduceBatch; i++) acc += v[i];
            }
            for (; j < cnt; j++) acc += __builtin_nontemporal_load(src + int64_t(j) * q);
            if (w_bf16) {
                const uint32_t lo = uint32_t(f32_to_bf16_rne(acc[0])) | (uint32_t(f32_to_bf16_rne(acc[1])) << 16);
                const uint32_t hi = uint32_t(f32_to_bf16_rne(acc[2])) | (uint32_t(f32_to_bf16_rne(acc[3])) << 16);
                reinterpret_cast<uint2*>(W)[int64_t(s) * q + e] = make_uint2(lo, hi);
            } else {
                reinterpret_cast<f32x4*>(W)[int64_t(s) * q + e] = acc;
            }
        }
        return;
    }
    for (int64_t e = int64_t(blockIdx.y) * kThreads + threadIdx.x; e < w_elems; e += int64_t(gridDim.y) * kThreads) {
        const float* src = parts + int64_t(first) * w_elems + e;
        float acc = 0.f;
        int j = 0;
        for (; j + kReduceBatch <= cnt; j += kReduceBatch) {
            float v[kReduceBatch];
#pragma unroll
            for (int i = 0; i < kReduceBatch; i++) v[i] = src[int64_t(j + i) * w_elems];
#pragma unroll
            for (int i = 0; i < kReduceBatch; i++) acc += v[i];
        }
        for (; j < cnt; j++) acc += src[int64_t(j) * w_elems];
        if (w_bf16) reinterpret_cast<uint16_t*>(W)[int64_t(s) * w_elems + e] = f32_to_bf16_rne(acc);
        else W[int64_t(s) * w_elems + e] = acc;
    }
}

// ----------------------------------------------------------- outputs

struct Unpack {
    int32_t n;
    int32_t bits[26];
};

// (dn: the counts from the join's header, the host's being bounds)
__global__ void k_write_keys(const uint64_t* __restrict__ seg_key, int64_t n_w, Unpack up, int32_t* __restrict__ out,
                             const WsHeader* __restrict__ dn) {
    const int64_t s = int64_t(blockIdx.x) * blockDim.x + threadIdx.x;
    if (dn) n_w = min(n_w, dn->n_w);
    if (s >= n_w) return;
    uint64_t k = seg_key[s];
    for (int c = up.n - 1; c >= 0; c--) {
        const int b = up.bits[c];
        out[s * up.n + c] = int32_t(b ? (k & ((uint64_t(1) << b) - 1)) : 0);
        k = b < 64 ? (k >> b) : 0;
    }
}

__global__ void k_write_pairs(const int32_t* __restrict__ pu, const int32_t* __restrict__ pv, int64_t n,
                              int32_t* __restrict__ out, const WsHeader* __restrict__ dn) {
    const int64_t p = int64_t(blockIdx.x) * blockDim.x + threadIdx.x;
    if (dn) n = min(n, dn->n_pairs);
    if (p >= n) return;
    out[2 * p] = pu[p];
    out[2 * p + 1] = pv[p];
}

inline unsigned blocks_for(int64_t n) { return unsigned((n + kThreads - 1) / kThreads); }

template <typename T, bool PF>
hipError_t gemm_dispatch(const Plan& p, const GemmArgs& g, dim3 grid, hipStream_t s) {
    // about 16 workgroups per CU; beyond that a workgroup loops over (short) units
    constexpr unsigned kGemmGrid = 4096;
    if (!PF) grid.x = std::min<unsigned>(grid.x, std::max<unsigned>(1, kGemmGrid / grid.y));
    const size_t tab = sizeof(int32_t) * size_t(kBM + kBN + 2 * int64_t(g.K));
    if (tab > 96 * 1024) return hipErrorInvalidConfiguration;
    const dim3 block{unsigned(kThreads)};
    if (p.a_kfast && p.b_kfast) return launch_k(k_gemm<T, true, true, PF>, grid, block, tab, s, g);
    if (p.a_kfast) return launch_k(k_gemm<T, true, false, PF>, grid, block, tab, s, g);
    if (p.b_kfast) return launch_k(k_gemm<T, false, true, PF>, grid, block, tab, s, g);
    return launch_k(k_gemm<T, false, false, PF>, grid, block, tab, s, g);
}

// Prefetch pays when units run many K chunks (pairs per unit x chunks per pair).
template <typename T>
hipError_t gemm_dispatch(const Plan& p, const GemmArgs& g, dim3 grid, int64_t n_pairs, int64_t n_units,
                         hipStream_t s) {
    const int64_t chunks = (p.nK + kBK - 1) / kBK;
    const bool pf = n_pairs * chunks >= 4 * std::max<int64_t>(n_units, 1);
    return pf ? gemm_dispatch<T, true>(p, g, grid, s) : gemm_dispatch<T, false>(p, g, grid, s);
}

}  // namespace

namespace {

// Whether the plan's contraction kernel reads offset table t.
bool table_used(const Plan& p, int t) {
    if (p.kclass == KC_VEC) return t >= T_EU;
    return !p.fast && t < T_EU;
}

// The tables the contraction reads (the others marked off = -1), their
// largest and total entry counts.
TableSet table_set(const Plan& p, int64_t* largest, int64_t* total) {
    TableSet ts{};
    *largest = 0;
    *total = 0;
    for (int t = 0; t < T_COUNT; t++) {
        ts.d[t] = p.dims[t];
        ts.off[t] = table_used(p, t) ? p.table_off[t] : -1;
        if (ts.off[t] < 0) continue;
        *largest = std::max<int64_t>(*largest, p.dims[t].count());
        *total += p.dims[t].count();
    }
    return ts;
}

}  // namespace

hipError_t launch_tables(const Plan& p, int32_t* tables, hipStream_t s) {
    int64_t mx, total;
    const TableSet ts = table_set(p, &mx, &total);
    if (total == 0) return hipSuccess;
    const unsigned gx = unsigned(std::min<int64_t>((mx + kThreads - 1) / kThreads, 1024));
    k_tables<<<dim3(gx, T_COUNT), kThreads, 0, s>>>(ts, tables);
    return hipGetLastError();
}

// One unit per key (no key longer than the cap): the unit table is the
// segment table, with no partial tiles and no split keys.
// (dev_nw: the key count from the header, n_w a bound)
__global__ void k_key_units(const int32_t* __restrict__ seg_start, int64_t n_w, Unit* __restrict__ units,
                            WsHeader* hdr, int dev_nw) {
    const int64_t s = int64_t(blockIdx.x) * blockDim.x + threadIdx.x;
    if (dev_nw) n_w = min(n_w, hdr->n_w);
    if (s > n_w) return;
    if (s == n_w) {
        hdr->n_units = int32_t(n_w);
        hdr->n_parts = 0;
        hdr->n_split = 0;
        return;
    }
    Unit u;
    u.seg = int32_t(s);
    u.p0 = seg_start[s];
    u.p1 = seg_start[s + 1];
    u.slot = -1;
    units[s] = u;
}

hipError_t launch_units(const Plan& p, const Layout& L, char* ws, int64_t n_pairs, int64_t n_w, int64_t p_unit,
                        bool longest_first, hipStream_t s, bool dev_counts) {
    WsHeader* hdr = reinterpret_cast<WsHeader*>(ws + L.hdr);
    int32_t* seg_start = reinterpret_cast<int32_t*>(ws + L.seg_start);
    int32_t* nunits = reinterpret_cast<int32_t*>(ws + L.seg_units);
    int32_t* nparts = reinterpret_cast<int32_t*>(ws + L.part_off);
    int32_t* nsplit = reinterpret_cast<int32_t*>(ws + L.flags);
    int32_t* tmp = reinterpret_cast<int32_t*>(ws + L.scan_tmp);
    hipError_t e;
    int32_t* tables = reinterpret_cast<int32_t*>(ws + L.tables);
    if (n_w <= kOrderMax) {
        // the tables too, when small (one launch for both)
        int64_t mx, total;
        const TableSet ts = table_set(p, &mx, &total);
        const bool with_tables = total > 0 && total <= kUnitsTableMax;
        if (total > kUnitsTableMax && (e = launch_tables(p, tables, s)) != hipSuccess) return e;
        k_units_small<<<1, kUnitsThreads, 0, s>>>(seg_start, n_w, std::max<int64_t>(p_unit, 1),
                                                   longest_first && p.kclass == KC_GEMM ? 1 : 0,
                                                   reinterpret_cast<Unit*>(ws + L.unit_desc),
                                                   reinterpret_cast<int32_t*>(ws + L.split_list), nparts, hdr, ts,
                                                   with_tables ? tables : nullptr, dev_counts ? 1 : 0);
        return hipGetLastError();
    }
    if ((e = launch_tables(p, tables, s)) != hipSuccess) return e;
    if (p_unit >= n_pairs) {  // no key can be longer than the cap
        k_key_units<<<blocks_for(n_w + 1), kThreads, 0, s>>>(seg_start, n_w, reinterpret_cast<Unit*>(ws + L.unit_desc),
                                                             hdr, dev_counts ? 1 : 0);
        if ((e = hipGetLastError()) != hipSuccess) return e;
        if (longest_first && p.kclass == KC_GEMM && n_w <= kOrderMax) {
            k_order_units<<<1, kOrderBins, 0, s>>>(reinterpret_cast<Unit*>(ws + L.unit_desc), hdr);
            e = hipGetLastError();
        }
        return e;
    }
    if (dev_counts) return hipErrorInvalidValue;  // device key counts: one-workgroup table or one unit per key
    k_seg_units<<<blocks_for(n_w + 1), kThreads, 0, s>>>(seg_start, n_w, p_unit, nunits, nparts, nsplit);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    if ((e = scan_exclusive_i32(nunits, nunits, n_w + 1, tmp, s)) != hipSuccess) return e;
    if ((e = scan_exclusive_i32(nparts, nparts, n_w + 1, tmp, s)) != hipSuccess) return e;
    if ((e = scan_exclusive_i32(nsplit, nsplit, n_w + 1, tmp, s)) != hipSuccess) return e;
    k_fill_units<<<blocks_for(n_w + 1), kThreads, 0, s>>>(seg_start, n_w, nunits, nparts, nsplit,
                                                          reinterpret_cast<Unit*>(ws + L.unit_desc),
                                                          reinterpret_cast<int32_t*>(ws + L.split_list), hdr);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    // one workgroup per output block and unit: dispatch the longest first
    if (longest_first && p.kclass == KC_GEMM && n_w + n_pairs / p_unit + 1 <= kOrderMax) {
        k_order_units<<<1, kOrderBins, 0, s>>>(reinterpret_cast<Unit*>(ws + L.unit_desc), hdr);
        e = hipGetLastError();
    }
    return e;
}

hipError_t launch_range_units(const Plan& p, const Layout& L, char* ws, int64_t n_w, int64_t n_u, int32_t R,
                              hipStream_t s) {
    (void)p;
    const int64_t n = std::max<int64_t>(int64_t(R) * n_w, n_w + 1);
    k_range_units<<<blocks_for(n), kThreads, 0, s>>>(
        reinterpret_cast<const int32_t*>(ws + L.seg_start), reinterpret_cast<const int32_t*>(ws + L.pu), n_w, n_u, R,
        reinterpret_cast<Unit*>(ws + L.unit_desc), reinterpret_cast<int32_t*>(ws + L.part_off),
        reinterpret_cast<int32_t*>(ws + L.split_list), reinterpret_cast<WsHeader*>(ws + L.hdr));
    return hipGetLastError();
}

hipError_t launch_contract(const Plan& p, const Layout& L, char* ws, const void* u_tiles, const void* v_tiles,
                           float* w_tiles, int64_t n_pairs, int64_t n_w, int64_t unit_bound, hipStream_t s) {
    (void)n_w;
    if (unit_bound <= 0) return hipSuccess;
    const int32_t* tb = reinterpret_cast<const int32_t*>(ws + L.tables);
    const int32_t* pu = reinterpret_cast<const int32_t*>(ws + L.pu);
    const int32_t* pv = reinterpret_cast<const int32_t*>(ws + L.pv);
    const Unit* units = reinterpret_cast<const Unit*>(ws + L.unit_desc);
    const WsHeader* hdr = reinterpret_cast<const WsHeader*>(ws + L.hdr);
    float* parts = reinterpret_cast<float*>(ws + L.partials);
    if (p.kclass == KC_GEMM && p.fast)
        return launch_gemm_fast(p, L, ws, u_tiles, v_tiles, w_tiles, n_pairs, unit_bound, s);
    if (p.kclass == KC_GEMM) {
        GemmArgs g{};
        g.A = p.swap ? v_tiles : u_tiles;
        g.B = p.swap ? u_tiles : v_tiles;
        g.pa = p.swap ? pv : pu;
        g.pb = p.swap ? pu : pv;
        g.a_elems = p.tile_elems[p.swap ? 1 : 0];
        g.b_elems = p.tile_elems[p.swap ? 0 : 1];
        g.w_elems = p.tile_elems[2];
        g.tAM = tb + p.table_off[T_AM];
        g.tAK = tb + p.table_off[T_AK];
        g.tBK = tb + p.table_off[T_BK];
        g.tBN = tb + p.table_off[T_BN];
        g.tWM = tb + p.table_off[T_WM];
        g.tWN = tb + p.table_off[T_WN];
        g.tAB = tb + p.table_off[T_AB];
        g.tBB = tb + p.table_off[T_BB];
        g.tWB = tb + p.table_off[T_WB];
        g.M = int32_t(p.swap ? p.nN : p.nM);
        g.N = int32_t(p.swap ? p.nM : p.nN);
        g.K = int32_t(p.nK);
        g.nB = int32_t(p.nB);
        g.mblocks = (g.M + kBM - 1) / kBM;
        g.nblocks = (g.N + kBN - 1) / kBN;
        g.vec_a = p.vec_a;
        g.vec_b = p.vec_b;
        g.units = units;
        g.hdr = hdr;
        g.W = w_tiles;
        g.partials = parts;
        const int64_t gy = int64_t(g.nB) * g.mblocks * g.nblocks;
        if (gy > 65535) return hipErrorInvalidConfiguration;
        dim3 grid{unsigned(unit_bound), unsigned(gy), 1u};
        return p.dtype == TRE_BF16 ? gemm_dispatch<uint16_t>(p, g, grid, n_pairs, unit_bound, s)
                                   : gemm_dispatch<float>(p, g, grid, n_pairs, unit_bound, s);
    }
    // with vec_swap the kernel's first (vector) operand is V: the product is
    // symmetric, so only the roles of the pointers and tables change
    const bool sw = p.vec_swap;
    VecArgs a{};
    a.U = sw ? v_tiles : u_tiles;
    a.V = sw ? u_tiles : v_tiles;
    a.pu = sw ? pv : pu;
    a.pv = sw ? pu : pv;
    a.u_elems = p.tile_elems[sw ? 1 : 0];
    a.v_elems = p.tile_elems[sw ? 0 : 1];
    a.w_elems = p.tile_elems[2];
    a.tEU = tb + p.table_off[sw ? T_EV : T_EU];
    a.tEV = tb + p.table_off[sw ? T_EU : T_EV];
    a.tKU = tb + p.table_off[sw ? T_KV : T_KU];
    a.tKV = tb + p.table_off[sw ? T_KU : T_KV];
    a.K = int32_t(p.nK);
    a.units = units;
    a.hdr = hdr;
    a.W = w_tiles;
    a.partials = parts;
    a.w_bf16 = p.opt.w_bf16;
    a.y_scalar = p.vec_vbcast && p.nK == 1 && a.v_elems == 1;
    const int ept = p.vec_ept;
    const int64_t threads = (p.tile_elems[2] + ept - 1) / ept;
    dim3 grid;
    if (threads <= kThreads / 2) {
        int tpu = 1;
        while (tpu < threads) tpu <<= 1;
        a.tpu = tpu;
        a.upb = kThreads / tpu;
        grid = dim3{unsigned((unit_bound + a.upb - 1) / a.upb), 1u, 1u};
    } else {
        a.tpu = int32_t(threads);
        a.upb = 1;
        const int64_t gy = (threads + kThreads - 1) / kThreads;
        if (gy > 65535) return hipErrorInvalidConfiguration;
        grid = dim3{unsigned(unit_bound), unsigned(gy), 1u};
    }
    if (p.dtype == TRE_BF16) {
        return ept == 8 ? vec_dispatch<uint16_t, 8>(p, a, grid, s) : vec_dispatch<uint16_t, 1>(p, a, grid, s);
    }
    return ept == 4 ? vec_dispatch<float, 4>(p, a, grid, s) : vec_dispatch<float, 1>(p, a, grid, s);
}

hipError_t launch_reduce(const Plan& p, const Layout& L, char* ws, float* w_tiles, int64_t split_bound,
                         hipStream_t s) {
    if (split_bound <= 0) return hipSuccess;
    const int64_t we = p.tile_elems[2];
    const int64_t lanes = we % 4 == 0 ? we / 4 : we;
    const unsigned gy = unsigned(std::min<int64_t>((lanes + kThreads - 1) / kThreads, 65535));
    k_reduce<<<dim3(unsigned(split_bound), gy), kThreads, 0, s>>>(
        reinterpret_cast<const int32_t*>(ws + L.split_list), reinterpret_cast<const WsHeader*>(ws + L.hdr),
        reinterpret_cast<const int32_t*>(ws + L.part_off), reinterpret_cast<const float*>(ws + L.partials), w_tiles,
        we, p.opt.w_bf16);
    return hipGetLastError();
}

hipError_t launch_write_outputs(const Plan& p, const Layout& L, char* ws, int32_t* w_keys, int32_t* pairs_out,
                                int64_t n_pairs, int64_t n_w, hipStream_t s, bool dev_counts) {
    const WsHeader* dn = dev_counts ? reinterpret_cast<const WsHeader*>(ws + L.hdr) : nullptr;
    if (w_keys && p.nk[2] > 0 && n_w > 0) {
        Unpack up{};
        up.n = p.nk[2];
        for (int c = 0; c < p.nk[2]; c++) up.bits[c] = p.w_bits[c];
        k_write_keys<<<blocks_for(n_w), kThreads, 0, s>>>(reinterpret_cast<const uint64_t*>(ws + L.seg_key), n_w, up,
                                                           w_keys, dn);
        hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    if (pairs_out && n_pairs > 0) {
        k_write_pairs<<<blocks_for(n_pairs), kThreads, 0, s>>>(reinterpret_cast<const int32_t*>(ws + L.pu),
                                                                reinterpret_cast<const int32_t*>(ws + L.pv), n_pairs,
                                                                pairs_out, dn);
        return hipGetLastError();
    }
    return hipSuccess;
}

// The counts of an asynchronous call, from the join's header: counts[0] the
// pairs, [1] the output keys, [2] a tre_status (key errors as on the host,
// pairs beyond the workspace's capacity), [3] zero.
__global__ void k_counts_out(const WsHeader* __restrict__ hdr, int64_t max_pairs, int64_t* __restrict__ counts) {
    if (threadIdx.x != 0 || blockIdx.x != 0) return;
    auto key_status = [](int32_t f) {
        return (f & 4) ? int64_t(TRE_E_KEYRANGE) : (f & 1) ? int64_t(TRE_E_UNSORTED) : (f & 2) ? int64_t(TRE_E_DUPKEY) : 0;
    };
    int64_t st = key_status(hdr->err_u);
    if (st == 0) st = key_status(hdr->err_v);
    const int64_t n_pairs = hdr->n_pairs;
    if (st == 0 && n_pairs > max_pairs) st = TRE_E_WORKSPACE;
    counts[0] = n_pairs;
    counts[1] = n_pairs > 0 ? hdr->n_w : 0;
    counts[2] = st;
    counts[3] = 0;
}

// The counts of a call that knew them on the host.
__global__ void k_counts_set(int64_t n_pairs, int64_t n_w, int64_t status, int64_t* __restrict__ counts) {
    if (threadIdx.x != 0 || blockIdx.x != 0) return;
    counts[0] = n_pairs;
    counts[1] = n_w;
    counts[2] = status;
    counts[3] = 0;
}

hipError_t launch_counts_out(const Layout& L, char* ws, int64_t max_pairs, int64_t* counts, hipStream_t s) {
    k_counts_out<<<1, 64, 0, s>>>(reinterpret_cast<const WsHeader*>(ws + L.hdr), max_pairs, counts);
    return hipGetLastError();
}

hipError_t launch_counts_set(int64_t n_pairs, int64_t n_w, int64_t status, int64_t* counts, hipStream_t s) {
    k_counts_set<<<1, 64, 0, s>>>(n_pairs, n_w, status, counts);
    return hipGetLastError();
}

}  // namespace tre
