// Stable LSD radix sort of (uint64 or uint32 key, payload) pairs over the low
// `bits` bits of the key, in passes of at most 8-bit digits (a 20-bit key takes
// three passes of 7 bits).  Payload: uint32 (a permutation) or uint64 (a
// packed pair, optionally split into two int32 arrays by the last pass).
// Passes ping-pong between the two buffers; the result stays where the last
// pass wrote it (radix_result_in_alt tells which).
//
// Per pass: (1) every 256-thread workgroup counts the digits of its
// 4096-item tile in LDS, (2) a device-wide exclusive scan over the
// digit-major count matrix gives each (digit, tile) its output base, (3)
// each workgroup ranks its tile locally and writes it out through LDS:
//   - wave w owns the contiguous quarter [1024 w, 1024 w + 1024) of the tile
//     and walks it in 16 rounds of 64 items; an item's rank among equal
//     digits of its wave comes from one ballot per digit bit (a 64-lane
//     match mask) plus a per-(wave, digit) counter in LDS,
//   - after one barrier the counters become per-digit wave prefixes and a
//     scan over the digits gives the tile-local start of every digit,
//   - items are placed in LDS in their tile-local sorted position, and the
//     workgroup copies the tile out in that order: each digit's run is one
//     contiguous stretch of the output, so the stores are coalesced.
// Equal digits keep their input order (wave, round, lane order is index
// order), so the sort is stable and the result deterministic.
#include "tre_internal.h"

namespace tre {

namespace {

constexpr int kThreads = 256;
constexpr int kWaves = kThreads / 64;
constexpr int kIpt = 16;
constexpr int kTile = kThreads * kIpt;  // 4096 items
constexpr int kPerWave = kTile / kWaves;
constexpr int kMaxBits = 8;
constexpr int kRadix = 1 << kMaxBits;
constexpr int kDpt = kRadix / kThreads;  // digits per thread in the prefix step
static_assert(kDpt >= 1 && kDpt * kThreads == kRadix, "radix must be a multiple of the workgroup size");

// Item count: the host's n, or min(*dn, n) when the count lives in device
// memory (the grid is then sized for n, the capacity).
__device__ inline int64_t item_count(int64_t n, const int64_t* dn) { return dn ? min(*dn, n) : n; }

template <typename KT>
__global__ __launch_bounds__(kThreads) void k_digit_hist(const KT* __restrict__ keys, int64_t cap,
                                                         const int64_t* __restrict__ dn, int shift, int dbits,
                                                         int32_t* __restrict__ hist, int64_t n_tiles) {
    __shared__ int32_t cnt[kRadix];
    const int64_t n = item_count(cap, dn);
    const int radix = 1 << dbits;
    for (int d = threadIdx.x; d < radix; d += kThreads) cnt[d] = 0;
    __syncthreads();
    const int64_t base = int64_t(blockIdx.x) * kTile;
    const uint64_t mask = uint64_t(radix - 1);
    // all of the thread's loads in flight before the first count
    KT k[kIpt];
#pragma unroll
    for (int r = 0; r < kIpt; r++) {
        const int64_t i = base + int64_t(r) * kThreads + threadIdx.x;
        k[r] = i < n ? keys[i] : KT(0);
    }
#pragma unroll
    for (int r = 0; r < kIpt; r++)
        if (base + int64_t(r) * kThreads + threadIdx.x < n) atomicAdd(&cnt[(k[r] >> shift) & mask], 1);
    __syncthreads();
    for (int d = threadIdx.x; d < radix; d += kThreads) hist[int64_t(d) * n_tiles + blockIdx.x] = cnt[d];
}

// SPLIT (uint64 payloads only): write the payload's high and low halves to
// two int32 arrays instead of vout.  KT: uint64 keys, or uint32 keys when
// the sorted bits fit (less traffic per pass).
template <typename KT, typename VT, bool SPLIT>
__global__ __launch_bounds__(kThreads) void k_digit_scatter(const KT* __restrict__ kin, const VT* __restrict__ vin,
                                                            KT* __restrict__ kout, VT* __restrict__ vout,
                                                            int32_t* __restrict__ hi_out, int32_t* __restrict__ lo_out,
                                                            int64_t cap, const int64_t* __restrict__ dn, int shift,
                                                            int dbits, const int32_t* __restrict__ offs,
                                                            int64_t n_tiles) {
    const int64_t n = item_count(cap, dn);
    if (int64_t(blockIdx.x) * kTile >= n) return;  // tiles past the count (their counts are 0)
    __shared__ KT skey[kTile];
    __shared__ VT sval[kTile];
    __shared__ int32_t wcnt[kWaves][kRadix];  // per-(wave, digit) counts, then wave prefixes
    __shared__ int32_t dstart[kRadix];        // tile-local start of each digit
    __shared__ int32_t gbase[kRadix];         // output position of (digit, this tile)
    __shared__ int32_t wsum[kWaves];
    const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
    const int radix = 1 << dbits;
    for (int d = tid; d < kRadix; d += kThreads)
#pragma unroll
        for (int i = 0; i < kWaves; i++) wcnt[i][d] = 0;
    __syncthreads();

    const uint64_t lt = (lane == 0) ? 0ull : (~0ull >> (64 - lane));
    const uint64_t dmask = uint64_t(radix - 1);
    const int64_t tile0 = int64_t(blockIdx.x) * kTile;
    const int64_t item0 = tile0 + int64_t(w) * kPerWave + lane;
    KT key[kIpt];
    VT val[kIpt];
    int32_t rank[kIpt];
#pragma unroll
    for (int r = 0; r < kIpt; r++) {
        const int64_t i = item0 + int64_t(r) * 64;
        const bool valid = i < n;
        key[r] = valid ? kin[i] : KT(0);
        val[r] = valid ? vin[i] : VT(0);
    }
    // ranks among equal digits inside this wave's quarter, in index order
#pragma unroll
    for (int r = 0; r < kIpt; r++) {
        const bool valid = item0 + int64_t(r) * 64 < n;
        const int d = int((uint64_t(key[r]) >> shift) & dmask);
        uint64_t mask = __ballot(valid);
        for (int b = 0; b < dbits; b++) {
            const bool bit = (d >> b) & 1;
            const uint64_t bb = __ballot(bit);
            mask &= bit ? bb : ~bb;
        }
        const int32_t before = valid ? wcnt[w][d] : 0;
        rank[r] = before + __popcll(mask & lt);
        // the lowest lane of each digit group advances the counter; every lane
        // of the group has read it above (one wavefront, LDS order kept)
        if (valid && (mask & lt) == 0) wcnt[w][d] = before + __popcll(mask);
    }
    __syncthreads();
    // per digit: wave prefixes and the tile total; then tile-local starts.
    // Thread t owns the kDpt consecutive digits [kDpt t, kDpt t + kDpt).
    int32_t tot[kDpt];
    int32_t sum = 0;
#pragma unroll
    for (int j = 0; j < kDpt; j++) {
        const int d = tid * kDpt + j;
        int32_t acc = 0;
#pragma unroll
        for (int i = 0; i < kWaves; i++) {
            const int32_t c = wcnt[i][d];
            wcnt[i][d] = acc;
            acc += c;
        }
        tot[j] = acc;
        sum += acc;
        gbase[d] = d < radix ? offs[int64_t(d) * n_tiles + blockIdx.x] : 0;
    }
    // exclusive scan of the per-thread sums over the workgroup
    int32_t incl = sum;
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
        const int32_t y = __shfl_up(incl, o);
        if (lane >= o) incl += y;
    }
    if (lane == 63) wsum[w] = incl;
    __syncthreads();
    int32_t run = incl - sum;
    for (int i = 0; i < w; i++) run += wsum[i];
#pragma unroll
    for (int j = 0; j < kDpt; j++) {
        dstart[tid * kDpt + j] = run;
        run += tot[j];
    }
    __syncthreads();
    // place every item at its tile-local sorted position
#pragma unroll
    for (int r = 0; r < kIpt; r++) {
        if (item0 + int64_t(r) * 64 < n) {
            const int d = int((uint64_t(key[r]) >> shift) & dmask);
            const int pos = dstart[d] + wcnt[w][d] + rank[r];
            skey[pos] = key[r];
            sval[pos] = val[r];
        }
    }
    __syncthreads();
    // copy out in sorted order: consecutive positions of one digit are
    // consecutive output positions
    const int cnt = int(min<int64_t>(kTile, n - tile0));
    for (int q = tid; q < cnt; q += kThreads) {
        const KT k = skey[q];
        const int d = int((uint64_t(k) >> shift) & dmask);
        const int64_t dest = int64_t(gbase[d]) + (q - dstart[d]);
        kout[dest] = k;
        if constexpr (SPLIT) {
            hi_out[dest] = int32_t(uint64_t(sval[q]) >> 32);
            lo_out[dest] = int32_t(uint64_t(sval[q]) & 0xffffffffu);
        } else {
            vout[dest] = sval[q];
        }
    }
}

int sort_passes(int bits) { return bits <= 0 ? 0 : (bits + kMaxBits - 1) / kMaxBits; }

template <typename KT, typename VT>
hipError_t sort_impl(KT* keys, VT* vals, KT* keys_alt, VT* vals_alt, int64_t n, const int64_t* dn, int bits,
                     int32_t* hist, int32_t* scan_tmp, int32_t* split_hi, int32_t* split_lo, hipStream_t s) {
    if (n <= 1 || bits <= 0) return hipSuccess;
    const int64_t nt = (n + kTile - 1) / kTile;
    const int passes = sort_passes(bits);
    const int dbits = (bits + passes - 1) / passes;
    KT *ki = keys, *ko = keys_alt;
    VT *vi = vals, *vo = vals_alt;
    for (int p = 0; p < passes; p++) {
        const int shift = dbits * p;
        k_digit_hist<KT><<<dim3(unsigned(nt)), kThreads, 0, s>>>(ki, n, dn, shift, dbits, hist, nt);
        hipError_t e = scan_exclusive_i32(hist, hist, (int64_t(1) << dbits) * nt, scan_tmp, s);
        if (e != hipSuccess) return e;
        if (split_hi && p == passes - 1)
            k_digit_scatter<KT, VT, true><<<dim3(unsigned(nt)), kThreads, 0, s>>>(
                ki, vi, ko, vo, split_hi, split_lo, n, dn, shift, dbits, hist, nt);
        else
            k_digit_scatter<KT, VT, false><<<dim3(unsigned(nt)), kThreads, 0, s>>>(
                ki, vi, ko, vo, nullptr, nullptr, n, dn, shift, dbits, hist, nt);
        std::swap(ki, ko);
        std::swap(vi, vo);
    }
    return hipGetLastError();
}

}  // namespace

int64_t radix_hist_elems(int64_t n) { return int64_t(kRadix) * ((n + kTile - 1) / kTile) + 64; }

bool radix_result_in_alt(int64_t n, int bits) { return n > 1 && (sort_passes(bits) & 1); }

hipError_t radix_sort_u64(uint64_t* keys, uint32_t* vals, uint64_t* keys_alt, uint32_t* vals_alt, int64_t n,
                          int bits, int32_t* hist, int32_t* scan_tmp, hipStream_t s) {
    return sort_impl<uint64_t, uint32_t>(keys, vals, keys_alt, vals_alt, n, nullptr, bits, hist, scan_tmp, nullptr,
                                         nullptr, s);
}

hipError_t radix_sort_u64_pairs(uint64_t* keys, uint64_t* vals, uint64_t* keys_alt, uint64_t* vals_alt, int64_t n,
                                const int64_t* dn, int bits, int32_t* hist, int32_t* scan_tmp, int32_t* split_hi,
                                int32_t* split_lo, hipStream_t s) {
    return sort_impl<uint64_t, uint64_t>(keys, vals, keys_alt, vals_alt, n, dn, bits, hist, scan_tmp, split_hi,
                                         split_lo, s);
}

hipError_t radix_sort_u32_pairs(uint32_t* keys, uint64_t* vals, uint32_t* keys_alt, uint64_t* vals_alt, int64_t n,
                                const int64_t* dn, int bits, int32_t* hist, int32_t* scan_tmp, int32_t* split_hi,
                                int32_t* split_lo, hipStream_t s) {
    if (bits > 32) return hipErrorInvalidValue;
    return sort_impl<uint32_t, uint64_t>(keys, vals, keys_alt, vals_alt, n, dn, bits, hist, scan_tmp, split_hi,
                                         split_lo, s);
}

}  // namespace tre
