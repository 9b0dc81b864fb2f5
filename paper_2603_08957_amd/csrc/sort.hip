// Stable LSD radix sort of (uint64 key, payload) pairs over the low `bits`
// bits of the key, with up to 11-bit digits (so a 20-bit key takes two
// passes).  Payload: uint32 (a permutation) or uint64 (a packed pair).
//
// Per pass: (1) every 256-thread workgroup counts the digits of its
// 8192-item tile in LDS, (2) a device-wide exclusive scan over the digit-major
// count matrix gives each (digit, tile) its output base, (3) each workgroup
// walks its tile in 32 rounds of 256 items in index order and ranks every item
// among equal digits with one wavefront ballot per digit bit (a 64-lane match
// mask); wave totals meet in LDS.  Equal keys keep their input order, so the
// result is deterministic.
#include "tre_internal.h"

namespace tre {

namespace {

constexpr int kThreads = 256;
constexpr int kIpt = 32;
constexpr int kTile = kThreads * kIpt;
constexpr int kMaxBits = 11;
constexpr int kMaxRadix = 1 << kMaxBits;

__global__ __launch_bounds__(kThreads) void k_digit_hist(const uint64_t* __restrict__ keys, int64_t n, int shift,
                                                         int dbits, int32_t* __restrict__ hist, int64_t n_tiles) {
    __shared__ int32_t cnt[kMaxRadix];
    const int radix = 1 << dbits;
    for (int d = threadIdx.x; d < radix; d += kThreads) cnt[d] = 0;
    __syncthreads();
    const int64_t base = int64_t(blockIdx.x) * kTile;
    const uint64_t mask = uint64_t(radix - 1);
#pragma unroll 4
    for (int r = 0; r < kIpt; r++) {
        const int64_t i = base + int64_t(r) * kThreads + threadIdx.x;
        if (i < n) atomicAdd(&cnt[(keys[i] >> shift) & mask], 1);
    }
    __syncthreads();
    for (int d = threadIdx.x; d < radix; d += kThreads) hist[int64_t(d) * n_tiles + blockIdx.x] = cnt[d];
}

template <typename VT>
__global__ __launch_bounds__(kThreads) void k_digit_scatter(const uint64_t* __restrict__ kin, const VT* __restrict__ vin,
                                                            uint64_t* __restrict__ kout, VT* __restrict__ vout,
                                                            int64_t n, int shift, int dbits,
                                                            const int32_t* __restrict__ offs, int64_t n_tiles) {
    __shared__ int32_t base[kMaxRadix];
    __shared__ int32_t wcnt[kThreads / 64][kMaxRadix];
    const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
    const int radix = 1 << dbits;
    for (int d = tid; d < radix; d += kThreads) {
        base[d] = offs[int64_t(d) * n_tiles + blockIdx.x];
#pragma unroll
        for (int i = 0; i < kThreads / 64; i++) wcnt[i][d] = 0;
    }
    __syncthreads();
    const uint64_t lt = (lane == 0) ? 0ull : (~0ull >> (64 - lane));
    const uint64_t dmask = uint64_t(radix - 1);
    const int64_t tile0 = int64_t(blockIdx.x) * kTile;
    for (int r = 0; r < kIpt; r++) {
        const int64_t i = tile0 + int64_t(r) * kThreads + tid;
        const bool valid = i < n;
        const uint64_t key = valid ? kin[i] : 0ull;
        const VT val = valid ? vin[i] : VT(0);
        const int d = int((key >> shift) & dmask);
        uint64_t mask = __ballot(valid);
        for (int b = 0; b < dbits; b++) {
            const bool bit = (d >> b) & 1;
            const uint64_t bb = __ballot(bit);
            mask &= bit ? bb : ~bb;
        }
        const int rank = __popcll(mask & lt);
        if (valid && rank == 0) wcnt[w][d] = __popcll(mask);
        __syncthreads();
        if (valid) {
            int32_t pre = 0;
            for (int j = 0; j < w; j++) pre += wcnt[j][d];
            const int64_t dest = int64_t(base[d]) + pre + rank;
            kout[dest] = key;
            vout[dest] = val;
        }
        __syncthreads();
        for (int dd = tid; dd < radix; dd += kThreads) {
            int32_t add = 0;
#pragma unroll
            for (int j = 0; j < kThreads / 64; j++) {
                add += wcnt[j][dd];
                wcnt[j][dd] = 0;
            }
            base[dd] += add;
        }
        __syncthreads();
    }
}

template <typename VT>
hipError_t sort_impl(uint64_t* keys, VT* vals, uint64_t* keys_alt, VT* vals_alt, int64_t n, int bits, int32_t* hist,
                     int32_t* scan_tmp, hipStream_t s) {
    if (n <= 1 || bits <= 0) return hipSuccess;
    const int64_t nt = (n + kTile - 1) / kTile;
    const int passes = (bits + kMaxBits - 1) / kMaxBits;
    const int dbits = (bits + passes - 1) / passes;
    uint64_t *ki = keys, *ko = keys_alt;
    VT *vi = vals, *vo = vals_alt;
    for (int p = 0; p < passes; p++) {
        const int shift = dbits * p;
        k_digit_hist<<<dim3(unsigned(nt)), kThreads, 0, s>>>(ki, n, shift, dbits, hist, nt);
        hipError_t e = scan_exclusive_i32(hist, hist, (int64_t(1) << dbits) * nt, scan_tmp, s);
        if (e != hipSuccess) return e;
        k_digit_scatter<VT><<<dim3(unsigned(nt)), kThreads, 0, s>>>(ki, vi, ko, vo, n, shift, dbits, hist, nt);
        std::swap(ki, ko);
        std::swap(vi, vo);
    }
    if (ki != keys) {
        hipError_t e = hipMemcpyAsync(keys, ki, sizeof(uint64_t) * size_t(n), hipMemcpyDeviceToDevice, s);
        if (e != hipSuccess) return e;
        e = hipMemcpyAsync(vals, vi, sizeof(VT) * size_t(n), hipMemcpyDeviceToDevice, s);
        if (e != hipSuccess) return e;
    }
    return hipGetLastError();
}

}  // namespace

int64_t radix_hist_elems(int64_t n) { return int64_t(kMaxRadix) * ((n + kTile - 1) / kTile) + 64; }

hipError_t radix_sort_u64(uint64_t* keys, uint32_t* vals, uint64_t* keys_alt, uint32_t* vals_alt, int64_t n,
                          int bits, int32_t* hist, int32_t* scan_tmp, hipStream_t s) {
    return sort_impl<uint32_t>(keys, vals, keys_alt, vals_alt, n, bits, hist, scan_tmp, s);
}

hipError_t radix_sort_u64_pairs(uint64_t* keys, uint64_t* vals, uint64_t* keys_alt, uint64_t* vals_alt, int64_t n,
                                int bits, int32_t* hist, int32_t* scan_tmp, hipStream_t s) {
    return sort_impl<uint64_t>(keys, vals, keys_alt, vals_alt, n, bits, hist, scan_tmp, s);
}

}  // namespace tre
