// Stable LSD radix sort of (uint64 key, uint32 payload) pairs, 8-bit digits.
//
// Per pass: (1) every 256-thread workgroup counts the digits of its 4096-item
// tile in LDS, (2) a device-wide exclusive scan over the digit-major count
// matrix gives each (digit, tile) its output base, (3) each workgroup walks
// its tile in 16 rounds of 256 items in index order and ranks every item among
// equal digits with eight wavefront ballots (a 64-lane match mask), wave
// totals meet in LDS -- so equal keys keep their input order and the result
// is deterministic.  Only the low `bits` bits of the key take part.
#include "tre_internal.h"

namespace tre {

namespace {

constexpr int kThreads = 256;
constexpr int kIpt = 16;
constexpr int kTile = kThreads * kIpt;
constexpr int kRadix = 256;

__global__ __launch_bounds__(kThreads) void k_digit_hist(const uint64_t* __restrict__ keys, int64_t n, int shift,
                                                         int64_t* __restrict__ hist, int64_t n_tiles) {
    __shared__ int32_t cnt[kRadix];
    cnt[threadIdx.x] = 0;
    __syncthreads();
    const int64_t base = int64_t(blockIdx.x) * kTile;
#pragma unroll 4
    for (int r = 0; r < kIpt; r++) {
        int64_t i = base + int64_t(r) * kThreads + threadIdx.x;
        if (i < n) atomicAdd(&cnt[(keys[i] >> shift) & (kRadix - 1)], 1);
    }
    __syncthreads();
    hist[int64_t(threadIdx.x) * n_tiles + blockIdx.x] = cnt[threadIdx.x];
}

__global__ __launch_bounds__(kThreads) void k_digit_scatter(const uint64_t* __restrict__ kin,
                                                            const uint32_t* __restrict__ vin,
                                                            uint64_t* __restrict__ kout, uint32_t* __restrict__ vout,
                                                            int64_t n, int shift, const int64_t* __restrict__ offs,
                                                            int64_t n_tiles) {
    __shared__ int64_t base[kRadix];
    __shared__ int32_t wcnt[kThreads / 64][kRadix];
    const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
    base[tid] = offs[int64_t(tid) * n_tiles + blockIdx.x];
#pragma unroll
    for (int i = 0; i < kThreads / 64; i++) wcnt[i][tid] = 0;
    __syncthreads();
    const uint64_t lt = (lane == 0) ? 0ull : (~0ull >> (64 - lane));
    const int64_t tile0 = int64_t(blockIdx.x) * kTile;
    for (int r = 0; r < kIpt; r++) {
        const int64_t i = tile0 + int64_t(r) * kThreads + tid;
        const bool valid = i < n;
        const uint64_t key = valid ? kin[i] : 0ull;
        const uint32_t val = valid ? vin[i] : 0u;
        const int d = int((key >> shift) & (kRadix - 1));
        uint64_t mask = __ballot(valid);
#pragma unroll
        for (int b = 0; b < 8; b++) {
            const bool bit = (d >> b) & 1;
            const uint64_t bb = __ballot(bit);
            mask &= bit ? bb : ~bb;
        }
        const int rank = __popcll(mask & lt);
        if (valid && rank == 0) wcnt[w][d] = __popcll(mask);
        __syncthreads();
        if (valid) {
            int64_t pre = 0;
            for (int j = 0; j < w; j++) pre += wcnt[j][d];
            const int64_t dest = base[d] + pre + rank;
            kout[dest] = key;
            vout[dest] = val;
        }
        __syncthreads();
        int64_t add = 0;
#pragma unroll
        for (int j = 0; j < kThreads / 64; j++) {
            add += wcnt[j][tid];
            wcnt[j][tid] = 0;
        }
        base[tid] += add;
        __syncthreads();
    }
}

}  // namespace

int64_t radix_hist_elems(int64_t n) { return int64_t(kRadix) * ((n + kTile - 1) / kTile) + 64; }

hipError_t radix_sort_u64(uint64_t* keys, uint32_t* vals, uint64_t* keys_alt, uint32_t* vals_alt, int64_t n,
                          int bits, int64_t* hist, int64_t* scan_tmp, hipStream_t s) {
    if (n <= 1 || bits <= 0) return hipSuccess;
    const int64_t nt = (n + kTile - 1) / kTile;
    const int passes = (bits + 7) / 8;
    uint64_t *ki = keys, *ko = keys_alt;
    uint32_t *vi = vals, *vo = vals_alt;
    for (int p = 0; p < passes; p++) {
        const int shift = 8 * p;
        k_digit_hist<<<dim3(unsigned(nt)), kThreads, 0, s>>>(ki, n, shift, hist, nt);
        hipError_t e = scan_exclusive_i64(hist, hist, kRadix * nt, scan_tmp, s);
        if (e != hipSuccess) return e;
        k_digit_scatter<<<dim3(unsigned(nt)), kThreads, 0, s>>>(ki, vi, ko, vo, n, shift, hist, nt);
        std::swap(ki, ko);
        std::swap(vi, vo);
    }
    if (ki != keys) {
        hipError_t e = hipMemcpyAsync(keys, ki, sizeof(uint64_t) * size_t(n), hipMemcpyDeviceToDevice, s);
        if (e != hipSuccess) return e;
        e = hipMemcpyAsync(vals, vi, sizeof(uint32_t) * size_t(n), hipMemcpyDeviceToDevice, s);
        if (e != hipSuccess) return e;
    }
    return hipGetLastError();
}

}  // namespace tre
