// Device-wide exclusive prefix sum (int32 / int64), used for pair counts,
// radix-sort digit offsets, segment heads and work-unit offsets.
//
// A tile of 4096 items per 256-thread workgroup: each thread owns 16
// consecutive items, wavefront-level inclusive scans of the per-thread sums
// run on 64-wide DPP-friendly shuffles, and wave totals meet in LDS.  Inputs
// longer than one tile take a reduce -> scan-of-sums -> rescan pass, applied
// recursively to the block sums (up to 32768 items: one workgroup, one
// launch).  In-place operation (in == out) is allowed.
#include "tre_internal.h"

namespace tre {

namespace {

constexpr int kThreads = 256;
constexpr int kIpt = 16;
constexpr int kTile = kThreads * kIpt;

template <typename T>
__device__ inline T wave_inclusive(T x) {
    const int lane = threadIdx.x & 63;
#pragma unroll
    for (int d = 1; d < 64; d <<= 1) {
        T y = __shfl_up(x, d, 64);
        if (lane >= d) x += y;
    }
    return x;
}

// Exclusive scan of the 256 per-thread values of a workgroup; returns the
// thread's exclusive prefix and writes the workgroup total to *total.
template <typename T>
__device__ inline T block_exclusive(T v, T* total) {
    __shared__ T wsum[kThreads / 64];
    const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
    T inc = wave_inclusive(v);
    if (lane == 63) wsum[w] = inc;
    __syncthreads();
    T before = 0, all = 0;
#pragma unroll
    for (int i = 0; i < kThreads / 64; i++) {
        T s = wsum[i];
        if (i < w) before += s;
        all += s;
    }
    __syncthreads();
    *total = all;
    return before + inc - v;
}

template <typename T>
__global__ __launch_bounds__(kThreads) void k_tile_sum(const T* __restrict__ in, int64_t n, T* __restrict__ sums) {
    const int64_t base = int64_t(blockIdx.x) * kTile + int64_t(threadIdx.x) * kIpt;
    T s = 0;
#pragma unroll
    for (int i = 0; i < kIpt; i++)
        if (base + i < n) s += in[base + i];
    T total;
    (void)block_exclusive(s, &total);
    if (threadIdx.x == 0) sums[blockIdx.x] = total;
}

template <typename T>
__global__ __launch_bounds__(kThreads) void k_tile_scan(const T* in, T* out, int64_t n, const T* __restrict__ tile_off) {
    const int64_t base = int64_t(blockIdx.x) * kTile + int64_t(threadIdx.x) * kIpt;
    T v[kIpt];
    T s = 0;
#pragma unroll
    for (int i = 0; i < kIpt; i++) {
        v[i] = (base + i < n) ? in[base + i] : T(0);
        s += v[i];
    }
    T total;
    T run = block_exclusive(s, &total) + (tile_off ? tile_off[blockIdx.x] : T(0));
#pragma unroll
    for (int i = 0; i < kIpt; i++) {
        if (base + i < n) out[base + i] = run;
        run += v[i];
    }
}

// Inputs of a few tiles: one workgroup of 1024 threads walks them in
// chunks of 16384 items (16 consecutive items per thread), carrying the
// running total, so the scan is one launch instead of three.
constexpr int kOneThreads = 1024;
constexpr int64_t kOneChunk = int64_t(kOneThreads) * kIpt;
constexpr int64_t kOneMax = 2 * kOneChunk;

template <typename T>
__global__ __launch_bounds__(kOneThreads) void k_scan_one(const T* in, T* out, int64_t n) {
    __shared__ T wsum[kOneThreads / 64];
    const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
    T carry = 0;
    for (int64_t c0 = 0; c0 < n; c0 += kOneChunk) {
        const int64_t base = c0 + int64_t(threadIdx.x) * kIpt;
        T v[kIpt];
        T sum = 0;
#pragma unroll
        for (int i = 0; i < kIpt; i++) {
            v[i] = (base + i < n) ? in[base + i] : T(0);
            sum += v[i];
        }
        const T inc = wave_inclusive(sum);
        if (lane == 63) wsum[w] = inc;
        __syncthreads();
        T before = 0, all = 0;
#pragma unroll
        for (int i = 0; i < kOneThreads / 64; i++) {
            const T x = wsum[i];
            if (i < w) before += x;
            all += x;
        }
        __syncthreads();
        T run = carry + before + inc - sum;
#pragma unroll
        for (int i = 0; i < kIpt; i++) {
            if (base + i < n) out[base + i] = run;
            run += v[i];
        }
        carry += all;
    }
}

template <typename T>
hipError_t scan_rec(const T* in, T* out, int64_t n, T* tmp, hipStream_t s) {
    if (n <= 0) return hipSuccess;
    const int64_t nt = (n + kTile - 1) / kTile;
    if (nt == 1) {
        k_tile_scan<T><<<1, kThreads, 0, s>>>(in, out, n, nullptr);
        return hipGetLastError();
    }
    if (n <= kOneMax) {
        k_scan_one<T><<<1, kOneThreads, 0, s>>>(in, out, n);
        return hipGetLastError();
    }
    T* sums = tmp;
    T* rest = tmp + (nt + 63) / 64 * 64;
    k_tile_sum<T><<<dim3(unsigned(nt)), kThreads, 0, s>>>(in, n, sums);
    hipError_t e = scan_rec<T>(sums, sums, nt, rest, s);
    if (e != hipSuccess) return e;
    k_tile_scan<T><<<dim3(unsigned(nt)), kThreads, 0, s>>>(in, out, n, sums);
    return hipGetLastError();
}

}  // namespace

size_t scan_tmp_elems(int64_t n) {
    size_t total = 64;
    while (n > kTile) {
        int64_t nt = (n + kTile - 1) / kTile;
        total += size_t((nt + 63) / 64 * 64);
        n = nt;
    }
    return total;
}

hipError_t scan_exclusive_i64(const int64_t* in, int64_t* out, int64_t n, int64_t* tmp, hipStream_t s) {
    return scan_rec<int64_t>(in, out, n, tmp, s);
}

hipError_t scan_exclusive_i32(const int32_t* in, int32_t* out, int64_t n, int32_t* tmp, hipStream_t s) {
    return scan_rec<int32_t>(in, out, n, tmp, s);
}

}  // namespace tre
