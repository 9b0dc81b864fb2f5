// Chain glue between two EinSums and input preparation:
//   - fp32 -> bf16 round-to-nearest-even cast of an intermediate relation,
//   - the STACK re-composition of Sec. 6 for one promoted label whose tile
//     grows from t_in to group * t_in (rows land at key % group, absent rows
//     stay zero),
//   - materialising dense tiles from scalar entries,
//   - a zero fill used instead of memset so the calls stay graph-capturable.
#include "tre_internal.h"

namespace tre {

namespace {

constexpr int kThreads = 256;

inline unsigned grid_for(int64_t n, int64_t per_thread = 1) {
    int64_t b = (n + kThreads * per_thread - 1) / (kThreads * per_thread);
    return unsigned(std::max<int64_t>(1, std::min<int64_t>(b, int64_t(1) << 20)));
}

__global__ void k_cast(const float* __restrict__ x, uint16_t* __restrict__ y, int64_t n) {
    const int64_t stride = int64_t(gridDim.x) * kThreads * 4;
    for (int64_t i = (int64_t(blockIdx.x) * kThreads + threadIdx.x) * 4; i < n; i += stride) {
        if (i + 4 <= n) {
            const float4 v = *reinterpret_cast<const float4*>(x + i);
            ushort4 o;
            o.x = f32_to_bf16_rne(v.x);
            o.y = f32_to_bf16_rne(v.y);
            o.z = f32_to_bf16_rne(v.z);
            o.w = f32_to_bf16_rne(v.w);
            *reinterpret_cast<ushort4*>(y + i) = o;
        } else {
            for (int64_t j = i; j < n; j++) y[j] = f32_to_bf16_rne(x[j]);
        }
    }
}

__global__ void k_fill_zero(uint32_t* __restrict__ p, int64_t n_words) {
    const int64_t stride = int64_t(gridDim.x) * kThreads * 4;
    for (int64_t i = (int64_t(blockIdx.x) * kThreads + threadIdx.x) * 4; i < n_words; i += stride) {
        if (i + 4 <= n_words) *reinterpret_cast<uint4*>(p + i) = make_uint4(0, 0, 0, 0);
        else
            for (int64_t j = i; j < n_words; j++) p[j] = 0;
    }
}

template <typename T>
__global__ void k_scatter_entries(const int64_t* __restrict__ slot, const int64_t* __restrict__ off,
                                  const T* __restrict__ val, int64_t n, T* __restrict__ tiles, int64_t tile_elems) {
    const int64_t i = int64_t(blockIdx.x) * kThreads + threadIdx.x;
    if (i >= n) return;
    tiles[slot[i] * tile_elems + off[i]] = val[i];
}

__global__ void k_stack_heads(const int32_t* __restrict__ keys, int64_t n, int32_t group, int32_t* __restrict__ flags) {
    const int64_t i = int64_t(blockIdx.x) * kThreads + threadIdx.x;
    if (i > n) return;
    flags[i] = (i < n && (i == 0 || keys[i] / group != keys[i - 1] / group)) ? 1 : 0;
}

__global__ void k_stack_count(const int32_t* __restrict__ excl, int64_t n, int64_t* __restrict__ n_out) {
    *n_out = excl[n];
}

// Copy every input row to its place in the stacked output, in copy units of
// type C (16 bytes when rows allow it); row i lands in output tuple
// excl[i] - (row i is not the first of its group) at row keys[i] % group.
template <typename C>
__global__ void k_stack_rows(const int32_t* __restrict__ keys, int64_t n, const int32_t* __restrict__ excl,
                             const C* __restrict__ src, int64_t row_units, int32_t group, int32_t* __restrict__ out_keys,
                             C* __restrict__ dst) {
    const int64_t total = n * row_units;
    const int64_t stride = int64_t(gridDim.x) * kThreads;
    for (int64_t c = int64_t(blockIdx.x) * kThreads + threadIdx.x; c < total; c += stride) {
        const int64_t i = c / row_units, e = c - i * row_units;
        const int32_t k = keys[i];
        const bool head = i == 0 || keys[i - 1] / group != k / group;
        const int32_t oi = excl[i] - (head ? 0 : 1);
        if (e == 0 && head) out_keys[oi] = k / group;
        dst[(int64_t(oi) * group + (k % group)) * row_units + e] = src[c];
    }
}

}  // namespace

hipError_t launch_cast_bf16(const float* x, uint16_t* y, int64_t n, hipStream_t s) {
    if (n <= 0) return hipSuccess;
    k_cast<<<grid_for(n, 4), kThreads, 0, s>>>(x, y, n);
    return hipGetLastError();
}

// y = s * x elementwise (x may be y): a unary EinSum applied to every tuple's
// tile, such as the attention scores' 1 / sqrt(d_k).
__global__ void k_scale(const float* __restrict__ x, float* __restrict__ y, int64_t n, float sc) {
    const int64_t stride = int64_t(gridDim.x) * kThreads * 4;
    for (int64_t i = (int64_t(blockIdx.x) * kThreads + threadIdx.x) * 4; i < n; i += stride) {
        if (i + 4 <= n) {
            float4 v = *reinterpret_cast<const float4*>(x + i);
            v.x *= sc;
            v.y *= sc;
            v.z *= sc;
            v.w *= sc;
            *reinterpret_cast<float4*>(y + i) = v;
        } else {
            for (int64_t j = i; j < n; j++) y[j] = x[j] * sc;
        }
    }
}

hipError_t launch_scale(const float* x, float* y, int64_t n, float sc, hipStream_t s) {
    if (n <= 0) return hipSuccess;
    k_scale<<<grid_for(n, 4), kThreads, 0, s>>>(x, y, n, sc);
    return hipGetLastError();
}

hipError_t launch_fill_zero(void* p, size_t bytes, hipStream_t s) {
    if (bytes == 0) return hipSuccess;
    const int64_t words = int64_t((bytes + 3) / 4);
    k_fill_zero<<<grid_for(words, 4), kThreads, 0, s>>>(reinterpret_cast<uint32_t*>(p), words);
    return hipGetLastError();
}

hipError_t launch_tiles_from_entries(const int64_t* slot, const int64_t* off, const void* val, int64_t n,
                                     int elem_bytes, void* tiles, int64_t n_tiles, int64_t tile_elems,
                                     hipStream_t s) {
    hipError_t e = launch_fill_zero(tiles, size_t(n_tiles) * size_t(tile_elems) * size_t(elem_bytes), s);
    if (e != hipSuccess || n <= 0) return e;
    const unsigned g = unsigned((n + kThreads - 1) / kThreads);
    if (elem_bytes == 2)
        k_scatter_entries<uint16_t><<<g, kThreads, 0, s>>>(slot, off, reinterpret_cast<const uint16_t*>(val), n,
                                                            reinterpret_cast<uint16_t*>(tiles), tile_elems);
    else
        k_scatter_entries<uint32_t><<<g, kThreads, 0, s>>>(slot, off, reinterpret_cast<const uint32_t*>(val), n,
                                                            reinterpret_cast<uint32_t*>(tiles), tile_elems);
    return hipGetLastError();
}

hipError_t launch_stack(const int32_t* keys, int64_t n, const void* tiles, int64_t row_elems, int32_t group,
                        int32_t elem_bytes, int32_t* out_keys, void* out_tiles, int64_t n_out, char* ws,
                        hipStream_t s, int stage) {
    int32_t* flags = reinterpret_cast<int32_t*>(ws);
    int64_t* cnt = reinterpret_cast<int64_t*>(ws + ((sizeof(int32_t) * size_t(n + 1) + 255) / 256 * 256));
    int32_t* tmp = reinterpret_cast<int32_t*>(reinterpret_cast<char*>(cnt) + 256);
    hipError_t e;
    if (stage == 0) {
        k_stack_heads<<<unsigned((n + 1 + kThreads - 1) / kThreads), kThreads, 0, s>>>(keys, n, group, flags);
        if ((e = hipGetLastError()) != hipSuccess) return e;
        if ((e = scan_exclusive_i32(flags, flags, n + 1, tmp, s)) != hipSuccess) return e;
        k_stack_count<<<1, 1, 0, s>>>(flags, n, cnt);
        return hipGetLastError();
    }
    // flags now holds the exclusive scan of head flags: a head row's output
    // index is excl[i]; a non-head row shares the previous head's index
    e = launch_fill_zero(out_tiles, size_t(n_out) * size_t(group) * size_t(row_elems) * size_t(elem_bytes), s);
    if (e != hipSuccess) return e;
    if (n <= 0) return hipSuccess;
    const int64_t row_bytes = row_elems * elem_bytes;
    const bool wide = row_bytes % 16 == 0 && reinterpret_cast<uintptr_t>(tiles) % 16 == 0 &&
                      reinterpret_cast<uintptr_t>(out_tiles) % 16 == 0;
    const int64_t units = wide ? row_bytes / 16 : row_elems;
    const unsigned grid = unsigned(std::min<int64_t>((n * units + kThreads - 1) / kThreads, 65536));
    if (wide)
        k_stack_rows<uint4><<<grid, kThreads, 0, s>>>(keys, n, flags, reinterpret_cast<const uint4*>(tiles), units,
                                                       group, out_keys, reinterpret_cast<uint4*>(out_tiles));
    else if (elem_bytes == 2)
        k_stack_rows<uint16_t><<<grid, kThreads, 0, s>>>(keys, n, flags, reinterpret_cast<const uint16_t*>(tiles),
                                                          units, group, out_keys,
                                                          reinterpret_cast<uint16_t*>(out_tiles));
    else
        k_stack_rows<uint32_t><<<grid, kThreads, 0, s>>>(keys, n, flags, reinterpret_cast<const uint32_t*>(tiles),
                                                          units, group, out_keys,
                                                          reinterpret_cast<uint32_t*>(out_tiles));
    return hipGetLastError();
}

size_t stack_ws_bytes(int64_t n) {
    return (sizeof(int32_t) * size_t(n + 1) + 255) / 256 * 256 + 256 + sizeof(int64_t) * scan_tmp_elems(n + 1);
}

}  // namespace tre
