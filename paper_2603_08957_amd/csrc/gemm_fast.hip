// bf16 tile contraction for plain 2-D tiles: each workgroup owns a 128x128
// block of one output tile and accumulates sum over the pairs of its work
// unit of A_p (128 x K) * B_p (K x 128) on v_mfma_f32_32x32x16_bf16.
//
// 256 threads = 4 waves in a 2x2 grid, each wave a 64x64 sub-block (2x2 MFMA
// tiles, 64 fp32 accumulators per lane).  K advances in 64-deep chunks over
// the concatenation of all pairs of the unit; each chunk of A and B is staged
// in LDS as [row][k] (k contiguous, so every MFMA operand is one 16-byte LDS
// read).  An operand whose unit stride runs along rows (M for A, N for B) is
// transposed in registers on the way in: each thread loads four 16-byte row
// segments (4 k x 8 rows) and writes eight 8-byte k-runs.  The next chunk's
// global loads are issued before the current chunk's MFMAs, and LDS is
// double-buffered, so one barrier per chunk suffices.  LDS: 2 x 2 x 18 KB.
#include "tre_internal.h"

namespace tre {

namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef unsigned short u16x8 __attribute__((ext_vector_type(8)));
typedef float floatx16 __attribute__((ext_vector_type(16)));
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

constexpr int kThreads = 256;
constexpr int kB = 128;        // output block (rows and columns)
constexpr int kKC = 64;        // K chunk
constexpr int kPitch = kKC + 8;  // LDS row pitch in bf16 (144 bytes)
constexpr int kBuf = kB * kPitch;  // one operand chunk in LDS (elements)

struct FastArgs {
    const uint16_t* A;
    const uint16_t* B;
    const int32_t* pa;
    const int32_t* pb;
    int64_t a_elems, b_elems, w_elems;
    int64_t lda, ldb, ldw;
    int32_t K, nblocks;
    const Unit* units;
    const WsHeader* hdr;
    float* W;
    float* partials;
};

// Global -> registers for one 128 x 64 chunk of an operand whose element
// (r, k) sits at base[r*ld + k] (ROWFAST = false) or base[k*ld + r] (true).
template <bool ROWFAST>
__device__ inline void load_chunk(u32x4 (&v)[4], const uint16_t* __restrict__ base, int64_t ld, int r0, int k0) {
    const int t = threadIdx.x;
    if (!ROWFAST) {
        // 8 threads per row, 16 bytes each: rows r0 + 32*j + t/8
        const int r = t >> 3, kk = (t & 7) * 8;
#pragma unroll
        for (int j = 0; j < 4; j++)
            v[j] = *reinterpret_cast<const u32x4*>(base + int64_t(r0 + 32 * j + r) * ld + k0 + kk);
    } else {
        // a 4 (k) x 8 (row) block per thread: rb = t % 16 (8 rows), kb = t / 16 (4 k)
        const int rb = t & 15, kb = t >> 4;
#pragma unroll
        for (int q = 0; q < 4; q++)
            v[q] = *reinterpret_cast<const u32x4*>(base + int64_t(k0 + kb * 4 + q) * ld + r0 + rb * 8);
    }
}

__device__ inline uint32_t lo_pair(uint32_t x, uint32_t y) { return (x & 0xffffu) | (y << 16); }
__device__ inline uint32_t hi_pair(uint32_t x, uint32_t y) { return (x >> 16) | (y & 0xffff0000u); }

// Registers -> LDS [row][k] for the chunk loaded by load_chunk.
template <bool ROWFAST>
__device__ inline void store_chunk(uint16_t* __restrict__ lds, const u32x4 (&v)[4]) {
    const int t = threadIdx.x;
    if (!ROWFAST) {
        const int r = t >> 3, kk = (t & 7) * 8;
#pragma unroll
        for (int j = 0; j < 4; j++) *reinterpret_cast<u32x4*>(lds + (32 * j + r) * kPitch + kk) = v[j];
    } else {
        const int rb = t & 15, kb = t >> 4;
        const u32x4 w0 = v[0];
        const u32x4 w1 = v[1];
        const u32x4 w2 = v[2];
        const u32x4 w3 = v[3];
        // v[q] holds rows rb*8 .. rb*8+7 of k = kb*4 + q, two rows per dword
#pragma unroll
        for (int c = 0; c < 4; c++) {
            uint2 even, odd;  // rows 2c and 2c+1, k = kb*4 .. kb*4+3
            even.x = lo_pair(w0[c], w1[c]);
            even.y = lo_pair(w2[c], w3[c]);
            odd.x = hi_pair(w0[c], w1[c]);
            odd.y = hi_pair(w2[c], w3[c]);
            *reinterpret_cast<uint2*>(lds + (rb * 8 + 2 * c) * kPitch + kb * 4) = even;
            *reinterpret_cast<uint2*>(lds + (rb * 8 + 2 * c + 1) * kPitch + kb * 4) = odd;
        }
    }
}

__device__ inline bf16x8 frag(const uint16_t* lds, int row, int k) {
    return __builtin_bit_cast(bf16x8, *reinterpret_cast<const u16x8*>(lds + row * kPitch + k));
}

template <bool AROW, bool BROW>
__global__ __launch_bounds__(kThreads, 2) void k_gemm_fast(FastArgs g) {
    const int unit_id = blockIdx.x;
    if (unit_id >= g.hdr->n_units) return;
    const Unit un = g.units[unit_id];
    const int mblk = blockIdx.y / g.nblocks, nblk = blockIdx.y % g.nblocks;
    const int m0 = mblk * kB, n0 = nblk * kB;

    __shared__ __attribute__((aligned(16))) uint16_t lds[2][2][kBuf];  // [buffer][A/B]

    const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
    const int wm = w >> 1, wn = w & 1;
    floatx16 acc[2][2];
#pragma unroll
    for (int i = 0; i < 2; i++)
#pragma unroll
        for (int j = 0; j < 2; j++)
#pragma unroll
            for (int r = 0; r < 16; r++) acc[i][j][r] = 0.f;

    const int kc_per_pair = g.K / kKC;
    const int total = (un.p1 - un.p0) * kc_per_pair;
    u32x4 ra[4], rb[4];

    {
        const uint16_t* Ab = g.A + int64_t(g.pa[un.p0]) * g.a_elems;
        const uint16_t* Bb = g.B + int64_t(g.pb[un.p0]) * g.b_elems;
        load_chunk<AROW>(ra, Ab, g.lda, m0, 0);
        load_chunk<BROW>(rb, Bb, g.ldb, n0, 0);
    }
    store_chunk<AROW>(lds[0][0], ra);
    store_chunk<BROW>(lds[0][1], rb);
    __syncthreads();
    const int row = lane & 31, half = lane >> 5;
    for (int it = 0; it < total; it++) {
        const int buf = it & 1;
        if (it + 1 < total) {
            const int nx = it + 1;
            const int p = un.p0 + nx / kc_per_pair;
            const int k0 = (nx % kc_per_pair) * kKC;
            const uint16_t* Ab = g.A + int64_t(g.pa[p]) * g.a_elems;
            const uint16_t* Bb = g.B + int64_t(g.pb[p]) * g.b_elems;
            load_chunk<AROW>(ra, Ab, g.lda, m0, k0);
            load_chunk<BROW>(rb, Bb, g.ldb, n0, k0);
        }
        const uint16_t* As = lds[buf][0];
        const uint16_t* Bs = lds[buf][1];
#pragma unroll
        for (int ks = 0; ks < kKC; ks += 16) {
            const int k = ks + half * 8;
            bf16x8 a0 = frag(As, wm * 64 + row, k);
            bf16x8 a1 = frag(As, wm * 64 + 32 + row, k);
            bf16x8 b0 = frag(Bs, wn * 64 + row, k);
            bf16x8 b1 = frag(Bs, wn * 64 + 32 + row, k);
            acc[0][0] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a0, b0, acc[0][0], 0, 0, 0);
            acc[0][1] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a0, b1, acc[0][1], 0, 0, 0);
            acc[1][0] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a1, b0, acc[1][0], 0, 0, 0);
            acc[1][1] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a1, b1, acc[1][1], 0, 0, 0);
        }
        if (it + 1 < total) {
            store_chunk<AROW>(lds[buf ^ 1][0], ra);
            store_chunk<BROW>(lds[buf ^ 1][1], rb);
        }
        __syncthreads();
    }

    float* out = un.slot < 0 ? g.W + int64_t(un.seg) * g.w_elems : g.partials + int64_t(un.slot) * g.w_elems;
#pragma unroll
    for (int i = 0; i < 2; i++)
#pragma unroll
        for (int j = 0; j < 2; j++) {
            const int n = n0 + wn * 64 + j * 32 + (lane & 31);
#pragma unroll
            for (int r = 0; r < 16; r++) {
                const int m = m0 + wm * 64 + i * 32 + (r >> 2) * 8 + (lane >> 5) * 4 + (r & 3);
                out[int64_t(m) * g.ldw + n] = acc[i][j][r];
            }
        }
}

}  // namespace

hipError_t launch_gemm_fast(const Plan& p, const Layout& L, char* ws, const void* u_tiles, const void* v_tiles,
                            float* w_tiles, int64_t unit_bound, hipStream_t s) {
    FastArgs g{};
    const int32_t* pu = reinterpret_cast<const int32_t*>(ws + L.pu);
    const int32_t* pv = reinterpret_cast<const int32_t*>(ws + L.pv);
    g.A = reinterpret_cast<const uint16_t*>(p.swap ? v_tiles : u_tiles);
    g.B = reinterpret_cast<const uint16_t*>(p.swap ? u_tiles : v_tiles);
    g.pa = p.swap ? pv : pu;
    g.pb = p.swap ? pu : pv;
    g.a_elems = p.tile_elems[p.swap ? 1 : 0];
    g.b_elems = p.tile_elems[p.swap ? 0 : 1];
    g.w_elems = p.tile_elems[2];
    g.lda = p.fast_lda;
    g.ldb = p.fast_ldb;
    g.ldw = p.fast_ldw;
    g.K = int32_t(p.nK);
    const int64_t M = p.swap ? p.nN : p.nM, N = p.swap ? p.nM : p.nN;
    g.nblocks = int32_t(N / kB);
    g.units = reinterpret_cast<const Unit*>(ws + L.unit_desc);
    g.hdr = reinterpret_cast<const WsHeader*>(ws + L.hdr);
    g.W = w_tiles;
    g.partials = reinterpret_cast<float*>(ws + L.partials);
    const int64_t gy = (M / kB) * (N / kB);
    if (gy > 65535) return hipErrorInvalidConfiguration;
    dim3 grid{unsigned(unit_bound), unsigned(gy), 1u};
    if (p.fast_a_rowfast && p.fast_b_rowfast) k_gemm_fast<true, true><<<grid, kThreads, 0, s>>>(g);
    else if (p.fast_a_rowfast) k_gemm_fast<true, false><<<grid, kThreads, 0, s>>>(g);
    else if (p.fast_b_rowfast) k_gemm_fast<false, true><<<grid, kThreads, 0, s>>>(g);
    else k_gemm_fast<false, false><<<grid, kThreads, 0, s>>>(g);
    return hipGetLastError();
}

}  // namespace tre
