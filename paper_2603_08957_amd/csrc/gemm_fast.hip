// bf16 tile contraction for plain 2-D tiles: each workgroup owns a 128x128
// block of one output tile and accumulates sum over the pairs of its work
// unit of A_p (128 x K) * B_p (K x 128) on v_mfma_f32_32x32x16_bf16.
//
// 256 threads = 4 waves in a 2x2 grid, each wave a 64x64 sub-block (2x2 MFMA
// tiles, 64 fp32 accumulators per lane).  K advances in 64-deep chunks over
// the concatenation of all pairs of the unit.  Each chunk of A and B is
// staged in LDS as [row][k]: 128-byte rows of eight 16-byte granules, granule
// g of row r stored at g ^ ((r ^ (r >> 3)) & 7).  With that swizzle the MFMA
// operand reads (one 16-byte read per lane, 16 or 8 consecutive rows per LDS
// cycle), the plain copies and the transposing writes below are all free of
// bank conflicts.
//
// An operand whose unit stride runs along rows (M for A, N for B) is
// transposed in registers: a thread loads four 16-byte row segments (4 k x 8
// rows) and writes eight 8-byte k-runs; half of each wavefront writes the
// odd row of a row pair first so that both bank halves stay busy.
//
// Global loads run two chunks ahead in registers (two register sets used
// alternately) and LDS is double-buffered, so one barrier per chunk suffices.
// LDS: 2 buffers x 2 operands x 16 KB.
#include "tre_internal.h"

namespace tre {

namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef unsigned short u16x8 __attribute__((ext_vector_type(8)));
typedef float floatx16 __attribute__((ext_vector_type(16)));
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
typedef unsigned int u32x2 __attribute__((ext_vector_type(2)));

constexpr int kThreads = 256;
constexpr int kB = 128;          // output block (rows and columns)
constexpr int kKC = 64;          // K chunk
constexpr int kRow = kKC;        // LDS row length in bf16 (128 bytes)
constexpr int kBuf = kB * kRow;  // one operand chunk in LDS (elements)

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

__device__ inline int swz(int r) { return (r ^ (r >> 3)) & 7; }

// element offset in an LDS chunk of (row r, 16-byte granule g)
__device__ inline int lds_off(int r, int g) { return r * kRow + ((g ^ swz(r)) << 3); }

// Thread -> data maps.  Copy: row t/8 + 32j, granule t%8.  Transpose: row
// block rb (8 rows) and k quad kb, chosen so that 8 consecutive lanes read
// 128 contiguous bytes of one k row.
__device__ inline int tr_rb(int t) { return (t & 7) | (((t >> 4) & 1) << 3); }
__device__ inline int tr_kb(int t) { return ((t >> 3) & 1) | (((t >> 5) & 1) << 1) | ((t >> 6) << 2); }

// Global -> registers for one 128 x 64 chunk of an operand whose element
// (r, k) sits at base[r*ld + k] (ROWFAST = false) or base[k*ld + r] (true).
// NT: the operand is streamed (each tile read by one workgroup once), so its
// loads carry the non-temporal hint and do not push reused tiles out of L2.
template <bool NT>
__device__ inline u32x4 gload(const uint16_t* p) {
    if constexpr (NT) return __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(p));
    else return *reinterpret_cast<const u32x4*>(p);
}

// The per-lane part of the addresses is fixed for the whole unit: lane offset
// `lo` and the step between a thread's four loads (32 rows when k is
// contiguous, one k row when rows are); the per-chunk part is uniform.
template <bool ROWFAST>
__device__ inline int32_t lane_offset(int32_t ld) {
    const int t = threadIdx.x;
    if (!ROWFAST) return (t >> 3) * ld + (t & 7) * 8;
    return tr_kb(t) * 4 * ld + tr_rb(t) * 8;
}

template <bool ROWFAST>
__device__ inline int64_t chunk_offset(int64_t ld, int r0, int k0) {
    return ROWFAST ? int64_t(k0) * ld + r0 : int64_t(r0) * ld + k0;
}

template <bool ROWFAST, bool NT>
__device__ inline void load_chunk(u32x4 (&v)[4], const uint16_t* __restrict__ base, int32_t lo, int32_t step) {
    const uint16_t* p = base + lo;
#pragma unroll
    for (int j = 0; j < 4; j++) v[j] = gload<NT>(p + j * step);
}

__device__ inline uint32_t lo_pair(uint32_t x, uint32_t y) { return (x & 0xffffu) | (y << 16); }
__device__ inline uint32_t hi_pair(uint32_t x, uint32_t y) { return (x >> 16) | (y & 0xffff0000u); }

// Registers -> LDS [row][k] for the chunk loaded by load_chunk.
template <bool ROWFAST>
__device__ inline void store_chunk(uint16_t* __restrict__ lds, const u32x4 (&v)[4]) {
    const int t = threadIdx.x;
    if (!ROWFAST) {
        const int r = t >> 3, g = t & 7;
#pragma unroll
        for (int j = 0; j < 4; j++) *reinterpret_cast<u32x4*>(lds + lds_off(32 * j + r, g)) = v[j];
    } else {
        const int rb = tr_rb(t), kb = tr_kb(t);
        const int g = kb >> 1, h = (kb & 1) * 4;
        const bool odd_first = (t >> 4) & 1;
        // v[q] holds rows rb*8 .. rb*8+7 of k = kb*4 + q, two rows per dword;
        // piece e = the 4 k values of row rb*8 + e
#pragma unroll
        for (int c = 0; c < 4; c++) {
            u32x2 even, odd;
            even.x = lo_pair(v[0][c], v[1][c]);
            even.y = lo_pair(v[2][c], v[3][c]);
            odd.x = hi_pair(v[0][c], v[1][c]);
            odd.y = hi_pair(v[2][c], v[3][c]);
            const u32x2 first = odd_first ? odd : even;
            const u32x2 second = odd_first ? even : odd;
            const int r1 = rb * 8 + 2 * c + (odd_first ? 1 : 0);
            const int r2 = rb * 8 + 2 * c + (odd_first ? 0 : 1);
            *reinterpret_cast<u32x2*>(lds + lds_off(r1, g) + h) = first;
            *reinterpret_cast<u32x2*>(lds + lds_off(r2, g) + h) = second;
        }
    }
}

__device__ inline bf16x8 frag(const uint16_t* lds, int row, int g) {
    return __builtin_bit_cast(bf16x8, *reinterpret_cast<const u16x8*>(lds + lds_off(row, g)));
}

template <bool AROW, bool BROW, bool ANT, bool BNT>
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

    const int kc = g.K / kKC;
    const int total = (un.p1 - un.p0) * kc;
    float* out = un.slot < 0 ? g.W + int64_t(un.seg) * g.w_elems : g.partials + int64_t(un.slot) * g.w_elems;
    if (total == 0) {
        // an empty U range of a key: its partial tile is zero
        for (int e = threadIdx.x; e < kB * kB; e += kThreads)
            out[int64_t(m0 + e / kB) * g.ldw + n0 + e % kB] = 0.f;
        return;
    }
    // chunk c of the unit: pair p0 + c / kc, k offset (c % kc) * 64; indices
    // past the end reload the last chunk so the load pattern stays uniform
    const int32_t lo_a = lane_offset<AROW>(int32_t(g.lda)), lo_b = lane_offset<BROW>(int32_t(g.ldb));
    const int32_t st_a = AROW ? int32_t(g.lda) : 32 * int32_t(g.lda);
    const int32_t st_b = BROW ? int32_t(g.ldb) : 32 * int32_t(g.ldb);
    auto src_a = [&](int c) {
        c = min(c, total - 1);
        return g.A + int64_t(g.pa[un.p0 + c / kc]) * g.a_elems + chunk_offset<AROW>(g.lda, m0, (c % kc) * kKC);
    };
    auto src_b = [&](int c) {
        c = min(c, total - 1);
        return g.B + int64_t(g.pb[un.p0 + c / kc]) * g.b_elems + chunk_offset<BROW>(g.ldb, n0, (c % kc) * kKC);
    };

    u32x4 ra0[4], rb0[4], ra1[4], rb1[4];
    load_chunk<AROW, ANT>(ra0, src_a(0), lo_a, st_a);
    load_chunk<BROW, BNT>(rb0, src_b(0), lo_b, st_b);
    load_chunk<AROW, ANT>(ra1, src_a(1), lo_a, st_a);
    load_chunk<BROW, BNT>(rb1, src_b(1), lo_b, st_b);
    store_chunk<AROW>(lds[0][0], ra0);
    store_chunk<BROW>(lds[0][1], rb0);
    __syncthreads();

    const int row = lane & 31, half = lane >> 5;
    auto compute = [&](const uint16_t* As, const uint16_t* Bs) {
#pragma unroll
        for (int ks = 0; ks < kKC / 16; ks++) {
            const int gr = ks * 2 + half;
            bf16x8 a0 = frag(As, wm * 64 + row, gr);
            bf16x8 a1 = frag(As, wm * 64 + 32 + row, gr);
            bf16x8 b0 = frag(Bs, wn * 64 + row, gr);
            bf16x8 b1 = frag(Bs, wn * 64 + 32 + row, gr);
            acc[0][0] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a0, b0, acc[0][0], 0, 0, 0);
            acc[0][1] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a0, b1, acc[0][1], 0, 0, 0);
            acc[1][0] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a1, b0, acc[1][0], 0, 0, 0);
            acc[1][1] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a1, b1, acc[1][1], 0, 0, 0);
        }
    };

    for (int it = 0; it < total; it += 2) {
        // even chunk `it` in LDS buffer 0; chunk it+1 in ra1/rb1
        load_chunk<AROW, ANT>(ra0, src_a(it + 2), lo_a, st_a);
        load_chunk<BROW, BNT>(rb0, src_b(it + 2), lo_b, st_b);
        compute(lds[0][0], lds[0][1]);
        store_chunk<AROW>(lds[1][0], ra1);
        store_chunk<BROW>(lds[1][1], rb1);
        __syncthreads();
        if (it + 1 >= total) break;
        // odd chunk it+1 in LDS buffer 1; chunk it+2 in ra0/rb0
        load_chunk<AROW, ANT>(ra1, src_a(it + 3), lo_a, st_a);
        load_chunk<BROW, BNT>(rb1, src_b(it + 3), lo_b, st_b);
        compute(lds[1][0], lds[1][1]);
        store_chunk<AROW>(lds[0][0], ra0);
        store_chunk<BROW>(lds[0][1], rb0);
        __syncthreads();
    }

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
                            float* w_tiles, int64_t n_pairs, int64_t unit_bound, hipStream_t s) {
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
    // an operand whose tiles are each used by about one pair is streamed
    const int64_t n_a = p.swap ? L.n_v : L.n_u, n_b = p.swap ? L.n_u : L.n_v;
    const bool ant = 2 * n_a >= n_pairs, bnt = 2 * n_b >= n_pairs;
    const int sel = (p.fast_a_rowfast ? 8 : 0) | (p.fast_b_rowfast ? 4 : 0) | (ant ? 2 : 0) | (bnt ? 1 : 0);
#define TRE_FAST_CASE(X)                                                                                   \
    case X:                                                                                                \
        k_gemm_fast<bool(X & 8), bool(X & 4), bool(X & 2), bool(X & 1)><<<grid, kThreads, 0, s>>>(g); \
        break;
    switch (sel) {
        TRE_FAST_CASE(0) TRE_FAST_CASE(1) TRE_FAST_CASE(2) TRE_FAST_CASE(3)
        TRE_FAST_CASE(4) TRE_FAST_CASE(5) TRE_FAST_CASE(6) TRE_FAST_CASE(7)
        TRE_FAST_CASE(8) TRE_FAST_CASE(9) TRE_FAST_CASE(10) TRE_FAST_CASE(11)
        TRE_FAST_CASE(12) TRE_FAST_CASE(13) TRE_FAST_CASE(14) TRE_FAST_CASE(15)
    }
#undef TRE_FAST_CASE
    return hipGetLastError();
}

}  // namespace tre
