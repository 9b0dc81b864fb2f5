// One three-operand EinSum "U,V,X->W" whose two small operands each meet U on
// a promoted label of their own (a, b: U's last two labels) and share one
// demoted label r with the output -- the non-binary EinSum of Sec. 8, e.g.
// A[i,r] = sum_jk T[i,j,k] B[j,r] C[k,r] -- without the intermediate relation
// of the binary path.
//
// Relational part (Sec. 5's join and GROUP BY over three relations): every U
// tuple looks up the V tuple with its key on a and the X tuple with its key
// on b (binary search; V and X are keyed by that one label); matched U
// tuples are compacted, in U order, into triples (u, v, x) with their packed
// output key; a stable radix sort orders them by output key unless W's
// promoted labels are a prefix of U's key (then U order already is); head
// flags, a scan and compaction give the output keys and their segments.
//
// Tile part: with p, q the last two labels of U (p outer), a U tile is a
// matrix [M rows = U's other tile labels] x [tp * tq], and one triple
// contributes T (M x tp*tq) times the Khatri-Rao block KR[(p', q'), r] =
// P[p', r] * Q[q', r], P being the operand joined on p and Q the one joined
// on q.  k3_gemm computes that with fp32 MFMA (v_mfma_f32_16x16x4f32) per
// 32 x 64 output block: T is streamed through LDS in chunks of 128
// contracted elements (two stages, prefetched one chunk ahead in
// registers), P and Q of the triple are staged in LDS (Q transposed), and
// the B operand of each MFMA is formed in registers as P * Q, so KR is never
// stored.  When tq is 16, 32 or 64, k3_gemm_q is used instead: it contracts
// over q' with MFMA (Q held in registers for the whole triple) and scales by
// P[p', r] afterwards, one multiply-add per output element and p' (measured
// 0.52 ms against 0.63 ms for k3_gemm on the 4096^3 sparse 3-way workload).
// The triples are dealt to the resident workgroups in equal
// contiguous ranges; a workgroup accumulates each segment's part of its range
// in registers, and segments split between ranges are summed by k3_reduce in
// range order (no atomics on values).
#include "tre_internal.h"

#include <algorithm>
#include <cstring>

namespace tre {

namespace {

typedef float floatx4 __attribute__((ext_vector_type(4)));

constexpr int kThreads = 256;
constexpr int kRows = 32;              // output rows (m) per workgroup
constexpr int kCols = 64;              // output columns (r) per workgroup
constexpr int kChunk = 128;            // contracted elements per staged chunk
constexpr int kPitchT = kChunk + 4;    // floats per staged T row
constexpr int kMaxPQ = 64;             // tile extent limit of p and q
constexpr int kMaxRows = kMaxDims - 2; // row labels of U

inline unsigned blocks_for(int64_t n) { return unsigned((n + kThreads - 1) / kThreads); }

struct F3Desc {
    int32_t nm;                        // row labels (U's labels before p, q)
    int64_t M;                         // product of their tile extents
    int32_t tp, tq, R;                 // tile extents of p, q; extent of r
    int64_t te_u, te_p, te_q, te_w;    // tile elements of U, the p operand, the q operand, W
    int64_t p_sp, p_sr;                // strides of (p', r) in a tile of the p operand
    int64_t q_sq, q_sr;                // strides of (q', r) in a tile of the q operand
    int32_t msize[kMaxRows];           // tile extent of each row label (U order)
    int64_t mwst[kMaxRows];            // its stride in the W tile
    int64_t w_sr;                      // stride of r in the W tile
    int32_t ru, pos_p, pos_q;          // U key arity; positions of p and q in U's key
    int32_t rw;                        // W key arity
    int32_t wpos[kMaxDims], wbits[kMaxDims];  // W key attributes: position in U's key, bits
    int32_t wkey_bits;
    int32_t v_on_p;                    // V is the operand joined on p
    int32_t mblocks, rblocks;
    int32_t needs_sort;
    int32_t radix_u[kMaxDims];         // extent / tile of U's key attributes
    int32_t radix_p, radix_q;          // of the p and q key attributes
    int32_t masked;                    // W has exactly U's labels and r is summed
};

struct F3Header {
    int32_t err_u, err_p, err_q, pad0;
    int64_t n_tri;
    int64_t n_w;
    int64_t pad2[12];
};

// ------------------------------------------------------------ relational part

__device__ inline int64_t find_key(const int32_t* __restrict__ keys, int64_t n, int32_t k) {
    int64_t lo = 0, hi = n;
    while (lo < hi) {
        const int64_t mid = (lo + hi) >> 1;
        if (keys[mid] < k) lo = mid + 1;
        else hi = mid;
    }
    return (lo < n && keys[lo] == k) ? lo : -1;
}

// Per U tuple: the p- and q-operand tuples it meets (or -1) and the match
// flag (flag[n_u] = 0 closes the array for the scan).
__global__ void k3_match(const int32_t* __restrict__ u_keys, int64_t n_u, F3Desc d,
                         const int32_t* __restrict__ p_keys, int64_t n_p, const int32_t* __restrict__ q_keys,
                         int64_t n_q, int32_t* __restrict__ flag, int32_t* __restrict__ ip, int32_t* __restrict__ iq) {
    const int64_t s = int64_t(blockIdx.x) * blockDim.x + threadIdx.x;
    if (s > n_u) return;
    if (s == n_u) {
        flag[s] = 0;
        return;
    }
    const int32_t* key = u_keys + s * d.ru;
    const int64_t a = find_key(p_keys, n_p, key[d.pos_p]);
    const int64_t b = find_key(q_keys, n_q, key[d.pos_q]);
    ip[s] = int32_t(a);
    iq[s] = int32_t(b);
    flag[s] = (a >= 0 && b >= 0) ? 1 : 0;
}

__device__ inline uint64_t pack_w(const int32_t* key, const F3Desc& d) {
    uint64_t k = 0;
    for (int i = 0; i < d.rw; i++) k = (k << d.wbits[i]) | uint64_t(uint32_t(key[d.wpos[i]]));
    return k;
}

// Matched U tuples, in U order, become triples with their packed W key.
__global__ void k3_compact(const int32_t* __restrict__ u_keys, int64_t n_u, F3Desc d,
                           const int32_t* __restrict__ pos, const int32_t* __restrict__ ip,
                           const int32_t* __restrict__ iq, int32_t* __restrict__ tu, int32_t* __restrict__ tp,
                           int32_t* __restrict__ tq, uint64_t* __restrict__ wkey, uint32_t* __restrict__ perm) {
    const int64_t s = int64_t(blockIdx.x) * blockDim.x + threadIdx.x;
    if (s >= n_u || ip[s] < 0 || iq[s] < 0) return;
    const int64_t t = pos[s];
    tu[t] = int32_t(s);
    tp[t] = ip[s];
    tq[t] = iq[s];
    wkey[t] = pack_w(u_keys + s * d.ru, d);
    if (perm) perm[t] = uint32_t(t);
}

// When the p and q operands hold every key of their key spaces, every U
// tuple is a triple and its partners are its own key values (sorted strictly
// increasing keys of n = radix tuples are exactly 0 .. n - 1): triple s is
// U tuple s, no search, no scan.  Key values outside their range come only
// from keys that fail validation (reported by the host) and are clamped so
// nothing is read out of bounds.  `wkey` may be null (the masked form, whose
// output keys are U's keys).
__global__ void k3_dense(const int32_t* __restrict__ u_keys, int64_t n_u, F3Desc d, int32_t* __restrict__ tu,
                         int32_t* __restrict__ tp, int32_t* __restrict__ tq, uint64_t* __restrict__ wkey,
                         uint32_t* __restrict__ perm) {
    const int64_t s = int64_t(blockIdx.x) * blockDim.x + threadIdx.x;
    if (s >= n_u) return;
    const int32_t* key = u_keys + s * d.ru;
    tu[s] = int32_t(s);
    tp[s] = min(max(key[d.pos_p], 0), d.radix_p - 1);
    tq[s] = min(max(key[d.pos_q], 0), d.radix_q - 1);
    if (wkey) wkey[s] = pack_w(key, d);
    if (perm) perm[s] = uint32_t(s);
}

// Output keys of the masked form: U's keys, row for row.
__global__ void k3_copy_keys(const int32_t* __restrict__ u_keys, int64_t n, int32_t* __restrict__ out) {
    const int64_t i = int64_t(blockIdx.x) * blockDim.x + threadIdx.x;
    if (i < n) out[i] = u_keys[i];
}

// Triples in sorted order, from the permutation of the sort.
__global__ void k3_gather(const uint32_t* __restrict__ perm, int64_t n, const int32_t* __restrict__ tu,
                          const int32_t* __restrict__ tp, const int32_t* __restrict__ tq, int32_t* __restrict__ su,
                          int32_t* __restrict__ sp, int32_t* __restrict__ sq) {
    const int64_t t = int64_t(blockIdx.x) * blockDim.x + threadIdx.x;
    if (t >= n) return;
    const uint32_t o = perm[t];
    su[t] = tu[o];
    sp[t] = tp[o];
    sq[t] = tq[o];
}

__global__ void k3_heads(const uint64_t* __restrict__ wkey, int64_t n, int32_t* __restrict__ heads) {
    const int64_t t = int64_t(blockIdx.x) * blockDim.x + threadIdx.x;
    if (t > n) return;
    heads[t] = (t < n && (t == 0 || wkey[t] != wkey[t - 1])) ? 1 : 0;
}

// Segment starts (seg_start[n_w] = n) and keys; n_w into the header.
__global__ void k3_segments(const uint64_t* __restrict__ wkey, int64_t n, const int32_t* __restrict__ seg_of,
                            int32_t* __restrict__ seg_start, uint64_t* __restrict__ seg_key, F3Header* hdr) {
    const int64_t t = int64_t(blockIdx.x) * blockDim.x + threadIdx.x;
    if (t > n) return;
    if (t == n) {
        seg_start[seg_of[n]] = int32_t(n);
        hdr->n_w = seg_of[n];
        return;
    }
    if (t == 0 || wkey[t] != wkey[t - 1]) {
        seg_start[seg_of[t]] = int32_t(t);
        seg_key[seg_of[t]] = wkey[t];
    }
}

// ------------------------------------------------------------ tile part
//
// Work split: the items are (output block, triple) pairs, blk * nt + t, in
// that order (blk = mb * rblocks + rb), and workgroup b of the n_wg resident
// workgroups takes items [b * total / n_wg, (b + 1) * total / n_wg), so every
// workgroup gets the same number of triples to within one.  A workgroup
// walks its range as pieces, each the part of one (segment, block) inside
// the range, and accumulates a piece in registers.  A piece that is a whole
// (segment, block) is written to W; otherwise it goes to a block-sized
// partial slot -- slot 2b if the segment began in an earlier range, slot
// 2b + 1 if it only continues into a later one -- and k3_reduce sums the
// slots of every split (segment, block) in range order (no atomics).

struct F3Args {
    const float* U;
    const float* P;
    const float* Q;
    const int32_t* tu;
    const int32_t* tp;
    const int32_t* tq;
    const int32_t* seg_of;     // exclusive scan of the head flags: triple t is in segment seg_of[t + 1] - 1
    const int32_t* seg_start;  // [n_w + 1]
    int64_t nt;                // triples
    int64_t n_wg;              // workgroups of the launch
    int32_t brows, mblocks;    // output rows per block and row blocks
    float* W;
    float* part;               // [2 n_wg][brows][kCols]
    F3Desc d;
};

__device__ inline int64_t w_row_offset(const F3Desc& d, int64_t m) {
    int64_t off = 0;
#pragma unroll
    for (int i = kMaxRows - 1; i >= 0; i--) {
        if (i >= d.nm) continue;
        off += (m % d.msize[i]) * d.mwst[i];
        m /= d.msize[i];
    }
    return off;
}

// Where a piece's block of output goes.
struct Dest {
    float* base;  // the W tile of the segment, or a partial slot
    bool slot;    // slot: block-local [brows][kCols]
    int64_t row0;
    int col0;
    __device__ void put(const F3Desc& d, int lr, int lc, float v) const {
        const int64_t m = row0 + lr;
        const int r = col0 + lc;
        if (m >= d.M || r >= d.R) return;
        if (slot) base[lr * kCols + lc] = v;
        else base[w_row_offset(d, m) + int64_t(r) * d.w_sr] = v;
    }
};

// The workgroup holding item x.
__device__ inline int64_t wg_of(int64_t x, int64_t total, int64_t n_wg) { return ((x + 1) * n_wg - 1) / total; }

// Walk this workgroup's pieces: begin(mb, rb) before a piece, triple(t,
// t_next) for each of its triples (t_next = the piece's next triple or -1),
// end(Dest) after it.
template <typename Begin, typename Triple, typename End>
__device__ inline void for_each_piece(const F3Args& g, Begin begin, Triple triple, End end) {
    const F3Desc& d = g.d;
    const int64_t total = g.nt * int64_t(g.mblocks) * d.rblocks;
    const int64_t b = blockIdx.x;
    const int64_t i1 = (b + 1) * total / g.n_wg;
    for (int64_t i = b * total / g.n_wg; i < i1;) {
        const int64_t blk = i / g.nt;
        const int32_t t = int32_t(i - blk * g.nt);
        const int32_t q = g.seg_of[t + 1] - 1;
        const int32_t s0 = g.seg_start[q], s1 = g.seg_start[q + 1];
        const int64_t pend = min(i1, blk * g.nt + s1);
        const bool before = s0 < t, cont = blk * g.nt + s1 > i1;
        const int mb = int(blk / d.rblocks), rb = int(blk % d.rblocks);
        begin(mb, rb);
        const int32_t t_end = t + int32_t(pend - i);
        for (int32_t tt = t; tt < t_end; tt++) triple(tt, tt + 1 < t_end ? tt + 1 : -1);
        Dest dst;
        dst.row0 = int64_t(mb) * g.brows;
        dst.col0 = rb * kCols;
        dst.slot = before || cont;
        dst.base = !dst.slot ? g.W + int64_t(q) * d.te_w
                             : g.part + (2 * b + (before ? 0 : 1)) * int64_t(g.brows) * kCols;
        end(dst);
        i = pend;
    }
}

// T chunk loads: 32 rows x kChunk elements, 4 float4 per thread.
struct ChunkLoader {
    float4 pre[4];
    __device__ void load(const F3Desc& d, const float* Tt, int64_t row0, int64_t KK, int c) {
        const int tid = threadIdx.x;
#pragma unroll
        for (int i = 0; i < 4; i++) {
            const int idx = tid + kThreads * i, row = idx >> 5, c4 = idx & 31;
            const int64_t kk = int64_t(c) * kChunk + 4 * c4;
            const int64_t m = row0 + row;
            pre[i] = (m < d.M && kk < KK) ? *reinterpret_cast<const float4*>(Tt + m * KK + kk)
                                          : float4{0.f, 0.f, 0.f, 0.f};
        }
    }
    __device__ void store(float* st) const {
        const int tid = threadIdx.x;
#pragma unroll
        for (int i = 0; i < 4; i++) {
            const int idx = tid + kThreads * i, row = idx >> 5, c4 = idx & 31;
            *reinterpret_cast<float4*>(st + row * kPitchT + 4 * c4) = pre[i];
        }
    }
};

// Stage the block's columns of the triple's P tile ([tp][kCols]) and Q tile
// (transposed, [kCols][qpitch]) in LDS.
__device__ inline void stage_pq(const F3Desc& d, const float* Pt, const float* Qt, int col0, int tq, int qpitch,
                                float* sP, float* sQ) {
    const int tid = threadIdx.x;
    for (int e = tid; e < d.tp * kCols; e += kThreads) {
        const int pp = e / kCols, c = e % kCols, r = col0 + c;
        sP[e] = r < d.R ? Pt[pp * d.p_sp + int64_t(r) * d.p_sr] : 0.f;
    }
    for (int e = tid; e < tq * kCols; e += kThreads) {
        const int qq = e / kCols, c = e % kCols, r = col0 + c;
        sQ[c * qpitch + qq] = r < d.R ? Qt[qq * d.q_sq + int64_t(r) * d.q_sr] : 0.f;
    }
}

// The P and Q slices for k3_gemm_q, both row-major [rows][kCols] (Q not
// transposed).  When the block's columns all lie inside R, straight from
// memory into LDS (global_load_lds_dword: lane l of a wavefront lands at the
// instruction's LDS address + 4 l), every load issued before the wait at the
// next barrier and no registers held; otherwise through registers as above.
__device__ inline void stage_pq_rows(const F3Desc& d, const float* Pt, const float* Qt, int col0, int tq, float* sP,
                                     float* sQ) {
    const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
    if (col0 + kCols <= d.R) {
        const int64_t r = col0 + lane;
        for (int row = w; row < d.tp; row += kThreads / 64)
            __builtin_amdgcn_global_load_lds(
                (const __attribute__((address_space(1))) void*)(Pt + row * d.p_sp + r * d.p_sr),
                (__attribute__((address_space(3))) void*)(sP + row * kCols), 4, 0, 0);
        for (int row = w; row < tq; row += kThreads / 64)
            __builtin_amdgcn_global_load_lds(
                (const __attribute__((address_space(1))) void*)(Qt + row * d.q_sq + r * d.q_sr),
                (__attribute__((address_space(3))) void*)(sQ + row * kCols), 4, 0, 0);
        return;
    }
    const int tid = threadIdx.x;
    for (int e = tid; e < d.tp * kCols; e += kThreads) {
        const int r = col0 + e % kCols;
        sP[e] = r < d.R ? Pt[(e / kCols) * d.p_sp + int64_t(r) * d.p_sr] : 0.f;
    }
    for (int e = tid; e < tq * kCols; e += kThreads) {
        const int r = col0 + e % kCols;
        sQ[e] = r < d.R ? Qt[(e / kCols) * d.q_sq + int64_t(r) * d.q_sr] : 0.f;
    }
}

// Any tq (a multiple of 4).  Dynamic LDS: T stages [2][kRows][kPitchT], P
// slice [tp][kCols], Q slice transposed [kCols][tq + 4] (floats).  Waves:
// rows [16 mh, +16) and columns [32 rh, +32) of the block; the B operand of
// every MFMA is P[p', r] * Q[q', r] formed in registers.
__global__ __launch_bounds__(kThreads) void k3_gemm(F3Args g) {
    extern __shared__ float lds[];
    const F3Desc& d = g.d;
    float* sT = lds;
    float* sP = lds + 2 * kRows * kPitchT;
    const int qpitch = d.tq + 4;
    float* sQ = sP + d.tp * kCols;
    const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
    const int mh = w & 1, rh = w >> 1;
    const int n = lane & 15, gq = lane >> 4;
    const int64_t KK = int64_t(d.tp) * d.tq;
    const int nchunks = int((KK + kChunk - 1) / kChunk);
    floatx4 acc[2][2];
    int64_t row0 = 0;
    int col0 = 0;
    ChunkLoader ld;
    auto begin = [&](int mb, int rb) {
        row0 = int64_t(mb) * kRows;
        col0 = rb * kCols;
#pragma unroll
        for (int t = 0; t < 2; t++)
#pragma unroll
            for (int e = 0; e < 2; e++) acc[t][e] = floatx4{0.f, 0.f, 0.f, 0.f};
    };
    auto triple = [&](int32_t t, int32_t) {
        const float* Tt = g.U + int64_t(g.tu[t]) * d.te_u;
        __syncthreads();  // the previous triple is done with sP, sQ and both T stages
        stage_pq(d, g.P + int64_t(g.tp[t]) * d.te_p, g.Q + int64_t(g.tq[t]) * d.te_q, col0, d.tq, qpitch, sP, sQ);
        ld.load(d, Tt, row0, KK, 0);
        for (int c = 0; c < nchunks; c++) {
            float* st = sT + (c & 1) * kRows * kPitchT;
            ld.store(st);
            __syncthreads();
            if (c + 1 < nchunks) ld.load(d, Tt, row0, KK, c + 1);
            // this lane's contracted index at the chunk start, as (p', q')
            int64_t kk0 = int64_t(c) * kChunk + 4 * gq;
            int pp = int(kk0 / d.tq), qq = int(kk0 % d.tq);
            const float* arow = st + (16 * mh + n) * kPitchT + 4 * gq;
#pragma unroll 2
            for (int kq = 0; kq < kChunk / 16; kq++) {
                const float4 a4 = *reinterpret_cast<const float4*>(arow + 16 * kq);
                const bool ok = kk0 < KK;
                const int ppc = ok ? pp : 0, qqc = ok ? qq : 0;
#pragma unroll
                for (int tt = 0; tt < 2; tt++) {
                    const int cl = 32 * rh + 16 * tt + n;
                    const float pv = ok ? sP[ppc * kCols + cl] : 0.f;
                    const float4 q4 = *reinterpret_cast<const float4*>(sQ + cl * qpitch + qqc);
                    acc[tt][0] = __builtin_amdgcn_mfma_f32_16x16x4f32(a4.x, pv * q4.x, acc[tt][0], 0, 0, 0);
                    acc[tt][1] = __builtin_amdgcn_mfma_f32_16x16x4f32(a4.y, pv * q4.y, acc[tt][1], 0, 0, 0);
                    acc[tt][0] = __builtin_amdgcn_mfma_f32_16x16x4f32(a4.z, pv * q4.z, acc[tt][0], 0, 0, 0);
                    acc[tt][1] = __builtin_amdgcn_mfma_f32_16x16x4f32(a4.w, pv * q4.w, acc[tt][1], 0, 0, 0);
                }
                kk0 += 16;
                qq += 16;
                while (qq >= d.tq) {
                    qq -= d.tq;
                    pp++;
                }
            }
        }
    };
    auto end = [&](const Dest& dst) {
        // lane holds rows 4 gq + i, column n of each 16 x 16 tile
#pragma unroll
        for (int tt = 0; tt < 2; tt++) {
            const floatx4 v = acc[tt][0] + acc[tt][1];
#pragma unroll
            for (int i = 0; i < 4; i++) dst.put(d, 16 * mh + 4 * gq + i, 32 * rh + 16 * tt + n, v[i]);
        }
    };
    for_each_piece(g, begin, triple, end);
}

// tq = TQ in {16, 32, 64}, ordered the other way round: for every p' the
// MFMAs contract over q' only, Y[m, r] = sum_q' T[m, p', q'] Q[q', r], and
// the result is scaled by P[p', r] and added to the accumulator (acc +=
// P[p', r] * Y[m, r], one fused multiply-add per element and p').  The B
// operand of every MFMA is then a plain Q element, held in registers for the
// whole triple (lane group g of the 16x16x4 MFMA takes q' = g * TQ/4 + s for
// step s, so a lane's A values are contiguous in the staged T row and come
// in 16-byte LDS reads), and the scale-add of p' - 1 is issued after the
// MFMAs of p' so that it does not wait for them.  The first T chunk of the
// piece's next triple is loaded during the last chunk of the current one.
template <int TQ>
__global__ __launch_bounds__(kThreads, 3) void k3_gemm_q(F3Args g) {
    constexpr int kS = TQ / 4;           // MFMA steps per p'
    constexpr int kPpc = kChunk / TQ;    // p' rows per staged chunk
    static_assert(kS % 4 == 0 && kChunk % TQ == 0, "TQ must be 16, 32 or 64");
    extern __shared__ float lds[];
    const F3Desc& d = g.d;
    float* sT = lds;
    float* sP = lds + 2 * kRows * kPitchT;
    constexpr int qpitch = TQ + 4;
    float* sQ = sP + d.tp * kCols;
    const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
    const int mh = w & 1, rh = w >> 1;
    const int n = lane & 15, gq = lane >> 4;
    const int64_t KK = int64_t(d.tp) * TQ;
    const int nchunks = int((KK + kChunk - 1) / kChunk);
    const int cl0 = 32 * rh + n, cl1 = cl0 + 16;  // this lane's two columns in the block
    const floatx4 zero = {0.f, 0.f, 0.f, 0.f};
    floatx4 acc[2], yprev[2];
    float pvprev[2];
    int64_t row0 = 0;
    int col0 = 0;
    bool have_next = false;  // the first chunk of the next triple is in ld
    ChunkLoader ld;
    auto begin = [&](int mb, int rb) {
        row0 = int64_t(mb) * kRows;
        col0 = rb * kCols;
        have_next = false;
#pragma unroll
        for (int t = 0; t < 2; t++) {
            acc[t] = yprev[t] = zero;
            pvprev[t] = 0.f;
        }
    };
    auto triple = [&](int32_t t, int32_t t_next) {
        const float* Tt = g.U + int64_t(g.tu[t]) * d.te_u;
        __syncthreads();  // the previous triple is done with sP, sQ and both T stages
        stage_pq_rows(d, g.P + int64_t(g.tp[t]) * d.te_p, g.Q + int64_t(g.tq[t]) * d.te_q, col0, TQ, sP, sQ);
        if (!have_next) ld.load(d, Tt, row0, KK, 0);
        have_next = false;
        float qreg[2][kS];
        for (int c = 0; c < nchunks; c++) {
            float* st = sT + (c & 1) * kRows * kPitchT;
            ld.store(st);
            __syncthreads();
            if (c + 1 < nchunks) {
                ld.load(d, Tt, row0, KK, c + 1);
            } else if (t_next >= 0) {
                ld.load(d, g.U + int64_t(g.tu[t_next]) * d.te_u, row0, KK, 0);
                have_next = true;
            }
            if (c == 0) {
                // this lane's Q elements for the whole triple: q' = gq * kS + j
#pragma unroll
                for (int j = 0; j < kS; j++) {
                    qreg[0][j] = sQ[(gq * kS + j) * kCols + cl0];
                    qreg[1][j] = sQ[(gq * kS + j) * kCols + cl1];
                }
            }
            const float* arow = st + (16 * mh + n) * kPitchT + gq * kS;
#pragma unroll
            for (int pl = 0; pl < kPpc; pl++) {
                const int pg = c * kPpc + pl;  // p' of this row of the chunk
                float a[kS];
#pragma unroll
                for (int j = 0; j < kS; j += 4) {
                    const float4 v = *reinterpret_cast<const float4*>(arow + pl * TQ + j);
                    a[j] = v.x, a[j + 1] = v.y, a[j + 2] = v.z, a[j + 3] = v.w;
                }
                const int pc = min(pg, d.tp - 1);
                const float p0 = sP[pc * kCols + cl0], p1 = sP[pc * kCols + cl1];
                floatx4 y0 = __builtin_amdgcn_mfma_f32_16x16x4f32(a[0], qreg[0][0], zero, 0, 0, 0);
                floatx4 y1 = __builtin_amdgcn_mfma_f32_16x16x4f32(a[0], qreg[1][0], zero, 0, 0, 0);
#pragma unroll
                for (int j = 1; j < kS; j++) {
                    y0 = __builtin_amdgcn_mfma_f32_16x16x4f32(a[j], qreg[0][j], y0, 0, 0, 0);
                    y1 = __builtin_amdgcn_mfma_f32_16x16x4f32(a[j], qreg[1][j], y1, 0, 0, 0);
                }
                // scale-add of the previous p' while these MFMAs run
                acc[0] += pvprev[0] * yprev[0];
                acc[1] += pvprev[1] * yprev[1];
                yprev[0] = y0;
                yprev[1] = y1;
                pvprev[0] = pg < d.tp ? p0 : 0.f;
                pvprev[1] = pg < d.tp ? p1 : 0.f;
            }
        }
    };
    auto end = [&](const Dest& dst) {
        acc[0] += pvprev[0] * yprev[0];
        acc[1] += pvprev[1] * yprev[1];
#pragma unroll
        for (int tt = 0; tt < 2; tt++)
#pragma unroll
            for (int i = 0; i < 4; i++) dst.put(d, 16 * mh + 4 * gq + i, 32 * rh + 16 * tt + n, acc[tt][i]);
    };
    for_each_piece(g, begin, triple, end);
}

// Sum the slots of every split (segment, block): workgroup b - 1 of this
// launch looks at the boundary where range b starts; the first boundary
// inside a (segment, block) sums slot 2 b0 + 1, slots 2 b of the ranges
// inside it and slot 2 b1, in that order, into W.
__global__ __launch_bounds__(kThreads) void k3_reduce(F3Args g) {
    const F3Desc& d = g.d;
    const int64_t total = g.nt * int64_t(g.mblocks) * d.rblocks;
    const int64_t b = int64_t(blockIdx.x) + 1;
    const int64_t x = b * total / g.n_wg;
    if (x <= 0 || x >= total) return;
    const int64_t blk = x / g.nt;
    const int32_t t = int32_t(x - blk * g.nt);
    const int32_t q = g.seg_of[t + 1] - 1;
    const int32_t s0 = g.seg_start[q], s1 = g.seg_start[q + 1];
    if (s0 == t) return;  // the range starts with a segment: nothing split here
    const int64_t b0 = wg_of(blk * g.nt + s0, total, g.n_wg);
    if (b != b0 + 1) return;
    const int64_t b1 = wg_of(blk * g.nt + s1 - 1, total, g.n_wg);
    const int mb = int(blk / d.rblocks), rb = int(blk % d.rblocks);
    Dest dst;
    dst.base = g.W + int64_t(q) * d.te_w;
    dst.slot = false;
    dst.row0 = int64_t(mb) * g.brows;
    dst.col0 = rb * kCols;
    const int64_t bs = int64_t(g.brows) * kCols;
    // kRedPer elements per thread at a time, so each slot's loads are all in
    // flight together (the sum still runs slot by slot, in range order)
    constexpr int kRedPer = 8;
    for (int e0 = threadIdx.x; e0 < bs; e0 += kRedPer * kThreads) {
        float v[kRedPer];
#pragma unroll
        for (int i = 0; i < kRedPer; i++) {
            const int64_t e = e0 + i * kThreads;
            v[i] = e < bs ? g.part[(2 * b0 + 1) * bs + e] : 0.f;
        }
        for (int64_t bb = b0 + 1; bb <= b1; bb++) {
            const float* src = g.part + (bb < b1 ? 2 * bb : 2 * b1) * bs;
            float x[kRedPer];
#pragma unroll
            for (int i = 0; i < kRedPer; i++) {
                const int64_t e = e0 + i * kThreads;
                x[i] = e < bs ? src[e] : 0.f;
            }
#pragma unroll
            for (int i = 0; i < kRedPer; i++) v[i] += x[i];
        }
#pragma unroll
        for (int i = 0; i < kRedPer; i++) {
            const int64_t e = e0 + i * kThreads;
            if (e < bs) dst.put(d, int(e / kCols), int(e % kCols), v[i]);
        }
    }
}

// Masked form: W has U's labels, so every triple is its own output tuple, in
// U order, and with tiles of 1 on p and q its value is the U tile times one
// dot product over r:  W[t][e] = U[tu[t]][e] * sum_r P[tp[t]][r] Q[tq[t]][r].
// One wavefront per kMaskedBatch consecutive triples: the lanes stride over r
// (16-byte loads when R is a multiple of 4 and the tiles are 16-byte aligned),
// the batch's P and Q rows are all in flight at once, and a butterfly of lane
// exchanges sums each dot product in a fixed order.  Consecutive triples of
// one U row share their P row, which then comes from the cache.
constexpr int kMaskedBatch = 4;

__device__ inline float wave_sum(float v) {
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
    return v;
}

template <bool V4>
__global__ __launch_bounds__(kThreads) void k3_masked(const float* __restrict__ U, const float* __restrict__ P,
                                                      const float* __restrict__ Q, const int32_t* __restrict__ tu,
                                                      const int32_t* __restrict__ tp, const int32_t* __restrict__ tq,
                                                      int64_t nt, int64_t te_u, int64_t R, float* __restrict__ W) {
    const int lane = threadIdx.x & 63;
    const int64_t t0 = (int64_t(blockIdx.x) * (kThreads / 64) + (threadIdx.x >> 6)) * kMaskedBatch;
    if (t0 >= nt) return;
    const float* p[kMaskedBatch];
    const float* q[kMaskedBatch];
    float acc[kMaskedBatch];
#pragma unroll
    for (int b = 0; b < kMaskedBatch; b++) {
        const int64_t t = min(t0 + b, nt - 1);  // past the end: repeat the last triple, never written
        p[b] = P + int64_t(tp[t]) * R;
        q[b] = Q + int64_t(tq[t]) * R;
        acc[b] = 0.f;
    }
    if constexpr (V4) {
        for (int64_t r = 4 * lane; r < R; r += 256) {
            float4 x[kMaskedBatch], y[kMaskedBatch];
#pragma unroll
            for (int b = 0; b < kMaskedBatch; b++) {
                x[b] = *reinterpret_cast<const float4*>(p[b] + r);
                y[b] = *reinterpret_cast<const float4*>(q[b] + r);
            }
#pragma unroll
            for (int b = 0; b < kMaskedBatch; b++) {
                acc[b] = fmaf(x[b].x, y[b].x, acc[b]);
                acc[b] = fmaf(x[b].y, y[b].y, acc[b]);
                acc[b] = fmaf(x[b].z, y[b].z, acc[b]);
                acc[b] = fmaf(x[b].w, y[b].w, acc[b]);
            }
        }
    } else {
        for (int64_t r = lane; r < R; r += 64)
#pragma unroll
            for (int b = 0; b < kMaskedBatch; b++) acc[b] = fmaf(p[b][r], q[b][r], acc[b]);
    }
#pragma unroll
    for (int b = 0; b < kMaskedBatch; b++) {
        const float dot = wave_sum(acc[b]);
        const int64_t t = t0 + b;
        if (t >= nt) break;
        const float* u = U + int64_t(tu[t]) * te_u;
        float* w = W + t * te_u;
        for (int64_t e = lane; e < te_u; e += 64) w[e] = u[e] * dot;
    }
}

__global__ void k3_write_keys(const uint64_t* __restrict__ seg_key, int64_t n_w, F3Desc d, int32_t* __restrict__ out) {
    const int64_t q = int64_t(blockIdx.x) * blockDim.x + threadIdx.x;
    if (q >= n_w) return;
    uint64_t k = seg_key[q];
    for (int a = d.rw - 1; a >= 0; a--) {
        out[q * d.rw + a] = int32_t(k & ((uint64_t(1) << d.wbits[a]) - 1));
        k >>= d.wbits[a];
    }
}

// ------------------------------------------------------------ host side

tre_status dev_fail(hipError_t e, const char* where) {
    set_error(std::string("tre_execute3: ") + where + ": " + hipGetErrorString(e));
    return TRE_E_DEVICE;
}

// Phase times from the five marks (join | units | contraction | reduction).
void finish_timing(tre_timing* timing, PhaseTimer& tm, bool deferred, bool dense, KernelEvents& ke) {
    if (!timing) return;
    std::memset(timing, 0, sizeof(*timing));
    timing->deferred = deferred ? 1 : 0;
    timing->join_path = dense ? 6 : 0;  // U drives the join; dense: partners indexed by key value
    if (deferred) {
        // the contraction kernel's own start and end, read later
        if (ke.launched) {
            timing->events[0] = reinterpret_cast<void*>(ke.start);
            timing->events[1] = reinterpret_cast<void*>(ke.stop);
            timing->pending = 1;
            ke.keep = true;
        }
        return;
    }
    timing->join_ms = tm.between(0, 1);
    timing->units_ms = tm.between(1, 2);
    timing->contract_ms = tm.between(2, 3);
    timing->reduce_ms = tm.between(3, 4);
    timing->total_ms = timing->join_ms + tm.between(1, 4);
}

tre_status fail(tre_status st, const char* msg) {
    set_error(std::string("tre_execute3: ") + msg);
    return st;
}

int32_t bit_width(int64_t x) {
    int32_t b = 0;
    while (x > 0) {
        b++;
        x >>= 1;
    }
    return b;
}

bool read_operand(const char*& c, std::string& op) {
    op.clear();
    while (*c >= 'a' && *c <= 'z') op.push_back(*c++);
    if (op.empty() || op.size() > size_t(kMaxDims)) return false;
    for (size_t i = 0; i < op.size(); i++)
        for (size_t j = i + 1; j < op.size(); j++)
            if (op[i] == op[j]) return false;
    return true;
}

tre_status parse3(const char* einsum, const char* upper, const int64_t* extent, const int32_t* tile, F3Desc& d) {
    std::memset(&d, 0, sizeof(d));
    if (!einsum || !upper || !extent || !tile) return fail(TRE_E_ARG, "null argument");
    std::string u, v, x, w;
    const char* c = einsum;
    if (!read_operand(c, u) || *c++ != ',' || !read_operand(c, v) || *c++ != ',' || !read_operand(c, x) ||
        c[0] != '-' || c[1] != '>')
        return fail(TRE_E_PARSE, "expected \"U,V,X->W\" with lower-case labels, none repeated in an operand");
    c += 2;
    if (!read_operand(c, w) || *c != '\0') return fail(TRE_E_PARSE, "bad output operand");
    bool up[26] = {};
    for (const char* k = upper; *k; k++) {
        if (*k < 'a' || *k > 'z') return fail(TRE_E_PARSE, "promoted labels must be lower-case letters");
        up[*k - 'a'] = true;
    }
    if (v.size() != 2 || x.size() != 2) return fail(TRE_E_SPLIT, "the two small operands have two labels each");
    char r = 0;
    for (char a : v)
        if (x.find(a) != std::string::npos) {
            if (r) return fail(TRE_E_SPLIT, "the small operands share exactly one label");
            r = a;
        }
    if (!r) return fail(TRE_E_SPLIT, "the small operands share exactly one label");
    const char a = v[0] == r ? v[1] : v[0];
    const char b = x[0] == r ? x[1] : x[0];
    const size_t nu = u.size();
    if (u.find(r) != std::string::npos || a == b || nu < 2 || !((u[nu - 2] == a && u[nu - 1] == b) ||
                                                                 (u[nu - 2] == b && u[nu - 1] == a)))
        return fail(TRE_E_SPLIT, "V and X must meet U on U's last two labels, one each, and share a label not in U");
    // W = U's other labels plus r, or exactly U's labels (masked form)
    d.masked = (w == u) ? 1 : 0;
    if (!d.masked) {
        if (w.size() != nu - 1 || w.find(r) == std::string::npos)
            return fail(TRE_E_SPLIT, "W holds U's labels other than the joined two plus the shared label, or U's labels");
        for (size_t i = 0; i + 2 < nu; i++)
            if (w.find(u[i]) == std::string::npos)
                return fail(TRE_E_SPLIT,
                            "W holds U's labels other than the joined two plus the shared label, or U's labels");
    }
    for (int l = 0; l < 26; l++)
        if (up[l] && u.find(char('a' + l)) == std::string::npos && char('a' + l) != r)
            return fail(TRE_E_SPLIT, "a promoted label is not in the expression");
    if (!up[a - 'a'] || !up[b - 'a'] || up[r - 'a'])
        return fail(TRE_E_SPLIT, "the joined labels must be promoted and the shared label demoted");
    auto tsz = [&](char l) -> int64_t { return up[l - 'a'] ? int64_t(tile[l - 'a']) : extent[l - 'a']; };
    for (char l : u + std::string(1, r)) {
        const int64_t e = extent[l - 'a'], t = tsz(l);
        if (e < 1 || t < 1 || t > e || e % t) return fail(TRE_E_SHAPE, "every tile size must divide its extent");
    }
    if (extent[r - 'a'] > (int64_t(1) << 30)) return fail(TRE_E_SHAPE, "shared label extent too large");
    const char p = u[nu - 2], q = u[nu - 1];
    d.tp = int32_t(tsz(p));
    d.tq = int32_t(tsz(q));
    d.R = int32_t(extent[r - 'a']);
    if (d.masked) {
        if (d.tp != 1 || d.tq != 1) return fail(TRE_E_SHAPE, "masked form: the joined labels take tiles of 1");
    } else if (d.tp > kMaxPQ || d.tq > kMaxPQ || d.tq % 4) {
        return fail(TRE_E_SHAPE, "tiles of U's last two labels must be at most 64, the last a multiple of 4");
    }
    d.nm = int32_t(nu - 2);
    d.M = 1;
    for (int i = 0; i < d.nm; i++) {
        d.msize[i] = int32_t(tsz(u[i]));
        d.M *= d.msize[i];
    }
    d.te_u = d.M * d.tp * d.tq;
    if (d.te_u > (int64_t(1) << 31)) return fail(TRE_E_SHAPE, "U tile too large");
    d.v_on_p = (a == p);
    // strides of the small operands' tiles (row-major over their two labels)
    const std::string& pop = d.v_on_p ? v : x;
    const std::string& qop = d.v_on_p ? x : v;
    d.te_p = int64_t(d.tp) * d.R;
    d.te_q = int64_t(d.tq) * d.R;
    d.p_sp = pop[0] == r ? 1 : d.R;
    d.p_sr = pop[0] == r ? d.tp : 1;
    d.q_sq = qop[0] == r ? 1 : d.R;
    d.q_sr = qop[0] == r ? d.tq : 1;
    // W strides (the masked form's W tile is laid out as U's)
    int64_t st = 1;
    int64_t wst[26] = {};
    for (int i = int(w.size()) - 1; i >= 0; i--) {
        wst[w[i] - 'a'] = st;
        st *= (w[i] == r) ? d.R : tsz(w[i]);
    }
    d.te_w = st;
    d.w_sr = d.masked ? 0 : wst[r - 'a'];
    for (int i = 0; i < d.nm; i++) d.mwst[i] = wst[u[i] - 'a'];
    // keys
    int upos[26];
    for (char l : u)
        if (up[l - 'a']) {
            upos[l - 'a'] = d.ru;
            d.radix_u[d.ru++] = int32_t(extent[l - 'a'] / tsz(l));
        }
    d.pos_p = upos[p - 'a'];
    d.pos_q = upos[q - 'a'];
    d.radix_p = int32_t(extent[p - 'a'] / d.tp);
    d.radix_q = int32_t(extent[q - 'a'] / d.tq);
    d.needs_sort = 0;
    for (char l : w)
        if (up[l - 'a']) {
            d.wpos[d.rw] = upos[l - 'a'];
            d.wbits[d.rw] = bit_width(extent[l - 'a'] / tsz(l) - 1);
            d.wkey_bits += d.wbits[d.rw];
            if (d.wpos[d.rw] != d.rw) d.needs_sort = 1;
            d.rw++;
        }
    if (d.wkey_bits > 64) return fail(TRE_E_SHAPE, "output key space exceeds 64 bits");
    d.mblocks = int32_t((d.M + kRows - 1) / kRows);
    d.rblocks = (d.R + kCols - 1) / kCols;
    return TRE_OK;
}

constexpr int kMaxOcc = 8;  // workgroups per CU counted for the partial slots

// CUs of the current device (256 when it cannot be read).
int64_t device_cus() {
    int dev = 0, cus = 0;
    if (hipGetDevice(&dev) != hipSuccess || hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) !=
                                                 hipSuccess || cus < 1)
        return 256;
    return cus;
}

struct F3Layout {
    size_t hdr, flag, pos, ip, iq, tmp, tu, tp, tq, su, sp, sq, wkey, wkey_alt, perm, perm_alt, hist, heads, seg_of,
        seg_start, seg_key, part, total;
    int64_t max_wg;  // workgroups the partial slots are sized for
};

size_t align256(size_t x) { return (x + 255) / 256 * 256; }

F3Layout f3_layout(const F3Desc& d, int64_t n_u) {
    const int64_t n = std::max<int64_t>(n_u, 1);
    F3Layout L{};
    L.max_wg = device_cus() * kMaxOcc;
    size_t off = 0;
    auto take = [&](size_t b) {
        const size_t o = off;
        off += align256(std::max<size_t>(b, 1));
        return o;
    };
    L.hdr = take(sizeof(F3Header));
    L.flag = take(sizeof(int32_t) * size_t(n + 1));
    L.pos = take(sizeof(int32_t) * size_t(n + 1));
    L.ip = take(sizeof(int32_t) * size_t(n));
    L.iq = take(sizeof(int32_t) * size_t(n));
    L.tmp = take(sizeof(int64_t) * scan_tmp_elems(n + 1));
    L.tu = take(sizeof(int32_t) * size_t(n));
    L.tp = take(sizeof(int32_t) * size_t(n));
    L.tq = take(sizeof(int32_t) * size_t(n));
    L.su = take(d.needs_sort ? sizeof(int32_t) * size_t(n) : 0);
    L.sp = take(d.needs_sort ? sizeof(int32_t) * size_t(n) : 0);
    L.sq = take(d.needs_sort ? sizeof(int32_t) * size_t(n) : 0);
    L.wkey = take(sizeof(uint64_t) * size_t(n));
    L.wkey_alt = take(d.needs_sort ? sizeof(uint64_t) * size_t(n) : 0);
    L.perm = take(d.needs_sort ? sizeof(uint32_t) * size_t(n) : 0);
    L.perm_alt = take(d.needs_sort ? sizeof(uint32_t) * size_t(n) : 0);
    L.hist = take(d.needs_sort ? sizeof(int32_t) * size_t(radix_hist_elems(n)) : 0);
    L.heads = take(sizeof(int32_t) * size_t(n + 1));
    L.seg_of = take(sizeof(int32_t) * size_t(n + 1));
    L.seg_start = take(sizeof(int32_t) * size_t(n + 1));
    L.seg_key = take(sizeof(uint64_t) * size_t(n));
    L.part = take(sizeof(float) * size_t(2 * L.max_wg) * size_t(kRows * kCols));
    L.total = off;
    return L;
}

size_t gemm_lds_bytes(const F3Desc& d) {
    return sizeof(float) * (size_t(2) * kRows * kPitchT + size_t(d.tp) * kCols + size_t(kCols) * (d.tq + 4));
}

}  // namespace

}  // namespace tre

using namespace tre;

extern "C" {

size_t tre_execute3_workspace_bytes(const char* einsum, const char* upper, const int64_t* extent,
                                    const int32_t* tile, int64_t n_u) {
    F3Desc d;
    if (n_u < 0 || parse3(einsum, upper, extent, tile, d) != TRE_OK) return 0;
    return f3_layout(d, n_u).total;
}

tre_status tre_execute3(const char* einsum, const char* upper, const int64_t* extent, const int32_t* tile,
                        int32_t in_dtype, const int32_t* u_keys, int64_t n_u, const void* u_tiles,
                        const int32_t* v_keys, int64_t n_v, const void* v_tiles, const int32_t* x_keys,
                        int64_t n_x, const void* x_tiles, int32_t* w_keys, float* w_tiles, int64_t w_cap,
                        int64_t* n_w, int64_t* n_triples, void* ws, size_t ws_bytes, void* stream,
                        tre_timing* timing) {
    F3Desc d;
    tre_status st = parse3(einsum, upper, extent, tile, d);
    if (st != TRE_OK) return st;
    if (in_dtype != TRE_F32) return fail(TRE_E_DTYPE, "fp32 inputs only");
    if (!n_w || !n_triples || n_u < 0 || n_v < 0 || n_x < 0 || w_cap < 0)
        return fail(TRE_E_ARG, "null count pointer or negative size");
    *n_w = 0;
    *n_triples = 0;
    if (n_u > int64_t(0x7fffffff) || n_v > int64_t(0x7fffffff) || n_x > int64_t(0x7fffffff))
        return fail(TRE_E_SHAPE, "too many tuples");
    if (d.ru == 0 && n_u > 1) return fail(TRE_E_DUPKEY, "U without promoted labels holds at most one tuple");
    if (!ws || (reinterpret_cast<uintptr_t>(ws) & 255))
        return fail(TRE_E_ARG, "null workspace or workspace not 256-byte aligned");
    if (n_u > 0 && (!u_keys || !u_tiles || (reinterpret_cast<uintptr_t>(u_tiles) & 15)))
        return fail(TRE_E_ARG, "null U keys / tiles, or U tiles not 16-byte aligned");
    if ((n_v > 0 && (!v_keys || !v_tiles)) || (n_x > 0 && (!x_keys || !x_tiles)))
        return fail(TRE_E_ARG, "null V / X keys or tiles");
    const F3Layout L = f3_layout(d, n_u);
    if (ws_bytes < L.total) return fail(TRE_E_WORKSPACE, "workspace too small");
    hipStream_t s = reinterpret_cast<hipStream_t>(stream);
    char* wsb = reinterpret_cast<char*>(ws);
    auto at = [&](size_t o) { return reinterpret_cast<void*>(wsb + o); };
    F3Header* hdr = static_cast<F3Header*>(at(L.hdr));
    const int32_t* p_keys = d.v_on_p ? v_keys : x_keys;
    const int32_t* q_keys = d.v_on_p ? x_keys : v_keys;
    const int64_t n_p = d.v_on_p ? n_v : n_x, n_q = d.v_on_p ? n_x : n_v;
    // deferred timing: only the contraction kernel, by its own start / end
    // events; otherwise marks around every phase
    const bool deferred = timing && timing->deferred;
    PhaseTimer tm(timing != nullptr && !deferred);
    KernelEvents ke;
    if (deferred) {
        ke.start = event_acquire();
        ke.stop = event_acquire();
    }
    KernelEvents* kep = (ke.start && ke.stop) ? &ke : nullptr;
    hipError_t e;
    tm.mark(s);
    if ((e = launch_fill_zero(hdr, sizeof(F3Header), s)) != hipSuccess) return dev_fail(e, "header");
    if (n_u == 0) {
        if (timing) std::memset(timing, 0, sizeof(*timing));
        return TRE_OK;
    }
    {
        const ValJob jobs[3] = {{u_keys, n_u, d.ru, d.radix_u, &hdr->err_u, nullptr},
                                {p_keys, n_p, 1, &d.radix_p, &hdr->err_p, nullptr},
                                {q_keys, n_q, 1, &d.radix_q, &hdr->err_q, nullptr}};
        if ((e = launch_validate(jobs, 3, s)) != hipSuccess) return dev_fail(e, "validate");
    }
    int32_t* flag = static_cast<int32_t*>(at(L.flag));
    int32_t* pos = static_cast<int32_t*>(at(L.pos));
    int32_t* ip = static_cast<int32_t*>(at(L.ip));
    int32_t* iq = static_cast<int32_t*>(at(L.iq));
    int32_t* tu = static_cast<int32_t*>(at(L.tu));
    int32_t* tp = static_cast<int32_t*>(at(L.tp));
    int32_t* tq = static_cast<int32_t*>(at(L.tq));
    uint64_t* wkey = static_cast<uint64_t*>(at(L.wkey));
    uint32_t* perm = d.needs_sort ? static_cast<uint32_t*>(at(L.perm)) : nullptr;
    F3Header h{};
    auto key_errors = [&]() -> tre_status {
        const int32_t kerr = h.err_u | h.err_p | h.err_q;
        if (!kerr) return TRE_OK;
        set_error("tre_execute3: keys out of range, unsorted or repeated");
        return (kerr & 4) ? TRE_E_KEYRANGE : (kerr & 1) ? TRE_E_UNSORTED : TRE_E_DUPKEY;
    };
    // p and q operands holding every key: each U tuple is a triple (no
    // search, no count to read back; key checks are read with the key count,
    // or at the end in the masked form)
    const bool dense = n_p == d.radix_p && n_q == d.radix_q;
    int64_t nt = n_u;
    if (dense) {
        k3_dense<<<blocks_for(n_u), kThreads, 0, s>>>(u_keys, n_u, d, tu, tp, tq, d.masked ? nullptr : wkey,
                                                       d.masked ? nullptr : perm);
        if ((e = hipGetLastError()) != hipSuccess) return dev_fail(e, "dense triples");
    } else {
        k3_match<<<blocks_for(n_u + 1), kThreads, 0, s>>>(u_keys, n_u, d, p_keys, n_p, q_keys, n_q, flag, ip, iq);
        if ((e = hipGetLastError()) != hipSuccess) return dev_fail(e, "match");
        if ((e = scan_exclusive_i32(flag, pos, n_u + 1, static_cast<int32_t*>(at(L.tmp)), s)) != hipSuccess)
            return dev_fail(e, "scan");
        int32_t n_tri32 = 0;
        if ((e = hipMemcpyAsync(&h, hdr, sizeof(h), hipMemcpyDeviceToHost, s)) != hipSuccess ||
            (e = hipMemcpyAsync(&n_tri32, pos + n_u, sizeof(int32_t), hipMemcpyDeviceToHost, s)) != hipSuccess ||
            (e = hipStreamSynchronize(s)) != hipSuccess)
            return dev_fail(e, "triple count read-back");
        const tre_status ks = key_errors();
        if (ks != TRE_OK) return ks;
        nt = n_tri32;
    }
    *n_triples = nt;
    if (dense && d.masked) {
        // one output tuple per U tuple, keyed as U: nothing to group; the
        // contraction is enqueued before the one read-back (key checks)
        *n_w = n_u;
        if (n_u > w_cap || !w_tiles || (d.rw > 0 && !w_keys)) {
            // key errors take precedence, as on the searching path
            if ((e = hipMemcpyAsync(&h, hdr, sizeof(h), hipMemcpyDeviceToHost, s)) != hipSuccess ||
                (e = hipStreamSynchronize(s)) != hipSuccess)
                return dev_fail(e, "key check read-back");
            const tre_status ks = key_errors();
            if (ks != TRE_OK) return ks;
            if (n_u > w_cap) return fail(TRE_E_CAPACITY, "w_cap below the output key count");
            return fail(TRE_E_ARG, "null output buffers");
        }
        tm.mark(s);
        tm.mark(s);
        const float* P = static_cast<const float*>(d.v_on_p ? v_tiles : x_tiles);
        const float* Q = static_cast<const float*>(d.v_on_p ? x_tiles : v_tiles);
        const bool v4 = d.R % 4 == 0 && ((reinterpret_cast<uintptr_t>(P) | reinterpret_cast<uintptr_t>(Q)) & 15) == 0;
        const int64_t waves = (nt + kMaskedBatch - 1) / kMaskedBatch;
        const dim3 grid{unsigned((waves + kThreads / 64 - 1) / (kThreads / 64))};
        t_kernel_events = kep;
        e = launch_k(v4 ? k3_masked<true> : k3_masked<false>, grid, dim3(kThreads), 0, s,
                     static_cast<const float*>(u_tiles), P, Q, tu, tp, tq, nt, d.te_u, d.R, w_tiles);
        t_kernel_events = nullptr;
        if (e != hipSuccess) return dev_fail(e, "masked contract");
        tm.mark(s);
        if (d.rw > 0) {
            k3_copy_keys<<<blocks_for(n_u * d.ru), kThreads, 0, s>>>(u_keys, n_u * d.ru, w_keys);
            if ((e = hipGetLastError()) != hipSuccess) return dev_fail(e, "keys");
        }
        tm.mark(s);
        if ((e = hipMemcpyAsync(&h, hdr, sizeof(h), hipMemcpyDeviceToHost, s)) != hipSuccess ||
            (e = hipStreamSynchronize(s)) != hipSuccess)
            return dev_fail(e, "key check read-back");
        const tre_status ks = key_errors();
        if (ks != TRE_OK) return ks;
        finish_timing(timing, tm, deferred, dense, ke);
        return TRE_OK;
    }
    if (nt > 0) {
        if (!dense) {
            k3_compact<<<blocks_for(n_u), kThreads, 0, s>>>(u_keys, n_u, d, pos, ip, iq, tu, tp, tq, wkey, perm);
            if ((e = hipGetLastError()) != hipSuccess) return dev_fail(e, "compact");
        }
        if (d.needs_sort) {
            if ((e = radix_sort_u64(wkey, perm, static_cast<uint64_t*>(at(L.wkey_alt)),
                                    static_cast<uint32_t*>(at(L.perm_alt)), nt, d.wkey_bits,
                                    static_cast<int32_t*>(at(L.hist)), static_cast<int32_t*>(at(L.tmp)), s)) !=
                hipSuccess)
                return dev_fail(e, "sort");
            if (radix_result_in_alt(nt, d.wkey_bits)) {
                wkey = static_cast<uint64_t*>(at(L.wkey_alt));
                perm = static_cast<uint32_t*>(at(L.perm_alt));
            }
            int32_t *su = static_cast<int32_t*>(at(L.su)), *sp = static_cast<int32_t*>(at(L.sp)),
                    *sq = static_cast<int32_t*>(at(L.sq));
            k3_gather<<<blocks_for(nt), kThreads, 0, s>>>(perm, nt, tu, tp, tq, su, sp, sq);
            if ((e = hipGetLastError()) != hipSuccess) return dev_fail(e, "gather");
            tu = su;
            tp = sp;
            tq = sq;
        }
    }
    int32_t* heads = static_cast<int32_t*>(at(L.heads));
    int32_t* seg_of = static_cast<int32_t*>(at(L.seg_of));
    int32_t* seg_start = static_cast<int32_t*>(at(L.seg_start));
    uint64_t* seg_key = static_cast<uint64_t*>(at(L.seg_key));
    k3_heads<<<blocks_for(nt + 1), kThreads, 0, s>>>(wkey, nt, heads);
    if ((e = hipGetLastError()) != hipSuccess) return dev_fail(e, "heads");
    if ((e = scan_exclusive_i32(heads, seg_of, nt + 1, static_cast<int32_t*>(at(L.tmp)), s)) != hipSuccess)
        return dev_fail(e, "segment scan");
    k3_segments<<<blocks_for(nt + 1), kThreads, 0, s>>>(wkey, nt, seg_of, seg_start, seg_key, hdr);
    if ((e = hipGetLastError()) != hipSuccess) return dev_fail(e, "segments");
    // the join's end mark goes before the read-back, so reading the join
    // time after the wait needs no further wait
    tm.mark(s);
    if ((e = hipMemcpyAsync(&h, hdr, sizeof(h), hipMemcpyDeviceToHost, s)) != hipSuccess ||
        (e = hipStreamSynchronize(s)) != hipSuccess)
        return dev_fail(e, "key count read-back");
    if (dense) {
        const tre_status ks = key_errors();
        if (ks != TRE_OK) return ks;
    }
    const int64_t nw = h.n_w;
    *n_w = nw;
    if (nw > w_cap) return fail(TRE_E_CAPACITY, "w_cap below the output key count");
    if (nw > 0 && (!w_tiles || (d.rw > 0 && !w_keys))) return fail(TRE_E_ARG, "null output buffers");
    tm.mark(s);  // (no separate work-unit phase: ranges are computed in the kernel)
    if (d.masked) {
        // one output tuple per triple, already in U order
        if (nw != nt) return fail(TRE_E_DEVICE, "internal: masked form with a key count other than the triple count");
        if (nw > 0) {
            const float* P = static_cast<const float*>(d.v_on_p ? v_tiles : x_tiles);
            const float* Q = static_cast<const float*>(d.v_on_p ? x_tiles : v_tiles);
            const bool v4 = d.R % 4 == 0 && ((reinterpret_cast<uintptr_t>(P) | reinterpret_cast<uintptr_t>(Q)) & 15) == 0;
            const int64_t waves = (nt + kMaskedBatch - 1) / kMaskedBatch;
            const dim3 grid{unsigned((waves + kThreads / 64 - 1) / (kThreads / 64))};
            t_kernel_events = kep;
            e = launch_k(v4 ? k3_masked<true> : k3_masked<false>, grid, dim3(kThreads), 0, s,
                         static_cast<const float*>(u_tiles), P, Q, tu, tp, tq, nt, d.te_u, d.R, w_tiles);
            t_kernel_events = nullptr;
            if (e != hipSuccess) return dev_fail(e, "masked contract");
        }
        tm.mark(s);
        if (nw > 0 && d.rw > 0) {
            k3_write_keys<<<blocks_for(nw), kThreads, 0, s>>>(seg_key, nw, d, w_keys);
            if ((e = hipGetLastError()) != hipSuccess) return dev_fail(e, "keys");
        }
        tm.mark(s);
    } else {
        const void* fn = d.tq == 16   ? reinterpret_cast<const void*>(&k3_gemm_q<16>)
                         : d.tq == 32 ? reinterpret_cast<const void*>(&k3_gemm_q<32>)
                         : d.tq == 64 ? reinterpret_cast<const void*>(&k3_gemm_q<64>)
                                      : reinterpret_cast<const void*>(&k3_gemm);
        const size_t lds = gemm_lds_bytes(d);
        F3Args g{};
        if (nw > 0) {
            if (lds > 65536 &&
                (e = hipFuncSetAttribute(fn, hipFuncAttributeMaxDynamicSharedMemorySize, int(lds))) != hipSuccess)
                return dev_fail(e, "shared memory size");
            // one workgroup per resident slot, each with an equal share of the
            // (block, triple) items
            int occ = 0;
            if ((e = hipOccupancyMaxActiveBlocksPerMultiprocessor(&occ, fn, kThreads, lds)) != hipSuccess)
                return dev_fail(e, "occupancy");
            const int64_t items = nt * int64_t(d.mblocks) * d.rblocks;
            const int64_t n_wg =
                std::max<int64_t>(1, std::min<int64_t>({device_cus() * std::max(occ, 1), L.max_wg, items}));
            g.U = static_cast<const float*>(u_tiles);
            g.P = static_cast<const float*>(d.v_on_p ? v_tiles : x_tiles);
            g.Q = static_cast<const float*>(d.v_on_p ? x_tiles : v_tiles);
            g.tu = tu;
            g.tp = tp;
            g.tq = tq;
            g.seg_of = seg_of;
            g.seg_start = seg_start;
            g.nt = nt;
            g.n_wg = n_wg;
            g.brows = kRows;
            g.mblocks = d.mblocks;
            g.W = w_tiles;
            g.part = static_cast<float*>(at(L.part));
            g.d = d;
            const dim3 grid{unsigned(n_wg)};
            t_kernel_events = kep;
            e = launch_k(d.tq == 16   ? k3_gemm_q<16>
                         : d.tq == 32 ? k3_gemm_q<32>
                         : d.tq == 64 ? k3_gemm_q<64>
                                      : k3_gemm,
                         grid, dim3(kThreads), lds, s, g);
            t_kernel_events = nullptr;
            if (e != hipSuccess) return dev_fail(e, "contract");
        }
        tm.mark(s);
        if (nw > 0) {
            if (g.n_wg > 1) {
                k3_reduce<<<dim3(unsigned(g.n_wg - 1)), kThreads, 0, s>>>(g);
                if ((e = hipGetLastError()) != hipSuccess) return dev_fail(e, "reduce");
            }
            if (d.rw > 0) {
                k3_write_keys<<<blocks_for(nw), kThreads, 0, s>>>(seg_key, nw, d, w_keys);
                if ((e = hipGetLastError()) != hipSuccess) return dev_fail(e, "keys");
            }
        }
        tm.mark(s);
    }
    finish_timing(timing, tm, deferred, dense, ke);
    return TRE_OK;
}

}  // extern "C"
