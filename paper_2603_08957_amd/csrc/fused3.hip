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
// flags, a scan and compaction give the output keys and their segments, and
// segments are cut into bounded work units as in the binary path.
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
// stored.  A unit's triples accumulate in registers; split segments are
// summed by k3_reduce in unit order (no atomics on values).
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
constexpr int kTargetUnits = 2048;     // about 8 workgroups per CU on 256 CUs
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
};

struct F3Header {
    int32_t err_u, err_p, err_q, pad0;
    int64_t n_tri;
    int64_t n_w;
    int64_t n_units;
    int64_t n_slots;
    int32_t n_split;
    int32_t pad1;
    int64_t pad2[10];
};

struct F3Unit {
    int32_t seg, t0, t1, slot;  // triples [t0, t1) of segment seg; slot >= 0: partial tile
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

// Per segment: (units << 32) | partial slots, for one int64 scan.
__global__ void k3_unit_count(const int32_t* __restrict__ seg_start, int64_t n_w, int64_t per_unit,
                              int64_t* __restrict__ cnt) {
    const int64_t q = int64_t(blockIdx.x) * blockDim.x + threadIdx.x;
    if (q > n_w) return;
    if (q == n_w) {
        cnt[q] = 0;
        return;
    }
    const int64_t len = seg_start[q + 1] - seg_start[q];
    const int64_t nu = (len + per_unit - 1) / per_unit;
    cnt[q] = (nu << 32) | (nu > 1 ? nu : 0);
}

__global__ void k3_unit_fill(const int32_t* __restrict__ seg_start, int64_t n_w, int64_t per_unit,
                             const int64_t* __restrict__ pref, F3Unit* __restrict__ units,
                             int32_t* __restrict__ split_list, F3Header* hdr) {
    const int64_t q = int64_t(blockIdx.x) * blockDim.x + threadIdx.x;
    if (q > n_w) return;
    if (q == n_w) {
        hdr->n_units = pref[n_w] >> 32;
        hdr->n_slots = pref[n_w] & 0xffffffffll;
        return;
    }
    const int64_t s0 = seg_start[q], s1 = seg_start[q + 1];
    const int64_t nu = (s1 - s0 + per_unit - 1) / per_unit;
    const int64_t ub = pref[q] >> 32, sb = pref[q] & 0xffffffffll;
    for (int64_t k = 0; k < nu; k++) {
        const int64_t t0 = s0 + k * per_unit;
        units[ub + k] = F3Unit{int32_t(q), int32_t(t0), int32_t(min(t0 + per_unit, s1)), nu > 1 ? int32_t(sb + k) : -1};
    }
    // split segments in any order: each is summed on its own
    if (nu > 1) split_list[atomicAdd(&hdr->n_split, 1)] = int32_t(q);
}

// ------------------------------------------------------------ tile part

struct F3Args {
    const float* U;
    const float* P;
    const float* Q;
    const int32_t* tu;
    const int32_t* tp;
    const int32_t* tq;
    const F3Unit* units;
    const F3Header* hdr;
    float* W;
    float* part;
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

// Dynamic LDS: T stages [2][kRows][kPitchT], P slice [tp][kCols], Q slice
// transposed [kCols][tq + 4] (floats).
__global__ __launch_bounds__(kThreads) void k3_gemm(F3Args g) {
    extern __shared__ float lds[];
    const F3Desc& d = g.d;
    float* sT = lds;
    float* sP = lds + 2 * kRows * kPitchT;
    const int qpitch = d.tq + 4;
    float* sQ = sP + d.tp * kCols;

    const int64_t per_unit_blocks = int64_t(d.mblocks) * d.rblocks;
    const int64_t u = int64_t(blockIdx.x) / per_unit_blocks;
    if (u >= g.hdr->n_units) return;
    const int rem = int(int64_t(blockIdx.x) - u * per_unit_blocks);
    const int mb = rem / d.rblocks, rb = rem % d.rblocks;
    const F3Unit un = g.units[u];

    const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
    const int mh = w & 1, rh = w >> 1;  // wave: rows [16 mh, +16), columns [32 rh, +32)
    const int n = lane & 15, gq = lane >> 4;
    const int64_t KK = int64_t(d.tp) * d.tq;
    const int nchunks = int((KK + kChunk - 1) / kChunk);
    const int64_t row0 = int64_t(mb) * kRows;
    const int col0 = rb * kCols;

    floatx4 acc[2][2];
#pragma unroll
    for (int t = 0; t < 2; t++)
#pragma unroll
        for (int e = 0; e < 2; e++) acc[t][e] = floatx4{0.f, 0.f, 0.f, 0.f};

    for (int32_t t = un.t0; t < un.t1; t++) {
        const int64_t s = g.tu[t];
        const float* Tt = g.U + s * d.te_u;
        const float* Pt = g.P + int64_t(g.tp[t]) * d.te_p;
        const float* Qt = g.Q + int64_t(g.tq[t]) * d.te_q;
        __syncthreads();  // the previous triple is done with sP, sQ and both T stages
        for (int e = tid; e < d.tp * kCols; e += kThreads) {
            const int pp = e / kCols, c = e % kCols, r = col0 + c;
            sP[e] = r < d.R ? Pt[pp * d.p_sp + int64_t(r) * d.p_sr] : 0.f;
        }
        for (int e = tid; e < d.tq * kCols; e += kThreads) {
            const int qq = e / kCols, c = e % kCols, r = col0 + c;
            sQ[c * qpitch + qq] = r < d.R ? Qt[qq * d.q_sq + int64_t(r) * d.q_sr] : 0.f;
        }
        // chunk loads: 4 float4 per thread, row = idx / 32, float4 column idx % 32
        float4 pre[4];
        auto load_chunk = [&](int c) {
#pragma unroll
            for (int i = 0; i < 4; i++) {
                const int idx = tid + kThreads * i, row = idx >> 5, c4 = idx & 31;
                const int64_t kk = int64_t(c) * kChunk + 4 * c4;
                const int64_t m = row0 + row;
                pre[i] = (m < d.M && kk < KK) ? *reinterpret_cast<const float4*>(Tt + m * KK + kk)
                                              : float4{0.f, 0.f, 0.f, 0.f};
            }
        };
        load_chunk(0);
        for (int c = 0; c < nchunks; c++) {
            float* st = sT + (c & 1) * kRows * kPitchT;
#pragma unroll
            for (int i = 0; i < 4; i++) {
                const int idx = tid + kThreads * i, row = idx >> 5, c4 = idx & 31;
                *reinterpret_cast<float4*>(st + row * kPitchT + 4 * c4) = pre[i];
            }
            __syncthreads();
            if (c + 1 < nchunks) load_chunk(c + 1);
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
    }
    // lane holds rows 4 gq + i, column n of each 16 x 16 tile
    float* dst = un.slot >= 0 ? g.part + int64_t(un.slot) * d.te_w : g.W + int64_t(un.seg) * d.te_w;
#pragma unroll
    for (int tt = 0; tt < 2; tt++) {
        const int r = col0 + 32 * rh + 16 * tt + n;
        const floatx4 v = acc[tt][0] + acc[tt][1];
#pragma unroll
        for (int i = 0; i < 4; i++) {
            const int64_t m = row0 + 16 * mh + 4 * gq + i;
            if (m < d.M && r < d.R) dst[w_row_offset(d, m) + int64_t(r) * d.w_sr] = v[i];
        }
    }
}

// Sum the partial tiles of every split segment, in unit order.
__global__ __launch_bounds__(kThreads) void k3_reduce(const int32_t* __restrict__ split_list,
                                                      const int64_t* __restrict__ pref,
                                                      const int32_t* __restrict__ seg_start, int64_t per_unit,
                                                      const float* __restrict__ part, int64_t te_w,
                                                      int64_t chunks, const F3Header* hdr, float* __restrict__ W) {
    const int64_t i = int64_t(blockIdx.x) / chunks;
    if (i >= hdr->n_split) return;
    const int64_t q = split_list[i];
    const int64_t nu = (seg_start[q + 1] - seg_start[q] + per_unit - 1) / per_unit;
    const int64_t sb = pref[q] & 0xffffffffll;
    const int64_t e0 = (int64_t(blockIdx.x) % chunks) * kThreads * 4;
    for (int64_t e = e0 + threadIdx.x; e < min(e0 + kThreads * 4, te_w); e += kThreads) {
        float acc = 0.f;
        for (int64_t k = 0; k < nu; k++) acc += part[(sb + k) * te_w + e];
        W[q * te_w + e] = acc;
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
    // W = U's other labels plus r
    if (w.size() != nu - 1 || w.find(r) == std::string::npos)
        return fail(TRE_E_SPLIT, "W holds U's labels other than the joined two, plus the shared label");
    for (size_t i = 0; i + 2 < nu; i++)
        if (w.find(u[i]) == std::string::npos)
            return fail(TRE_E_SPLIT, "W holds U's labels other than the joined two, plus the shared label");
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
    if (d.tp > kMaxPQ || d.tq > kMaxPQ || d.tq % 4)
        return fail(TRE_E_SHAPE, "tiles of U's last two labels must be at most 64, the last a multiple of 4");
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
    // W strides
    int64_t st = 1;
    int64_t wst[26] = {};
    for (int i = int(w.size()) - 1; i >= 0; i--) {
        wst[w[i] - 'a'] = st;
        st *= (w[i] == r) ? d.R : tsz(w[i]);
    }
    d.te_w = st;
    d.w_sr = wst[r - 'a'];
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

int64_t target_units(const F3Desc& d) {
    return std::max<int64_t>(1, kTargetUnits / (int64_t(d.mblocks) * d.rblocks));
}

struct F3Layout {
    size_t hdr, flag, pos, ip, iq, tmp, tu, tp, tq, su, sp, sq, wkey, wkey_alt, perm, perm_alt, hist, heads, seg_of,
        seg_start, seg_key, cnt, units, split, part, total;
};

size_t align256(size_t x) { return (x + 255) / 256 * 256; }

F3Layout f3_layout(const F3Desc& d, int64_t n_u) {
    const int64_t n = std::max<int64_t>(n_u, 1);
    const int64_t T = target_units(d);
    F3Layout L{};
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
    L.cnt = take(sizeof(int64_t) * size_t(n + 1));
    L.units = take(sizeof(F3Unit) * size_t(T + n));
    L.split = take(sizeof(int32_t) * size_t(T));
    L.part = take(sizeof(float) * size_t(2 * T) * size_t(d.te_w));
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
                        tre_dtype in_dtype, const int32_t* u_keys, int64_t n_u, const void* u_tiles,
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
    const bool deferred = timing && timing->deferred;
    PhaseTimer tm(timing != nullptr);
    hipError_t e;
    tm.mark(s);
    if ((e = launch_fill_zero(hdr, sizeof(F3Header), s)) != hipSuccess) return dev_fail(e, "header");
    if (n_u == 0) {
        if (timing) std::memset(timing, 0, sizeof(*timing));
        return TRE_OK;
    }
    if ((e = launch_validate(u_keys, n_u, d.ru, d.radix_u, &hdr->err_u, s)) != hipSuccess ||
        (e = launch_validate(p_keys, n_p, 1, &d.radix_p, &hdr->err_p, s)) != hipSuccess ||
        (e = launch_validate(q_keys, n_q, 1, &d.radix_q, &hdr->err_q, s)) != hipSuccess)
        return dev_fail(e, "validate");
    int32_t* flag = static_cast<int32_t*>(at(L.flag));
    int32_t* pos = static_cast<int32_t*>(at(L.pos));
    int32_t* ip = static_cast<int32_t*>(at(L.ip));
    int32_t* iq = static_cast<int32_t*>(at(L.iq));
    k3_match<<<blocks_for(n_u + 1), kThreads, 0, s>>>(u_keys, n_u, d, p_keys, n_p, q_keys, n_q, flag, ip, iq);
    if ((e = hipGetLastError()) != hipSuccess) return dev_fail(e, "match");
    if ((e = scan_exclusive_i32(flag, pos, n_u + 1, static_cast<int32_t*>(at(L.tmp)), s)) != hipSuccess)
        return dev_fail(e, "scan");
    F3Header h{};
    int32_t n_tri32 = 0;
    if ((e = hipMemcpyAsync(&h, hdr, sizeof(h), hipMemcpyDeviceToHost, s)) != hipSuccess ||
        (e = hipMemcpyAsync(&n_tri32, pos + n_u, sizeof(int32_t), hipMemcpyDeviceToHost, s)) != hipSuccess ||
        (e = hipStreamSynchronize(s)) != hipSuccess)
        return dev_fail(e, "triple count read-back");
    const int32_t kerr = h.err_u | h.err_p | h.err_q;
    if (kerr) {
        set_error("tre_execute3: keys out of range, unsorted or repeated");
        return (kerr & 4) ? TRE_E_KEYRANGE : (kerr & 1) ? TRE_E_UNSORTED : TRE_E_DUPKEY;
    }
    const int64_t nt = n_tri32;
    *n_triples = nt;
    int32_t* tu = static_cast<int32_t*>(at(L.tu));
    int32_t* tp = static_cast<int32_t*>(at(L.tp));
    int32_t* tq = static_cast<int32_t*>(at(L.tq));
    uint64_t* wkey = static_cast<uint64_t*>(at(L.wkey));
    uint32_t* perm = d.needs_sort ? static_cast<uint32_t*>(at(L.perm)) : nullptr;
    if (nt > 0) {
        k3_compact<<<blocks_for(n_u), kThreads, 0, s>>>(u_keys, n_u, d, pos, ip, iq, tu, tp, tq, wkey, perm);
        if ((e = hipGetLastError()) != hipSuccess) return dev_fail(e, "compact");
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
    if ((e = hipMemcpyAsync(&h, hdr, sizeof(h), hipMemcpyDeviceToHost, s)) != hipSuccess ||
        (e = hipStreamSynchronize(s)) != hipSuccess)
        return dev_fail(e, "key count read-back");
    const int64_t nw = h.n_w;
    *n_w = nw;
    tm.mark(s);
    if (nw > w_cap) return fail(TRE_E_CAPACITY, "w_cap below the output key count");
    if (nw > 0 && (!w_tiles || (d.rw > 0 && !w_keys))) return fail(TRE_E_ARG, "null output buffers");
    // work units
    const int64_t T = target_units(d);
    const int64_t per_unit = std::max<int64_t>(1, (nt + T - 1) / T);
    int64_t* cnt = static_cast<int64_t*>(at(L.cnt));
    F3Unit* units = static_cast<F3Unit*>(at(L.units));
    int32_t* split = static_cast<int32_t*>(at(L.split));
    if (nw > 0) {
        k3_unit_count<<<blocks_for(nw + 1), kThreads, 0, s>>>(seg_start, nw, per_unit, cnt);
        if ((e = hipGetLastError()) != hipSuccess) return dev_fail(e, "unit count");
        if ((e = scan_exclusive_i64(cnt, cnt, nw + 1, static_cast<int64_t*>(at(L.tmp)), s)) != hipSuccess)
            return dev_fail(e, "unit scan");
        k3_unit_fill<<<blocks_for(nw + 1), kThreads, 0, s>>>(seg_start, nw, per_unit, cnt, units, split, hdr);
        if ((e = hipGetLastError()) != hipSuccess) return dev_fail(e, "units");
    }
    tm.mark(s);
    if (nw > 0) {
        // at most nt / per_unit + nw units; workgroups past the real count exit
        const int64_t unit_bound = nt / per_unit + nw;
        const int64_t blocks = unit_bound * d.mblocks * d.rblocks;
        if (blocks > int64_t(0x7fffffff)) return fail(TRE_E_SHAPE, "too many output blocks");
        F3Args g{};
        g.U = static_cast<const float*>(u_tiles);
        g.P = static_cast<const float*>(d.v_on_p ? v_tiles : x_tiles);
        g.Q = static_cast<const float*>(d.v_on_p ? x_tiles : v_tiles);
        g.tu = tu;
        g.tp = tp;
        g.tq = tq;
        g.units = units;
        g.hdr = hdr;
        g.W = w_tiles;
        g.part = static_cast<float*>(at(L.part));
        g.d = d;
        const size_t lds = gemm_lds_bytes(d);
        if (lds > 65536 &&
            (e = hipFuncSetAttribute(reinterpret_cast<const void*>(&k3_gemm),
                                     hipFuncAttributeMaxDynamicSharedMemorySize, int(lds))) != hipSuccess)
            return dev_fail(e, "shared memory size");
        k3_gemm<<<dim3(unsigned(blocks)), kThreads, lds, s>>>(g);
        if ((e = hipGetLastError()) != hipSuccess) return dev_fail(e, "contract");
    }
    tm.mark(s);
    if (nw > 0) {
        const int64_t chunks = (d.te_w + kThreads * 4 - 1) / (kThreads * 4);
        k3_reduce<<<dim3(unsigned(T * chunks)), kThreads, 0, s>>>(split, cnt, seg_start, per_unit,
                                                                   static_cast<const float*>(at(L.part)), d.te_w,
                                                                   chunks, hdr, w_tiles);
        if ((e = hipGetLastError()) != hipSuccess) return dev_fail(e, "reduce");
        if (d.rw > 0) {
            k3_write_keys<<<blocks_for(nw), kThreads, 0, s>>>(seg_key, nw, d, w_keys);
            if ((e = hipGetLastError()) != hipSuccess) return dev_fail(e, "keys");
        }
    }
    tm.mark(s);
    if (timing) {
        std::memset(timing, 0, sizeof(*timing));
        timing->deferred = deferred ? 1 : 0;
        timing->join_ms = tm.between(0, 1);
        timing->total_ms = timing->join_ms;
        if (deferred && tm.on) {
            // the events after the join go to the caller; the first is ours
            for (int i = 0; i < 4; i++) timing->events[i] = reinterpret_cast<void*>(tm.ev[i + 1]);
            timing->pending = 1;
            tm.keep = true;
            (void)hipEventDestroy(tm.ev[0]);
        } else {
            timing->units_ms = tm.between(1, 2);
            timing->contract_ms = tm.between(2, 3);
            timing->reduce_ms = tm.between(3, 4);
            timing->total_ms += tm.between(1, 4);
        }
    }
    return TRE_OK;
}

}  // extern "C"
