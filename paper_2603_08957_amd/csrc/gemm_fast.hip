// Tile contraction for plain 2-D tiles, bf16 or fp32: each workgroup owns a
// 128x128 block of one output tile and accumulates sum over the pairs of its
// work unit of A_p (128 x K) * B_p (K x 128) on v_mfma_f32_32x32x16_bf16
// (bf16) or v_mfma_f32_32x32x2_f32 (fp32).
//
// 256 threads = 4 waves in a 2x2 grid, each wave a 64x64 sub-block (2x2 MFMA
// tiles, 64 fp32 accumulators per lane).  K advances over the concatenation
// of all pairs of the unit.  The ring geometry below is in bytes and is the
// same for both element types; a stage holds half as many k for fp32.
//
// Global memory is copied straight into LDS by global_load_lds_dwordx4 (16
// bytes per lane, lane l to LDS base + 16 l), so no registers hold staged
// data and no VALU work transposes it.  Each operand has its own ring of LDS
// stages, shaped by the direction of its unit stride so that every copy
// instruction moves eight whole 128-byte lines:
//   KFAST (k contiguous): a stage is a K = 64 chunk, [row][64 k] with
//     128-byte rows, 16 KB, three stages; the 16-byte granule G of row r sits
//     in slot G ^ ((r ^ (r >> 3)) & 7).  Read with ds_read_b128.
//   RFAST (rows contiguous): a stage is a K = 32 chunk, [k][128 rows] with
//     256-byte k-rows, 8 KB, four stages; granule g of k-row k sits in slot
//     g ^ (4 (k & 3)).  Read with ds_read_b64_tr_b16, which hands each lane
//     4 consecutive k of one row.
//   fp32: KFAST stages are K = 32 ([row][32 k], 128-byte rows, same
//     swizzle), RFAST stages K = 16 ([k][128 rows], 512-byte k-rows, granule
//     g of k-row k in slot g ^ (8 ((k >> 3) & 1))).  The MFMA takes one k per
//     lane and half-wave per step; the k of a tick are taken in the order
//     k = 8 half + s (s = 0 .. 7) in both operands, so a KFAST lane reads its
//     8 k with two ds_read_b128 and an RFAST lane with eight ds_read_b32 at
//     one base address.
// The swizzles are applied by choosing, per lane, which global granule goes
// to the lane's fixed LDS slot; all reads are free of bank conflicts and
// every global access covers whole contiguous row segments.  With one ring
// of each kind a workgroup takes 80 KB of LDS (two per CU).
//
// The main loop advances in ticks (K = 32 bf16, 16 fp32): an RFAST ring is refilled every
// tick three ticks ahead, a KFAST ring every second tick four ticks ahead,
// so only the stage being computed on is ever read while the others fill.
// The copies are issued from inline assembly (the compiler's own wait
// insertion would drain every outstanding copy before the first LDS read);
// the kernel waits for them explicitly (vmcnt) before each barrier and
// drains them before it leaves the loop.
#include "tre_internal.h"

#include <type_traits>

namespace tre {

namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef unsigned short u16x8 __attribute__((ext_vector_type(8)));
typedef float floatx16 __attribute__((ext_vector_type(16)));

constexpr int kThreads = 256;
constexpr int kB = 128;  // output block (rows and columns)

struct FastArgs {
    const void* A;
    const void* B;
    const int32_t* pa;
    const int32_t* pb;
    int64_t a_elems, b_elems, w_elems;
    int64_t lda, ldb, ldw;
    int32_t K, mblocks, nblocks;
    const int32_t* ridx;  // pacing: U's tile index of each pair, and U's tile count
    int64_t n_r;
    const Unit* units;
    const WsHeader* hdr;
    float* W;  // bf16 bits when w_bf16 (partials stay fp32)
    float* partials;
    int32_t w_bf16;
};

typedef short v4i16 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) v4i16 lds_v4i16;
typedef __attribute__((address_space(3))) char lds_char;
typedef __attribute__((address_space(4))) int32_t const_i32;

// s_waitcnt immediate: vmcnt(n) with expcnt and lgkmcnt left alone
constexpr int vmcnt_only(int n) { return (n & 15) | ((n >> 4) << 14) | (7 << 4) | (15 << 8); }

// ring geometry of one operand of element type T
template <typename T, bool RF>
struct Ring {
    static constexpr int kK = (RF ? 64 : 128) / int(sizeof(T));  // K per stage
    static constexpr int kStageBytes = RF ? 8192 : 16384;
    static constexpr int kStages = RF ? 4 : 3;
    static constexpr int kBytes = kStages * kStageBytes;
    static constexpr int kPerWave = kStageBytes / 1024 / 4;  // copy instructions per wave per refill
};

// K of one tick of the main loop
template <typename T>
constexpr int kTickK = 64 / int(sizeof(T));

__device__ inline uint64_t uniform64(uint64_t x) {
    const uint32_t lo = __builtin_amdgcn_readfirstlane(uint32_t(x));
    const uint32_t hi = __builtin_amdgcn_readfirstlane(uint32_t(x >> 32));
    return (uint64_t(hi) << 32) | lo;
}

template <bool NT>
__device__ inline void dma16(uint32_t lds_addr, const void* base, uint32_t voff) {
    const uint32_t m = __builtin_amdgcn_readfirstlane(lds_addr);
    const uint64_t b = uniform64(reinterpret_cast<uint64_t>(base));
    if constexpr (NT)
        asm volatile("s_mov_b32 m0, %0\n\tglobal_load_lds_dwordx4 %1, %2 nt" ::"s"(m), "v"(voff), "s"(b) : "m0");
    else
        asm volatile("s_mov_b32 m0, %0\n\tglobal_load_lds_dwordx4 %1, %2" ::"s"(m), "v"(voff), "s"(b) : "m0");
}

// Byte offset, from the stage's chunk origin, of the 16 bytes this lane
// copies for copy instruction q of an operand with leading dimension ld
// (elements); the copy lands at stage offset q * 1024 + 16 * lane.
template <typename T, bool RF>
__device__ inline uint32_t dma_src(int lane, int q, int64_t ld) {
    constexpr int E = int(sizeof(T));
    if (!RF) {  // 8 rows x 128 B; row & 7 == lane >> 3, (row >> 3) & 7 == q & 7
        const int row = 8 * q + (lane >> 3);
        return uint32_t(row * ld * E + (((lane & 7) ^ (lane >> 3) ^ (q & 7)) << 4));
    }
    if constexpr (E == 2) {
        const int krow = 4 * q + (lane >> 4);  // 4 k-rows x 256 B; krow & 3 == lane >> 4
        return uint32_t(krow * ld * E + (((lane & 15) ^ ((lane >> 4) << 2)) << 4));
    } else {
        const int krow = 2 * q + (lane >> 5);  // 2 k-rows x 512 B
        return uint32_t(krow * ld * E + (((lane & 31) ^ (((krow >> 3) & 1) << 3)) << 4));
    }
}

// Element offset inside a tile of the chunk origin (rows r0.., k0..).
template <bool RF>
__device__ inline int64_t dma_origin(int64_t ld, int r0, int k0) {
    return RF ? int64_t(k0) * ld + r0 : int64_t(r0) * ld + k0;
}

// Stage offsets of this lane's MFMA operand reads for the 32-row tile at row
// rb (a multiple of 32), one per k-step of 16 inside a stage.  KFAST: the
// 16-byte read of k-step s.  RFAST: the first of the two 8-byte transposing
// reads (k 0..3 and 4..7 of the lane's eight; the second is 4 k-rows on).
template <bool RF>
__device__ inline void frag_offsets(int lane, int rb, uint32_t (&off)[4]) {
    if (!RF) {
        const int r = rb + (lane & 31);
        const int x = (r ^ (r >> 3)) & 7, h = lane >> 5;
#pragma unroll
        for (int s = 0; s < 4; s++) off[s] = uint32_t(r * 128 + (((2 * s + h) ^ x) << 4));
    } else {
        const int i = lane & 15, G = lane >> 4;
        const int krow = 8 * (G >> 1) + (i >> 2);
        const int gran = ((rb >> 3) ^ ((i >> 2) << 2)) + 2 * (G & 1) + ((i & 3) >> 1);
        off[0] = uint32_t(krow * 256 + gran * 16 + 8 * (i & 1));
        off[1] = off[0] + 16 * 256;
        off[2] = off[3] = 0;
    }
}

template <bool RF>
__device__ inline bf16x8 frag_read(const char* stage, uint32_t off) {
    if (!RF) return __builtin_bit_cast(bf16x8, *reinterpret_cast<const u16x8*>(stage + off));
    const v4i16 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_v4i16*)(stage + off));
    const v4i16 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_v4i16*)(stage + off + 4 * 256));
    const v4i16 both[2] = {lo, hi};
    return __builtin_bit_cast(bf16x8, both);
}

typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) f32x4 lds_f32x4;
typedef __attribute__((address_space(3))) float lds_f32;

// fp32: stage offsets of the lane's reads for the 32-row tile at rb.
//   KFAST: off[2 p + j] = granule j of the lane's 8 k in tick half p.
//   RFAST: off[0] = the first of the lane's 8 k-rows (the others follow at
//          512-byte steps).
template <bool RF>
__device__ inline void frag_offsets_f32(int lane, int rb, uint32_t (&off)[4]) {
    const int h = lane >> 5;
    if (!RF) {
        const int r = rb + (lane & 31);
        const int x = (r ^ (r >> 3)) & 7;
#pragma unroll
        for (int p = 0; p < 2; p++)
#pragma unroll
            for (int j = 0; j < 2; j++) off[2 * p + j] = uint32_t(r * 128 + (((4 * p + 2 * h + j) ^ x) << 4));
    } else {
        const int c = rb + (lane & 31);
        off[0] = uint32_t(8 * h * 512 + ((((c >> 2) ^ (h << 3))) << 4) + 4 * (c & 3));
        off[1] = off[2] = off[3] = 0;
    }
}

// The lane's 8 fp32 operand values of tick half p (k = 8 half + s).
template <bool RF>
__device__ inline void frag8_f32(const char* stage, const uint32_t (&off)[4], int p, float (&v)[8]) {
    if (!RF) {
        const f32x4 a = *(const lds_f32x4*)((lds_char*)stage + off[2 * p]);
        const f32x4 b = *(const lds_f32x4*)((lds_char*)stage + off[2 * p + 1]);
#pragma unroll
        for (int i = 0; i < 4; i++) {
            v[i] = a[i];
            v[4 + i] = b[i];
        }
    } else {
        (void)p;
#pragma unroll
        for (int i = 0; i < 8; i++) v[i] = *(const lds_f32*)((lds_char*)stage + off[0] + i * 512);
    }
}

// Copy cursor of one operand: walks the unit's pairs stage by stage; past
// the end it copies the last stage again (never read).
template <typename T, bool RF, bool NT>
struct Cursor {
    using R = Ring<T, RF>;
    const T* base;         // operand tiles, offset to the block's chunk origin
    const const_i32* idx;  // tile index of each pair of the unit
    int64_t elems, step;   // tile elements; element step from one stage to the next
    int np, per_pair;      // pairs; stages per pair
    int ip = 0, ik = 0, stage = 0;
    int32_t next = 0;
    const T* cur = nullptr;
    uint32_t src[R::kPerWave];

    __device__ void init(const T* b, const const_i32* ix, int64_t e, int64_t ld, int K, int npairs, int lane, int w) {
        base = b;
        idx = ix;
        elems = e;
        step = RF ? int64_t(R::kK) * ld : R::kK;
        np = npairs;
        per_pair = K / R::kK;
        cur = base + int64_t(idx[0]) * elems;
        next = idx[min(1, np - 1)];
#pragma unroll
        for (int j = 0; j < R::kPerWave; j++) src[j] = dma_src<T, RF>(lane, R::kPerWave * w + j, ld);
    }
    __device__ void issue(uint32_t ring_lds, int w) {
        const uint32_t l0 = ring_lds + stage * R::kStageBytes + R::kPerWave * w * 1024;
#pragma unroll
        for (int j = 0; j < R::kPerWave; j++) dma16<NT>(l0 + j * 1024, cur, src[j]);
        stage = stage == R::kStages - 1 ? 0 : stage + 1;
        if (++ik < per_pair) {
            cur += step;
            return;
        }
        ik = 0;
        if (ip + 1 < np) {
            ip++;
            cur = base + int64_t(next) * elems;
            next = idx[min(ip + 1, np - 1)];
        } else {
            cur -= (per_pair - 1) * step;
        }
    }
};

template <typename T, bool AROW, bool BROW>
struct DmaShape {
    using RA = Ring<T, AROW>;
    using RB = Ring<T, BROW>;
    static constexpr int kLds = RA::kBytes + RB::kBytes;
    static constexpr int kOcc = 163840 / kLds;
    // Copies still allowed in flight when a tick's data must have landed (see
    // the schedule above): with one RFAST ring, the two previous ticks'
    // copies; with two KFAST rings, the previous refill (even ticks) or the
    // two previous refills (odd ticks, which need no new data).
    static constexpr int kWait0 = (AROW || BROW) ? 8 : 8;
    static constexpr int kWait1 = (AROW || BROW) ? 8 : 16;
};

// Pacing hooks of run_unit: called by every thread at the first tick of
// each pair and after the last one.  NoPace does nothing.
struct NoPace {
    __device__ void at_pair(int) {}
    __device__ void at_end() {}
};

// Cooperative pacing for the persistent variant (below).  The reused
// operand's index range is cut into `windows` windows; done[q] counts the
// workgroups of this XCD and round that have moved past window q.  Before a
// workgroup's pairs enter window w, it waits until `thr` peers are past
// window w - 1 - ahead, so the workgroups sharing an L2 stay within a few
// windows of each other.  The wait is bounded: after kMaxPolls polls it
// goes on regardless, so pacing can only cost time, never correctness.
struct Pace {
    static constexpr int kMaxPolls = 4096;
    int32_t* done;
    const const_i32* ridx;  // reused operand's tile index of each pair of the unit
    int64_t n_r;            // tiles of the reused operand
    int windows, ahead, thr, cur;
    __device__ int window_of(int32_t i) const { return int(int64_t(i) * windows / n_r); }
    __device__ void pass_to(int w) {
        for (int q = cur < 0 ? 0 : cur; q < w; q++) atomicAdd(done + q, 1);
    }
    __device__ void at_pair(int p) {
        if (threadIdx.x != 0) return;
        const int w = window_of(ridx[p]);
        if (w == cur) return;
        pass_to(w);
        cur = w;
        const int q = w - 1 - ahead;
        if (q < 0) return;
        for (int it = 0; it < kMaxPolls; it++) {
            if (__hip_atomic_load(done + q, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) >= thr) break;
            __builtin_amdgcn_s_sleep(2);
        }
    }
    __device__ void at_end() {
        if (threadIdx.x == 0) pass_to(windows);
    }
};

// One work unit: sum over its pairs of A_p B_p into the 128x128 block
// (m0, n0) of its output tile, written to W (whole key) or a partial slot.
template <typename T, bool AROW, bool BROW, bool ANT, bool BNT, class Pacer>
__device__ inline void run_unit(const FastArgs& g, const Unit& un, int m0, int n0, char* lds, Pacer& pc) {
    using SH = DmaShape<T, AROW, BROW>;
    using RA = Ring<T, AROW>;
    using RB = Ring<T, BROW>;
    constexpr bool F32 = sizeof(T) == 4;
    const uint32_t lds_a = uint32_t(reinterpret_cast<uintptr_t>((lds_char*)(lds)));
    const uint32_t lds_b = lds_a + RA::kBytes;

    const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
    const int wm = w >> 1, wn = w & 1;
    floatx16 acc[2][2];
#pragma unroll
    for (int i = 0; i < 2; i++)
#pragma unroll
        for (int j = 0; j < 2; j++)
#pragma unroll
            for (int r = 0; r < 16; r++) acc[i][j][r] = 0.f;

    const int np = un.p1 - un.p0;
    const int tpp = g.K / kTickK<T>;  // ticks per pair
    const int ticks = np * tpp;
    float* out = un.slot < 0 ? g.W + int64_t(un.seg) * g.w_elems : g.partials + int64_t(un.slot) * g.w_elems;
    uint16_t* out16 = (g.w_bf16 && un.slot < 0) ? reinterpret_cast<uint16_t*>(g.W) + int64_t(un.seg) * g.w_elems
                                                 : nullptr;
    if (ticks == 0) {
        for (int e = threadIdx.x; e < kB * kB; e += kThreads) {
            const int64_t o = int64_t(m0 + e / kB) * g.ldw + n0 + e % kB;
            if (out16) out16[o] = 0;
            else out[o] = 0.f;
        }
        pc.at_end();
        return;
    }
    // the pair list is read-only here; reading it through the constant
    // address space keeps the (uniform) index loads on the scalar unit
    Cursor<T, AROW, ANT> ca;
    Cursor<T, BROW, BNT> cb;
    ca.init(reinterpret_cast<const T*>(g.A) + dma_origin<AROW>(g.lda, m0, 0), (const const_i32*)(g.pa + un.p0),
            g.a_elems, g.lda, g.K, np, lane, w);
    cb.init(reinterpret_cast<const T*>(g.B) + dma_origin<BROW>(g.ldb, n0, 0), (const const_i32*)(g.pb + un.p0),
            g.b_elems, g.ldb, g.K, np, lane, w);

    uint32_t oa[2][4], ob[2][4];
#pragma unroll
    for (int t = 0; t < 2; t++) {
        if constexpr (F32) {
            frag_offsets_f32<AROW>(lane, wm * 64 + t * 32, oa[t]);
            frag_offsets_f32<BROW>(lane, wn * 64 + t * 32, ob[t]);
        } else {
            frag_offsets<AROW>(lane, wm * 64 + t * 32, oa[t]);
            frag_offsets<BROW>(lane, wn * 64 + t * 32, ob[t]);
        }
    }

    // refills of tick tau: KFAST rings on even ticks (stage tau / 2 + 2),
    // then RFAST rings (stage tau + 3); the prologue runs ticks -4 .. -1
    auto refill = [&](int tau_parity, bool rf_too) {
        if (tau_parity == 0) {
            if (!AROW) ca.issue(lds_a, w);
            if (!BROW) cb.issue(lds_b, w);
        }
        if (rf_too) {
            if (AROW) ca.issue(lds_a, w);
            if (BROW) cb.issue(lds_b, w);
        }
    };
    refill(0, false);  // tick -4
    refill(1, true);   // tick -3
    refill(0, true);   // tick -2
    refill(1, true);   // tick -1

    int sa = 0, sb = 0;  // ring stage being read
    auto tick = [&](auto parity) {
        constexpr int p = decltype(parity)::value;
        __builtin_amdgcn_s_waitcnt(vmcnt_only(p == 0 ? SH::kWait0 : SH::kWait1));
        __syncthreads();
        refill(p, true);
        const char* As = lds + sa * RA::kStageBytes;
        const char* Bs = lds + RA::kBytes + sb * RB::kStageBytes;
        if constexpr (F32) {
            float a[2][8], b[2][8];
#pragma unroll
            for (int t = 0; t < 2; t++) {
                frag8_f32<AROW>(As, oa[t], p, a[t]);
                frag8_f32<BROW>(Bs, ob[t], p, b[t]);
            }
#pragma unroll
            for (int s = 0; s < 8; s++) {
                acc[0][0] = __builtin_amdgcn_mfma_f32_32x32x2f32(a[0][s], b[0][s], acc[0][0], 0, 0, 0);
                acc[0][1] = __builtin_amdgcn_mfma_f32_32x32x2f32(a[0][s], b[1][s], acc[0][1], 0, 0, 0);
                acc[1][0] = __builtin_amdgcn_mfma_f32_32x32x2f32(a[1][s], b[0][s], acc[1][0], 0, 0, 0);
                acc[1][1] = __builtin_amdgcn_mfma_f32_32x32x2f32(a[1][s], b[1][s], acc[1][1], 0, 0, 0);
            }
        } else {
            bf16x8 a[2][2], b[2][2];
#pragma unroll
            for (int s = 0; s < 2; s++)
#pragma unroll
                for (int t = 0; t < 2; t++) {
                    a[s][t] = frag_read<AROW>(As, oa[t][AROW ? s : 2 * p + s]);
                    b[s][t] = frag_read<BROW>(Bs, ob[t][BROW ? s : 2 * p + s]);
                }
#pragma unroll
            for (int s = 0; s < 2; s++) {
                acc[0][0] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[s][0], b[s][0], acc[0][0], 0, 0, 0);
                acc[0][1] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[s][0], b[s][1], acc[0][1], 0, 0, 0);
                acc[1][0] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[s][1], b[s][0], acc[1][0], 0, 0, 0);
                acc[1][1] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[s][1], b[s][1], acc[1][1], 0, 0, 0);
            }
        }
        // advance the read stages: RFAST every tick, KFAST after odd ticks
        if (AROW || p == 1) sa = sa == RA::kStages - 1 ? 0 : sa + 1;
        if (BROW || p == 1) sb = sb == RB::kStages - 1 ? 0 : sb + 1;
    };
    // K is a multiple of 64, so a unit has an even number of ticks
    for (int t = 0; t < ticks; t += 2) {
        if (t % tpp == 0) pc.at_pair(t / tpp);
        tick(std::integral_constant<int, 0>{});
        tick(std::integral_constant<int, 1>{});
    }
    pc.at_end();
    // the copies issued past the end must land before the workgroup leaves
    // (its LDS may be handed to another workgroup)
    __builtin_amdgcn_s_waitcnt(vmcnt_only(0));

    // non-temporal stores: an output block is written once per launch, and
    // keeping its lines out of L2 leaves room for the reused operand's tiles
#pragma unroll
    for (int i = 0; i < 2; i++)
#pragma unroll
        for (int j = 0; j < 2; j++) {
            const int n = n0 + wn * 64 + j * 32 + (lane & 31);
#pragma unroll
            for (int r = 0; r < 16; r++) {
                const int m = m0 + wm * 64 + i * 32 + (r >> 2) * 8 + (lane >> 5) * 4 + (r & 3);
                if (out16) __builtin_nontemporal_store(f32_to_bf16_rne(acc[i][j][r]), out16 + int64_t(m) * g.ldw + n);
                else __builtin_nontemporal_store(acc[i][j][r], out + int64_t(m) * g.ldw + n);
            }
        }
}

template <typename T, bool AROW, bool BROW, bool ANT, bool BNT>
__global__ __launch_bounds__(kThreads, (DmaShape<T, AROW, BROW>::kOcc)) void k_gemm_dma(FastArgs g) {
    // Workgroup -> (unit, row block, column block).  Workgroups are dealt to
    // the 8 XCDs round-robin; the column blocks of one (unit, row block) take
    // consecutive slots of one XCD, so they share the A tile in its L2.
    const int64_t xcd = blockIdx.x % 8, slot = blockIdx.x / 8;
    const int64_t grp = (slot / g.nblocks) * 8 + xcd;
    const int nblk = int(slot % g.nblocks), mblk = int(grp % g.mblocks);
    const int64_t unit_id = grp / g.mblocks;
    if (unit_id >= g.hdr->n_units) return;
    __shared__ __attribute__((aligned(1024))) char lds[DmaShape<T, AROW, BROW>::kLds];
    NoPace pc;
    run_unit<T, AROW, BROW, ANT, BNT>(g, g.units[unit_id], mblk * kB, nblk * kB, lds, pc);
}

// Persistent, paced variant for one 128x128 block per key (M = N = 128):
// `n_wg` workgroups, all resident at once; workgroup b takes units b, b +
// n_wg, b + 2 n_wg, ... (one per round).  Units of one round start together,
// and pacing keeps the workgroups of an XCD within a few windows of the
// reused operand, so its tiles stay in that XCD's L2 without cutting keys
// into ranges (no partial tiles).  pace: rounds x 8 x windows counters,
// zeroed by the host before the launch.
template <typename T, bool AROW, bool BROW, bool ANT, bool BNT>
__global__ __launch_bounds__(kThreads, (DmaShape<T, AROW, BROW>::kOcc)) void k_gemm_paced(FastArgs g, int32_t* pace,
                                                                                      int32_t n_wg, int32_t windows,
                                                                                      int32_t ahead, int32_t slack_div) {
    __shared__ __attribute__((aligned(1024))) char lds[DmaShape<T, AROW, BROW>::kLds];
    const int64_t n_units = g.hdr->n_units;
    const int xcd = int(blockIdx.x % 8);
    for (int64_t round = 0;; round++) {
        const int64_t unit_id = blockIdx.x + round * n_wg;
        if (unit_id >= n_units) break;
        // workgroups of this XCD that have a unit in this round
        const int64_t left = n_units - round * n_wg - xcd;
        const int64_t active = min<int64_t>((left + 7) / 8, (n_wg - xcd + 7) / 8);
        const Unit un = g.units[unit_id];
        Pace pc;
        pc.done = pace + (round * 8 + xcd) * windows;
        pc.ridx = (const const_i32*)(g.ridx + un.p0);
        pc.n_r = g.n_r;
        pc.windows = windows;
        pc.ahead = ahead;
        pc.thr = int(max<int64_t>(active - active / slack_div, 1));
        pc.cur = -1;
        __syncthreads();  // the previous unit's LDS reads are done
        run_unit<T, AROW, BROW, ANT, BNT>(g, un, 0, 0, lds, pc);
    }
}

}  // namespace

namespace {

FastArgs fast_args(const Plan& p, const Layout& L, char* ws, const void* u_tiles, const void* v_tiles,
                   float* w_tiles) {
    FastArgs g{};
    const int32_t* pu = reinterpret_cast<const int32_t*>(ws + L.pu);
    const int32_t* pv = reinterpret_cast<const int32_t*>(ws + L.pv);
    g.A = p.swap ? v_tiles : u_tiles;
    g.B = p.swap ? u_tiles : v_tiles;
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
    g.mblocks = int32_t(M / kB);
    g.nblocks = int32_t(N / kB);
    g.ridx = pu;
    g.n_r = L.n_u;
    g.units = reinterpret_cast<const Unit*>(ws + L.unit_desc);
    g.hdr = reinterpret_cast<const WsHeader*>(ws + L.hdr);
    g.W = w_tiles;
    g.partials = reinterpret_cast<float*>(ws + L.partials);
    g.w_bf16 = p.opt.w_bf16;
    return g;
}

// kernel variant: operand layouts, and which operand is streamed (each tile
// used by about one pair, so its copies carry the non-temporal hint)
int fast_variant(const Plan& p, const Layout& L, int64_t n_pairs) {
    const int64_t n_a = p.swap ? L.n_v : L.n_u, n_b = p.swap ? L.n_u : L.n_v;
    const bool ant = 2 * n_a >= n_pairs, bnt = 2 * n_b >= n_pairs;
    return (p.fast_a_rowfast ? 8 : 0) | (p.fast_b_rowfast ? 4 : 0) | (ant ? 2 : 0) | (bnt ? 1 : 0);
}

}  // namespace

hipError_t launch_gemm_fast(const Plan& p, const Layout& L, char* ws, const void* u_tiles, const void* v_tiles,
                            float* w_tiles, int64_t n_pairs, int64_t unit_bound, hipStream_t s) {
    const FastArgs g = fast_args(p, L, ws, u_tiles, v_tiles, w_tiles);
    const int64_t groups = unit_bound * g.mblocks;
    const int64_t blocks = (groups + 7) / 8 * 8 * g.nblocks;
    if (blocks > int64_t(0x7fffffff)) return hipErrorInvalidConfiguration;
    dim3 grid{unsigned(blocks), 1u, 1u};
    hipError_t e = hipErrorInvalidValue;
#define TRE_FAST_CASE(X)                                                                                      \
    case X:                                                                                                   \
        if (p.dtype == TRE_BF16)                                                                              \
            e = launch_k(k_gemm_dma<uint16_t, bool(X & 8), bool(X & 4), bool(X & 2), bool(X & 1)>, grid,        \
                         dim3(kThreads), 0, s, g);                                                            \
        else                                                                                                  \
            e = launch_k(k_gemm_dma<float, bool(X & 8), bool(X & 4), bool(X & 2), bool(X & 1)>, grid,           \
                         dim3(kThreads), 0, s, g);                                                            \
        break;
    switch (fast_variant(p, L, n_pairs)) {
        TRE_FAST_CASE(0) TRE_FAST_CASE(1) TRE_FAST_CASE(2) TRE_FAST_CASE(3)
        TRE_FAST_CASE(4) TRE_FAST_CASE(5) TRE_FAST_CASE(6) TRE_FAST_CASE(7)
        TRE_FAST_CASE(8) TRE_FAST_CASE(9) TRE_FAST_CASE(10) TRE_FAST_CASE(11)
        TRE_FAST_CASE(12) TRE_FAST_CASE(13) TRE_FAST_CASE(14) TRE_FAST_CASE(15)
    }
#undef TRE_FAST_CASE
    return e;
}

int64_t gemm_paced_slots(const Plan& p) {
    int dev = 0, cus = 0;
    if (hipGetDevice(&dev) != hipSuccess ||
        hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || cus <= 0)
        return 0;
    const int occ = (p.fast_a_rowfast || p.fast_b_rowfast) ? 2 : 1;  // 80 / 64 KB vs 96 KB of LDS
    return int64_t(cus) * occ;
}

hipError_t launch_gemm_paced(const Plan& p, const Layout& L, char* ws, const void* u_tiles, const void* v_tiles,
                             float* w_tiles, int64_t n_pairs, int64_t n_wg, int32_t windows, hipStream_t s) {
    const FastArgs g = fast_args(p, L, ws, u_tiles, v_tiles, w_tiles);
    if (g.mblocks != 1 || g.nblocks != 1 || n_wg <= 0 || n_wg > int64_t(0x7fffffff)) return hipErrorInvalidValue;
    int32_t* pace = reinterpret_cast<int32_t*>(ws + L.pace);
    // a workgroup waits until 3/4 of its XCD's peers have left the window
    // before the one it enters
    constexpr int32_t kAhead = 0, kSlackDiv = 4;
    dim3 grid{unsigned(n_wg), 1u, 1u};
    hipError_t e = hipErrorInvalidValue;
#define TRE_PACED_CASE(X)                                                                                      \
    case X:                                                                                                    \
        if (p.dtype == TRE_BF16)                                                                               \
            e = launch_k(k_gemm_paced<uint16_t, bool(X & 8), bool(X & 4), bool(X & 2), bool(X & 1)>, grid,      \
                         dim3(kThreads), 0, s, g, pace, int32_t(n_wg), windows, kAhead, kSlackDiv);             \
        else                                                                                                   \
            e = launch_k(k_gemm_paced<float, bool(X & 8), bool(X & 4), bool(X & 2), bool(X & 1)>, grid,         \
                         dim3(kThreads), 0, s, g, pace, int32_t(n_wg), windows, kAhead, kSlackDiv);             \
        break;
    switch (fast_variant(p, L, n_pairs)) {
        TRE_PACED_CASE(0) TRE_PACED_CASE(1) TRE_PACED_CASE(2) TRE_PACED_CASE(3)
        TRE_PACED_CASE(4) TRE_PACED_CASE(5) TRE_PACED_CASE(6) TRE_PACED_CASE(7)
        TRE_PACED_CASE(8) TRE_PACED_CASE(9) TRE_PACED_CASE(10) TRE_PACED_CASE(11)
        TRE_PACED_CASE(12) TRE_PACED_CASE(13) TRE_PACED_CASE(14) TRE_PACED_CASE(15)
    }
#undef TRE_PACED_CASE
    return e;
}

}  // namespace tre
