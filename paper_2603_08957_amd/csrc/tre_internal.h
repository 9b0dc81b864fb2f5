// Internal declarations shared by the host planner and the gfx950 kernels.
#pragma once

#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>

#include <cstddef>
#include <cstdint>
#include <string>

#include "../../include/tre.h"

namespace tre {

// fp32 -> bf16 bits, round to nearest even, NaN kept quiet (the cast glue and
// the bf16 output of tre_contract)
__device__ inline uint16_t f32_to_bf16_rne(float f) {
    uint32_t u = __float_as_uint(f);
    if ((u & 0x7f800000u) == 0x7f800000u && (u & 0x007fffffu)) return uint16_t((u >> 16) | 0x40u);
    u += 0x7fffu + ((u >> 16) & 1u);
    return uint16_t(u >> 16);
}

// Exclusive scan of one int32 per thread over a workgroup of W threads
// (a multiple of 64); wsum holds W / 64 ints of LDS.  Every thread of the
// workgroup must call it.
template <int W>
__device__ inline int32_t block_scan_excl(int32_t v, int32_t* wsum, int32_t* total) {
    const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
    int32_t x = v;
#pragma unroll
    for (int d = 1; d < 64; d <<= 1) {
        const int32_t y = __shfl_up(x, d, 64);
        if (lane >= d) x += y;
    }
    if (lane == 63) wsum[w] = x;
    __syncthreads();
    int32_t before = 0, all = 0;
#pragma unroll
    for (int i = 0; i < W / 64; i++) {
        const int32_t s = wsum[i];
        if (i < w) before += s;
        all += s;
    }
    __syncthreads();
    *total = all;
    return before + x - v;
}

constexpr int kMaxDims = 8;
constexpr int kMaxURanges = 64;
constexpr int64_t kPaceCounters = int64_t(1) << 20;  // int32 pacing counters in the workspace

// Row-major index decomposition: index x over sizes (last fastest) maps to
// sum_i coord_i(x) * stride_i.  Used to build per-role offset tables.
struct Dims {
    int32_t n = 0;
    int32_t size[kMaxDims] = {};
    int32_t stride[kMaxDims] = {};
    int64_t count() const {
        int64_t c = 1;
        for (int i = 0; i < n; i++) c *= size[i];
        return c;
    }
};

// Offset tables (int32 element offsets inside one tile).
//   GEMM: A/B are the two operands as the MFMA kernel sees them (A = U unless
//   the plan swaps), W the output tile.
//   VEC : EU/EV map a W-tile element (in W memory order) to the U / V offset
//   of its non-contracted part; KU/KV map the contracted index.
enum TableId { T_AM, T_AK, T_BK, T_BN, T_WM, T_WN, T_AB, T_BB, T_WB, T_EU, T_EV, T_KU, T_KV, T_COUNT };

enum KernelClass { KC_GEMM = 0, KC_VEC = 1 };

struct Plan {
    std::string einsum;
    tre_dtype dtype = TRE_F32;
    tre_options opt{};
    // parsed labels
    int nl[3] = {0, 0, 0};
    int lab[3][26] = {};
    bool up[26] = {};
    bool used[26] = {};
    int64_t ext[26] = {};
    int64_t tsz[26] = {};  // extent of the label inside a tile
    int nk[3] = {0, 0, 0};
    int klab[3][26] = {};
    int64_t tile_elems[3] = {1, 1, 1};
    int32_t radix[3][26] = {};  // per key attribute: extent / t
    // join key: join labels in V's key order, packed most significant first
    int n_join = 0;
    int join_pos_u[26] = {}, join_pos_v[26] = {}, join_bits[26] = {};
    int join_total_bits = 0;
    bool v_needs_sort = false;
    // W key: attributes in W key order, each from U (0) or V (1)
    int w_src[26] = {}, w_pos[26] = {}, w_bits[26] = {};
    int w_total_bits = 0;
    bool group_needs_sort = false;
    // join driven by V: W's key is V's key prefix and V's remaining key
    // attributes are the join labels, which U's key starts with; each V tuple
    // then meets one run of U tuples and the pairs come out in (W key, u, v)
    // order with no sort (see classify)
    bool v_outer = false;
    // tile roles
    char role[26] = {};
    int64_t nB = 1, nM = 1, nN = 1, nK = 1;
    KernelClass kclass = KC_VEC;
    bool swap = false;     // GEMM: A operand is V
    bool a_kfast = false;  // GEMM: A's unit-stride dim is a K dim
    bool b_kfast = false;
    bool vec_a = false;    // GEMM: 8-wide vector loads legal along A's fast dim
    bool vec_b = false;
    // 128x128 fast path (bf16, fp32): A(m,k) = A[k*lda + m] if a_rowfast else A[m*lda + k];
    // B(n,k) = B[k*ldb + n] if b_rowfast else B[n*ldb + k]; W(m,n) = W[m*ldw + n]
    // vector class: W elements per thread (1, 4 for fp32, 8 for bf16) and
    // whether V's element is the same for a whole group of them
    int vec_ept = 1;
    bool vec_vbcast = false;
    bool vec_swap = false;  // vector class: the kernel's vector operand is V and its broadcast one U
    bool fast = false;
    bool fast_a_rowfast = false, fast_b_rowfast = false;
    int64_t fast_lda = 0, fast_ldb = 0, fast_ldw = 0;
    Dims dims[T_COUNT];
    int64_t table_off[T_COUNT] = {};
    int64_t table_total = 0;
};

// Workspace layout (byte offsets from the workspace base).
struct Layout {
    int64_t n_u = 0, n_v = 0, max_pairs = 0;
    int64_t part_cap = 0;  // partial tiles
    size_t hdr, vjk, vjk_alt, vperm, vperm_alt, ucnt, ulo, scan_tmp, pu, pv, pu_alt, pv_alt, wk, wk_alt, pidx,
        pidx_alt, hist, flags, seg_start, seg_key, unit_desc, seg_units, part_off, split_list, tables, pace, partials;
    size_t total = 0;
};

// Header at the start of the workspace (device memory).
struct WsHeader {
    int32_t err_u;       // bit 0 unsorted, bit 1 duplicate, bit 2 range
    int32_t err_v;
    int32_t pad0[2];
    int64_t n_pairs;
    int64_t n_w;
    int64_t n_units;
    int64_t n_split;
    int64_t n_parts;
    int64_t pad1[9];
};

// Work unit: a run of pairs [p0, p1) of one segment; slot >= 0 means the
// unit writes a partial tile that the segmented reduction sums.
struct Unit {
    int32_t seg;
    int32_t p0;
    int32_t p1;
    int32_t slot;
};

Layout make_layout(const Plan& p, int64_t n_u, int64_t n_v, int64_t max_pairs);
bool u_ranges_possible(const Plan& p);

// ----- launchers (defined in the .hip files) -----
// scan.hip
size_t scan_tmp_elems(int64_t n);
hipError_t scan_exclusive_i64(const int64_t* in, int64_t* out, int64_t n, int64_t* tmp, hipStream_t s);
hipError_t scan_exclusive_i32(const int32_t* in, int32_t* out, int64_t n, int32_t* tmp, hipStream_t s);

// sort.hip: stable LSD radix sort of (uint64 key, payload) over the low
// `bits` bits.  The passes alternate between the primary and the alt
// buffers; the sorted result is in the alt buffers iff
// radix_result_in_alt(n, bits).  The pair variant can split the uint64
// payload (hi, lo) into two int32 arrays instead (split_hi non-null).  The
// pair variants also take the item count from device memory: with dn
// non-null they sort min(*dn, n) items, n being the capacity the grids and
// the histogram matrix are sized for (passes and buffers as for n).
int64_t radix_hist_elems(int64_t n);
bool radix_result_in_alt(int64_t n, int bits);
hipError_t radix_sort_u64(uint64_t* keys, uint32_t* vals, uint64_t* keys_alt, uint32_t* vals_alt, int64_t n,
                          int bits, int32_t* hist, int32_t* scan_tmp, hipStream_t s);
hipError_t radix_sort_u64_pairs(uint64_t* keys, uint64_t* vals, uint64_t* keys_alt, uint64_t* vals_alt, int64_t n,
                                const int64_t* dn, int bits, int32_t* hist, int32_t* scan_tmp, int32_t* split_hi,
                                int32_t* split_lo, hipStream_t s);
hipError_t radix_sort_u32_pairs(uint32_t* keys, uint64_t* vals, uint32_t* keys_alt, uint64_t* vals_alt, int64_t n,
                                const int64_t* dn, int bits, int32_t* hist, int32_t* scan_tmp, int32_t* split_hi,
                                int32_t* split_lo, hipStream_t s);

// join.hip
hipError_t launch_validate(const int32_t* keys, int64_t n, int r, const int32_t* radix, int32_t* err_flag,
                           hipStream_t s, const int64_t* dn = nullptr);
// several relations (at most three) in one launch; jobs with no rows or no
// key attributes are skipped
struct ValJob {
    const int32_t* keys;
    int64_t n;
    int r;
    const int32_t* radix;  // host, r entries
    int32_t* err;          // device flag word (bits 1 unsorted, 2 duplicate, 4 range)
    const int64_t* dn;     // optional device row count
};
hipError_t launch_validate(const ValJob* jobs, int n_jobs, hipStream_t s);
hipError_t launch_join(const Plan& p, const Layout& L, char* ws, const int32_t* u_keys, const int32_t* v_keys,
                       hipStream_t s, int stage);
// A V-driven join where U's key is the join labels and U holds every key of
// that key space: U's index is the join key itself, one pair per V tuple,
// written by the GROUP BY stage (the pair count is n_v, known on the host).
// Taken when V drives the plan's join, and also when U does but V's key
// starts with the join labels: V's order is then (u, v) order as well.
bool v_dense(const Plan& p, int64_t n_u);
// The same with U driving: V's key is the join labels and V holds every key of
// that key space (one pair per U tuple, the pair count n_u known on the host)
bool u_dense(const Plan& p, int64_t n_v);
// The whole join (runs, offsets, expansion, segments) in one workgroup when
// the pairs come out grouped by W key, the driving relation has at most 4096
// tuples and the capacity (min(workspace pairs, pair bound)) is at most 4096
// pairs
bool small_join_ok(const Plan& p, int64_t n_u, int64_t n_v, int64_t cap);
hipError_t launch_join_small(const Plan& p, const Layout& L, char* ws, const int32_t* u_keys, const int32_t* v_keys,
                             int64_t cap, hipStream_t s);
// V without promoted labels (one tuple) and W keyed by U's key as it is:
// every U tuple is one pair and one group, written without counting
bool keyed_by_u(const Plan& p);
hipError_t launch_keyed_by_u(const Plan& p, const Layout& L, char* ws, const int32_t* u_keys, hipStream_t s,
                             const int64_t* n_dev = nullptr);
// GROUP BY stage: the pair count is read on the device from the workspace
// header (written by launch_join), clamped to the capacity `cap` (at most
// L.max_pairs) that every grid is sized for, so the host launches it
// without waiting
hipError_t launch_group(const Plan& p, const Layout& L, char* ws, const int32_t* u_keys, const int32_t* v_keys,
                        int64_t cap, hipStream_t s);

// contract.hip
hipError_t launch_tables(const Plan& p, int32_t* tables, hipStream_t s);
// longest_first: reorder the units by decreasing length (GEMM class, at most
// a few thousand units) for a dispatch in that order
// dev_counts: n_pairs and n_w are upper bounds and the kernels read the
// join's counts from the workspace header (no read-back before the launch;
// one-workgroup unit tables or one unit per key only)
hipError_t launch_units(const Plan& p, const Layout& L, char* ws, int64_t n_pairs, int64_t n_w, int64_t p_unit,
                        bool longest_first, hipStream_t s, bool dev_counts = false);
// U-range units: unit r * n_w + s holds the pairs of key s whose U index lies
// in [r * n_u / R, (r + 1) * n_u / R); its partial tile is slot s * R + r.
hipError_t launch_range_units(const Plan& p, const Layout& L, char* ws, int64_t n_w, int64_t n_u, int32_t R,
                              hipStream_t s);
hipError_t launch_contract(const Plan& p, const Layout& L, char* ws, const void* u_tiles, const void* v_tiles,
                           float* w_tiles, int64_t n_pairs, int64_t n_w, int64_t unit_bound, hipStream_t s);
hipError_t launch_gemm_fast(const Plan& p, const Layout& L, char* ws, const void* u_tiles, const void* v_tiles,
                            float* w_tiles, int64_t n_pairs, int64_t unit_bound, hipStream_t s);
// Persistent paced variant (one unit per key, one 128x128 block per W tile):
// n_wg workgroups, all resident at once; pacing counters in L.pace, zeroed by
// the caller (rounds x 8 x windows int32, rounds = ceil(n_units / n_wg)).
int64_t gemm_paced_slots(const Plan& p);
hipError_t launch_gemm_paced(const Plan& p, const Layout& L, char* ws, const void* u_tiles, const void* v_tiles,
                             float* w_tiles, int64_t n_pairs, int64_t n_wg, int32_t windows, hipStream_t s);
hipError_t launch_reduce(const Plan& p, const Layout& L, char* ws, float* w_tiles, int64_t split_bound,
                         hipStream_t s);
hipError_t launch_write_outputs(const Plan& p, const Layout& L, char* ws, int32_t* w_keys, int32_t* pairs_out,
                                int64_t n_pairs, int64_t n_w, hipStream_t s, bool dev_counts = false);
hipError_t launch_counts_out(const Layout& L, char* ws, int64_t max_pairs, int64_t* counts, hipStream_t s);
hipError_t launch_counts_set(int64_t n_pairs, int64_t n_w, int64_t status, int64_t* counts, hipStream_t s);

// glue.hip
hipError_t launch_cast_bf16(const float* x, uint16_t* y, int64_t n, hipStream_t s);
hipError_t launch_scale(const float* x, float* y, int64_t n, float sc, hipStream_t s);
hipError_t launch_tiles_from_entries(const int64_t* slot, const int64_t* off, const void* val, int64_t n,
                                     int elem_bytes, void* tiles, int64_t n_tiles, int64_t tile_elems,
                                     hipStream_t s);
hipError_t launch_fill_zero(void* p, size_t bytes, hipStream_t s);
hipError_t launch_stack(const int32_t* keys, int64_t n, const void* tiles, int64_t row_elems, int32_t group,
                        int32_t elem_bytes, int32_t* out_keys, void* out_tiles, int64_t n_out, char* ws,
                        hipStream_t s, int stage);
size_t stack_ws_bytes(int64_t n);

void set_error(const std::string& msg);

// Timing events from a per-device pool (created on first use, reused after
// release).
hipEvent_t event_acquire();
void event_release(hipEvent_t e);

// Start and end events of one kernel, recorded by the kernel's own dispatch
// (hipExtLaunchKernel): no marker packets on the stream, so timing a kernel
// this way adds next to nothing to the launch sequence.  While
// t_kernel_events is set, the contraction kernel launches attach it.
struct KernelEvents {
    hipEvent_t start = nullptr, stop = nullptr;
    bool launched = false;
    bool keep = false;  // handed to a tre_timing (released by tre_timing_read)
    KernelEvents() = default;
    KernelEvents(const KernelEvents&) = delete;
    KernelEvents& operator=(const KernelEvents&) = delete;
    ~KernelEvents();  // back to the pool unless kept
};
extern thread_local KernelEvents* t_kernel_events;

template <typename T>
struct same_type {
    using type = T;
};

// Launch `kernel` (<<<>>> semantics); with t_kernel_events set, through
// hipExtLaunchKernel with its start / stop events.
template <typename... KArgs>
inline hipError_t launch_k(void (*kernel)(KArgs...), dim3 grid, dim3 block, size_t shmem, hipStream_t s,
                           typename same_type<KArgs>::type... args) {
    KernelEvents* ke = t_kernel_events;
    if (!ke) {
        kernel<<<grid, block, shmem, s>>>(args...);
        return hipGetLastError();
    }
    void* argv[] = {static_cast<void*>(&args)...};
    const hipError_t e = hipExtLaunchKernel(reinterpret_cast<const void*>(kernel), grid, block, argv, shmem, s,
                                            ke->start, ke->stop, 0);
    if (e == hipSuccess) ke->launched = true;
    return e;
}

// hipEvent timer.  In deferred mode the events are handed to the caller's
// tre_timing (keep = true) and read and released later by tre_timing_read.
struct PhaseTimer {
    static constexpr int kMax = 5;
    bool on = false;
    bool keep = false;  // set once the events are handed to a deferred tre_timing
    hipEvent_t ev[kMax] = {};
    int n = 0;
    explicit PhaseTimer(bool enable) : on(enable) {}
    ~PhaseTimer() {
        if (keep) return;
        for (auto& e : ev) event_release(e);
    }
    // events are taken when first recorded, so a deferred timer hands over
    // exactly the events it recorded
    void mark(hipStream_t s) {
        if (!on || n >= kMax) return;
        ev[n] = event_acquire();
        if (!ev[n]) {
            on = false;
            return;
        }
        (void)hipEventRecord(ev[n++], s);
    }
    float between(int a, int b) {
        float ms = 0.f;
        if (on && b < n) {
            (void)hipEventSynchronize(ev[b]);
            (void)hipEventElapsedTime(&ms, ev[a], ev[b]);
        }
        return ms;
    }
};

inline float event_elapsed(void* a, void* b) {
    float ms = 0.f;
    if (a && b) {
        (void)hipEventSynchronize(reinterpret_cast<hipEvent_t>(b));
        (void)hipEventElapsedTime(&ms, reinterpret_cast<hipEvent_t>(a), reinterpret_cast<hipEvent_t>(b));
    }
    return ms;
}


}  // namespace tre

// Opaque plan handle of the C ABI.
struct tre_plan_s {
    tre::Plan p;
};
