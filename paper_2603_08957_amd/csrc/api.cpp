// C-ABI entry points: argument checks, workspace layout, phase ordering,
// the join's one count read-back, capacity checks and timing.
#include <algorithm>
#include <cmath>
#include <cstring>

#include "tre_internal.h"

using namespace tre;

namespace {

constexpr uint64_t kMagic = 0x7472655f6a6f696eull;  // "tre_join"
constexpr int kTargetWorkgroups = 2048;              // 8 per CU on 256 CUs
constexpr int64_t kAsyncMaxKeys = 4096;              // output keys of the one-workgroup unit table

tre_status dev_fail(hipError_t e, const char* where) {
    set_error(std::string(where) + ": " + hipGetErrorString(e));
    return TRE_E_DEVICE;
}

tre_status key_error(int32_t flags) {
    if (flags & 4) return TRE_E_KEYRANGE;
    if (flags & 1) return TRE_E_UNSORTED;
    if (flags & 2) return TRE_E_DUPKEY;
    return TRE_OK;
}

int64_t blocks_per_unit(const Plan& p) {
    if (p.kclass == KC_GEMM) {
        const int64_t M = p.swap ? p.nN : p.nM, N = p.swap ? p.nM : p.nN;
        if (p.fast) return (M / 128) * (N / 128);
        return p.nB * ((M + 63) / 64) * ((N + 63) / 64);
    }
    return (p.tile_elems[2] + 255) / 256;
}

// Number of U-index ranges for the 128x128 path (0 or 1 = off).  Worth
// it when the U tiles are reused by many keys (pairs per U tuple high) but do
// not fit in one XCD's 4 MB L2: cutting every key's pairs into ranges of U and
// dispatching range by range lets the workgroups resident on an XCD share
// about 2 MB of U tiles, which stay in its L2 while the V tiles stream past,
// at the price of one partial tile per (key, range).
int32_t choose_u_ranges(const Plan& p, const Layout& L, int64_t n_u, int64_t n_pairs, int64_t n_w) {
    if (!(p.kclass == KC_GEMM && p.fast) || p.opt.u_ranges < 0 || n_u < 2 || n_w < 1) return 0;
    int64_t R;
    if (p.opt.u_ranges > 0) {
        R = p.opt.u_ranges;
    } else {
        const int64_t u_bytes = n_u * p.tile_elems[0] * (p.dtype == TRE_BF16 ? 2 : 4);
        const int64_t reuse = n_pairs / n_u;
        if (u_bytes <= (int64_t(16) << 20) || reuse < 64 || n_w * blocks_per_unit(p) < kTargetWorkgroups) return 0;
        // ~2 MB of U per range: measured best on the 262,144-vertex chain
        // (4 MB ranges thrash the L2, 1 MB ranges pay for twice the partials)
        R = (u_bytes + (int64_t(2) << 20) - 1) >> 21;
    }
    R = std::min<int64_t>({R, n_u, kMaxURanges});
    while (R > 1 && R * n_w > L.part_cap) R /= 2;
    return R > 1 ? int32_t(R) : 0;
}

// Windows for the paced persistent kernel (0 = not used).  It applies where
// U ranges would (U tiles reused by many keys and too big for one L2) when a W
// tile is one 128x128 block, and is preferred there: it keeps U tiles in L2
// without partial tiles.  `slots` = workgroups resident at once.
int32_t choose_pacing(const Plan& p, int64_t n_u, int64_t n_pairs, int64_t n_w, int64_t slots) {
    if (!(p.kclass == KC_GEMM && p.fast) || blocks_per_unit(p) != 1 || p.opt.pace_windows < 0 ||
        p.opt.max_pairs_per_unit > 0 || n_u < 2 || n_w < 1 || slots <= 0)
        return 0;
    int64_t W;
    if (p.opt.pace_windows > 0) {
        W = p.opt.pace_windows;
    } else {
        if (p.opt.u_ranges != 0) return 0;  // an explicit U-range request wins
        const int64_t u_bytes = n_u * p.tile_elems[0] * (p.dtype == TRE_BF16 ? 2 : 4);
        const int64_t reuse = n_pairs / n_u;
        if (u_bytes <= (int64_t(16) << 20) || reuse < 64 || n_w < slots) return 0;
        // ~5.5 MB of U per window: measured best on the 262,144-vertex chain
        // (12 windows of its 64 MB; 16 or 10 windows are 0.5% slower, 8 and
        // 24 windows 1-3%: small windows wait more often, large ones miss L2)
        constexpr int64_t kWindowBytes = int64_t(11) << 19;
        W = (u_bytes + kWindowBytes - 1) / kWindowBytes;
    }
    W = std::max<int64_t>(1, std::min<int64_t>({W, n_u, 256}));
    const int64_t n_wg = std::min(n_w, slots);
    const int64_t rounds = (n_w + n_wg - 1) / n_wg;
    if (rounds * 8 * W > kPaceCounters) return 0;
    return int32_t(W);
}

// Workgroups one unit occupies: its output blocks (GEMM), or its threads /
// 256 for the vector class (several small units share a workgroup).
double unit_workgroups(const Plan& p) {
    if (p.kclass == KC_GEMM) return double(blocks_per_unit(p));
    const int64_t threads = (p.tile_elems[2] + p.vec_ept - 1) / p.vec_ept;
    if (threads > 128) return double((threads + 255) / 256);
    int64_t t = 1;
    while (t < threads) t <<= 1;
    return double(t) / 256.0;
}

// Unit length cap.  GEMM-class units are dispatched longest first, so once
// the keys' output blocks fill every resident slot (two workgroups per CU)
// one unit per key is the better schedule: measured on the block-sparse
// product (1,024 blocks of 6.4 pairs on average), cutting keys into units of
// 4-8 pairs cost 10% more in contraction and partial-tile sums.
int64_t choose_unit(const Plan& p, const Layout& L, int64_t n_pairs, int64_t n_w) {
    const double uw = unit_workgroups(p);
    int dev = 0, cus = 0;
    const int64_t fill = (hipGetDevice(&dev) == hipSuccess &&
                          hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) == hipSuccess && cus > 0)
                             ? 2 * int64_t(cus)
                             : int64_t(kTargetWorkgroups);
    int64_t pu;
    if (p.opt.max_pairs_per_unit > 0) {
        pu = p.opt.max_pairs_per_unit;
    } else if (double(n_w) * uw >= kTargetWorkgroups || (p.kclass == KC_GEMM && double(n_w) * uw >= fill)) {
        pu = std::max<int64_t>(n_pairs, 1);  // enough output blocks: one unit per key
    } else {
        pu = std::max<int64_t>(4, int64_t(std::ceil(double(n_pairs) * uw / kTargetWorkgroups)));
    }
    // partial tiles of split keys must fit: at most 2 * n_pairs / pu of them
    const int64_t need = (2 * n_pairs + L.part_cap - 2) / std::max<int64_t>(L.part_cap - 1, 1);
    return std::max<int64_t>(pu, std::max<int64_t>(need, 1));
}

// Most pairs a join of n_u and n_v tuples (unique keys) can make: the cross
// product, or one pair per tuple of the other side when one side's key is
// made of join labels only.  The GROUP BY grids are sized for min(this,
// workspace capacity).
int64_t pair_bound(const Plan& p, int64_t n_u, int64_t n_v) {
    int64_t b = (n_v > 0 && n_u > INT64_MAX / n_v) ? INT64_MAX : n_u * n_v;
    if (p.nk[0] == p.n_join) b = std::min(b, n_v);  // a V tuple meets at most one U tuple
    if (p.nk[1] == p.n_join) b = std::min(b, n_u);
    return b;
}

}  // namespace

namespace {

// What the join leaves for its read-back.
struct JoinState {
    int64_t max_pairs = 0;
    int64_t cap = 0;      // pairs the GROUP BY grids are sized for
    bool counts_known = false;  // pair and key counts known on the host (no read-back needed for them)
    bool small = false;
    int32_t path = 0;     // tre_timing.join_path
};

// tre_join up to its read-back: argument checks, workspace layout and every
// join launch.  `out` gets the sizes and the internal fields.
tre_status join_enqueue(tre_plan_t plan, const int32_t* u_keys, int64_t n_u, const int32_t* v_keys, int64_t n_v,
                        void* ws, size_t ws_bytes, hipStream_t s, tre_join_result* out, JoinState* st,
                        const int64_t* n_u_dev = nullptr) {
    if (!plan || !out || n_u < 0 || n_v < 0 || !ws) {
        set_error("tre_join: null plan/out/workspace or negative size");
        return TRE_E_ARG;
    }
    const Plan& p = plan->p;
    std::memset(out, 0, sizeof(*out));
    out->n_u = n_u;
    out->n_v = n_v;
    if ((p.nk[0] > 0 && n_u > 0 && !u_keys) || (p.nk[1] > 0 && n_v > 0 && !v_keys)) {
        set_error("tre_join: null key array");
        return TRE_E_ARG;
    }
    if (reinterpret_cast<uintptr_t>(ws) % 256) {
        set_error("tre_join: workspace must be 256-byte aligned");
        return TRE_E_ARG;
    }
    if ((p.nk[0] == 0 && n_u > 1) || (p.nk[1] == 0 && n_v > 1)) {
        set_error("tre_join: a relation without promoted labels holds at most one tuple");
        return TRE_E_DUPKEY;
    }
    if (n_u >= INT32_MAX || n_v >= INT32_MAX) {
        set_error("tre_join: more than 2^31 - 1 tuples");
        return TRE_E_SHAPE;
    }
    const int64_t max_pairs = tre_workspace_max_pairs(plan, n_u, n_v, ws_bytes);
    if (max_pairs < 0) {
        set_error("tre_join: workspace smaller than tre_workspace_bytes(plan, n_u, n_v, 0)");
        return TRE_E_WORKSPACE;
    }
    st->max_pairs = max_pairs;
    out->internal[0] = kMagic;
    out->internal[1] = reinterpret_cast<uint64_t>(plan);
    out->internal[2] = reinterpret_cast<uint64_t>(ws);
    out->internal[3] = uint64_t(ws_bytes);
    out->internal[4] = uint64_t(max_pairs);
    const Layout L = make_layout(p, n_u, n_v, max_pairs);
    char* w = reinterpret_cast<char*>(ws);
    hipError_t e = launch_fill_zero(w + L.hdr, sizeof(WsHeader), s);
    if (e != hipSuccess) return dev_fail(e, "header");
    WsHeader* hdr = reinterpret_cast<WsHeader*>(w + L.hdr);
    if (p.opt.validate_keys) {
        const ValJob jobs[2] = {{u_keys, n_u, p.nk[0], p.radix[0], &hdr->err_u, n_u_dev},
                                {v_keys, n_v, p.nk[1], p.radix[1], &hdr->err_v, nullptr}};
        if ((e = launch_validate(jobs, 2, s)) != hipSuccess) return dev_fail(e, "validate");
    }
    if (n_u > 0 && n_v == 1 && keyed_by_u(p)) {
        // one pair and one group per U tuple: nothing to count
        if (n_u > max_pairs) {
            out->n_pairs = n_u;
            set_error("tre_join: workspace too small for the matched pairs (see n_pairs)");
            return TRE_E_WORKSPACE;
        }
        if ((e = launch_keyed_by_u(p, L, w, u_keys, s, n_u_dev)) != hipSuccess) return dev_fail(e, "join");
        st->cap = n_u;
        st->counts_known = true;
        st->path = 4;
        out->n_pairs = n_u;
        out->n_w = n_u;
        return TRE_OK;
    }
    // the join counts the pairs into the header; the GROUP BY stage reads
    // that count on the device (its grids are sized for the workspace's
    // capacity), so one read-back at the end returns the key checks, the
    // pair count and the key count together
    const bool vd = n_u > 0 && n_v > 0 && v_dense(p, n_u), ud = n_u > 0 && n_v > 0 && u_dense(p, n_v);
    if ((vd || ud) && (vd ? n_v : n_u) > max_pairs) {
        // one pair per tuple of the driving relation, known without the device
        out->n_pairs = vd ? n_v : n_u;
        set_error("tre_join: workspace too small for the matched pairs (see n_pairs)");
        return TRE_E_WORKSPACE;
    }
    const int64_t cap = std::min(max_pairs, pair_bound(p, n_u, n_v));
    st->cap = (n_u > 0 && n_v > 0) ? std::max<int64_t>(cap, 0) : 0;
    st->small = n_u > 0 && n_v > 0 && small_join_ok(p, n_u, n_v, cap);
    if (st->small) {
        if ((e = launch_join_small(p, L, w, u_keys, v_keys, cap, s)) != hipSuccess) return dev_fail(e, "join");
    } else if (n_u > 0 && n_v > 0 && max_pairs > 0) {
        if ((e = launch_join(p, L, w, u_keys, v_keys, s, 0)) != hipSuccess) return dev_fail(e, "join");
        if ((e = launch_group(p, L, w, u_keys, v_keys, cap, s)) != hipSuccess) return dev_fail(e, "group");
    } else if (n_u > 0 && n_v > 0) {
        // no room for any pair: count only, to report the size needed
        if ((e = launch_join(p, L, w, u_keys, v_keys, s, 0)) != hipSuccess) return dev_fail(e, "join");
    }
    st->path = st->small                               ? 5
               : vd                                     ? 3
               : ud                                     ? 6
               : (p.v_outer && p.nk[0] == p.n_join)     ? 2
               : p.v_outer                              ? 1
                                                        : 0;
    return TRE_OK;
}

// The join's read-back: key checks and, unless known on the host, the pair
// and key counts.  With key checks off and counts known, nothing to wait for.
tre_status join_finish(const Plan& p, const JoinState& st, tre_join_result* out, hipStream_t s) {
    if (st.counts_known && !p.opt.validate_keys) return TRE_OK;
    const Layout L = make_layout(p, out->n_u, out->n_v, st.max_pairs);
    const char* w = reinterpret_cast<const char*>(out->internal[2]);
    WsHeader h{};
    hipError_t e;
    if ((e = hipMemcpyAsync(&h, w + L.hdr, sizeof(h), hipMemcpyDeviceToHost, s)) != hipSuccess)
        return dev_fail(e, "count read-back");
    if ((e = hipStreamSynchronize(s)) != hipSuccess) return dev_fail(e, "join sync");
    tre_status ks = key_error(h.err_u);
    if (ks == TRE_OK) ks = key_error(h.err_v);
    if (ks != TRE_OK) {
        set_error(std::string("tre_join: invalid keys in ") + (key_error(h.err_u) != TRE_OK ? "U" : "V"));
        return ks;
    }
    if (st.counts_known) return TRE_OK;
    const int64_t n_pairs = (out->n_u > 0 && out->n_v > 0) ? h.n_pairs : 0;
    out->n_pairs = n_pairs;
    if (n_pairs > st.max_pairs) {
        set_error("tre_join: workspace too small for the matched pairs (see n_pairs)");
        return TRE_E_WORKSPACE;
    }
    if (n_pairs >= INT32_MAX) {
        set_error("tre_join: more than 2^31 - 1 pairs");
        return TRE_E_SHAPE;
    }
    out->n_w = n_pairs > 0 ? h.n_w : 0;
    return TRE_OK;
}

void join_timing(tre_timing* timing, int32_t path) {
    if (!timing) return;
    const int32_t deferred = timing->deferred;
    std::memset(timing, 0, sizeof(*timing));
    timing->deferred = deferred;
    timing->join_path = path;
}

// tre_contract's launches, for the join's counts n_pairs and n_w.  With
// `dev` those are upper bounds and every kernel reads the join's counts from
// the workspace header (the caller has checked that the bounds need no U
// ranges and take a one-workgroup unit table or one unit per key).
tre_status contract_enqueue(tre_plan_t plan, const tre_join_result* jr, int64_t n_pairs, int64_t n_w,
                            const void* u_tiles, const void* v_tiles, int32_t* w_keys, void* w_out,
                            int32_t* pairs_out, hipStream_t s, tre_timing* timing, bool dev = false) {
    // W's element type is the plan's (fp32, or bf16 bits with w_bf16); the
    // kernels take the array as float* and store 16-bit elements through it
    // when the plan says bf16
    float* w_tiles = static_cast<float*>(w_out);
    const Plan& p = plan->p;
    if (n_pairs == 0) return TRE_OK;
    if (!u_tiles || !v_tiles || !w_tiles || (p.nk[2] > 0 && !w_keys)) {
        set_error("tre_contract: null tile or key buffer");
        return TRE_E_ARG;
    }
    if ((reinterpret_cast<uintptr_t>(u_tiles) | reinterpret_cast<uintptr_t>(v_tiles) |
         reinterpret_cast<uintptr_t>(w_tiles)) & 15) {
        set_error("tre_contract: tile arrays must be 16-byte aligned");
        return TRE_E_ARG;
    }
    char* w = reinterpret_cast<char*>(jr->internal[2]);
    const Layout L = make_layout(p, jr->n_u, jr->n_v, int64_t(jr->internal[4]));
    // deferred timing: only the contraction kernel, by its own start / end
    // events (no marker packets); otherwise marks around every phase
    const bool deferred = timing && timing->deferred;
    PhaseTimer tm(timing != nullptr && !deferred);
    KernelEvents ke;
    if (deferred) {
        ke.start = event_acquire();
        ke.stop = event_acquire();
    }
    tm.mark(s);
    const int64_t slots = (p.kclass == KC_GEMM && p.fast) ? gemm_paced_slots(p) : 0;
    const int32_t pace = choose_pacing(p, jr->n_u, n_pairs, n_w, slots);
    const int32_t R = (pace || dev) ? 0 : choose_u_ranges(p, L, jr->n_u, n_pairs, n_w);
    // (a keyless one-tuple V with W keyed by U: one pair per key, nothing
    // to cut and no partial tiles to sum)
    const bool one_pair_keys = jr->n_v <= 1 && keyed_by_u(p);
    const int64_t p_unit = (R > 1 || pace || one_pair_keys) ? n_pairs : choose_unit(p, L, n_pairs, n_w);
    hipError_t e;
    // (launch_units writes the tile offset tables itself)
    if (R > 1) {
        if ((e = launch_tables(p, reinterpret_cast<int32_t*>(w + L.tables), s)) != hipSuccess)
            return dev_fail(e, "tables");
        e = launch_range_units(p, L, w, n_w, jr->n_u, R, s);
    } else {
        e = launch_units(p, L, w, n_pairs, n_w, p_unit, !pace, s, dev);
    }
    if (e != hipSuccess) return dev_fail(e, "units");
    tm.mark(s);
    const int64_t unit_bound = R > 1 ? int64_t(R) * n_w : n_w + n_pairs / p_unit + 1;
    if (pace) {
        // one unit per key; every workgroup of the grid is resident at once
        const int64_t n_wg = std::min(n_w, slots);
        const int64_t rounds = (n_w + n_wg - 1) / n_wg;
        if ((e = launch_fill_zero(w + L.pace, sizeof(int32_t) * size_t(rounds * 8 * pace), s)) != hipSuccess)
            return dev_fail(e, "pace");
        if (ke.start && ke.stop) t_kernel_events = &ke;
        e = launch_gemm_paced(p, L, w, u_tiles, v_tiles, w_tiles, n_pairs, n_wg, pace, s);
    } else {
        if (ke.start && ke.stop) t_kernel_events = &ke;
        e = launch_contract(p, L, w, u_tiles, v_tiles, w_tiles, n_pairs, n_w, unit_bound, s);
    }
    t_kernel_events = nullptr;
    if (e != hipSuccess) return dev_fail(e, "contract");
    tm.mark(s);
    if (R > 1 || p_unit < n_pairs) {
        const int64_t split_bound = R > 1 ? n_w : std::min<int64_t>(n_w, n_pairs / (p_unit + 1) + 1);
        if ((e = launch_reduce(p, L, w, w_tiles, split_bound, s)) != hipSuccess) return dev_fail(e, "reduce");
    }
    if ((e = launch_write_outputs(p, L, w, w_keys, pairs_out, n_pairs, n_w, s, dev)) != hipSuccess)
        return dev_fail(e, "outputs");
    tm.mark(s);
    if (timing) {
        timing->contract_path = pace ? 3 : R > 1 ? 4 : (p.kclass == KC_VEC ? 1 : p.fast ? 2 : 0);
        if (deferred) {
            if (ke.launched) {
                timing->events[0] = reinterpret_cast<void*>(ke.start);
                timing->events[1] = reinterpret_cast<void*>(ke.stop);
                timing->pending = 1;
                ke.keep = true;
            }
        } else {
            timing->units_ms = tm.between(0, 1);
            timing->contract_ms = tm.between(1, 2);
            timing->reduce_ms = tm.between(2, 3);
            timing->total_ms += tm.between(0, 3);
        }
        WsHeader h{};
        if (!deferred && hipMemcpy(&h, w + L.hdr, sizeof(h), hipMemcpyDeviceToHost) == hipSuccess) {
            timing->n_units = h.n_units;
            timing->n_split_segments = h.n_split;
            timing->n_partials = h.n_parts;
        }
    }
    return TRE_OK;
}

// Upper bounds on a join's pair and output key counts, from the sizes alone
// (exact when the host knows them), and whether the contraction can be
// enqueued on them with the counts read on the device: no pacing and no U
// ranges at the bounds, and a one-workgroup unit table or one unit per key
// (the paced persistent grid takes one unit per key and reads their count).
struct AsyncBounds {
    int64_t pairs = 0, keys = 0;
    bool ok = false;
};

AsyncBounds async_bounds(const Plan& p, int64_t n_u, int64_t n_v, int64_t max_pairs) {
    AsyncBounds b;
    if (n_u > 0 && n_v == 1 && keyed_by_u(p)) {
        b.pairs = b.keys = n_u;
    } else {
        int64_t w_space = 1;
        for (int c = 0; c < p.nk[2] && w_space <= (int64_t(1) << 40); c++) w_space *= p.radix[2][c];
        b.pairs = (n_u > 0 && n_v > 0) ? std::max<int64_t>(0, std::min(max_pairs, pair_bound(p, n_u, n_v))) : 0;
        b.keys = std::min(b.pairs, w_space);
    }
    if (b.pairs <= 0) {
        b.ok = true;
        return b;
    }
    const Layout L = make_layout(p, n_u, n_v, max_pairs);
    const int64_t slots = (p.kclass == KC_GEMM && p.fast) ? gemm_paced_slots(p) : 0;
    if (choose_pacing(p, n_u, b.pairs, b.keys, slots) != 0) {
        b.ok = true;  // one unit per key; the persistent grid reads the unit count on the device
        return b;
    }
    if (choose_u_ranges(p, L, n_u, b.pairs, b.keys) != 0) return b;
    const int64_t p_unit = choose_unit(p, L, b.pairs, b.keys);
    b.ok = b.keys <= kAsyncMaxKeys || p_unit >= b.pairs;
    return b;
}

}  // namespace

extern "C" {

tre_status tre_join(tre_plan_t plan, const int32_t* u_keys, int64_t n_u, const int32_t* v_keys, int64_t n_v,
                    void* ws, size_t ws_bytes, void* stream, tre_join_result* out, tre_timing* timing) {
    hipStream_t s = reinterpret_cast<hipStream_t>(stream);
    PhaseTimer tm(timing != nullptr && !timing->deferred);  // (deferred timing covers the contraction only)
    tm.mark(s);
    JoinState st;
    tre_status r = join_enqueue(plan, u_keys, n_u, v_keys, n_v, ws, ws_bytes, s, out, &st);
    if (r != TRE_OK) return r;
    // the end mark goes before the read-back, so reading the join time after
    // the wait needs no further wait
    tm.mark(s);
    if ((r = join_finish(plan->p, st, out, s)) != TRE_OK) return r;
    join_timing(timing, st.path);
    if (timing) {
        timing->join_ms = tm.between(0, 1);
        timing->total_ms = timing->join_ms;
    }
    return TRE_OK;
}

tre_status tre_contract(tre_plan_t plan, const tre_join_result* jr, const void* u_tiles, const void* v_tiles,
                        int32_t* w_keys, int64_t w_cap, void* w_out, int32_t* pairs_out, int64_t pair_cap,
                        void* stream, tre_timing* timing) {
    if (!plan || !jr) {
        set_error("tre_contract: null plan or join result");
        return TRE_E_ARG;
    }
    if (jr->internal[0] != kMagic || jr->internal[1] != reinterpret_cast<uint64_t>(plan)) {
        set_error("tre_contract: join result was not produced by tre_join with this plan");
        return TRE_E_STATE;
    }
    if (w_cap < jr->n_w || (pairs_out && pair_cap < jr->n_pairs)) {
        set_error("tre_contract: output capacity below n_w / n_pairs");
        return TRE_E_CAPACITY;
    }
    return contract_enqueue(plan, jr, jr->n_pairs, jr->n_w, u_tiles, v_tiles, w_keys, w_out, pairs_out,
                            reinterpret_cast<hipStream_t>(stream), timing);
}

tre_status tre_join_keys(tre_plan_t plan, const tre_join_result* jr, int32_t* w_keys, int64_t w_cap, void* stream) {
    if (!plan || !jr) {
        set_error("tre_join_keys: null plan or join result");
        return TRE_E_ARG;
    }
    if (jr->internal[0] != kMagic || jr->internal[1] != reinterpret_cast<uint64_t>(plan)) {
        set_error("tre_join_keys: join result was not produced by tre_join with this plan");
        return TRE_E_STATE;
    }
    const Plan& p = plan->p;
    if (w_cap < jr->n_w) {
        set_error("tre_join_keys: output capacity below n_w");
        return TRE_E_CAPACITY;
    }
    if (p.nk[2] == 0 || jr->n_w == 0) return TRE_OK;
    if (!w_keys) {
        set_error("tre_join_keys: null key buffer");
        return TRE_E_ARG;
    }
    char* w = reinterpret_cast<char*>(jr->internal[2]);
    const Layout L = make_layout(p, jr->n_u, jr->n_v, int64_t(jr->internal[4]));
    const hipError_t e = launch_write_outputs(p, L, w, w_keys, nullptr, jr->n_pairs, jr->n_w,
                                              reinterpret_cast<hipStream_t>(stream));
    return e == hipSuccess ? TRE_OK : dev_fail(e, "keys");
}

tre_status tre_timing_read(tre_timing* t) {
    if (!t) return TRE_E_ARG;
    if (!t->pending) return TRE_OK;
    // the contraction kernel's start and end
    t->contract_ms = event_elapsed(t->events[0], t->events[1]);
    t->total_ms += t->contract_ms;
    for (auto& e : t->events) {
        event_release(reinterpret_cast<hipEvent_t>(e));
        e = nullptr;
    }
    t->pending = 0;
    return TRE_OK;
}

tre_status tre_execute(tre_plan_t plan, const int32_t* u_keys, int64_t n_u, const void* u_tiles,
                       const int32_t* v_keys, int64_t n_v, const void* v_tiles, int32_t* w_keys, void* w_tiles,
                       int64_t w_cap, int64_t* n_w, int32_t* pairs_out, int64_t pair_cap, int64_t* n_pairs,
                       void* ws, size_t ws_bytes, void* stream, tre_timing* timing) {
    tre_join_result jr{};
    tre_status st = tre_join(plan, u_keys, n_u, v_keys, n_v, ws, ws_bytes, stream, &jr, timing);
    if (n_pairs) *n_pairs = jr.n_pairs;
    if (n_w) *n_w = jr.n_w;
    if (st != TRE_OK) return st;
    return tre_contract(plan, &jr, u_tiles, v_tiles, w_keys, w_cap, w_tiles, pairs_out, pair_cap, stream, timing);
}

tre_status tre_output_bounds(tre_plan_t plan, int64_t n_u, int64_t n_v, size_t ws_bytes, int64_t* pairs_bound,
                             int64_t* keys_bound, int32_t* async_ok) {
    if (!plan || n_u < 0 || n_v < 0 || !pairs_bound || !keys_bound || !async_ok) {
        set_error("tre_output_bounds: null argument or negative size");
        return TRE_E_ARG;
    }
    const int64_t max_pairs = tre_workspace_max_pairs(plan, n_u, n_v, ws_bytes);
    if (max_pairs < 0) {
        set_error("tre_output_bounds: workspace smaller than tre_workspace_bytes(plan, n_u, n_v, 0)");
        return TRE_E_WORKSPACE;
    }
    const AsyncBounds b = async_bounds(plan->p, n_u, n_v, max_pairs);
    *pairs_bound = b.pairs;
    *keys_bound = b.keys;
    *async_ok = b.ok ? 1 : 0;
    return TRE_OK;
}

tre_status tre_execute_async(tre_plan_t plan, const int32_t* u_keys, int64_t n_u, const int64_t* n_u_dev,
                             const void* u_tiles, const int32_t* v_keys, int64_t n_v, const void* v_tiles,
                             int32_t* w_keys, void* w_tiles, int64_t w_cap, int32_t* pairs_out, int64_t pair_cap,
                             int64_t* counts, void* ws, size_t ws_bytes, void* stream, tre_timing* timing) {
    if (!plan || !counts || n_u < 0 || n_v < 0) {
        set_error("tre_execute_async: null plan / counts or negative size");
        return TRE_E_ARG;
    }
    const Plan& p = plan->p;
    hipStream_t s = reinterpret_cast<hipStream_t>(stream);
    if (n_u_dev && !(n_v == 1 && keyed_by_u(p))) {
        set_error("tre_execute_async: a device-side U count needs a keyless one-tuple V with W keyed by U");
        return TRE_E_ARG;
    }
    const int64_t max_pairs = tre_workspace_max_pairs(plan, n_u, n_v, ws_bytes);
    if (max_pairs < 0) {
        set_error("tre_execute_async: workspace smaller than tre_workspace_bytes(plan, n_u, n_v, 0)");
        return TRE_E_WORKSPACE;
    }
    const AsyncBounds b = async_bounds(p, n_u, n_v, max_pairs);
    if (!b.ok) {
        if (n_u_dev) {
            set_error("tre_execute_async: a device-side U count needs an output within the device-count launches");
            return TRE_E_ARG;
        }
        // the counts are needed on the host: the synchronous call, then the
        // counts and the status to the device
        int64_t nw = 0, np = 0;
        const tre_status st = tre_execute(plan, u_keys, n_u, u_tiles, v_keys, n_v, v_tiles, w_keys, w_tiles, w_cap,
                                          &nw, pairs_out, pair_cap, &np, ws, ws_bytes, stream, timing);
        if (st == TRE_E_ARG || st == TRE_E_DEVICE || st == TRE_E_STATE) return st;
        const hipError_t e = launch_counts_set(np, nw, int64_t(st), counts, s);
        return e == hipSuccess ? st : dev_fail(e, "counts");
    }
    if (w_cap < b.keys || (pairs_out && pair_cap < b.pairs)) {
        set_error("tre_execute_async: output capacity below the bounds of tre_output_bounds");
        return TRE_E_CAPACITY;
    }
    tre_join_result jr{};
    JoinState js;
    PhaseTimer tm(timing != nullptr && !timing->deferred);
    tm.mark(s);
    tre_status st = join_enqueue(plan, u_keys, n_u, v_keys, n_v, ws, ws_bytes, s, &jr, &js, n_u_dev);
    if (st != TRE_OK) return st;
    tm.mark(s);
    join_timing(timing, js.path);
    if ((st = contract_enqueue(plan, &jr, b.pairs, b.keys, u_tiles, v_tiles, w_keys, w_tiles, pairs_out, s, timing,
                               true)) != TRE_OK)
        return st;
    const Layout L = make_layout(p, n_u, n_v, max_pairs);
    const hipError_t e = launch_counts_out(L, static_cast<char*>(ws), max_pairs, counts, s);
    if (e != hipSuccess) return dev_fail(e, "counts");
    if (timing && !timing->deferred) {
        const float jm = tm.between(0, 1);
        timing->join_ms = jm;
        timing->total_ms += jm;
    }
    return TRE_OK;
}

tre_status tre_cast_f32_bf16(const float* x, uint16_t* y, int64_t n, void* stream) {
    if (n < 0 || (n > 0 && (!x || !y))) return TRE_E_ARG;
    hipError_t e = launch_cast_bf16(x, y, n, reinterpret_cast<hipStream_t>(stream));
    return e == hipSuccess ? TRE_OK : dev_fail(e, "cast");
}

tre_status tre_scale_f32(const float* x, float* y, int64_t n, float scale, void* stream) {
    if (n < 0 || (n > 0 && (!x || !y))) return TRE_E_ARG;
    if (n > 0 && ((reinterpret_cast<uintptr_t>(x) | reinterpret_cast<uintptr_t>(y)) & 15)) {
        set_error("tre_scale_f32: arrays must be 16-byte aligned");
        return TRE_E_ARG;
    }
    hipError_t e = launch_scale(x, y, n, scale, reinterpret_cast<hipStream_t>(stream));
    return e == hipSuccess ? TRE_OK : dev_fail(e, "scale");
}

size_t tre_stack_workspace_bytes(int64_t n) { return n < 0 ? 0 : stack_ws_bytes(n); }

tre_status tre_stack_rows(const int32_t* keys, int64_t n, const void* tiles, int64_t row_elems, int32_t group,
                          int32_t elem_bytes, int32_t* out_keys, void* out_tiles, int64_t out_cap, int64_t* n_out,
                          void* ws, size_t ws_bytes, void* stream) {
    if (n < 0 || row_elems < 1 || group < 1 || (elem_bytes != 2 && elem_bytes != 4) || !n_out || !ws ||
        (n > 0 && (!keys || !tiles))) {
        set_error("tre_stack_rows: bad argument");
        return TRE_E_ARG;
    }
    if (ws_bytes < stack_ws_bytes(n)) return TRE_E_WORKSPACE;
    hipStream_t s = reinterpret_cast<hipStream_t>(stream);
    char* w = reinterpret_cast<char*>(ws);
    *n_out = 0;
    if (n == 0) return TRE_OK;
    hipError_t e = launch_stack(keys, n, tiles, row_elems, group, elem_bytes, nullptr, nullptr, 0, w, s, 0);
    if (e != hipSuccess) return dev_fail(e, "stack count");
    int64_t cnt = 0;
    const size_t cnt_off = (sizeof(int32_t) * size_t(n + 1) + 255) / 256 * 256;
    if ((e = hipMemcpyAsync(&cnt, w + cnt_off, sizeof(cnt), hipMemcpyDeviceToHost, s)) != hipSuccess)
        return dev_fail(e, "stack read-back");
    if ((e = hipStreamSynchronize(s)) != hipSuccess) return dev_fail(e, "stack sync");
    *n_out = cnt;
    if (cnt > out_cap || !out_keys || !out_tiles) {
        set_error("tre_stack_rows: output capacity below the number of stacked keys");
        return TRE_E_CAPACITY;
    }
    e = launch_stack(keys, n, tiles, row_elems, group, elem_bytes, out_keys, out_tiles, cnt, w, s, 1);
    return e == hipSuccess ? TRE_OK : dev_fail(e, "stack");
}

tre_status tre_tiles_from_entries(const int64_t* slot, const int64_t* offset, const void* value, int64_t n_entries,
                                  int32_t elem_bytes, void* tiles, int64_t n_tiles, int64_t tile_elems,
                                  void* stream) {
    if (n_entries < 0 || n_tiles < 0 || tile_elems < 1 || (elem_bytes != 2 && elem_bytes != 4) ||
        (n_entries > 0 && (!slot || !offset || !value)) || (n_tiles > 0 && !tiles)) {
        set_error("tre_tiles_from_entries: bad argument");
        return TRE_E_ARG;
    }
    hipError_t e = launch_tiles_from_entries(slot, offset, value, n_entries, elem_bytes, tiles, n_tiles, tile_elems,
                                             reinterpret_cast<hipStream_t>(stream));
    return e == hipSuccess ? TRE_OK : dev_fail(e, "tiles_from_entries");
}

}  // extern "C"
