// Host planner: parse one binary EinSum with its promoted labels and tile
// sizes, assign every label its relational and tile role, and size the
// workspace.  No device work happens here.
//
// Roles follow Sec. 5 of the paper (Eq. "eqn_tr" / "eqn-TRA"):
//   promoted labels shared by U and V    -> join attributes,
//   promoted labels of W                 -> GROUP BY attributes,
//   promoted labels not in W             -> summed by the GROUP BY (upper-agg),
// and the tile part of every label (the whole demoted label, or l' of a
// promoted label with tile size t) takes a role of the per-pair kernel K:
//   in U, V and W -> batch, in U and W -> M, in V and W -> N,
//   in U and V    -> K (contracted inside the tile),
//   in one input only and not in W -> pre-sum (folded into K with a zero
//   stride in the other operand).
#include <algorithm>
#include <cstring>
#include <new>
#include <vector>

#include "tre_internal.h"

namespace tre {

static thread_local std::string g_last_error;
void set_error(const std::string& msg) { g_last_error = msg; }

static int bits_for(int64_t radix) {
    int b = 0;
    while ((int64_t(1) << b) < radix) b++;
    return b;
}

static int find(const int* arr, int n, int x) {
    for (int i = 0; i < n; i++)
        if (arr[i] == x) return i;
    return -1;
}

static tre_status parse(Plan& p, const char* einsum, const char* upper, const int64_t* extent, const int32_t* tile) {
    int op = 0;
    bool arrow = false;
    for (const char* s = einsum; *s; ++s) {
        char c = *s;
        if (c == ' ') continue;
        if (c == ',') {
            if (op != 0) { set_error("more than two inputs"); return TRE_E_PARSE; }
            op = 1;
            continue;
        }
        if (c == '-') {
            if (s[1] != '>' || op != 1 || arrow) { set_error("expected one '->' after two inputs"); return TRE_E_PARSE; }
            arrow = true;
            op = 2;
            ++s;
            continue;
        }
        if (c < 'a' || c > 'z') { set_error(std::string("bad character '") + c + "'"); return TRE_E_PARSE; }
        int l = c - 'a';
        if (find(p.lab[op], p.nl[op], l) >= 0) { set_error("label repeated within an operand"); return TRE_E_PARSE; }
        p.lab[op][p.nl[op]++] = l;
        p.used[l] = true;
    }
    if (!arrow) { set_error("missing '->'"); return TRE_E_PARSE; }
    for (int i = 0; i < p.nl[2]; i++) {
        int l = p.lab[2][i];
        if (find(p.lab[0], p.nl[0], l) < 0 && find(p.lab[1], p.nl[1], l) < 0) {
            set_error("output label not in any input");
            return TRE_E_PARSE;
        }
    }
    for (const char* s = upper ? upper : ""; *s; ++s) {
        if (*s < 'a' || *s > 'z' || !p.used[*s - 'a']) {
            set_error("promoted label not used by the EinSum");
            return TRE_E_SPLIT;
        }
        p.up[*s - 'a'] = true;
    }
    for (int l = 0; l < 26; l++) {
        if (!p.used[l]) continue;
        if (extent[l] < 1 || extent[l] > INT32_MAX) { set_error("extent out of range"); return TRE_E_SHAPE; }
        p.ext[l] = extent[l];
        if (p.up[l]) {
            int64_t t = tile ? tile[l] : 1;
            if (t < 1 || t > extent[l] || extent[l] % t) { set_error("tile size must divide the extent"); return TRE_E_SHAPE; }
            p.tsz[l] = t;
        } else {
            p.tsz[l] = extent[l];
        }
    }
    for (int o = 0; o < 3; o++) {
        p.tile_elems[o] = 1;
        for (int i = 0; i < p.nl[o]; i++) {
            int l = p.lab[o][i];
            p.tile_elems[o] *= p.tsz[l];
            if (p.up[l]) {
                p.radix[o][p.nk[o]] = int32_t(p.ext[l] / p.tsz[l]);
                p.klab[o][p.nk[o]++] = l;
            }
        }
        if (p.tile_elems[o] > (int64_t(1) << 30)) { set_error("tile larger than 2^30 elements"); return TRE_E_SHAPE; }
    }
    return TRE_OK;
}

static int64_t stride_in(const Plan& p, int op, int l) {
    int64_t s = 1;
    for (int i = p.nl[op] - 1; i >= 0; i--) {
        if (p.lab[op][i] == l) return s;
        s *= p.tsz[p.lab[op][i]];
    }
    return -1;  // not present
}

static void push(Dims& d, int64_t size, int64_t stride) {
    d.size[d.n] = int32_t(size);
    d.stride[d.n] = int32_t(stride);
    d.n++;
}

static std::vector<int32_t> host_table(const Dims& d) {
    std::vector<int32_t> t(size_t(d.count()));
    for (int64_t x = 0; x < d.count(); x++) {
        int64_t rem = x, off = 0;
        for (int i = d.n - 1; i >= 0; i--) {
            off += (rem % d.size[i]) * d.stride[i];
            rem /= d.size[i];
        }
        t[size_t(x)] = int32_t(off);
    }
    return t;
}

// True when the table is made of aligned runs of 8 consecutive offsets.
static bool runs_of_8(const std::vector<int32_t>& t) {
    if (t.size() % 8) return false;
    for (size_t g = 0; g < t.size(); g += 8) {
        if (t[g] % 8) return false;
        for (int j = 1; j < 8; j++)
            if (t[g + j] != t[g] + j) return false;
    }
    return true;
}

static bool all_mult_8(const std::vector<int32_t>& t) {
    for (int32_t x : t)
        if (x % 8) return false;
    return true;
}

static tre_status classify(Plan& p) {
    // ---- join key (join labels in V's key order) ----
    p.n_join = 0;
    for (int b = 0; b < p.nk[1]; b++) {
        int l = p.klab[1][b];
        int a = find(p.klab[0], p.nk[0], l);
        if (a < 0) continue;
        p.join_pos_u[p.n_join] = a;
        p.join_pos_v[p.n_join] = b;
        p.join_bits[p.n_join] = bits_for(p.radix[1][b]);
        p.join_total_bits += p.join_bits[p.n_join];
        p.n_join++;
    }
    p.v_needs_sort = false;
    for (int i = 0; i < p.n_join; i++)
        if (p.join_pos_v[i] != i) p.v_needs_sort = true;
    if (p.join_total_bits > 64) { set_error("join key wider than 64 bits"); return TRE_E_SHAPE; }
    // ---- W key ----
    bool prefix_of_u = true;
    for (int c = 0; c < p.nk[2]; c++) {
        int l = p.klab[2][c];
        int a = find(p.klab[0], p.nk[0], l);
        if (a >= 0) {
            p.w_src[c] = 0;
            p.w_pos[c] = a;
            p.w_bits[c] = bits_for(p.radix[0][a]);
        } else {
            int b = find(p.klab[1], p.nk[1], l);
            if (b < 0) { set_error("promoted W label missing from both inputs"); return TRE_E_SPLIT; }
            p.w_src[c] = 1;
            p.w_pos[c] = b;
            p.w_bits[c] = bits_for(p.radix[1][b]);
        }
        if (!(p.w_src[c] == 0 && p.w_pos[c] == c)) prefix_of_u = false;
        p.w_total_bits += p.w_bits[c];
    }
    if (p.w_total_bits > 64) { set_error("W key wider than 64 bits"); return TRE_E_SHAPE; }
    // pairs come out of the join in (u, v) order: already grouped when W's
    // promoted labels are a prefix of U's key
    p.group_needs_sort = !(p.nk[2] == 0 || prefix_of_u);
    // Otherwise the join can be driven by V instead when V's key is W's key
    // followed by the join labels and U's key starts with the same join
    // labels in the same order.  V's tuples of one W key then carry distinct
    // join keys in increasing order, each meets one run of U tuples (U is
    // sorted by its join attributes first), and those runs increase with the
    // join key, so walking V and expanding each tuple's U run gives the pairs
    // in the canonical (W key, u, v) order directly.
    if (p.group_needs_sort && p.nk[1] == p.nk[2] + p.n_join) {
        bool ok = true;
        for (int c = 0; c < p.nk[2] && ok; c++) ok = p.w_src[c] == 1 && p.w_pos[c] == c;
        for (int i = 0; i < p.n_join && ok; i++) ok = p.join_pos_v[i] == p.nk[2] + i && p.join_pos_u[i] == i;
        if (ok) {
            p.v_outer = true;
            p.group_needs_sort = false;
            p.v_needs_sort = false;
        }
    }

    // ---- tile roles ----
    std::vector<int> bl, ml, nl, kl, pul, pvl;
    for (int i = 0; i < p.nl[2]; i++) {
        int l = p.lab[2][i];
        bool inU = find(p.lab[0], p.nl[0], l) >= 0, inV = find(p.lab[1], p.nl[1], l) >= 0;
        if (inU && inV) { p.role[l] = 'b'; bl.push_back(l); }
        else if (inU) { p.role[l] = 'm'; ml.push_back(l); }
        else { p.role[l] = 'n'; nl.push_back(l); }
    }
    for (int i = 0; i < p.nl[0]; i++) {
        int l = p.lab[0][i];
        if (find(p.lab[2], p.nl[2], l) >= 0) continue;
        if (find(p.lab[1], p.nl[1], l) >= 0) { p.role[l] = 'k'; kl.push_back(l); }
        else { p.role[l] = 'p'; pul.push_back(l); }
    }
    for (int i = 0; i < p.nl[1]; i++) {
        int l = p.lab[1][i];
        if (find(p.lab[2], p.nl[2], l) >= 0 || find(p.lab[0], p.nl[0], l) >= 0) continue;
        p.role[l] = 'p';
        pvl.push_back(l);
    }
    if (bl.size() > kMaxDims || ml.size() > kMaxDims || nl.size() > kMaxDims ||
        kl.size() + pul.size() + pvl.size() > kMaxDims) {
        set_error("too many labels in one role");
        return TRE_E_SHAPE;
    }
    auto prod = [&](const std::vector<int>& v) {
        int64_t x = 1;
        for (int l : v) x *= p.tsz[l];
        return x;
    };
    p.nB = prod(bl);
    p.nM = prod(ml);
    p.nN = prod(nl);
    p.nK = prod(kl) * prod(pul) * prod(pvl);
    if (p.nK > (int64_t(1) << 30)) { set_error("contracted extent too large"); return TRE_E_SHAPE; }

    p.kclass = (p.nM >= 16 && p.nN >= 16 && p.nK >= 8) ? KC_GEMM : KC_VEC;
    // GEMM output stores are coalesced along the kernel's N; when W's unit
    // stride label belongs to M, swap the operands so it becomes N.
    p.swap = false;
    if (p.kclass == KC_GEMM) {
        for (int i = p.nl[2] - 1; i >= 0; i--) {
            int l = p.lab[2][i];
            if (p.tsz[l] == 1) continue;
            p.swap = p.role[l] == 'm';
            break;
        }
    }
    const int A = p.swap ? 1 : 0, B = p.swap ? 0 : 1;
    const std::vector<int>& Ml = p.swap ? nl : ml;
    const std::vector<int>& Nl = p.swap ? ml : nl;
    for (auto& d : p.dims) d = Dims{};
    for (int l : bl) {
        push(p.dims[T_AB], p.tsz[l], stride_in(p, A, l));
        push(p.dims[T_BB], p.tsz[l], stride_in(p, B, l));
        push(p.dims[T_WB], p.tsz[l], stride_in(p, 2, l));
    }
    for (int l : Ml) {
        push(p.dims[T_AM], p.tsz[l], stride_in(p, A, l));
        push(p.dims[T_WM], p.tsz[l], stride_in(p, 2, l));
    }
    for (int l : Nl) {
        push(p.dims[T_BN], p.tsz[l], stride_in(p, B, l));
        push(p.dims[T_WN], p.tsz[l], stride_in(p, 2, l));
    }
    for (int l : kl) {
        push(p.dims[T_AK], p.tsz[l], stride_in(p, A, l));
        push(p.dims[T_BK], p.tsz[l], stride_in(p, B, l));
        push(p.dims[T_KU], p.tsz[l], stride_in(p, 0, l));
        push(p.dims[T_KV], p.tsz[l], stride_in(p, 1, l));
    }
    for (int l : pul) {
        push(p.dims[T_AK], p.tsz[l], A == 0 ? stride_in(p, 0, l) : 0);
        push(p.dims[T_BK], p.tsz[l], B == 0 ? stride_in(p, 0, l) : 0);
        push(p.dims[T_KU], p.tsz[l], stride_in(p, 0, l));
        push(p.dims[T_KV], p.tsz[l], 0);
    }
    for (int l : pvl) {
        push(p.dims[T_AK], p.tsz[l], A == 1 ? stride_in(p, 1, l) : 0);
        push(p.dims[T_BK], p.tsz[l], B == 1 ? stride_in(p, 1, l) : 0);
        push(p.dims[T_KU], p.tsz[l], 0);
        push(p.dims[T_KV], p.tsz[l], stride_in(p, 1, l));
    }
    // W element (memory order) -> U / V offsets of its batch, M and N parts
    for (int i = 0; i < p.nl[2]; i++) {
        int l = p.lab[2][i];
        int64_t su = stride_in(p, 0, l), sv = stride_in(p, 1, l);
        push(p.dims[T_EU], p.tsz[l], su < 0 ? 0 : su);
        push(p.dims[T_EV], p.tsz[l], sv < 0 ? 0 : sv);
    }
    int64_t off = 0;
    for (int t = 0; t < T_COUNT; t++) {
        p.table_off[t] = off;
        off += (p.dims[t].count() + 63) / 64 * 64;
    }
    p.table_total = off;

    // Vector class: EPT consecutive W elements per thread when U's offsets run
    // contiguously in aligned groups of EPT and V's either do too or stay
    // constant over each group (V broadcast), or the same with U and V
    // exchanged (U broadcast: the kernel then reads V as its vector operand);
    // otherwise one element.
    if (p.kclass == KC_VEC) {
        auto tEU = host_table(p.dims[T_EU]), tEV = host_table(p.dims[T_EV]);
        auto tKU = host_table(p.dims[T_KU]), tKV = host_table(p.dims[T_KV]);
        const int ept = p.dtype == TRE_BF16 ? 8 : 4;
        auto grouped = [&](const std::vector<int32_t>& t, bool& contiguous, bool& constant) {
            contiguous = constant = t.size() % ept == 0;
            for (size_t g = 0; g < t.size() && (contiguous || constant); g += ept) {
                if (t[g] % ept) contiguous = false;
                for (int j = 1; j < ept; j++) {
                    if (t[g + j] != t[g] + j) contiguous = false;
                    if (t[g + j] != t[g]) constant = false;
                }
            }
        };
        auto aligned = [&](const std::vector<int32_t>& t) {
            for (int32_t x : t)
                if (x % ept) return false;
            return true;
        };
        bool u_cont, u_const, v_cont, v_const;
        grouped(tEU, u_cont, u_const);
        grouped(tEV, v_cont, v_const);
        const bool u_ok = u_cont && p.tile_elems[0] % ept == 0 && aligned(tKU);
        const bool v_vec = v_cont && p.tile_elems[1] % ept == 0 && aligned(tKV);
        if (u_ok && p.tile_elems[2] % ept == 0 && (v_vec || v_const)) {
            p.vec_ept = ept;
            p.vec_vbcast = !v_vec;
        } else if (v_vec && u_const && p.tile_elems[2] % ept == 0) {
            p.vec_ept = ept;
            p.vec_vbcast = true;
            p.vec_swap = true;
        }
    }
    // GEMM staging: which dim of A / B has unit stride, and whether 8-wide
    // aligned vector loads along it are legal
    if (p.kclass == KC_GEMM) {
        auto tAM = host_table(p.dims[T_AM]), tAK = host_table(p.dims[T_AK]), tBK = host_table(p.dims[T_BK]),
             tBN = host_table(p.dims[T_BN]), tAB = host_table(p.dims[T_AB]), tBB = host_table(p.dims[T_BB]);
        auto has_unit = [](const std::vector<int32_t>& t) { return t.size() > 1 && t[1] - t[0] == 1; };
        p.a_kfast = has_unit(tAK) || !has_unit(tAM);
        p.b_kfast = has_unit(tBK) || !has_unit(tBN);
        bool te_a = p.tile_elems[A] % 8 == 0, te_b = p.tile_elems[B] % 8 == 0;
        p.vec_a = te_a && all_mult_8(tAB) &&
                  (p.a_kfast ? (runs_of_8(tAK) && all_mult_8(tAM)) : (runs_of_8(tAM) && all_mult_8(tAK)));
        p.vec_b = te_b && all_mult_8(tBB) &&
                  (p.b_kfast ? (runs_of_8(tBK) && all_mult_8(tBN)) : (runs_of_8(tBN) && all_mult_8(tBK)));
        // Fast path: bf16 (K a multiple of 64) or fp32 (K a multiple of 32),
        // no batch, 128-multiple M/N, every operand a plain 2-D row-major
        // matrix (one unit stride, one leading dimension) and W stored with N
        // fastest.
        auto affine = [](const std::vector<int32_t>& t, int64_t& s) {
            s = t.size() > 1 ? t[1] - t[0] : 0;
            for (size_t i = 0; i < t.size(); i++)
                if (t[i] != int64_t(i) * s) return false;
            return true;
        };
        auto tWM = host_table(p.dims[T_WM]), tWN = host_table(p.dims[T_WN]);
        const int64_t M = p.swap ? p.nN : p.nM, N = p.swap ? p.nM : p.nN;
        int64_t sAM, sAK, sBN, sBK, sWM, sWN;
        const int64_t kq = p.dtype == TRE_BF16 ? 64 : 32;
        bool ok = p.nB == 1 && M % 128 == 0 && N % 128 == 0 && p.nK % kq == 0 &&
                  affine(tAM, sAM) && affine(tAK, sAK) && affine(tBN, sBN) && affine(tBK, sBK) &&
                  affine(tWM, sWM) && affine(tWN, sWN) && sWN == 1 && sWM >= N;
        if (ok) {
            if (sAK == 1 && sAM >= p.nK) { p.fast_a_rowfast = false; p.fast_lda = sAM; }
            else if (sAM == 1 && sAK >= M) { p.fast_a_rowfast = true; p.fast_lda = sAK; }
            else ok = false;
            if (sBK == 1 && sBN >= p.nK) { p.fast_b_rowfast = false; p.fast_ldb = sBN; }
            else if (sBN == 1 && sBK >= N) { p.fast_b_rowfast = true; p.fast_ldb = sBK; }
            else ok = false;
            p.fast_ldw = sWM;
            // 16-byte copies: rows must start on 16-byte boundaries
            ok = ok && p.fast_lda % 8 == 0 && p.fast_ldb % 8 == 0;
        }
        p.fast = ok;
    }
    return TRE_OK;
}

static size_t align256(size_t x) { return (x + 255) / 256 * 256; }

// Whether the 128x128 path may cut keys into U ranges (each (key, range)
// leaving a partial tile): asked for explicitly, or where the paced
// persistent grid cannot run instead -- several 128x128 blocks per W tile,
// pacing switched off, or a unit length cap.  Where pacing can run, the
// automatic choice takes it, and a U-range fallback (output keys beyond
// what the pacing counters cover) sizes its ranges to the partial tiles the
// workspace holds.
bool u_ranges_possible(const Plan& p) {
    if (!(p.kclass == KC_GEMM && p.fast) || p.opt.u_ranges < 0) return false;
    const int64_t M = p.swap ? p.nN : p.nM, N = p.swap ? p.nM : p.nN;
    return p.opt.u_ranges > 0 || (M / 128) * (N / 128) != 1 || p.opt.pace_windows < 0 ||
           p.opt.max_pairs_per_unit > 0;
}

Layout make_layout(const Plan& p, int64_t n_u, int64_t n_v, int64_t max_pairs) {
    Layout L;
    L.n_u = n_u;
    L.n_v = n_v;
    L.max_pairs = max_pairs;
    const int64_t P = std::max<int64_t>(max_pairs, 1);
    const int64_t wtile_bytes = p.tile_elems[2] * 4;
    // partial tiles: only keys split across several units need them
    int64_t cap = std::max<int64_t>(16, (int64_t(1) << 30) / wtile_bytes);
    cap = std::min<int64_t>(cap, 4096);
    cap = std::min<int64_t>(cap, P + 1);
    if (u_ranges_possible(p)) {
        // U-range mode: up to kMaxURanges partial tiles per output key, at
        // most 4 GiB of them
        int64_t wspace = 1;
        for (int c = 0; c < p.nk[2] && wspace < (int64_t(1) << 40); c++) wspace *= p.radix[2][c];
        const int64_t n_w_max = std::min<int64_t>(P, wspace);
        const int64_t range_cap = std::min<int64_t>(kMaxURanges * n_w_max, (int64_t(4) << 30) / wtile_bytes);
        cap = std::max<int64_t>(cap, range_cap);
    }
    L.part_cap = cap;
    const int64_t units_max = std::max<int64_t>(2 * P + 2, cap);
    size_t off = 0;
    auto take = [&](size_t bytes) {
        size_t o = off;
        off += align256(bytes);
        return o;
    };
    int64_t sort_n = std::max<int64_t>(p.v_needs_sort ? n_v : 0, p.group_needs_sort ? P : 0);
    L.hdr = take(sizeof(WsHeader));
    L.vjk = take(sizeof(uint64_t) * size_t(std::max<int64_t>(n_v, 1)));
    L.vjk_alt = take(p.v_needs_sort ? sizeof(uint64_t) * size_t(n_v) : 0);
    L.vperm = take(p.v_needs_sort ? sizeof(uint32_t) * size_t(n_v) : 0);
    L.vperm_alt = take(p.v_needs_sort ? sizeof(uint32_t) * size_t(n_v) : 0);
    const int64_t n_outer = p.v_outer ? n_v : n_u;  // the relation whose tuples find their runs
    L.ucnt = take(sizeof(int64_t) * size_t(n_outer + 1));
    L.ulo = take(sizeof(int64_t) * size_t(std::max<int64_t>(n_outer, 1)));
    int64_t scan_n = std::max<int64_t>({n_outer + 1, P + 1, radix_hist_elems(std::max<int64_t>(sort_n, 1))});
    L.scan_tmp = take(sizeof(int64_t) * scan_tmp_elems(scan_n));
    L.pu = take(sizeof(int32_t) * size_t(P));
    L.pv = take(sizeof(int32_t) * size_t(P));
    L.pu_alt = take(0);
    L.pv_alt = take(0);
    L.wk = take(sizeof(uint64_t) * size_t(P));
    L.wk_alt = take(p.group_needs_sort ? sizeof(uint64_t) * size_t(P) : 0);
    L.pidx = take(p.group_needs_sort ? sizeof(uint64_t) * size_t(P) : 0);      // packed (u, v) per pair
    L.pidx_alt = take(p.group_needs_sort ? sizeof(uint64_t) * size_t(P) : 0);
    L.hist = take(sizeof(int32_t) * size_t(radix_hist_elems(std::max<int64_t>(sort_n, 1))));
    L.flags = take(sizeof(int32_t) * size_t(P + 1));
    L.seg_start = take(sizeof(int32_t) * size_t(P + 1));
    L.seg_key = take(sizeof(uint64_t) * size_t(P));
    L.unit_desc = take(sizeof(Unit) * size_t(units_max));
    L.seg_units = take(sizeof(int32_t) * size_t(P + 1));
    L.part_off = take(sizeof(int32_t) * size_t(P + 1));
    L.split_list = take(sizeof(int32_t) * size_t(P + 1));
    L.tables = take(sizeof(int32_t) * size_t(p.table_total));
    L.pace = take((p.kclass == KC_GEMM && p.fast) ? sizeof(int32_t) * size_t(kPaceCounters) : 0);
    L.partials = take(sizeof(float) * size_t(cap) * size_t(p.tile_elems[2]));
    L.total = off;
    return L;
}

}  // namespace tre

using namespace tre;

extern "C" {

tre_status tre_plan(const char* einsum, const char* upper, const int64_t* extent, const int32_t* tile,
                    int32_t in_dtype, const tre_options* opt, tre_plan_t* out) {
    if (!einsum || !extent || !out) {
        set_error("null argument");
        return TRE_E_ARG;
    }
    *out = nullptr;
    if (in_dtype != TRE_F32 && in_dtype != TRE_BF16) {
        set_error("in_dtype must be TRE_F32 or TRE_BF16");
        return TRE_E_DTYPE;
    }
    auto* h = new (std::nothrow) tre_plan_s();
    if (!h) return TRE_E_ARG;
    Plan& p = h->p;
    p.einsum = einsum;
    p.dtype = in_dtype == TRE_BF16 ? TRE_BF16 : TRE_F32;
    p.opt.validate_keys = 1;
    if (opt) {
        p.opt = *opt;
        if (p.opt.max_pairs_per_unit < 0) {
            delete h;
            set_error("max_pairs_per_unit must be >= 0");
            return TRE_E_ARG;
        }
    }
    tre_status st = parse(p, einsum, upper, extent, tile);
    if (st == TRE_OK) st = classify(p);
    if (st == TRE_OK && p.opt.w_bf16 && p.kclass == KC_GEMM && !p.fast) {
        set_error("w_bf16: bf16 output is written by the vector class and the 128x128 path only");
        st = TRE_E_DTYPE;
    }
    if (st != TRE_OK) {
        delete h;
        return st;
    }
    *out = h;
    return TRE_OK;
}

tre_status tre_plan_get_info(tre_plan_t plan, tre_plan_info* info) {
    if (!plan || !info) return TRE_E_ARG;
    const Plan& p = plan->p;
    std::memset(info, 0, sizeof(*info));
    for (int o = 0; o < 3; o++) {
        info->key_arity[o] = p.nk[o];
        info->tile_elems[o] = p.tile_elems[o];
        for (int a = 0; a < p.nk[o]; a++) info->key_labels[o][a] = char('a' + p.klab[o][a]);
    }
    info->n_join = p.n_join;
    info->kernel_class = (p.kclass == KC_GEMM && p.fast) ? 2 : p.kclass;
    info->batch = p.nB;
    info->m = p.nM;
    info->n = p.nN;
    info->k = p.nK;
    info->flops_per_pair = 2 * p.nB * p.nM * p.nN * p.nK;
    for (int l = 0; l < 26; l++) info->roles[l] = p.used[l] ? p.role[l] : '.';
    info->group_needs_sort = p.group_needs_sort;
    info->v_needs_sort = p.v_needs_sort;
    info->w_dtype = p.opt.w_bf16 ? TRE_BF16 : TRE_F32;
    info->join_outer = p.v_outer ? 1 : 0;
    return TRE_OK;
}

void tre_plan_destroy(tre_plan_t plan) { delete plan; }

size_t tre_workspace_bytes(tre_plan_t plan, int64_t n_u, int64_t n_v, int64_t max_pairs) {
    if (!plan || n_u < 0 || n_v < 0 || max_pairs < 0) return 0;
    return make_layout(plan->p, n_u, n_v, max_pairs).total;
}

int64_t tre_workspace_max_pairs(tre_plan_t plan, int64_t n_u, int64_t n_v, size_t ws_bytes) {
    if (!plan || n_u < 0 || n_v < 0) return -1;
    int64_t lo = 0, hi = int64_t(INT32_MAX) - 1;
    if (make_layout(plan->p, n_u, n_v, 0).total > ws_bytes) return -1;
    while (lo < hi) {
        int64_t mid = lo + (hi - lo + 1) / 2;
        if (make_layout(plan->p, n_u, n_v, mid).total <= ws_bytes) lo = mid;
        else hi = mid - 1;
    }
    return lo;
}

const char* tre_status_str(tre_status s) {
    switch (s) {
        case TRE_OK: return "TRE_OK";
        case TRE_E_ARG: return "TRE_E_ARG";
        case TRE_E_PARSE: return "TRE_E_PARSE";
        case TRE_E_SPLIT: return "TRE_E_SPLIT";
        case TRE_E_SHAPE: return "TRE_E_SHAPE";
        case TRE_E_DTYPE: return "TRE_E_DTYPE";
        case TRE_E_UNSORTED: return "TRE_E_UNSORTED";
        case TRE_E_DUPKEY: return "TRE_E_DUPKEY";
        case TRE_E_KEYRANGE: return "TRE_E_KEYRANGE";
        case TRE_E_CAPACITY: return "TRE_E_CAPACITY";
        case TRE_E_WORKSPACE: return "TRE_E_WORKSPACE";
        case TRE_E_DEVICE: return "TRE_E_DEVICE";
        case TRE_E_STATE: return "TRE_E_STATE";
    }
    return "TRE_E_UNKNOWN";
}

const char* tre_last_error(void) { return g_last_error.c_str(); }

const char* tre_version(void) { return "tre 0.1 gfx950"; }

}  // extern "C"
