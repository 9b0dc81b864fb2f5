/*
 * tre_oracle.c -- plain CPU oracle for one binary upper-case-lower-case EinSum.
 *
 * TEST INFRASTRUCTURE, NOT PART OF THE PRODUCT.  Only the tests, the smoke
 * check and the CPU-baseline leg of the benchmark load this file's library.
 * It shares no code, header, table or constant with the HIP library.
 *
 * What it computes (Tang et al., "Automated Tensor-Relational Decomposition
 * for Large-Scale Sparse Tensor Computation", PVLDB 19(6), 2026):
 *
 *   A binary EinSum  W[lW] = sum over the labels not in W of  U[lU] * V[lV]
 *   (the general binary form, Sec. 3, Eq. "Einsum", with (+, *) as the pair of
 *   aggregation and join operators).  Each operand is held as a tensor
 *   relation (Sec. 4.2): the promoted (upper-case) labels index tuples, the
 *   demoted (lower-case) labels index a dense tile stored in each tuple.
 *   A promoted label l may carry a tile size t_l: the global index is
 *   g = t_l * L + l', L is the tuple attribute and l' indexes the tile.
 *   t_l = 1 is the paper's plain promoted label; a demoted label keeps its
 *   whole extent inside the tile.
 *
 *   The tensor-relational evaluation (Sec. 5, Eq. "eqn-TRA" and the SQL form
 *   SELECT upper(W), SUM(K(valU, valV)) FROM U NATURAL JOIN V GROUP BY upper(W))
 *   equals the dense EinSum for every decomposition (Sec. 4.2, the
 *   equivalence class of decompositions).  So this oracle computes the plain
 *   definition, on scalars:
 *
 *   1. orc_expand: every relation is expanded to scalar COO with global
 *      coordinates (the point lookup of Sec. 4.2: coordinate = key * t + offset).
 *   2. orc_join: key-level join on the shared promoted labels and GROUP BY on
 *      W's promoted labels (Sec. 5), giving the matched pair list in the
 *      canonical order (w_key, u, v) and the sorted output key set.
 *   3. orc_eval: for every U entry and every V entry that agree on all the
 *      labels the two operands share, add the product into the W coordinate
 *      built from the two entries, in fp64, together with the sum of the
 *      absolute values of the products (the magnitude used for the
 *      componentwise error bound).
 *
 * Everything is single-threaded, fp64, and deliberately simple: sorting with
 * qsort_r and binary search are the only "algorithms" used.
 */
#define _GNU_SOURCE
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#define ORC_OK 0
#define ORC_E_ARG 1
#define ORC_E_PARSE 2
#define ORC_E_SPLIT 3
#define ORC_E_SHAPE 4
#define ORC_E_UNSORTED 5
#define ORC_E_DUPKEY 6
#define ORC_E_KEYRANGE 7
#define ORC_E_NOMEM 8

typedef struct {
    int nl[3];          /* number of labels of U (0), V (1), W (2) */
    int lab[3][26];     /* label ids (0..25) in operand string order */
    int up[26];         /* 1 when the label is promoted (upper case) */
    int used[26];
    int64_t ext[26];    /* extent of the label in the full tensor */
    int64_t t[26];      /* extent inside a tile */
    int nk[3];          /* key arity: number of promoted labels of the operand */
    int klab[3][26];    /* promoted labels in operand string order */
    int64_t tile_elems[3];
} orc_plan;

int64_t orc_plan_size(void) { return (int64_t)sizeof(orc_plan); }

static int has_label(const orc_plan *p, int op, int l) {
    for (int i = 0; i < p->nl[op]; i++)
        if (p->lab[op][i] == l) return 1;
    return 0;
}

/* Parse "ab,bc->ca" plus the promoted label set and the per-letter extents and
 * tile sizes.  Returns ORC_OK or an error category. */
int orc_plan_make(const char *einsum, const char *upper, const int64_t *ext,
                  const int32_t *tile, orc_plan *p) {
    if (!einsum || !ext || !p) return ORC_E_ARG;
    memset(p, 0, sizeof(*p));
    int op = 0, seen_arrow = 0;
    const char *s = einsum;
    while (*s) {
        char c = *s;
        if (c == ' ') { s++; continue; }
        if (c == ',') {
            if (op != 0 || seen_arrow) return ORC_E_PARSE;
            op = 1; s++; continue;
        }
        if (c == '-') {
            if (s[1] != '>' || op != 1 || seen_arrow) return ORC_E_PARSE;
            seen_arrow = 1; op = 2; s += 2; continue;
        }
        if (c < 'a' || c > 'z') return ORC_E_PARSE;
        int l = c - 'a';
        if (has_label(p, op, l)) return ORC_E_PARSE; /* repeated within an operand */
        p->lab[op][p->nl[op]++] = l;
        p->used[l] = 1;
        s++;
    }
    if (!seen_arrow) return ORC_E_PARSE;
    for (int i = 0; i < p->nl[2]; i++) {
        int l = p->lab[2][i];
        if (!has_label(p, 0, l) && !has_label(p, 1, l)) return ORC_E_PARSE;
    }
    if (upper) {
        for (const char *u = upper; *u; u++) {
            if (*u < 'a' || *u > 'z') return ORC_E_SPLIT;
            int l = *u - 'a';
            if (!p->used[l]) return ORC_E_SPLIT;
            p->up[l] = 1;
        }
    }
    for (int l = 0; l < 26; l++) {
        if (!p->used[l]) continue;
        if (ext[l] < 1) return ORC_E_SHAPE;
        p->ext[l] = ext[l];
        if (p->up[l]) {
            int64_t t = tile ? (int64_t)tile[l] : 1;
            if (t < 1 || t > ext[l] || ext[l] % t != 0) return ORC_E_SHAPE;
            p->t[l] = t;
        } else {
            p->t[l] = ext[l];
        }
    }
    for (int o = 0; o < 3; o++) {
        p->tile_elems[o] = 1;
        for (int i = 0; i < p->nl[o]; i++) {
            int l = p->lab[o][i];
            p->tile_elems[o] *= p->t[l];
            if (p->up[l]) p->klab[o][p->nk[o]++] = l;
        }
    }
    return ORC_OK;
}

void orc_plan_desc(const orc_plan *p, int32_t *nl, int32_t *nk, int64_t *tile_elems,
                   int32_t *labels, int32_t *klabels) {
    for (int o = 0; o < 3; o++) {
        nl[o] = p->nl[o];
        nk[o] = p->nk[o];
        tile_elems[o] = p->tile_elems[o];
        for (int i = 0; i < 26; i++) {
            labels[o * 26 + i] = i < p->nl[o] ? p->lab[o][i] : -1;
            klabels[o * 26 + i] = i < p->nk[o] ? p->klab[o][i] : -1;
        }
    }
}

/* A relation's keys must be strictly increasing in lexicographic order (one
 * tuple per key, Sec. 4.2) and every attribute in [0, extent / t). */
int orc_check_keys(const orc_plan *p, int op, const int32_t *keys, int64_t n) {
    int r = p->nk[op];
    if (r == 0) return n <= 1 ? ORC_OK : ORC_E_DUPKEY;
    for (int64_t i = 0; i < n; i++) {
        for (int a = 0; a < r; a++) {
            int l = p->klab[op][a];
            int32_t k = keys[i * r + a];
            if (k < 0 || (int64_t)k >= p->ext[l] / p->t[l]) return ORC_E_KEYRANGE;
        }
    }
    for (int64_t i = 1; i < n; i++) {
        int c = 0;
        for (int a = 0; a < r && c == 0; a++) {
            int32_t x = keys[(i - 1) * r + a], y = keys[i * r + a];
            c = (x < y) ? -1 : (x > y ? 1 : 0);
        }
        if (c == 0) return ORC_E_DUPKEY;
        if (c > 0) return ORC_E_UNSORTED;
    }
    return ORC_OK;
}

static double bf16_to_double(uint16_t b) {
    uint32_t bits = (uint32_t)b << 16;
    float f;
    memcpy(&f, &bits, 4);
    return (double)f;
}

/* fp32 -> bf16 with round-to-nearest-even on the 16 dropped bits; NaN stays
 * a quiet NaN.  (The standard bit-level formulation of IEEE RNE.) */
void orc_f32_to_bf16(const float *x, uint16_t *y, int64_t n) {
    for (int64_t i = 0; i < n; i++) {
        uint32_t bits;
        memcpy(&bits, &x[i], 4);
        if ((bits & 0x7f800000u) == 0x7f800000u && (bits & 0x007fffffu)) {
            y[i] = (uint16_t)((bits >> 16) | 0x0040u);
            continue;
        }
        uint32_t lsb = (bits >> 16) & 1u;
        bits += 0x7fffu + lsb;
        y[i] = (uint16_t)(bits >> 16);
    }
}

/* Step 1: expand a relation to scalar COO.  dtype: 0 = fp32, 1 = bf16,
 * 2 = fp64.  coords is [nnz x nl] in operand label order (global indices),
 * tuple[] records the source tuple.  With coords == NULL only counts.
 * Exact zeros (either sign) are not emitted: a zero contributes nothing to a
 * sum of products. */
int64_t orc_expand(const orc_plan *p, int op, const int32_t *keys, int64_t n,
                   const void *tiles, int dtype, int64_t *coords, double *vals,
                   int64_t *tuple, int64_t cap) {
    int nl = p->nl[op], r = p->nk[op];
    int64_t te = p->tile_elems[op];
    int64_t nnz = 0;
    int64_t off[26];
    for (int64_t tu = 0; tu < n; tu++) {
        for (int64_t e = 0; e < te; e++) {
            double v;
            if (dtype == 0) v = (double)((const float *)tiles)[tu * te + e];
            else if (dtype == 1) v = bf16_to_double(((const uint16_t *)tiles)[tu * te + e]);
            else v = ((const double *)tiles)[tu * te + e];
            if (v == 0.0) continue;
            if (coords) {
                if (nnz >= cap) return -1;
                /* row-major decomposition of e over the operand's tile labels */
                int64_t rem = e;
                for (int i = nl - 1; i >= 0; i--) {
                    int64_t sz = p->t[p->lab[op][i]];
                    off[i] = rem % sz;
                    rem /= sz;
                }
                int ka = 0;
                for (int i = 0; i < nl; i++) {
                    int l = p->lab[op][i];
                    int64_t g = off[i];
                    if (p->up[l]) {
                        g += (int64_t)keys[tu * r + ka] * p->t[l];
                        ka++;
                    }
                    coords[nnz * nl + i] = g;
                }
                vals[nnz] = v;
                if (tuple) tuple[nnz] = tu;
            }
            nnz++;
        }
    }
    return nnz;
}

/* ---------------------------------------------------------------- sorting */

typedef struct {
    const int32_t *rows;   /* int32 rows of length w */
    int w;
} row_ctx;

static int cmp_rows(const void *a, const void *b, void *c) {
    const row_ctx *x = (const row_ctx *)c;
    int64_t i = *(const int64_t *)a, j = *(const int64_t *)b;
    const int32_t *ri = x->rows + i * x->w, *rj = x->rows + j * x->w;
    for (int k = 0; k < x->w; k++) {
        if (ri[k] != rj[k]) return ri[k] < rj[k] ? -1 : 1;
    }
    return (i < j) ? -1 : (i > j ? 1 : 0);
}

/* Key set of a relation given as scalar COO: the distinct promoted-label
 * projections (coordinate / t) of its entries, sorted lexicographically. */
int orc_keys_from_coo(const orc_plan *p, int op, const int64_t *coords, int64_t nnz,
                      int64_t *n_out, int32_t **keys_out) {
    int nl = p->nl[op], r = p->nk[op];
    *n_out = 0;
    *keys_out = NULL;
    if (nnz == 0) return ORC_OK;
    if (r == 0) {
        *n_out = 1;
        *keys_out = (int32_t *)malloc(4);
        return *keys_out ? ORC_OK : ORC_E_NOMEM;
    }
    int32_t *rows = (int32_t *)malloc(sizeof(int32_t) * (size_t)(nnz * r));
    int64_t *idx = (int64_t *)malloc(sizeof(int64_t) * (size_t)nnz);
    if (!rows || !idx) { free(rows); free(idx); return ORC_E_NOMEM; }
    for (int64_t e = 0; e < nnz; e++) {
        int ka = 0;
        for (int i = 0; i < nl; i++) {
            int l = p->lab[op][i];
            if (p->up[l]) rows[e * r + ka++] = (int32_t)(coords[e * nl + i] / p->t[l]);
        }
        idx[e] = e;
    }
    row_ctx c = {rows, r};
    qsort_r(idx, (size_t)nnz, sizeof(int64_t), cmp_rows, &c);
    int32_t *out = (int32_t *)malloc(sizeof(int32_t) * (size_t)(nnz * r));
    if (!out) { free(rows); free(idx); return ORC_E_NOMEM; }
    int64_t m = 0;
    for (int64_t e = 0; e < nnz; e++) {
        const int32_t *row = rows + idx[e] * r;
        if (m > 0 && memcmp(out + (m - 1) * r, row, sizeof(int32_t) * (size_t)r) == 0) continue;
        memcpy(out + m * r, row, sizeof(int32_t) * (size_t)r);
        m++;
    }
    free(rows);
    free(idx);
    *n_out = m;
    *keys_out = out;
    return ORC_OK;
}

/* ---------------------------------------------------------- step 2: join */

/* Key-level natural join on the promoted labels the operands share, followed
 * by GROUP BY on W's promoted labels.  Output:
 *   pairs  [npairs x 2] (u, v) in order of (w_key, u, v),
 *   wkeys  [nw x nk(W)] sorted, distinct.
 * Memory is malloc'ed; release with orc_free. */
int orc_join(const orc_plan *p, const int32_t *ukeys, int64_t nu, const int32_t *vkeys,
             int64_t nv, int64_t *npairs_out, int32_t **pairs_out, int64_t *nw_out,
             int32_t **wkeys_out) {
    int ru = p->nk[0], rv = p->nk[1], rw = p->nk[2];
    *npairs_out = 0; *nw_out = 0; *pairs_out = NULL; *wkeys_out = NULL;
    if (nu == 0 || nv == 0) return ORC_OK;
    /* join labels: promoted in both (a label has one case in the EinSum) */
    int ju[26], jv[26], nj = 0;
    for (int a = 0; a < ru; a++)
        for (int b = 0; b < rv; b++)
            if (p->klab[0][a] == p->klab[1][b]) { ju[nj] = a; jv[nj] = b; nj++; }
    /* where each W key attribute comes from */
    int wsrc[26], wpos[26];
    for (int c = 0; c < rw; c++) {
        int l = p->klab[2][c];
        wsrc[c] = -1;
        for (int a = 0; a < ru; a++) if (p->klab[0][a] == l) { wsrc[c] = 0; wpos[c] = a; }
        if (wsrc[c] < 0)
            for (int b = 0; b < rv; b++) if (p->klab[1][b] == l) { wsrc[c] = 1; wpos[c] = b; }
        if (wsrc[c] < 0) return ORC_E_SPLIT; /* upper in W but lower in both inputs */
    }
    /* V tuples ordered by join key */
    int32_t *vj = (int32_t *)malloc(sizeof(int32_t) * (size_t)(nv * (nj ? nj : 1)));
    int64_t *vidx = (int64_t *)malloc(sizeof(int64_t) * (size_t)nv);
    if (!vj || !vidx) { free(vj); free(vidx); return ORC_E_NOMEM; }
    for (int64_t v = 0; v < nv; v++) {
        for (int k = 0; k < nj; k++) vj[v * nj + k] = vkeys[v * rv + jv[k]];
        vidx[v] = v;
    }
    row_ctx cv = {vj, nj};
    if (nj) qsort_r(vidx, (size_t)nv, sizeof(int64_t), cmp_rows, &cv);
    /* count and collect pairs: for each u, the run of V tuples with equal join key */
    int64_t cap = 1024, np = 0;
    int32_t *pr = (int32_t *)malloc(sizeof(int32_t) * (size_t)(cap * (rw + 2)));
    if (!pr) { free(vj); free(vidx); return ORC_E_NOMEM; }
    int32_t key[26];
    for (int64_t u = 0; u < nu; u++) {
        for (int k = 0; k < nj; k++) key[k] = ukeys[u * ru + ju[k]];
        /* lower bound of key in the sorted V join keys */
        int64_t lo = 0, hi = nv;
        while (lo < hi) {
            int64_t mid = (lo + hi) / 2;
            const int32_t *row = vj + vidx[mid] * nj;
            int c = 0;
            for (int k = 0; k < nj && c == 0; k++) c = row[k] < key[k] ? -1 : (row[k] > key[k] ? 1 : 0);
            if (c < 0) lo = mid + 1; else hi = mid;
        }
        for (int64_t s = lo; s < nv; s++) {
            const int32_t *row = vj + vidx[s] * nj;
            if (nj && memcmp(row, key, sizeof(int32_t) * (size_t)nj) != 0) break;
            int64_t v = vidx[s];
            if (np == cap) {
                cap *= 2;
                int32_t *q = (int32_t *)realloc(pr, sizeof(int32_t) * (size_t)(cap * (rw + 2)));
                if (!q) { free(pr); free(vj); free(vidx); return ORC_E_NOMEM; }
                pr = q;
            }
            int32_t *rec = pr + np * (rw + 2);
            for (int c = 0; c < rw; c++)
                rec[c] = wsrc[c] == 0 ? ukeys[u * ru + wpos[c]] : vkeys[v * rv + wpos[c]];
            rec[rw] = (int32_t)u;
            rec[rw + 1] = (int32_t)v;
            np++;
        }
    }
    free(vj);
    free(vidx);
    /* canonical order (w_key, u, v) */
    int64_t *ord = (int64_t *)malloc(sizeof(int64_t) * (size_t)(np ? np : 1));
    int32_t *pairs = (int32_t *)malloc(sizeof(int32_t) * (size_t)(2 * (np ? np : 1)));
    int32_t *wk = (int32_t *)malloc(sizeof(int32_t) * (size_t)((np ? np : 1) * (rw ? rw : 1)));
    if (!ord || !pairs || !wk) { free(ord); free(pairs); free(wk); free(pr); return ORC_E_NOMEM; }
    for (int64_t i = 0; i < np; i++) ord[i] = i;
    row_ctx cp = {pr, rw + 2};
    qsort_r(ord, (size_t)np, sizeof(int64_t), cmp_rows, &cp);
    int64_t nw = 0;
    for (int64_t i = 0; i < np; i++) {
        const int32_t *rec = pr + ord[i] * (rw + 2);
        pairs[2 * i] = rec[rw];
        pairs[2 * i + 1] = rec[rw + 1];
        if (nw == 0 || (rw > 0 && memcmp(wk + (nw - 1) * rw, rec, sizeof(int32_t) * (size_t)rw) != 0)) {
            if (rw > 0) memcpy(wk + nw * rw, rec, sizeof(int32_t) * (size_t)rw);
            if (nw == 0 || rw > 0) nw++;
        }
    }
    free(pr);
    free(ord);
    *npairs_out = np;
    *pairs_out = pairs;
    *nw_out = nw;
    *wkeys_out = wk;
    return ORC_OK;
}

void orc_free(void *x) { free(x); }

/* ---------------------------------------------------------- step 3: eval */

typedef struct {
    const int64_t *coords;
    int nl;
    int ns;
    const int *pos;   /* positions (within the operand) of the shared labels */
} coo_ctx;

static int cmp_coo(const void *a, const void *b, void *c) {
    const coo_ctx *x = (const coo_ctx *)c;
    int64_t i = *(const int64_t *)a, j = *(const int64_t *)b;
    for (int k = 0; k < x->ns; k++) {
        int64_t ci = x->coords[i * x->nl + x->pos[k]], cj = x->coords[j * x->nl + x->pos[k]];
        if (ci != cj) return ci < cj ? -1 : 1;
    }
    return (i < j) ? -1 : (i > j ? 1 : 0);
}

/* Value-level evaluation.  For each pair of entries (one of U, one of V) whose
 * coordinates agree on every label the operands share, add the product into
 * the W entry whose coordinates are taken from the two entries.  Output W is
 * given by its key list (sorted, [nw x nk(W)]); acc and mag are
 * [nw x tile_elems(W)] and are overwritten.  Contributions that fall outside
 * the listed keys are counted in *n_outside (a full evaluation must find 0;
 * an evaluation restricted to sampled output keys skips them). */
int orc_eval(const orc_plan *p, const int64_t *ucoo, const double *uval, int64_t nu,
             const int64_t *vcoo, const double *vval, int64_t nv, const int32_t *wkeys,
             int64_t nw, double *acc, double *mag, int64_t *n_outside) {
    int nlu = p->nl[0], nlv = p->nl[1], nlw = p->nl[2], rw = p->nk[2];
    int64_t tw = p->tile_elems[2];
    memset(acc, 0, sizeof(double) * (size_t)(nw * tw));
    memset(mag, 0, sizeof(double) * (size_t)(nw * tw));
    *n_outside = 0;
    if (nu == 0 || nv == 0 || nw == 0) return ORC_OK;
    int su[26], sv[26], ns = 0;
    for (int a = 0; a < nlu; a++)
        for (int b = 0; b < nlv; b++)
            if (p->lab[0][a] == p->lab[1][b]) { su[ns] = a; sv[ns] = b; ns++; }
    /* each W label takes its coordinate from U if present there, else from V */
    int wsrc[26], wpos[26];
    for (int c = 0; c < nlw; c++) {
        int l = p->lab[2][c];
        wsrc[c] = -1;
        for (int a = 0; a < nlu; a++) if (p->lab[0][a] == l) { wsrc[c] = 0; wpos[c] = a; }
        if (wsrc[c] < 0)
            for (int b = 0; b < nlv; b++) if (p->lab[1][b] == l) { wsrc[c] = 1; wpos[c] = b; }
    }
    /* iterate over the operand with fewer entries; index the other one by its
     * shared-label coordinates */
    int outer_is_u = nu <= nv;
    const int64_t *oc = outer_is_u ? ucoo : vcoo, *ic = outer_is_u ? vcoo : ucoo;
    const double *ov = outer_is_u ? uval : vval, *iv = outer_is_u ? vval : uval;
    int64_t no = outer_is_u ? nu : nv, ni = outer_is_u ? nv : nu;
    int nlo = outer_is_u ? nlu : nlv, nli = outer_is_u ? nlv : nlu;
    const int *po = outer_is_u ? su : sv, *pi = outer_is_u ? sv : su;
    int64_t *idx = (int64_t *)malloc(sizeof(int64_t) * (size_t)ni);
    if (!idx) return ORC_E_NOMEM;
    for (int64_t i = 0; i < ni; i++) idx[i] = i;
    coo_ctx cc = {ic, nli, ns, pi};
    if (ns) qsort_r(idx, (size_t)ni, sizeof(int64_t), cmp_coo, &cc);
    int64_t want[26];
    int32_t wk[26];
    for (int64_t o = 0; o < no; o++) {
        for (int k = 0; k < ns; k++) want[k] = oc[o * nlo + po[k]];
        int64_t lo = 0, hi = ni;
        while (lo < hi) {
            int64_t mid = (lo + hi) / 2;
            int c = 0;
            for (int k = 0; k < ns && c == 0; k++) {
                int64_t x = ic[idx[mid] * nli + pi[k]];
                c = x < want[k] ? -1 : (x > want[k] ? 1 : 0);
            }
            if (c < 0) lo = mid + 1; else hi = mid;
        }
        for (int64_t s = lo; s < ni; s++) {
            int64_t i = idx[s];
            int match = 1;
            for (int k = 0; k < ns && match; k++) match = ic[i * nli + pi[k]] == want[k];
            if (!match) break;
            const int64_t *cu = outer_is_u ? oc + o * nlo : ic + i * nli;
            const int64_t *cv = outer_is_u ? ic + i * nli : oc + o * nlo;
            double prod = ov[o] * iv[i];
            /* W coordinate -> (key, offset in tile) */
            int64_t offw = 0;
            int ka = 0;
            for (int c = 0; c < nlw; c++) {
                int l = p->lab[2][c];
                int64_t g = wsrc[c] == 0 ? cu[wpos[c]] : cv[wpos[c]];
                if (p->up[l]) {
                    wk[ka++] = (int32_t)(g / p->t[l]);
                    offw = offw * p->t[l] + g % p->t[l];
                } else {
                    offw = offw * p->t[l] + g;
                }
            }
            /* binary search for the key */
            int64_t a = 0, b = nw, found = -1;
            while (a < b) {
                int64_t m = (a + b) / 2;
                int c = 0;
                for (int k = 0; k < rw && c == 0; k++) {
                    int32_t x = wkeys[m * rw + k];
                    c = x < wk[k] ? -1 : (x > wk[k] ? 1 : 0);
                }
                if (c == 0) { found = m; break; }
                if (c < 0) a = m + 1; else b = m;
            }
            if (rw == 0) found = 0;
            if (found < 0) { (*n_outside)++; continue; }
            acc[found * tw + offw] += prod;
            mag[found * tw + offw] += fabs(prod);
        }
    }
    free(idx);
    return ORC_OK;
}

/* ------------------------------------------------------ repartition */

/*
 * orc_repartition -- the same tensor under a second decomposition (Sec. 6,
 * "changing representation" between two EinSums: decompose every tuple on
 * all labels promoted in either decomposition, ALLINTS, then re-compose with
 * the STACK aggregate grouped by the target's promoted labels).
 *
 * Written as its plain definition, element by element:
 *   - the target holds one tuple for every target tile that contains at
 *     least one position of a source tile (zero values included: a stored
 *     tile joins like any other, so every position it covers is carried);
 *   - every target element equals the source element at the same global
 *     coordinate, and 0 where no source tile covers the coordinate.
 * labels: the tensor's labels in string order (no repeats).  up_in / up_out:
 * promoted labels of the two decompositions.  ext[26]: extents; tin / tout
 * [26]: tile sizes of promoted labels (a demoted label keeps its extent).
 * Keys are int32 [n x r] in label-string order of the promoted labels.
 * Tile values are doubles; outputs are malloc'd (free with orc_free).
 */
typedef struct {
    int nl;
    int lab[26];
    int64_t ext[26], tin[26], tout[26];   /* per position in `labels` */
    int pin[26], pout[26];                /* promoted in source / target */
    int rin, rout;
    int64_t te_in, te_out;
} rp_desc;

static int rp_make(const char *labels, const char *up_in, const char *up_out, const int64_t *ext,
                   const int32_t *tin, const int32_t *tout, rp_desc *d) {
    memset(d, 0, sizeof(*d));
    int seen[26] = {0};
    for (const char *c = labels; *c; c++) {
        if (*c < 'a' || *c > 'z' || seen[*c - 'a'] || d->nl == 26) return ORC_E_PARSE;
        seen[*c - 'a'] = 1;
        d->lab[d->nl++] = *c - 'a';
    }
    int inup[26] = {0}, outup[26] = {0};
    for (const char *c = up_in; *c; c++) {
        if (*c < 'a' || *c > 'z' || !seen[*c - 'a']) return ORC_E_SPLIT;
        inup[*c - 'a'] = 1;
    }
    for (const char *c = up_out; *c; c++) {
        if (*c < 'a' || *c > 'z' || !seen[*c - 'a']) return ORC_E_SPLIT;
        outup[*c - 'a'] = 1;
    }
    d->te_in = d->te_out = 1;
    for (int i = 0; i < d->nl; i++) {
        int l = d->lab[i];
        d->ext[i] = ext[l];
        if (ext[l] < 1) return ORC_E_SHAPE;
        d->pin[i] = inup[l];
        d->pout[i] = outup[l];
        d->tin[i] = inup[l] ? tin[l] : ext[l];
        d->tout[i] = outup[l] ? tout[l] : ext[l];
        if (d->tin[i] < 1 || ext[l] % d->tin[i] || d->tout[i] < 1 || ext[l] % d->tout[i]) return ORC_E_SHAPE;
        d->rin += inup[l];
        d->rout += outup[l];
        d->te_in *= d->tin[i];
        d->te_out *= d->tout[i];
    }
    return ORC_OK;
}

static int cmp_keyrow(const void *a, const void *b, void *c) {
    int r = *(const int *)c;
    const int32_t *x = (const int32_t *)a, *y = (const int32_t *)b;
    for (int k = 0; k < r; k++) {
        if (x[k] != y[k]) return x[k] < y[k] ? -1 : 1;
    }
    return 0;
}

/* global coordinate of element e of source tuple `key` on label position i */
static void rp_coords(const rp_desc *d, const int32_t *key, int64_t e, int64_t *g) {
    int64_t rem = e;
    for (int i = d->nl - 1; i >= 0; i--) {
        g[i] = rem % d->tin[i];
        rem /= d->tin[i];
    }
    int ka = 0;
    for (int i = 0; i < d->nl; i++)
        if (d->pin[i]) g[i] += (int64_t)key[ka++] * d->tin[i];
}

/* target key and target offset of global coordinate g */
static int64_t rp_target(const rp_desc *d, const int64_t *g, int32_t *tkey) {
    int64_t off = 0;
    int ka = 0;
    for (int i = 0; i < d->nl; i++) {
        if (d->pout[i]) tkey[ka++] = (int32_t)(g[i] / d->tout[i]);
        off = off * d->tout[i] + g[i] % d->tout[i];
    }
    return off;
}

int orc_repartition(const char *labels, const char *up_in, const char *up_out, const int64_t *ext,
                    const int32_t *tin, const int32_t *tout, const int32_t *keys_in, int64_t n_in,
                    const double *tiles_in, int64_t *n_out, int32_t **keys_out, double **tiles_out) {
    rp_desc d;
    int st = rp_make(labels, up_in, up_out, ext, tin, tout, &d);
    if (st != ORC_OK) return st;
    *n_out = 0;
    *keys_out = NULL;
    *tiles_out = NULL;
    const int rout = d.rout;
    const int64_t total = n_in * d.te_in;
    /* the target key of every source position, then sorted and made unique */
    int32_t *all = (int32_t *)malloc(sizeof(int32_t) * (size_t)(total > 0 ? total : 1) * (size_t)(rout > 0 ? rout : 1));
    if (!all) return ORC_E_NOMEM;
    int64_t g[26];
    for (int64_t s = 0; s < n_in; s++) {
        for (int64_t e = 0; e < d.te_in; e++) {
            rp_coords(&d, keys_in + s * d.rin, e, g);
            rp_target(&d, g, all + (s * d.te_in + e) * rout);
        }
    }
    int64_t nk = 0;
    if (total > 0) {
        if (rout > 0) {
            qsort_r(all, (size_t)total, sizeof(int32_t) * (size_t)rout, cmp_keyrow, (void *)&rout);
            for (int64_t i = 0; i < total; i++) {
                if (nk == 0 || cmp_keyrow(all + (nk - 1) * rout, all + i * rout, (void *)&rout) != 0) {
                    memmove(all + nk * rout, all + i * rout, sizeof(int32_t) * (size_t)rout);
                    nk++;
                }
            }
        } else {
            nk = 1;
        }
    }
    double *tiles = (double *)calloc((size_t)(nk > 0 ? nk : 1) * (size_t)d.te_out, sizeof(double));
    if (!tiles) {
        free(all);
        return ORC_E_NOMEM;
    }
    int32_t tkey[26];
    for (int64_t s = 0; s < n_in; s++) {
        for (int64_t e = 0; e < d.te_in; e++) {
            rp_coords(&d, keys_in + s * d.rin, e, g);
            int64_t off = rp_target(&d, g, tkey);
            int64_t a = 0, b = nk, found = rout == 0 ? 0 : -1;
            while (found < 0 && a < b) {
                int64_t m = (a + b) / 2;
                int c = cmp_keyrow(all + m * rout, tkey, (void *)&rout);
                if (c == 0) found = m;
                else if (c < 0) a = m + 1;
                else b = m;
            }
            if (found < 0) {  /* cannot happen: every position's key was listed */
                free(all);
                free(tiles);
                return ORC_E_ARG;
            }
            tiles[found * d.te_out + off] = tiles_in[s * d.te_in + e];
        }
    }
    *n_out = nk;
    *keys_out = all;
    *tiles_out = tiles;
    return ORC_OK;
}
