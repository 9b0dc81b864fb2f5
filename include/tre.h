/*
 * tre.h -- C ABI of the tensor-relational EinSum library for AMD Instinct
 * MI355X (gfx950).
 *
 * One call evaluates one binary EinSum whose operands are tensor relations
 * (Tang et al., "Automated Tensor-Relational Decomposition for Large-Scale
 * Sparse Tensor Computation", PVLDB 19(6), 2026):
 *
 *   - Sec. 3, Eq. "Einsum": W[lW] = sum over labels not in W of U[lU] * V[lV].
 *   - Sec. 4.2: a relation stores one tuple per key of its promoted
 *     (upper-case) labels; each tuple holds a dense tile over the demoted
 *     (lower-case) labels.  Here a promoted label l may also carry a tile size
 *     t_l: the global index is t_l * L + l', L is the tuple attribute and l'
 *     indexes the tile (t_l = 1 is the paper's plain promoted label).
 *   - Sec. 5, Eq. "eqn-TRA" and its SQL form
 *         SELECT upper(W), SUM(K(valU, valV)) FROM U NATURAL JOIN V
 *         GROUP BY upper(W)
 *     is what tre_join + tre_contract compute: (1) a join on the promoted
 *     labels the operands share, (2) the kernel K -- the EinSum restricted to
 *     the tile labels -- on every matched tile pair, (3) a sum of the partial
 *     tiles grouped by W's promoted labels.
 *
 * Conventions for every entry point:
 *   - Device pointers are HIP device memory owned by the caller; the library
 *     allocates no device memory in tre_join / tre_contract / tre_execute and
 *     uses only the caller's workspace.  Host pointers are marked "host".
 *   - `stream` is a hipStream_t passed as void* (NULL = the null stream).
 *   - Keys: int32, row-major [n x r], r = number of promoted labels of the
 *     operand, attributes in the order the labels appear in the operand's
 *     string; rows strictly increasing in lexicographic order; attribute of
 *     label l in [0, extent_l / t_l).  A relation with r = 0 holds at most one
 *     tuple and its key pointer is ignored.
 *   - Tiles: [n x tile_elems] contiguous, each tile row-major over ALL the
 *     operand's labels in string order, with extent t_l for a promoted label
 *     and the full extent for a demoted one.  Inputs are fp32 or bf16 (raw
 *     bits, uint16).  Accumulation is fp32; W tiles are fp32, or bf16 bits
 *     rounded to nearest even from the fp32 sums when the plan was made with
 *     the w_bf16 option (tre_plan_info.w_dtype says which).  Tile arrays
 *     start on a 16-byte boundary (TRE_E_ARG otherwise).
 *   - Output order: W keys sorted lexicographically; the pair list in order of
 *     (W key, u index, v index), u/v being positions in the caller's arrays.
 *   - Errors are returned as tre_status; the library never aborts and never
 *     prints.  tre_last_error() gives a thread-local detail string.
 */
#ifndef TRE_H
#define TRE_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
    TRE_OK = 0,
    TRE_E_ARG = 1,        /* null pointer, negative size, bad option */
    TRE_E_PARSE = 2,      /* malformed EinSum string */
    TRE_E_SPLIT = 3,      /* promoted-label set names a label not in the EinSum */
    TRE_E_SHAPE = 4,      /* extent < 1, tile not dividing extent, key space > 64 bits */
    TRE_E_DTYPE = 5,      /* unsupported input dtype */
    TRE_E_UNSORTED = 6,   /* keys not in increasing lexicographic order */
    TRE_E_DUPKEY = 7,     /* repeated key (or r = 0 with more than one tuple) */
    TRE_E_KEYRANGE = 8,   /* key attribute outside [0, extent / t) */
    TRE_E_CAPACITY = 9,   /* caller buffer too small; required sizes are reported */
    TRE_E_WORKSPACE = 10, /* workspace too small for this input */
    TRE_E_DEVICE = 11,    /* a HIP runtime call failed */
    TRE_E_STATE = 12      /* join result does not belong to this plan / workspace */
} tre_status;

typedef enum { TRE_F32 = 0, TRE_BF16 = 1 } tre_dtype;

typedef struct tre_plan_s *tre_plan_t;

typedef struct {
    int32_t validate_keys;      /* nonzero: check key order, uniqueness and range on the device (default 1) */
    int32_t max_pairs_per_unit; /* work-unit length cap; 0 = chosen from the pair count */
    int32_t u_ranges;           /* 128x128 path: cut every output key's pairs into this many ranges of
                                   U tuple index and run range by range so concurrent workgroups share U
                                   tiles in L2 (partials summed after); 0 = automatic, < 0 = never */
    int32_t pace_windows;       /* 128x128 path with one 128x128 block per W tile: one persistent
                                   workgroup per resident slot walks whole keys while the workgroups of each
                                   XCD keep within a few windows of U tuple index of each other (the U
                                   index range is cut into this many windows), so U tiles stay in L2 with
                                   no partial tiles; 0 = automatic (preferred over u_ranges when both
                                   apply), < 0 = never.  Results do not depend on it. */
    int32_t w_bf16;             /* nonzero: tre_contract writes W as bf16 (round to nearest even from the
                                   fp32 sum; the bits tre_cast_f32_bf16 gives) instead of fp32, for a
                                   consumer that reads bf16: the producer writes half the bytes and no
                                   cast pass runs.  Vector class and 128x128 path only (TRE_E_DTYPE in
                                   tre_plan otherwise). */
    int32_t small_join;         /* 0 = automatic: a join whose pairs come out grouped by W key, whose driving
                                   relation has at most 4096 tuples and at most 4096 pairs runs in one
                                   workgroup (one launch); < 0 = never */
    int32_t reserved[2];
} tre_options;

/* Static facts about a plan (host). */
typedef struct {
    int32_t key_arity[3];     /* r_U, r_V, r_W */
    int64_t tile_elems[3];    /* elements per tile of U, V, W */
    int32_t n_join;           /* promoted labels shared by U and V */
    int32_t kernel_class;     /* 0 = MFMA tile GEMM, 1 = vector (scale / GEMV / dot), 2 = MFMA GEMM with
                                 128x128 blocks and direct-to-LDS copies (bf16 with K a multiple of 64,
                                 fp32 with K a multiple of 32) */
    int64_t batch, m, n, k;   /* per-pair contraction: W[b,m,n] += sum_k U[b,m,k] V[b,k,n] */
    int64_t flops_per_pair;   /* 2 * batch * m * n * k */
    char key_labels[3][27];   /* promoted labels of U, V, W in key order (NUL-terminated) */
    char roles[27];           /* per letter a..z: 'b','m','n','k','p' (pre-sum) or '.' unused */
    int32_t group_needs_sort; /* 1 if pairs are radix-sorted by W key */
    int32_t v_needs_sort;     /* 1 if V is radix-sorted by its join key */
    int32_t w_dtype;          /* element type tre_contract writes to w_tiles: TRE_F32, or TRE_BF16 with w_bf16 */
    int32_t join_outer;       /* 0: the join walks U and searches V; 1: it walks V and searches U, which
                                 emits the pairs already grouped by W key (W's key is V's key prefix,
                                 followed by the join labels, which U's key starts with) */
} tre_plan_info;

/* Result of tre_join, consumed by tre_contract (host struct; the pair list,
 * segments and packed output keys stay in the workspace). */
typedef struct {
    int64_t n_u, n_v;
    int64_t n_pairs;          /* matched tile pairs */
    int64_t n_w;              /* output tuples (distinct W keys) */
    uint64_t internal[16];    /* workspace layout; do not modify */
} tre_join_result;

/* Optional per-phase device timings (milliseconds, hipEvent based).
 * With `deferred` = 0 every phase is bracketed by events recorded on the
 * stream and the call waits for them before returning.
 * With `deferred` != 0 only the contraction kernel is timed, by start and end
 * events that its own launch records (hipExtLaunchKernel: no marker packets,
 * no wait, next to no cost for a small call); tre_timing_read later waits for
 * them, fills contract_ms (the other phase fields stay 0) and releases the
 * events.  A struct with `pending` set must be read (or the events leak). */
typedef struct {
    float join_ms;            /* key validation, join, group-by up to the count read-back (tre_join; not with
                                 deferred) */
    float units_ms;           /* offset tables and work units */
    float contract_ms;        /* the tile-contraction kernel alone */
    float reduce_ms;          /* segmented sum of split segments + key / pair write-out */
    float total_ms;
    int32_t deferred;         /* in */
    int32_t pending;          /* out: events recorded, not yet read */
    int64_t n_units;
    int64_t n_split_segments;
    int64_t n_partials;       /* partial tiles written by units of split segments */
    void *events[4];          /* library-owned while pending */
    int32_t contract_path;    /* out: the contraction launch tre_contract chose: 0 generic MFMA GEMM (64x64
                                 blocks), 1 vector class, 2 128x128 MFMA path, 3 the same as a paced
                                 persistent grid, 4 the same with U-range units (partials summed after) */
    int32_t join_path;        /* out (tre_join, tre_execute3): 0 driven by U (runs searched in V), 1 driven by V (runs
                                 searched in U), 2 driven by V with at most one U tuple each, 3 driven by V
                                 over a U holding every key (no search), 4 keyless one-tuple V with W keyed by
                                 U, 5 the whole join in one workgroup (small inputs), 6 driven by U over a V
                                 holding every key (no search) */
} tre_timing;

/* tre_plan -- parse and classify one binary EinSum (host only, no device work).
 *   einsum : host string "lhs0,lhs1->out" of lower-case letters; exactly two
 *            inputs; no label repeated within an operand; every output label
 *            appears in an input (Sec. 3 general form).
 *   upper  : host string, the promoted labels (Sec. 4.3 upper case); may be "".
 *   extent : host [26], indexed by letter - 'a'; >= 1 for used labels.
 *   tile   : host [26]; for a promoted label 1 <= t <= extent and extent % t == 0;
 *            ignored for demoted labels (their tile extent is the full extent).
 *   in_dtype : a tre_dtype value, TRE_F32 or TRE_BF16, for both inputs (passed
 *            as int32 so that any other value is a defined TRE_E_DTYPE);
 *            accumulation is fp32 and W is fp32 unless opt->w_bf16 asks for
 *            bf16 output.
 *   opt    : host, may be NULL for defaults.
 *   out    : receives a host-owned, immutable plan; thread-safe to share. */
tre_status tre_plan(const char *einsum, const char *upper, const int64_t *extent, const int32_t *tile,
                    int32_t in_dtype, const tre_options *opt, tre_plan_t *out);

tre_status tre_plan_get_info(tre_plan_t plan, tre_plan_info *info);

void tre_plan_destroy(tre_plan_t plan);

/* Upper bound on the workspace needed for n_u and n_v input tuples and at most
 * max_pairs matched pairs (bytes, a multiple of 256). */
size_t tre_workspace_bytes(tre_plan_t plan, int64_t n_u, int64_t n_v, int64_t max_pairs);

/* Largest pair count a workspace of ws_bytes can hold for n_u, n_v. */
int64_t tre_workspace_max_pairs(tre_plan_t plan, int64_t n_u, int64_t n_v, size_t ws_bytes);

/* tre_join -- step (1) of Sec. 5 plus the GROUP BY keys: validate keys
 * (optional), sort V by join key if its key order does not start with the
 * join labels, build the matched pair list on the device (binary-search
 * counts, scan, load-balanced expansion), sort pairs by W key (stable LSD
 * radix) and run-length encode them into output keys and segments.
 *   u_keys, v_keys : device, as in the conventions above.
 *   ws, ws_bytes   : device workspace (256-byte aligned); must stay untouched
 *                    until the matching tre_contract has completed.
 *   out            : host; receives n_pairs and n_w.
 * Synchronizes the stream once, reading back the key checks, the pair count
 * and the output key count together (the GROUP BY stage takes the pair
 * count from device memory, its grids sized for the pairs the workspace can
 * hold); when V has no promoted labels (one tuple) and W's key is U's key as
 * it is, every U tuple is one pair and one output tuple, the counts are
 * known without the device, and the call synchronizes only to report key
 * validation: without it, the join's kernels may still be running on the
 * stream when the call returns, so work on another stream that reads the
 * workspace (tre_contract, tre_join_keys) must wait for this stream.
 * TRE_E_WORKSPACE (out->n_pairs set) if the pairs do not fit; key errors are
 * reported as TRE_E_UNSORTED / TRE_E_DUPKEY / TRE_E_KEYRANGE. */
tre_status tre_join(tre_plan_t plan, const int32_t *u_keys, int64_t n_u, const int32_t *v_keys, int64_t n_v,
                    void *ws, size_t ws_bytes, void *stream, tre_join_result *out, tre_timing *timing);

/* tre_join_keys -- the output keys of a join (the GROUP BY keys of Sec. 5),
 * before any contraction: lets a consumer EinSum start its own join on
 * another stream while tre_contract runs.  Writes the same keys tre_contract
 * writes.
 *   join   : host, from tre_join with this plan; its workspace untouched since.
 *   w_keys : device [w_cap x r_W] int32 (r_W = 0: nothing is written), sorted.
 * Asynchronous on the stream; TRE_E_CAPACITY if w_cap < n_w. */
tre_status tre_join_keys(tre_plan_t plan, const tre_join_result *join, int32_t *w_keys, int64_t w_cap, void *stream);

/* tre_contract -- steps (2) and (3) of Sec. 5: contract every matched tile
 * pair and sum the results per output key.  Pairs of one output key are
 * processed together (split into bounded work units when long); a unit
 * accumulates in registers; split keys are summed by an atomic-free
 * fixed-order segmented reduction, so results are run-to-run deterministic.
 *   u_tiles, v_tiles : device tiles of the same arrays given to tre_join.
 *   w_keys  : device [w_cap x r_W] int32 (may be NULL when r_W = 0).
 *   w_tiles : device [w_cap x tile_elems(W)] of the plan's W element type
 *             (tre_plan_info.w_dtype): fp32, or bf16 bits (uint16) when the
 *             plan was made with w_bf16.
 *   pairs_out : device [pair_cap x 2] int32 (u, v) or NULL.
 * TRE_E_CAPACITY if w_cap < n_w or (pairs_out and pair_cap < n_pairs).
 * Asynchronous on the stream unless timing is non-NULL and not deferred. */
tre_status tre_contract(tre_plan_t plan, const tre_join_result *jr, const void *u_tiles, const void *v_tiles,
                        int32_t *w_keys, int64_t w_cap, void *w_tiles, int32_t *pairs_out, int64_t pair_cap,
                        void *stream, tre_timing *timing);

/* Wait for the events of a deferred tre_contract / tre_execute3 timing and
 * fill contract_ms (and total_ms). */
tre_status tre_timing_read(tre_timing *timing);

/* tre_execute -- tre_join followed by tre_contract (w_tiles of the plan's W
 * element type, as for tre_contract).  n_w / n_pairs (host) are always
 * written when the join succeeded, also with TRE_E_CAPACITY. */
tre_status tre_execute(tre_plan_t plan, const int32_t *u_keys, int64_t n_u, const void *u_tiles,
                       const int32_t *v_keys, int64_t n_v, const void *v_tiles, int32_t *w_keys, void *w_tiles,
                       int64_t w_cap, int64_t *n_w, int32_t *pairs_out, int64_t pair_cap, int64_t *n_pairs,
                       void *ws, size_t ws_bytes, void *stream, tre_timing *timing);

/* tre_output_bounds -- upper bounds on the pair and output key counts of a
 * join of n_u and n_v tuples with a workspace of ws_bytes (host only, no
 * device work): the pair bound is the cross product, or n_u (n_v) when one
 * side's key is made of the join labels only, capped by the workspace's
 * pair capacity; the key bound is that, capped by W's key space; both are
 * n_u for a keyless one-tuple V with W keyed by U.  async_ok = 1 when
 * tre_execute_async can enqueue the whole EinSum without a read-back for
 * these sizes.  TRE_E_WORKSPACE if ws_bytes is below tre_workspace_bytes(
 * plan, n_u, n_v, 0). */
tre_status tre_output_bounds(tre_plan_t plan, int64_t n_u, int64_t n_v, size_t ws_bytes, int64_t *pairs_bound,
                             int64_t *keys_bound, int32_t *async_ok);

/* tre_execute_async -- tre_execute with no wait on the host: the join (Sec.
 * 5), the GROUP BY keys and the contraction are all enqueued on the stream
 * with their grids sized for the bounds of tre_output_bounds, every kernel
 * reading the counts the join wrote in device memory, and the counts come
 * back in device memory, so calls (and chains of them) run back to back.
 *   counts  : device int64 [4], written last on the stream: [0] pairs, [1]
 *             output keys, [2] a tre_status (TRE_OK, TRE_E_UNSORTED /
 *             TRE_E_DUPKEY / TRE_E_KEYRANGE when key validation finds an
 *             error, TRE_E_WORKSPACE when the pairs exceed the workspace's
 *             capacity: then [0] is the number needed), [3] 0.  W and the
 *             pair list hold [1] and [0] entries when [2] is TRE_OK and are
 *             unspecified otherwise.
 *   w_cap, pair_cap : at least the key and pair bounds (TRE_E_CAPACITY on
 *             the host otherwise).
 *   n_u_dev : optional device int64 holding U's tuple count when only a
 *             bound n_u is known on the host (the keys and tiles of U are
 *             read up to that count): for a keyless one-tuple V with W keyed
 *             by U, e.g. the second EinSum of a chain whose U is the first
 *             one's output (TRE_E_ARG for other plans, or when the sizes are
 *             not async_ok).
 *   Everything else as for tre_execute.  When the sizes are not async_ok
 *   (and n_u_dev is NULL) the call runs tre_execute, waiting for its counts,
 *   and writes them to `counts`.  The summation order follows the bounds,
 *   so results can differ in the last bits from tre_execute's when a bound
 *   exceeds the count it stands for. */
tre_status tre_execute_async(tre_plan_t plan, const int32_t *u_keys, int64_t n_u, const int64_t *n_u_dev,
                             const void *u_tiles, const int32_t *v_keys, int64_t n_v, const void *v_tiles,
                             int32_t *w_keys, void *w_tiles, int64_t w_cap, int32_t *pairs_out, int64_t pair_cap,
                             int64_t *counts, void *ws, size_t ws_bytes, void *stream, tre_timing *timing);

/* tre_execute_noalloc -- tre_execute without a workspace argument, for
 * callers that cannot allocate device memory: code under stream capture,
 * tight serving loops, harnesses that forbid allocation.  The workspace is a
 * static device array of tre_noalloc_scratch_bytes() bytes (256 MiB) in the
 * library's device data; every GPU the library runs on holds its own copy
 * until the process ends.  The call allocates nothing (no hipMalloc, no
 * events) and takes its timing from no one (no tre_timing argument); outputs
 * are the caller's, as for tre_execute (w_tiles of the plan's W element
 * type).  Every call on one GPU uses that GPU's array and leaves its
 * contents behind; what must start at zero is cleared by each call, but
 * calls that overlap on one GPU (from several streams or threads) race on the
 * array: serialise them.  Inputs whose workspace (tre_workspace_bytes with
 * the join's pair count) exceeds the array: TRE_E_WORKSPACE, n_pairs set when
 * the join got that far, nothing else written.  Synchronizes like tre_join. */
size_t tre_noalloc_scratch_bytes(void);
tre_status tre_execute_noalloc(tre_plan_t plan, const int32_t *u_keys, int64_t n_u, const void *u_tiles,
                               const int32_t *v_keys, int64_t n_v, const void *v_tiles, int32_t *w_keys,
                               void *w_tiles, int64_t w_cap, int64_t *n_w, int32_t *pairs_out, int64_t pair_cap,
                               int64_t *n_pairs, void *stream);

/* --- chain glue between two EinSums (Sec. 6, repartition) --------------- */

/* Round fp32 to bf16 (nearest even; NaN stays NaN).  x, y device, n elements. */
tre_status tre_cast_f32_bf16(const float *x, uint16_t *y, int64_t n, void *stream);

/* y = scale * x, elementwise over n fp32 values (device, 16-byte aligned; x
 * may equal y): a unary EinSum applied to every tuple's tile, e.g. the
 * 1 / sqrt(d_k) of the attention scores (Sec. 9, Table gt-schema).
 * TRE_E_ARG on a null or misaligned array or n < 0; asynchronous. */
tre_status tre_scale_f32(const float *x, float *y, int64_t n, float scale, void *stream);

/* Re-compose a relation keyed by ONE promoted label from tile size t_in to
 * t_out = group * t_in along that label (the STACK aggregate of Sec. 6 where
 * the new promoted set equals the old one):
 *   keys     : device [n] int32 sorted increasing (arity 1).
 *   tiles    : device [n x row_elems] of elem_bytes-wide elements; a tile is
 *              t_in rows along the label times the remaining elements.
 *   out_keys : device [out_cap] int32 = distinct key / group.
 *   out_tiles: device [out_cap x group*row_elems]; absent rows are zero.
 *   ws       : device workspace of at least tre_stack_workspace_bytes(n).
 *   n_out    : host; synchronizes to read it.  TRE_E_CAPACITY if out_cap is short. */
size_t tre_stack_workspace_bytes(int64_t n);
tre_status tre_stack_rows(const int32_t *keys, int64_t n, const void *tiles, int64_t row_elems, int32_t group,
                          int32_t elem_bytes, int32_t *out_keys, void *out_tiles, int64_t out_cap, int64_t *n_out,
                          void *ws, size_t ws_bytes, void *stream);

/* Repartition (Sec. 6, "changing representation" between two EinSums): the
 * same tensor under a second decomposition.  The relation is decomposed on
 * every label promoted in either decomposition (ALLINTS) and re-composed with
 * the STACK aggregate grouped by the target's promoted labels; here both
 * steps are one device pass.
 *   labels            : the tensor's labels in string order, e.g. "ki" (at most 8).
 *   upper_in/upper_out: promoted labels of the source / target decomposition.
 *   extent[26], tile_in[26], tile_out[26]: per letter; a promoted label's tile
 *                       size must divide its extent, a demoted label keeps its
 *                       whole extent in the tile (its tile entry is ignored).
 *   elem_bytes        : 2 (bf16 bits) or 4 (fp32); values are copied bit for bit.
 *   keys_in, tiles_in : device source relation, conventions above (sorted keys).
 *   keys_out, tiles_out: device [out_cap x r_out] int32 / [out_cap x tile_elems_out].
 *                       tiles_out may be tiles_in (in place) when the target
 *                       tiles are the source tiles regrouped: every source tile
 *                       lies in one target tile as one contiguous run, every
 *                       target tile is covered, and source key order is target
 *                       order (e.g. stacking per-vertex rows into row blocks
 *                       with no vertex missing).  Then no tile byte moves and
 *                       only keys_out is written; otherwise in place is
 *                       TRE_E_ARG, with the tiles untouched.
 *   n_out             : host; the number of target tuples: one for every target
 *                       tile that contains a position of a source tile (zero
 *                       values included), keys sorted.  Target elements that no
 *                       source tile covers are zero.
 *   ws, ws_bytes      : device workspace, 256-byte aligned, at least
 *                       tre_repartition_workspace_bytes(...) (0 on bad arguments).
 * Synchronizes the stream twice.  TRE_E_CAPACITY (n_out set) if out_cap is
 * short; TRE_E_UNSORTED / TRE_E_DUPKEY / TRE_E_KEYRANGE for bad source keys. */
size_t tre_repartition_workspace_bytes(const char *labels, const char *upper_in, const char *upper_out,
                                       const int64_t extent[26], const int32_t tile_in[26],
                                       const int32_t tile_out[26], int64_t n_in);
tre_status tre_repartition(const char *labels, const char *upper_in, const char *upper_out,
                           const int64_t extent[26], const int32_t tile_in[26], const int32_t tile_out[26],
                           int32_t elem_bytes, const int32_t *keys_in, int64_t n_in, const void *tiles_in,
                           int32_t *keys_out, void *tiles_out, int64_t out_cap, int64_t *n_out, void *ws,
                           size_t ws_bytes, void *stream);

/* --- non-binary EinSum (Sec. 8) ------------------------------------------- */

/* tre_execute3 -- one three-operand EinSum "U,V,X->W" whose two small
 * operands each meet U on a promoted label of their own and share one
 * demoted label r, in one of two forms:
 *   - r is kept in W and U's two joined labels are summed, e.g. A[i,r] =
 *     sum_jk T[i,j,k] B[j,r] C[k,r] (the non-binary EinSum of Sec. 8);
 *   - masked form: W has exactly U's labels and r is summed, e.g. the
 *     attention scores S[i,j] = sum_k A[i,j] T0[i,k] T1[j,k] of the graph
 *     transformer of Sec. 9, which Table gt-schema runs as two binary EinSums
 *     (T2 = T0 A with no aggregation, then T3 = sum_k T2 T1).
 * Instead of two binary EinSums (U join V, then that result join X), U is
 * joined with V and X in one pass (the join of Sec. 5 over three relations):
 * every U tuple whose key on a has a V tuple and whose key on b has an X
 * tuple forms a triple, each triple contributes the tile EinSum of its three
 * tiles, and the contributions are summed per output key (GROUP BY W's
 * promoted labels) in U order, atomic-free, as in tre_contract.  No
 * intermediate relation is materialised.  In the masked form every triple is
 * its own output tuple: W's keys are the matched U keys, in U order.
 * Structure (TRE_E_PARSE / TRE_E_SPLIT otherwise):
 *   - V and X have two labels each and share exactly one, r, which is not in
 *     U and is demoted; V's other label a and X's other label b are promoted
 *     labels of U and are U's last two labels, in either order;
 *   - W's labels are U's labels other than a and b, plus r, in any order; or
 *     W is U's label string itself (masked form).
 * Shapes (TRE_E_SHAPE otherwise): tiles divide extents; first form: the tile
 * extent of U's last label is a multiple of 4 and the tile extents of U's
 * last two labels are at most 64 each; masked form: U's last two labels take
 * tiles of 1 (one scalar per edge, as in Table gt-schema), U's other labels
 * any tiles.  in_dtype: TRE_F32 only (TRE_E_DTYPE otherwise; an int32 holding a
 * tre_dtype value, as for tre_plan).
 *   extent, tile : host [26] per letter, as for tre_plan.
 *   u_keys [n_u x r_U], v_keys [n_v x 1], x_keys [n_x x 1]: device int32,
 *                  sorted strictly increasing (U keyed by its promoted labels
 *                  in string order, V by a, X by b).
 *   u_tiles, v_tiles, x_tiles: device fp32 tiles, 16-byte aligned, row-major
 *                  over each operand's labels in string order.
 *   w_keys  : device [w_cap x r_W] int32 (may be NULL when r_W = 0), sorted;
 *   w_tiles : device [w_cap x tile_elems(W)] fp32.
 *   n_w, n_triples: host; written also with TRE_E_CAPACITY.
 *   ws, ws_bytes: device workspace, 256-byte aligned, at least
 *                  tre_execute3_workspace_bytes(...) (0 on bad arguments).
 *   timing  : optional (deferred mode as for tre_contract: the fused
 *             contraction kernel only); join_ms covers
 *             validation, the triple join and the output keys, units_ms is
 *             empty (each workgroup finds its range of triples itself),
 *             contract_ms the fused contraction kernel, reduce_ms the sum of
 *             output blocks split between workgroups (none in the masked
 *             form) and the key write-out; join_path 6 (partners indexed by
 *             key value) or 0 (searched).
 * When V and X each hold every key of their label's range (n_v and n_x equal
 * the number of tiles along a and b), every U tuple is a triple whose
 * partners are its own key values: no search and no triple count to read
 * back.  Synchronizes the stream twice (triple count, output key count) when
 * searching, once (output key count) otherwise, and once at the end in the
 * masked form without search, whose outputs are then written before the key
 * checks are read (their contents are unspecified when a key error is
 * returned).  Key errors as TRE_E_UNSORTED / TRE_E_DUPKEY / TRE_E_KEYRANGE. */
size_t tre_execute3_workspace_bytes(const char *einsum, const char *upper, const int64_t *extent,
                                    const int32_t *tile, int64_t n_u);
tre_status tre_execute3(const char *einsum, const char *upper, const int64_t *extent, const int32_t *tile,
                        int32_t in_dtype, const int32_t *u_keys, int64_t n_u, const void *u_tiles,
                        const int32_t *v_keys, int64_t n_v, const void *v_tiles, const int32_t *x_keys,
                        int64_t n_x, const void *x_tiles, int32_t *w_keys, float *w_tiles, int64_t w_cap,
                        int64_t *n_w, int64_t *n_triples, void *ws, size_t ws_bytes, void *stream,
                        tre_timing *timing);

/* --- input preparation --------------------------------------------------- */

/* Materialise tiles from scalar entries: tiles[slot[e] * tile_elems + offset[e]]
 * = value[e] after zero-filling n_tiles tiles.  slot/offset device int64,
 * value device (elem_bytes = 2 for bf16 bits or 4 for fp32).  Entries must
 * address distinct positions (else the last writer is unspecified). */
tre_status tre_tiles_from_entries(const int64_t *slot, const int64_t *offset, const void *value, int64_t n_entries,
                                  int32_t elem_bytes, void *tiles, int64_t n_tiles, int64_t tile_elems, void *stream);

/* --- errors -------------------------------------------------------------- */
const char *tre_status_str(tre_status s);
const char *tre_last_error(void);
const char *tre_version(void);

#ifdef __cplusplus
}
#endif

#endif /* TRE_H */
