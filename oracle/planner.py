"""Oracle for the decomposition planner: the cost model of Sec. 7 evaluated
on every plan of a small program by exhaustive enumeration (no dynamic
programme), so the cheapest plans are known exactly.

TEST INFRASTRUCTURE, NOT PART OF THE PRODUCT (see the package docstring).

A program is a dict:
  {"inputs": {name: {"labels": "ij", "extents": {...}, "nnz": T,
                     "distinct": {label: V}, "elem_bytes": 4,
                     "tiled": {label: {t: V_t}}   (optional)}},
   "einsums": [(name, "U,V->W", left name, right name), ...]}   (topological)
A plan gives every EinSum its promoted labels with a tile size each
({label: t}; t = 1 is the paper's promotion, t > 1 splits the label as
t L + l', the paper's model on the reshaped tensor); a label has one case
and tile in the whole EinSum, and U, V and W are decomposed by that choice
restricted to their labels.  Inputs come in the decomposition their
consumer uses; an EinSum result consumed in another decomposition pays
C_repart.  Everything follows the formulas printed in Sec. 7 (Eq.
eqn-count for tuple counts, the textbook join estimate, the aggregation
estimate with its three cases, C_join, C_agg, C_repart) with V(l) taken at
the label's tile size, and the readings stated in the planner's
documentation: C_add = one flop per W tile element, flops of the kernel = 2
x the product of the tile extents of all labels of U and V, a key attribute
takes 4 bytes, EinSum results hold 4-byte elements, result statistics from
the classical estimators on the purely relational form (Algorithm
GetStats), and a repartition's intermediate at the smaller tile of a label
promoted on both sides.  Only the paper's terms are here: the product
planner's own additions (a per-call latency and a span term) are not part of
Sec. 7 and are checked in the product's tests by hand counts.
"""
from __future__ import annotations

import itertools
import math


def eqn_count(nnz, slice_counts):
    """Eq. eqn-count: n (1 - exp(-T / n)), n = product of the slice counts."""
    n = 1.0
    for x in slice_counts:
        n = n * x
    if nnz <= 0:
        return 0.0
    return n * (1.0 - math.exp(-nnz / n))


def _vt(t, l, size):
    """V of label l at tile size ``size``."""
    if size == 1:
        return t["distinct"][l]
    return t["tiled"][l][size]


def _rename(t, letters):
    old = t["labels"]
    m = {old[i]: letters[i] for i in range(len(old))}
    return {"labels": letters,
            "extents": {m[l]: x for l, x in t["extents"].items()},
            "nnz": t["nnz"],
            "distinct": {m[l]: x for l, x in t["distinct"].items()},
            "tiled": {m[l]: dict(x) for l, x in t.get("tiled", {}).items()},
            "elem_bytes": t["elem_bytes"]}


def derive(u, v, w, tu, tv):
    """Statistics of W = U (x) V over the purely relational form: join size by
    the textbook estimate, group count capped by the output labels' value
    counts, value counts (per tile size too) from the holder(s) of each
    label."""
    du, dv = tu["distinct"], tv["distinct"]
    div = 1.0
    for l in u:
        if l in v:
            div = div * max(du[l], dv[l])
    joined = tu["nnz"] * tv["nnz"] / div
    val, tiled = {}, {}
    for l in w:
        a, b = tu.get("tiled", {}).get(l, {}), tv.get("tiled", {}).get(l, {})
        if l in du and l in dv:
            val[l] = min(du[l], dv[l])
            tiled[l] = {s: min(a[s], b[s]) for s in a if s in b}
        elif l in du:
            val[l] = du[l]
            tiled[l] = dict(a)
        else:
            val[l] = dv[l]
            tiled[l] = dict(b)
    cap = 1.0
    for l in w:
        cap = cap * val[l]
    nnz = joined if joined < cap else cap
    ext = {}
    for l in w:
        ext[l] = tu["extents"][l] if l in tu["extents"] else tv["extents"][l]
    return {"labels": w, "extents": ext, "nnz": nnz, "distinct": {l: min(val[l], nnz) for l in w},
            "tiled": {l: {s: min(x, nnz) for s, x in tiled[l].items()} for l in w if tiled[l]}, "elem_bytes": 4}


def tile_elems(t, prom):
    e = 1
    for l in t["labels"]:
        e = e * (prom[l] if l in prom else t["extents"][l])
    return e


def row_bytes(t, prom):
    """Bytes of one tuple: 4 per key attribute plus the tile."""
    keys = sum(1 for l in t["labels"] if l in prom)
    return 4 * keys + t["elem_bytes"] * tile_elems(t, prom)


def count(t, prom):
    return eqn_count(t["nnz"], [_vt(t, l, prom[l]) for l in t["labels"] if l in prom])


def einsum_cost(tu, tv, tw, prom, p):
    """C_join + C_agg (Sec. 7.2) of one EinSum; inf past the memory cap.
    ``prom``: {label: tile} (a set means tiles of 1)."""
    if not isinstance(prom, dict):
        prom = {l: 1 for l in prom}
    call = tu["elem_bytes"] * tile_elems(tu, prom) + tv["elem_bytes"] * tile_elems(tv, prom) \
        + tw["elem_bytes"] * tile_elems(tw, prom)
    if call > p["max_call_bytes"]:
        return math.inf
    div = 1.0
    for l in tu["labels"]:
        if l in prom and l in tv["labels"]:
            div = div * max(_vt(tu, l, prom[l]), _vt(tv, l, prom[l]))
    t_join = count(tu, prom) * count(tv, prom) / div
    dem = 1
    seen = set()
    for t in (tu, tv):
        for l in t["labels"]:
            if l not in seen:
                seen.add(l)
                dem = dem * (prom[l] if l in prom else t["extents"][l])
    kernel = 2 * dem * p["c_flop"]
    c_join = t_join * ((row_bytes(tu, prom) + row_bytes(tv, prom)) * p["c_xfer"] + kernel + p["c_fixed"])
    groups = 1.0
    for l in tw["labels"]:
        if l not in prom:
            continue
        in_u, in_v = l in tu["distinct"], l in tv["distinct"]
        if in_u and in_v:
            groups = groups * min(_vt(tu, l, prom[l]), _vt(tv, l, prom[l]))
        elif in_u:
            groups = groups * _vt(tu, l, prom[l])
        else:
            groups = groups * _vt(tv, l, prom[l])
    t_agg = min(0.5 * t_join, groups)
    c_add = tile_elems(tw, prom) * p["c_flop"]
    c_agg = (t_join - t_agg) * (row_bytes(tw, prom) * p["c_xfer"] + c_add + p["c_fixed"])
    return c_join + c_agg


def repart(t, p_in, p_out, p):
    """C_repart (Sec. 7.2) between two decompositions ({label: tile}, or sets
    for tiles of 1) of the same tensor."""
    a = dict(p_in) if isinstance(p_in, dict) else {l: 1 for l in p_in}
    b = dict(p_out) if isinstance(p_out, dict) else {l: 1 for l in p_out}
    if a == b:
        return 0.0
    union = {}
    for l in t["labels"]:
        if l in a and l in b:
            union[l] = min(a[l], b[l])
        elif l in a:
            union[l] = a[l]
        elif l in b:
            union[l] = b[l]
    moved = 2 * count(t, union) - count(t, a) - count(t, b)
    return moved * (row_bytes(t, union) * p["c_xfer"] + p["c_fixed"])


def _sizes(t, l):
    return [1] + sorted(s for s in t.get("tiled", {}).get(l, {}) if 1 < s < t["extents"][l])


def all_plans(prog):
    """Every plan: per EinSum, each label demoted or promoted at one of the
    tile sizes its input statistics hold (both inputs' for a shared label)."""
    stats = {k: v for k, v in prog["inputs"].items()}
    per = []
    for name, e, left, right in prog["einsums"]:
        lhs, w = e.split("->")
        u, v = lhs.split(",")
        tu, tv = _rename(stats[left], u), _rename(stats[right], v)
        stats[name] = derive(u, v, w, tu, tv)
        letters = sorted(set(u) | set(v))
        opts = []
        for l in letters:
            if l in tu["labels"] and l in tv["labels"]:
                ss = [s for s in _sizes(tu, l) if s in _sizes(tv, l)]
            else:
                ss = _sizes(tu if l in tu["labels"] else tv, l)
            opts.append([None] + ss)
        choices = []
        for combo in itertools.product(*opts):
            choices.append({letters[i]: combo[i] for i in range(len(letters)) if combo[i] is not None})
        per.append((name, choices))
    for pick in itertools.product(*[c for _, c in per]):
        yield {per[i][0]: pick[i] for i in range(len(per))}


def total_cost(prog, plan, p):
    """The cost of one plan: every EinSum's C_join + C_agg plus C_repart on
    every EinSum-to-EinSum edge whose decompositions differ."""
    stats = {k: dict(v) for k, v in prog["inputs"].items()}
    produced = {}  # EinSum name -> (its W string, {promoted W label: tile})
    cost = 0.0
    for name, e, left, right in prog["einsums"]:
        lhs, w = e.split("->")
        u, v = lhs.split(",")
        tu = _rename(stats[left], u)
        tv = _rename(stats[right], v)
        tw = derive(u, v, w, tu, tv)
        stats[name] = tw
        prom = plan[name] if isinstance(plan[name], dict) else {l: 1 for l in plan[name]}
        cost += einsum_cost(tu, tv, tw, prom, p)
        for src, letters, t in ((left, u, tu), (right, v, tv)):
            if src in produced:
                src_w, src_prom = produced[src]
                as_mine = {letters[src_w.index(l)]: s for l, s in src_prom.items()}
                cost += repart(t, as_mine, {l: prom[l] for l in letters if l in prom}, p)
        produced[name] = (w, {l: prom[l] for l in w if l in prom})
    return cost


def best_plans(prog, p, k=1):
    """The k cheapest (cost, plan) pairs by exhaustive enumeration."""
    scored = [(total_cost(prog, plan, p), plan) for plan in all_plans(prog)]
    scored = [x for x in scored if not math.isinf(x[0])]
    scored.sort(key=lambda x: x[0])
    return scored[:k]
