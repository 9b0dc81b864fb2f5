"""Oracle for the decomposition planner: the cost model of Sec. 7 evaluated
on every plan of a small program by exhaustive enumeration (no dynamic
programme), so the cheapest plans are known exactly.

TEST INFRASTRUCTURE, NOT PART OF THE PRODUCT (see the package docstring).

A program is a dict:
  {"inputs": {name: {"labels": "ij", "extents": {...}, "nnz": T,
                     "distinct": {label: V}, "elem_bytes": 4}},
   "einsums": [(name, "U,V->W", left name, right name), ...]}   (topological)
A plan assigns every EinSum one set of promoted labels over its letters (a
label has one case in the whole EinSum); U, V and W are decomposed by that
set restricted to their labels.  Inputs come in the decomposition their
consumer uses; an EinSum result consumed in another decomposition pays
C_repart.  Everything follows the formulas printed in Sec. 7 (Eq.
eqn-count for tuple counts, the textbook join estimate, the aggregation
estimate with its three cases, C_join, C_agg, C_repart), with the readings
stated in the planner's documentation: C_add = one flop per W tile element,
flops of the kernel = 2 x the product of all demoted extents of U and V,
a key attribute takes 4 bytes, EinSum results hold 4-byte elements, and
result statistics come from the classical estimators on the purely
relational form (Algorithm GetStats).  The optional per-call latency
``c_call`` (0 unless given) is charged once per EinSum and once per
repartition that changes the decomposition.
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


def _rename(t, letters):
    old = t["labels"]
    return {"labels": letters,
            "extents": {letters[i]: t["extents"][old[i]] for i in range(len(old))},
            "nnz": t["nnz"],
            "distinct": {letters[i]: t["distinct"][old[i]] for i in range(len(old))},
            "elem_bytes": t["elem_bytes"]}


def derive(u, v, w, tu, tv):
    """Statistics of W = U (x) V over the purely relational form: join size by
    the textbook estimate, group count capped by the output labels' value
    counts, value counts from the holder(s) of each label."""
    du, dv = tu["distinct"], tv["distinct"]
    div = 1.0
    for l in u:
        if l in v:
            div = div * max(du[l], dv[l])
    joined = tu["nnz"] * tv["nnz"] / div
    val = {}
    for l in w:
        if l in du and l in dv:
            val[l] = min(du[l], dv[l])
        elif l in du:
            val[l] = du[l]
        else:
            val[l] = dv[l]
    cap = 1.0
    for l in w:
        cap = cap * val[l]
    nnz = joined if joined < cap else cap
    ext = {}
    for l in w:
        ext[l] = tu["extents"][l] if l in tu["extents"] else tv["extents"][l]
    return {"labels": w, "extents": ext, "nnz": nnz, "distinct": {l: min(val[l], nnz) for l in w}, "elem_bytes": 4}


def tile_elems(t, prom):
    e = 1
    for l in t["labels"]:
        if l not in prom:
            e = e * t["extents"][l]
    return e


def row_bytes(t, prom):
    """Bytes of one tuple: 4 per key attribute plus the tile."""
    keys = sum(1 for l in t["labels"] if l in prom)
    return 4 * keys + t["elem_bytes"] * tile_elems(t, prom)


def count(t, prom):
    return eqn_count(t["nnz"], [t["distinct"][l] for l in t["labels"] if l in prom])


def einsum_cost(tu, tv, tw, prom, p):
    """C_join + C_agg (Sec. 7.2) of one EinSum; inf past the memory cap."""
    call = tu["elem_bytes"] * tile_elems(tu, prom) + tv["elem_bytes"] * tile_elems(tv, prom) \
        + tw["elem_bytes"] * tile_elems(tw, prom)
    if call > p["max_call_bytes"]:
        return math.inf
    div = 1.0
    for l in tu["labels"]:
        if l in prom and l in tv["labels"]:
            div = div * max(tu["distinct"][l], tv["distinct"][l])
    t_join = count(tu, prom) * count(tv, prom) / div
    dem = 1
    seen = set()
    for t in (tu, tv):
        for l in t["labels"]:
            if l not in prom and l not in seen:
                seen.add(l)
                dem = dem * t["extents"][l]
    kernel = 2 * dem * p["c_flop"]
    c_join = t_join * ((row_bytes(tu, prom) + row_bytes(tv, prom)) * p["c_xfer"] + kernel + p["c_fixed"])
    groups = 1.0
    for l in tw["labels"]:
        if l not in prom:
            continue
        in_u, in_v = l in tu["distinct"], l in tv["distinct"]
        if in_u and in_v:
            groups = groups * min(tu["distinct"][l], tv["distinct"][l])
        elif in_u:
            groups = groups * tu["distinct"][l]
        else:
            groups = groups * tv["distinct"][l]
    t_agg = min(0.5 * t_join, groups)
    c_add = tile_elems(tw, prom) * p["c_flop"]
    c_agg = (t_join - t_agg) * (row_bytes(tw, prom) * p["c_xfer"] + c_add + p["c_fixed"])
    return c_join + c_agg + p.get("c_call", 0.0)


def repart(t, p_in, p_out, p):
    """C_repart (Sec. 7.2) between two promoted sets of the same tensor."""
    a, b = set(p_in), set(p_out)
    if a == b:
        return 0.0
    union = a | b
    moved = 2 * count(t, union) - count(t, a) - count(t, b)
    return moved * (row_bytes(t, union) * p["c_xfer"] + p["c_fixed"]) + p.get("c_call", 0.0)


def all_plans(prog):
    """Every plan: one promoted set per EinSum over its letters."""
    options = []
    for name, e, _, _ in prog["einsums"]:
        lhs = e.split("->")[0]
        letters = sorted(set(lhs.replace(",", "")))
        subs = []
        for r in range(len(letters) + 1):
            subs.extend(frozenset(c) for c in itertools.combinations(letters, r))
        options.append((name, subs))
    for combo in itertools.product(*[s for _, s in options]):
        yield {options[i][0]: combo[i] for i in range(len(options))}


def total_cost(prog, plan, p):
    """The cost of one plan: every EinSum's C_join + C_agg plus C_repart on
    every EinSum-to-EinSum edge whose decompositions differ."""
    stats = {k: dict(v) for k, v in prog["inputs"].items()}
    produced = {}  # EinSum name -> (its W string, promoted W labels)
    cost = 0.0
    for name, e, left, right in prog["einsums"]:
        lhs, w = e.split("->")
        u, v = lhs.split(",")
        tu = _rename(stats[left], u)
        tv = _rename(stats[right], v)
        tw = derive(u, v, w, tu, tv)
        stats[name] = tw
        prom = plan[name]
        cost += einsum_cost(tu, tv, tw, prom, p)
        for src, letters, t in ((left, u, tu), (right, v, tv)):
            if src in produced:
                src_w, src_prom = produced[src]
                as_mine = {letters[src_w.index(l)] for l in src_prom}
                cost += repart(t, as_mine, {l for l in letters if l in prom}, p)
        produced[name] = (w, {l for l in w if l in prom})
    return cost


def best_plans(prog, p, k=1):
    """The k cheapest (cost, plan) pairs by exhaustive enumeration."""
    scored = [(total_cost(prog, plan, p), plan) for plan in all_plans(prog)]
    scored = [x for x in scored if not math.isinf(x[0])]
    scored.sort(key=lambda x: x[0])
    return scored[:k]
