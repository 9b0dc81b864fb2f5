"""Host-side choice of the decomposition: the sparsity-aware cost model of
Sec. 7 and the dynamic programme of Sec. 8 (Algorithm ComputeMinCostForTree).

This is host logic only (no device work): it ranks, for a tree of binary
EinSums, the choices of promoted labels of every EinSum and returns the
cheapest ones, which the library then executes as written (a promoted label
takes a tile of 1, a demoted one its whole extent).

Plan space.  One promoted set P per EinSum over its labels, each promoted
label with a tile size (1, the paper's promotion, or a candidate size given
with the statistics; a label split as l = t L + l' is the paper's model on
the reshaped tensor), so that U, V and W are decomposed by P restricted to
their labels: a label shared by two
operands has one case in the whole EinSum, the consistency Algorithm 1
requires between W and its inputs extended to the contracted labels (which
the library also requires).  Input tensors are taken in whatever
decomposition their consumer uses (their cost table is 0 for every
decomposition, Sec. 8); an EinSum result whose decomposition differs from
its consumer's is repartitioned (C_repart).

Statistics.  Every tensor has T (non-zero count) and V(l) (non-empty slices
along label l), Sec. 7.1, and for a label l with candidate tile sizes t, V_t(l)
(non-empty slices of t consecutive indices).  For an EinSum result they are estimated from its
inputs' by the classical relational estimators on the purely relational form
(Algorithm GetStats): the join size T_U T_V / prod max(V_U(l), V_V(l)) over
the shared labels, the group count bounded by the product of the output
labels' value counts, and V(l) of the output taken from the input(s) holding
l (the smaller one for a shared label), capped by the output's T.

Costs (seconds).  With c_xfer per byte, c_flop per kernel flop and c_fixed
per tuple:
  T(P)      = n(P) (1 - exp(-T / n(P))),  n(P) = prod_{l in P} V(l)   (Eq. eqn-count)
  T_join    = T(P_U) T(P_V) / prod_{l in P_U and P_V} max(V_U(l), V_V(l))
  C_join    = T_join [(sizeof U + sizeof V) c_xfer + flops(K) c_flop + c_fixed]
  T_agg     = min(T_join / 2, prod_{l in P_W} (min(V_U, V_V) if shared, else the holder's V))
  C_agg     = (T_join - T_agg) [sizeof W c_xfer + C_add + c_fixed]
  C_repart  = (2 T(P_in u P) - T(P_in) - T(P)) [sizeof W_int c_xfer + c_fixed]
V(l) in these terms is V_t(l) at the label's tile size, and C_repart's
intermediate takes the smaller tile of a label promoted on both sides.
sizeof of a tuple = 4 bytes per promoted label + its tile (element bytes x
the tile extents: t for a promoted label, the extent for a demoted one);
flops(K) = 2 x the product of the tile extents of every label of U and V
(the dense tile contraction);
C_add, which the paper leaves undefined, is read as one flop per element of
a W tile.  A choice whose kernel call (one U, V and W tile) exceeds
``max_call_bytes`` is excluded (the memory constraint of Sec. 8).

One term is added to the paper's model: ``c_call``, a fixed latency per
EinSum and per repartition (kernel launches and the count read-backs of one
library call).  The paper's constants are per tuple and per byte, which on
a cluster dominate; on one GPU a small EinSum costs about one such latency
whatever its tuples, so plans that repartition more are slower than the
per-tuple terms say.  With ``c_call = 0`` (the default) the model is the
paper's.
"""
from __future__ import annotations

import heapq
import itertools
import math
from dataclasses import dataclass, field

PEAK_HBM_BYTES_S = 8.0e12
PEAK_FLOPS = {"f32": 157.3e12, "bf16": 2516.6e12}
KEY_BYTES = 4


@dataclass
class Stats:
    """A tensor's label string (in storage order), extents, non-zero count
    T, per-label non-empty slice counts V(l), element bytes, and optionally
    per label {t: V_t(l)} for candidate tile sizes t > 1."""
    labels: str
    extents: dict
    nnz: float
    distinct: dict
    elem_bytes: int = 4
    tiled: dict = field(default_factory=dict)

    def v(self, l: str, t: int = 1) -> float:
        return float(self.distinct[l]) if t == 1 else float(self.tiled[l][t])

    def tiles_of(self, l: str):
        """Tile sizes a promoted l may take: 1 and the candidates below its extent."""
        return [1] + sorted(t for t in self.tiled.get(l, {}) if 1 < t < self.extents[l])


@dataclass
class Costs:
    c_xfer: float
    c_flop: float
    c_fixed: float
    max_call_bytes: float = math.inf
    c_call: float = 0.0
    c_block: float = 0.0  # seconds per flop of one workgroup (a 64 x 64 block of a W tile)

    @classmethod
    def mi355x(cls, dtype: str = "f32", c_fixed: float = 2e-10, max_call_bytes: float = math.inf,
               c_call: float = 0.0, c_block: float = 0.0) -> "Costs":
        """c_xfer from the HBM bandwidth, c_flop from the dense peak of the
        kernel's input type, c_fixed a measured per-tuple overhead, c_call a
        measured per-call latency, c_block the time per flop of one of the
        two workgroups sharing a CU (2 x 256 / the dense peak on MI355X, see
        block_rate)."""
        return cls(1.0 / PEAK_HBM_BYTES_S, 1.0 / PEAK_FLOPS[dtype], c_fixed, max_call_bytes, c_call, c_block)

    @staticmethod
    def block_rate(dtype: str = "f32", cus: int = 256) -> float:
        """c_block for MI355X: one of two resident workgroups of one CU."""
        return 2.0 * cus / PEAK_FLOPS[dtype]


@dataclass
class EinSum:
    """One binary EinSum vertex: ``einsum`` "U,V->W" over its own letters,
    and the names of its two inputs (input tensors or earlier EinSums,
    matched to U and V position by position)."""
    name: str
    einsum: str
    left: str
    right: str

    def operands(self):
        lhs, w = self.einsum.split("->")
        u, v = lhs.split(",")
        return u, v, w


@dataclass
class Program:
    inputs: dict                      # name -> Stats
    einsums: list                     # EinSum in topological order; each result used once
    out_elem_bytes: int = 4           # EinSum results are fp32

    def consumers(self):
        c = {}
        for e in self.einsums:
            for side, src in ((0, e.left), (1, e.right)):
                if src in c:
                    raise ValueError(f"{src} is used more than once: split the program into trees first")
                c[src] = (e.name, side)
        return c


# ------------------------------------------------------------ statistics

def tuples(st: Stats, promoted) -> float:
    """Eq. eqn-count: expected non-empty tuples of the decomposition by
    ``promoted`` ({label: tile}) when the non-zeros are spread uniformly."""
    n = 1.0
    for l, t in promoted.items():
        n *= st.v(l, t)
    if st.nnz <= 0:
        return 0.0
    return n * (1.0 - math.exp(-st.nnz / n))


def result_stats(su: Stats, sv: Stats, e: EinSum, elem_bytes: int) -> Stats:
    """Classical estimates for the result of E over the purely relational
    form: join size, group count, per-label value counts (per tile size
    too, from the input(s) holding the label)."""
    u, v, w = e.operands()
    vu = {l: su.v(su.labels[i]) for i, l in enumerate(u)}
    vv = {l: sv.v(sv.labels[i]) for i, l in enumerate(v)}
    tu = {l: su.tiled.get(su.labels[i], {}) for i, l in enumerate(u)}
    tv = {l: sv.tiled.get(sv.labels[i], {}) for i, l in enumerate(v)}
    ext = {}
    for i, l in enumerate(u):
        ext[l] = su.extents[su.labels[i]]
    for i, l in enumerate(v):
        ext[l] = sv.extents[sv.labels[i]]
    shared = set(u) & set(v)
    denom = 1.0
    for l in shared:
        denom *= max(vu[l], vv[l])
    t_join = su.nnz * sv.nnz / denom
    vals, tiled = {}, {}
    for l in w:
        if l in vu and l in vv:
            vals[l] = min(vu[l], vv[l])
            tiled[l] = {t: min(tu[l][t], tv[l][t]) for t in tu[l] if t in tv[l]}
        else:
            vals[l] = vu[l] if l in vu else vv[l]
            tiled[l] = dict(tu[l] if l in vu else tv[l])
    groups = 1.0
    for l in w:
        groups *= vals[l]
    nnz = min(t_join, groups)
    return Stats(w, {l: ext[l] for l in w}, nnz, {l: min(vals[l], nnz) for l in w}, elem_bytes,
                 {l: {t: min(x, nnz) for t, x in tiled[l].items()} for l in w if tiled[l]})


def _restrict(st: Stats, P) -> dict:
    """The part of plan set P ({label: tile}) on st's labels."""
    return {l: P[l] for l in st.labels if l in P}


def tile_bytes(st: Stats, promoted) -> float:
    b = st.elem_bytes
    for l in st.labels:
        b *= promoted[l] if l in promoted else st.extents[l]
    return b


def tuple_bytes(st: Stats, promoted) -> float:
    return KEY_BYTES * len([l for l in st.labels if l in promoted]) + tile_bytes(st, promoted)


# ----------------------------------------------------------------- costs

def local_cost(su: Stats, sv: Stats, sw: Stats, P: dict, c: Costs) -> float:
    """C_join + C_agg of one EinSum whose operands' labels are already in the
    EinSum's own letters (su.labels = U's string, ...), promoted labels and
    their tiles P ({label: tile})."""
    pu, pv, pw = _restrict(su, P), _restrict(sv, P), _restrict(sw, P)
    call = tile_bytes(su, pu) + tile_bytes(sv, pv) + tile_bytes(sw, pw)
    if call > c.max_call_bytes:
        return math.inf
    denom = 1.0
    for l in set(pu) & set(pv):
        denom *= max(su.v(l, P[l]), sv.v(l, P[l]))
    t_join = tuples(su, pu) * tuples(sv, pv) / denom
    flops = 2.0
    for l in set(su.labels) | set(sv.labels):
        flops *= P[l] if l in P else (su.extents[l] if l in su.extents else sv.extents[l])
    c_join = t_join * ((tuple_bytes(su, pu) + tuple_bytes(sv, pv)) * c.c_xfer + flops * c.c_flop + c.c_fixed)
    groups = 1.0
    for l, t in pw.items():
        if l in su.distinct and l in sv.distinct:
            groups *= min(su.v(l, t), sv.v(l, t))
        else:
            groups *= su.v(l, t) if l in su.distinct else sv.v(l, t)
    t_agg = min(t_join / 2.0, groups)
    add = tile_bytes(sw, pw) / sw.elem_bytes  # elements of a W tile
    c_agg = (t_join - t_agg) * (tuple_bytes(sw, pw) * c.c_xfer + add * c.c_flop + c.c_fixed)
    # the span: one pair's kernel is the smallest piece of work, shared by the
    # workgroups of its W tile's 64 x 64 blocks (an added term, 0 = the paper)
    span = c.c_block * flops / max(1.0, add / 4096.0) if t_join > 0 else 0.0
    return c_join + c_agg + c.c_call + span


def repart_cost(st: Stats, p_in: dict, p_out: dict, c: Costs) -> float:
    """C_repart from promoted set p_in to p_out ({label: tile}) of the same
    tensor; the intermediate promotes every label of either, at the smaller
    tile where both promote it."""
    if p_in == p_out:
        return 0.0
    both = dict(p_in)
    for l, t in p_out.items():
        both[l] = min(t, both[l]) if l in both else t
    n_int = 2.0 * tuples(st, both) - tuples(st, p_in) - tuples(st, p_out)
    return n_int * (tuple_bytes(st, both) * c.c_xfer + c.c_fixed) + c.c_call


def _renamed(st: Stats, letters: str) -> Stats:
    """The same statistics under the consumer's letters (position by position)."""
    m = dict(zip(st.labels, letters))
    return Stats(letters, {m[l]: x for l, x in st.extents.items()}, st.nnz,
                 {m[l]: x for l, x in st.distinct.items()}, st.elem_bytes,
                 {m[l]: dict(x) for l, x in st.tiled.items()})


def _choices(su: Stats, sv: Stats, labels):
    """Every promoted set of the EinSum: each label demoted or promoted at one
    of its tile sizes (for a label of both inputs, sizes both have stats for)."""
    opts = []
    for l in labels:
        if l in su.distinct and l in sv.distinct:
            ts = [t for t in su.tiles_of(l) if t in sv.tiles_of(l)]
        else:
            ts = (su if l in su.distinct else sv).tiles_of(l)
        opts.append([None] + ts)
    for combo in itertools.product(*opts):
        yield {l: t for l, t in zip(labels, combo) if t is not None}


def _key(P: dict, letters) -> frozenset:
    return frozenset((l, t) for l, t in P.items() if l in letters)


# ------------------------------------------------------ dynamic programme

@dataclass(order=True)
class _Entry:
    cost: float
    plan: tuple = field(compare=False)  # ((einsum name, promoted {label: tile}), ...) of the subtree


def optimize(prog: Program, costs: Costs, k: int = 1):
    """The k cheapest plans of the program: a list of (cost, {EinSum name:
    {promoted label: tile}} in the EinSum's letters), cheapest first.  Each
    vertex keeps, per promoted set (with tiles) of its output, its k cheapest
    subtrees (Algorithm ComputeMinCostForTree with k-best lists); the root's
    lists are merged."""
    prog.consumers()  # checks the tree property
    stats = dict(prog.inputs)
    table = {}  # EinSum name -> {frozenset(promoted W labels in W letters): [entries]}
    for e in prog.einsums:
        u, v, w = e.operands()
        su = _renamed(stats[e.left], u)
        sv = _renamed(stats[e.right], v)
        sw = result_stats(su, sv, e, prog.out_elem_bytes)
        stats[e.name] = sw
        sw = _renamed(sw, w)
        best = {}
        for P in _choices(su, sv, list(dict.fromkeys(u + v))):
            local = local_cost(su, sv, sw, P, costs)
            if math.isinf(local):
                continue
            sides = []
            for src, st, letters in ((e.left, su, u), (e.right, sv, v)):
                need = {l: P[l] for l in letters if l in P}
                if src not in table:  # input tensor: taken in this decomposition
                    sides.append([_Entry(0.0, ())])
                    continue
                cands = []
                m = dict(zip(stats[src].labels, letters))
                for p_in, entries in table[src].items():
                    r = repart_cost(st, {m[l]: t for l, t in p_in}, need, costs)
                    for en in entries:
                        cands.append(_Entry(en.cost + r, en.plan))
                sides.append(heapq.nsmallest(k, cands))
            combos = heapq.nsmallest(k, (_Entry(a.cost + b.cost + local, a.plan + b.plan + ((e.name, P),))
                                         for a in sides[0] for b in sides[1]))
            key = _key(P, w)
            best[key] = heapq.nsmallest(k, best.get(key, []) + combos)
        table[e.name] = best
    root = prog.einsums[-1].name
    final = heapq.nsmallest(k, (en for entries in table[root].values() for en in entries))
    return [(en.cost, {name: dict(sorted(P.items())) for name, P in en.plan}) for en in final]


def _as_tiles(p) -> dict:
    """{label: tile} from a plan entry given as such a dict or as a string
    (or set) of promoted labels, each with a tile of 1."""
    return dict(p) if isinstance(p, dict) else {l: 1 for l in p}


def plan_cost(prog: Program, costs: Costs, plan: dict) -> float:
    """Total cost of one given plan ({EinSum name: {promoted label: tile}},
    or promoted label strings for tiles of 1)."""
    stats = dict(prog.inputs)
    out_p = {}
    total = 0.0
    for e in prog.einsums:
        u, v, w = e.operands()
        su = _renamed(stats[e.left], u)
        sv = _renamed(stats[e.right], v)
        sw0 = result_stats(su, sv, e, prog.out_elem_bytes)
        stats[e.name] = sw0
        P = _as_tiles(plan[e.name])
        total += local_cost(su, sv, _renamed(sw0, w), P, costs)
        for src, st, letters in ((e.left, su, u), (e.right, sv, v)):
            if src in out_p:
                m = dict(zip(stats[src].labels, letters))
                total += repart_cost(st, {m[l]: t for l, t in out_p[src].items()},
                                     {l: P[l] for l in letters if l in P}, costs)
        out_p[e.name] = {l: P[l] for l in w if l in P}
    return total


# ------------------------------------------------------- statistics from data

def stats_from_coo(labels: str, extents: dict, coords, elem_bytes: int = 4, tiles: dict | None = None) -> Stats:
    """T, V(l) and V_t(l) of a tensor from its non-zero coordinates ([nnz x d]
    ints, one column per label in ``labels``): the GetStats counts, computed
    directly; ``tiles`` gives candidate tile sizes per label."""
    import numpy as np

    coords = np.asarray(coords)
    tiled = {}
    for i, l in enumerate(labels):
        for t in (tiles or {}).get(l, []):
            if t > 1:
                tiled.setdefault(l, {})[t] = float(len(np.unique(coords[:, i] // t))) if len(coords) else 0.0
    return Stats(labels, dict(extents), float(len(coords)),
                 {l: float(len(np.unique(coords[:, i]))) if len(coords) else 0.0 for i, l in enumerate(labels)},
                 elem_bytes, tiled)
