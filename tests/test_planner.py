"""The decomposition planner (Sec. 7 cost model, Sec. 8 dynamic programme).

The oracle (oracle/planner.py) evaluates the cost model on every plan of a
small program; its pieces are pinned here against data and hand counts:
Eq. eqn-count against the stored tiles of a generated graph and against a
simulated sparse tensor, the join estimate against real join sizes of
uniform random relations, and the join / aggregation / repartition terms
against hand-counted cases.  The planner's dynamic programme must then find
exactly the oracle's cheapest plans.

The oracle holds only the paper's model.  The product planner adds two terms
of its own (a per-call latency c_call and a span term c_block, both 0 by
default); every comparison with the oracle runs them at 0, and the two terms
are pinned separately by hand counts against the product alone."""
import math

import numpy as np
import pytest

import workloads
from oracle import planner as op


def _costs(c_xfer=1e-12, c_flop=1e-14, c_fixed=1e-9, cap=math.inf):
    return {"c_xfer": c_xfer, "c_flop": c_flop, "c_fixed": c_fixed, "max_call_bytes": cap}


# ------------------------------------------------------------- oracle pins

def test_eqn_count_matches_generated_tiles():
    """The fp32 GNN graph (4096 vertices, 8 uniform out-edges each) in 64x64
    tiles: Eq. eqn-count predicts 4094.6 stored tiles of 4096; the generator
    stores 4094."""
    w = workloads.config(1)
    n_tiles = len(w["Y"]["keys"])
    pred = op.eqn_count(w["n_edges"], [64, 64])
    assert abs(pred - 4094.626) < 1e-3
    assert abs(n_tiles - pred) / pred < 2e-3


def test_eqn_count_simulated_sparse_tensor():
    """Non-zeros placed uniformly in a 40 x 30 x 50 tensor: the number of
    non-empty (i, j) slices averages n (1 - exp(-T / n)) with n = 1200."""
    rng = np.random.default_rng(3)
    a, b, c = 40, 30, 50
    for T in (300, 1200, 5000):
        got = []
        for _ in range(40):
            cells = rng.choice(a * b * c, size=T, replace=False)
            got.append(len(np.unique(cells // c)))
        pred = op.eqn_count(T, [a, b])
        assert abs(np.mean(got) - pred) / pred < 0.01, (T, np.mean(got), pred)


def test_join_estimate_uniform_relations():
    """Two relations whose join attribute is uniform over the same D values:
    the textbook estimate T_U T_V / D is the expected join size."""
    rng = np.random.default_rng(5)
    D, tu, tv = 60, 400, 300
    sizes = []
    for _ in range(200):
        ju = rng.integers(0, D, tu)
        jv = rng.integers(0, D, tv)
        sizes.append(int((np.bincount(ju, minlength=D) * np.bincount(jv, minlength=D)).sum()))
    assert abs(np.mean(sizes) / (tu * tv / D) - 1) < 0.02


def _dense_stats(labels, ext, nnz=1e12, elem=4):
    """A tensor so full that every slice is non-empty: T(P) = n(P)."""
    return {"labels": labels, "extents": dict(ext), "nnz": nnz, "distinct": {l: ext[l] for l in labels},
            "elem_bytes": elem}


def test_cross_product_hand_count():
    """No shared promoted label: the join is the cross product.  U keyed i
    (10 tuples), V keyed k (10 tuples), W = "" (one group): with only a
    per-tuple cost of 1, C_join = 100 and C_agg = 100 - min(50, 1) = 99."""
    tu = _dense_stats("ij", {"i": 10, "j": 3})
    tv = _dense_stats("jk", {"j": 3, "k": 10})
    tw = op.derive("ij", "jk", "", tu, tv)
    cost = op.einsum_cost(tu, tv, tw, {"i", "k"}, _costs(0.0, 0.0, 1.0))
    assert cost == pytest.approx(199.0, rel=1e-12)


def test_join_and_group_hand_count():
    """Shared promoted j with V_U(j) = 10, V_V(j) = 20 and 10 x 20 tuples:
    T_join = 10 * 20 / 20 = 10; groups of W keyed k (V_V(k) = 1): T_agg =
    min(5, 1) = 1.  Per-tuple cost 1: C = 10 + 9 = 19.  Adding 1 per byte:
    U tuples are 4 + 4 * 5 bytes (key j, tile over i), V tuples 2 * 4 + 4
    (keys j and k, a one-element tile), W tuples 4 + 4 * 5 (key k, tile over
    i) -> + 10 * (24 + 12) + 9 * 24 = 595 in all."""
    tu = {"labels": "ij", "extents": {"i": 5, "j": 10}, "nnz": 1e12, "distinct": {"i": 5, "j": 10}, "elem_bytes": 4}
    tv = {"labels": "jk", "extents": {"j": 20, "k": 1}, "nnz": 1e12, "distinct": {"j": 20, "k": 1}, "elem_bytes": 4}
    tw = op.derive("ij", "jk", "ki", tu, tv)
    base = op.einsum_cost(tu, tv, tw, {"j", "k"}, _costs(0.0, 0.0, 1.0))
    assert base == pytest.approx(19.0, rel=1e-12)
    withb = op.einsum_cost(tu, tv, tw, {"j", "k"}, _costs(1.0, 0.0, 1.0))
    assert withb == pytest.approx(19.0 + 10 * 36 + 9 * 24, rel=1e-12)


def test_kernel_flops_and_memory_cap():
    """All labels demoted: one pair whose kernel is the whole 8x6x7 product
    (2 * 336 flops); a cap below the three tiles' bytes excludes it."""
    tu = _dense_stats("ij", {"i": 8, "j": 6})
    tv = _dense_stats("jk", {"j": 6, "k": 7})
    tw = op.derive("ij", "jk", "ik", tu, tv)
    c = op.einsum_cost(tu, tv, tw, set(), _costs(0.0, 1.0, 0.0))
    # one join tuple, one group: T_agg = min(1/2, 1) = 1/2 -> C_add on half a tuple
    assert c == pytest.approx(2 * 8 * 6 * 7 + 0.5 * 8 * 7, rel=1e-12)
    tiles = 4 * (8 * 6 + 6 * 7 + 8 * 7)
    assert op.einsum_cost(tu, tv, tw, set(), _costs(cap=tiles)) < math.inf
    assert op.einsum_cost(tu, tv, tw, set(), _costs(cap=tiles - 1)) == math.inf


def _product_stats(t):
    from paper_2603_08957_amd import planner as pl

    return pl.Stats(t["labels"], t["extents"], t["nnz"], t["distinct"], t["elem_bytes"], t.get("tiled", {}))


def test_per_call_latency_product_hand_count():
    """Product-only term: c_call is charged once per EinSum and once per
    repartition that changes the decomposition, nothing else changes.  Hand
    count on U [i 4][j 3] x V [j 3][k 5] dense, i promoted: the paper's terms
    with c_xfer = c_flop = 0 and c_fixed = 1 are the tuples touched, 4 join
    tuples and (4 - min(2, 4)) = 2 aggregated, 6 in all."""
    from paper_2603_08957_amd import planner as pl

    tu = _dense_stats("ij", {"i": 4, "j": 3})
    tv = _dense_stats("jk", {"j": 3, "k": 5})
    su, sv = _product_stats(tu), _product_stats(tv)
    sw = pl.result_stats(su, sv, pl.EinSum("E", "ij,jk->ik", "U", "V"), 4)
    base = pl.local_cost(su, sv, sw, {"i": 1}, pl.Costs(0.0, 0.0, 1.0))
    assert base == pytest.approx(4 + 2, rel=1e-12)
    assert pl.local_cost(su, sv, sw, {"i": 1}, pl.Costs(0.0, 0.0, 1.0, c_call=7.0)) == pytest.approx(base + 7.0,
                                                                                                      rel=1e-12)
    assert pl.repart_cost(sw, {"i": 1}, {"i": 1}, pl.Costs(0.0, 0.0, 1.0, c_call=7.0)) == 0.0
    r = pl.repart_cost(sw, {"i": 1}, {"k": 1}, pl.Costs(0.0, 0.0, 1.0))
    assert r > 0
    assert pl.repart_cost(sw, {"i": 1}, {"k": 1}, pl.Costs(0.0, 0.0, 1.0, c_call=7.0)) == pytest.approx(r + 7.0,
                                                                                                         rel=1e-12)


def test_span_term_product_hand_count():
    """Product-only term: one pair's kernel flops over the 64 x 64 blocks of
    its W tile, times c_block; none without pairs.  Here U [i 128][j 32] and
    V [j 32][k 256] dense, nothing promoted: one pair, 2*128*32*256 flops, a
    W tile of 128 x 256 = 8 blocks; with j promoted at a tile of 8 there are
    4 pairs of 2*128*8*256 flops and the same 8 blocks."""
    from paper_2603_08957_amd import planner as pl

    tu = dict(_dense_stats("ij", {"i": 128, "j": 32}), tiled={"j": {8: 4}})
    tv = dict(_dense_stats("jk", {"j": 32, "k": 256}), tiled={"j": {8: 4}})
    su, sv = _product_stats(tu), _product_stats(tv)
    sw = pl.result_stats(su, sv, pl.EinSum("E", "ij,jk->ik", "U", "V"), 4)
    for prom, flops in (({}, 2 * 128 * 32 * 256), ({"j": 8}, 2 * 128 * 8 * 256)):
        c0 = pl.local_cost(su, sv, sw, prom, pl.Costs(1e-12, 1e-14, 1e-9))
        c1 = pl.local_cost(su, sv, sw, prom, pl.Costs(1e-12, 1e-14, 1e-9, c_block=1e-9))
        assert c1 - c0 == pytest.approx(1e-9 * flops / 8, rel=1e-12)
    assert pl.Costs.block_rate("f32") == pytest.approx(512 / 157.3e12)


def test_product_terms_zero_is_the_papers_model():
    """With c_call = c_block = 0 the product prices every EinSum and
    repartition as the oracle does (hand-built cases of each kind)."""
    from paper_2603_08957_amd import planner as pl

    c = _costs(3e-12, 2e-14, 5e-9)
    C = pl.Costs(c["c_xfer"], c["c_flop"], c["c_fixed"])
    tu = dict(_dense_stats("ij", {"i": 128, "j": 32}), tiled={"j": {8: 4}})
    tv = dict(_dense_stats("jk", {"j": 32, "k": 256}), tiled={"j": {8: 4}})
    tw = op.derive("ij", "jk", "ik", tu, tv)
    su, sv = _product_stats(tu), _product_stats(tv)
    sw = pl.result_stats(su, sv, pl.EinSum("E", "ij,jk->ik", "U", "V"), 4)
    for prom in ({}, {"i": 1}, {"j": 8}, {"i": 1, "k": 1}, {"i": 1, "j": 1, "k": 1}):
        assert pl.local_cost(su, sv, sw, prom, C) == pytest.approx(op.einsum_cost(tu, tv, tw, prom, c), rel=1e-12)
    for a, b in (({"i": 1}, {"k": 1}), ({}, {"i": 1, "k": 1}), ({"i": 1}, {"i": 1})):
        assert pl.repart_cost(sw, a, b, C) == pytest.approx(op.repart(tw, a, b, c), rel=1e-12)


def test_repart_properties():
    t = {"labels": "abc", "extents": {"a": 9, "b": 7, "c": 5}, "nnz": 120.0, "distinct": {"a": 9, "b": 7, "c": 5},
         "elem_bytes": 4}
    p = _costs()
    assert op.repart(t, {"a"}, {"a"}, p) == 0.0
    for x, y in (({"a"}, {"b"}), ({"a"}, {"a", "c"}), (set(), {"a", "b", "c"})):
        assert op.repart(t, x, y, p) > 0
        assert op.repart(t, x, y, p) == pytest.approx(op.repart(t, y, x, p), rel=1e-12)
    # moving to a superset creates T(union) - T(in) tuples and aggregates none away beyond T(out)
    p1 = _costs(0.0, 0.0, 1.0)
    want = 2 * op.eqn_count(120, [9, 7]) - op.eqn_count(120, [9]) - op.eqn_count(120, [9, 7])
    assert op.repart(t, {"a"}, {"a", "b"}, p1) == pytest.approx(want, rel=1e-12)


# ---------------------------------------------------- planner vs the oracle

def _rand_tensor(rng, labels, ext, tiles=None):
    """Random statistics; ``tiles`` maps a label to candidate tile sizes
    (V_t drawn between V / t and min(V, extent / t))."""
    cells = 1
    for l in labels:
        cells *= ext[l]
    nnz = float(rng.integers(1, cells + 1))
    distinct = {l: float(rng.integers(max(1, int(ext[l] * 0.3)), ext[l] + 1)) for l in labels}
    tiled = {}
    for l in labels:
        for t in (tiles or {}).get(l, []):
            lo, hi = math.ceil(distinct[l] / t), min(distinct[l], ext[l] // t)
            tiled.setdefault(l, {})[t] = float(rng.integers(lo, max(lo, hi) + 1))
    return {"labels": labels, "extents": {l: ext[l] for l in labels}, "nnz": nnz, "distinct": distinct,
            "elem_bytes": int(rng.choice([2, 4])), "tiled": tiled}


def _rand_program(rng, with_tiles=False):
    """A chain of 1-3 binary EinSums over 2-3 labels per operand; the next
    EinSum consumes the previous result on the left or the right.  With
    ``with_tiles`` the extents are multiples of 4 and some labels carry
    candidate tile sizes 2 and 4."""
    letters = list("abcdefgh")
    if with_tiles:
        ext = {l: 4 * int(rng.integers(1, 10)) for l in letters}
        cand = {l: [2, 4] for l in letters if rng.random() < 0.5}
    else:
        ext = {l: int(rng.integers(2, 40)) for l in letters}
        cand = {}
    rng.shuffle(letters)
    n_e = int(rng.integers(1, 4 if not with_tiles else 3))
    inputs, einsums = {}, []
    u = "".join(letters[:2])
    cur = "x0"
    inputs["x0"] = _rand_tensor(rng, u, ext, cand)
    cur_labels = u
    pool = letters[2:]
    for i in range(n_e):
        shared = cur_labels[int(rng.integers(0, len(cur_labels)))]
        new = pool.pop() if pool else letters[0]
        v = shared + new if rng.random() < 0.5 else new + shared
        if rng.random() < 0.3 and pool:
            v = v + pool.pop()
        keep = [l for l in cur_labels + v if (l != shared or rng.random() < 0.3)]
        w = "".join(dict.fromkeys(keep))
        w = "".join(rng.permutation(list(w)))
        name_v = f"y{i}"
        inputs[name_v] = _rand_tensor(rng, v, ext, cand)
        if rng.random() < 0.5:
            einsums.append((f"e{i}", f"{cur_labels},{v}->{w}", cur, name_v))
        else:
            einsums.append((f"e{i}", f"{v},{cur_labels}->{w}", name_v, cur))
        cur, cur_labels = f"e{i}", w
    return {"inputs": inputs, "einsums": einsums}


def _to_product(prog, c, c_call=0.0, c_block=0.0):
    """The program and costs for the product planner; c_call and c_block
    are the product's own terms (0 = the paper's model, the oracle's)."""
    from paper_2603_08957_amd import planner as pl

    inputs = {k: pl.Stats(t["labels"], t["extents"], t["nnz"], t["distinct"], t["elem_bytes"], t.get("tiled", {}))
              for k, t in prog["inputs"].items()}
    einsums = [pl.EinSum(n, e, a, b) for n, e, a, b in prog["einsums"]]
    return pl.Program(inputs, einsums), pl.Costs(c["c_xfer"], c["c_flop"], c["c_fixed"], c["max_call_bytes"],
                                                 c_call, c_block)


@pytest.mark.parametrize("seed", range(60))
def test_planner_matches_exhaustive_search(seed):
    """The dynamic programme's k = 4 cheapest plans have the oracle's four
    smallest costs, and the oracle prices each of them the same."""
    from paper_2603_08957_amd import planner as pl

    rng = np.random.default_rng(900 + seed)
    prog = _rand_program(rng)
    cap = math.inf if seed % 3 else float(rng.integers(200, 20000))
    c = _costs(10 ** rng.uniform(-13, -10), 10 ** rng.uniform(-15, -12), 10 ** rng.uniform(-11, -8), cap)
    want = op.best_plans(prog, c, k=4)
    P, C = _to_product(prog, c)
    got = pl.optimize(P, C, k=4)
    assert len(got) == len(want)
    for (gc, gplan), (wc, _) in zip(got, want):
        assert gc == pytest.approx(wc, rel=1e-9)
        assert op.total_cost(prog, gplan, c) == pytest.approx(gc, rel=1e-9)
        assert pl.plan_cost(P, C, gplan) == pytest.approx(gc, rel=1e-9)


@pytest.mark.parametrize("seed", range(30))
def test_planner_with_tiles_matches_exhaustive_search(seed):
    """Labels with candidate tile sizes: each EinSum picks, per label,
    demoted or promoted at tile 1, 2 or 4; the dynamic programme still
    finds the oracle's four cheapest plans."""
    from paper_2603_08957_amd import planner as pl

    rng = np.random.default_rng(7100 + seed)
    prog = _rand_program(rng, with_tiles=True)
    cap = math.inf if seed % 3 else float(rng.integers(200, 20000))
    c = _costs(10 ** rng.uniform(-13, -10), 10 ** rng.uniform(-15, -12), 10 ** rng.uniform(-11, -8), cap)
    want = op.best_plans(prog, c, k=4)
    P, C = _to_product(prog, c)
    got = pl.optimize(P, C, k=4)
    assert len(got) == len(want)
    for (gc, gplan), (wc, _) in zip(got, want):
        assert gc == pytest.approx(wc, rel=1e-9)
        assert op.total_cost(prog, gplan, c) == pytest.approx(gc, rel=1e-9)


@pytest.mark.parametrize("seed", range(30))
def test_planner_with_product_terms_is_exact(seed):
    """With the product's own terms switched on (c_call, c_block) the dynamic
    programme's four cheapest plans are still the four cheapest under the
    product's pricing of whole plans, found by listing every plan (the
    oracle's enumeration supplies the list; the prices are the product's,
    whose extra terms are pinned by the hand counts above)."""
    from paper_2603_08957_amd import planner as pl

    rng = np.random.default_rng(4200 + seed)
    prog = _rand_program(rng, with_tiles=bool(seed % 2))
    c = _costs(10 ** rng.uniform(-13, -10), 10 ** rng.uniform(-15, -12), 10 ** rng.uniform(-11, -8))
    P, C = _to_product(prog, c, 10 ** rng.uniform(-6, -3), 10 ** rng.uniform(-13, -10))
    priced = sorted(pl.plan_cost(P, C, plan) for plan in op.all_plans(prog))
    priced = [x for x in priced if not math.isinf(x)][:4]
    got = pl.optimize(P, C, k=4)
    assert [g for g, _ in got] == pytest.approx(priced, rel=1e-9)


def test_tiled_count_matches_generated_tiles():
    """The 4096-vertex graph's adjacency at tile 64 on both labels: the
    tiled statistics (64 non-empty 64-slices per label) give Eq. eqn-count's
    4094.6 tuples, the generator stores 4094 tiles."""
    from paper_2603_08957_amd import planner as pl

    w = workloads.config(1, y_layout="jk")
    st = pl.stats_from_coo("jk", {"j": 4096, "k": 4096}, w["Y"]["coo"][0], 4, {"j": [64], "k": [64]})
    assert st.v("j", 64) == 64 and st.v("k", 64) == 64
    t = {"labels": "jk", "extents": st.extents, "nnz": st.nnz, "distinct": st.distinct, "tiled": st.tiled,
         "elem_bytes": 4}
    assert op.count(t, {"j": 64, "k": 64}) == pytest.approx(op.eqn_count(32768, [64, 64]), rel=1e-12)
    assert abs(len(w["Y"]["keys"]) - op.count(t, {"j": 64, "k": 64})) < 1.0
    # tile-1 counts are the distinct-coordinate counts
    assert op.count(t, {"j": 1}) == pytest.approx(op.eqn_count(32768, [st.v("j")]), rel=1e-12)


def test_tiled_kernel_and_tuple_sizes():
    """A label promoted at tile t contributes t to the kernel's extents and
    to the tile bytes, and one key attribute."""
    tu = {"labels": "ij", "extents": {"i": 8, "j": 12}, "nnz": 1e12, "distinct": {"i": 8, "j": 12},
          "tiled": {"j": {4: 3}}, "elem_bytes": 4}
    tv = {"labels": "jk", "extents": {"j": 12, "k": 5}, "nnz": 1e12, "distinct": {"j": 12, "k": 5},
          "tiled": {"j": {4: 3}}, "elem_bytes": 4}
    tw = op.derive("ij", "jk", "ik", tu, tv)
    assert op.row_bytes(tu, {"j": 4}) == 4 + 4 * 8 * 4
    # 3 x 3 / 3 = 3 join tuples of a 2 * 8 * 4 * 5-flop kernel; one group
    # (W has no promoted label), T_agg = min(3 / 2, 1) = 1, so 2 adds of an
    # 8 x 5 tile
    c = op.einsum_cost(tu, tv, tw, {"j": 4}, _costs(0.0, 1.0, 0.0))
    assert c == pytest.approx(3 * 2 * 8 * 4 * 5 + (3 - 1) * 8 * 5, rel=1e-12)


def test_planner_rejects_reused_results():
    from paper_2603_08957_amd import planner as pl

    s = pl.Stats("ij", {"i": 4, "j": 4}, 8.0, {"i": 4, "j": 4})
    prog = pl.Program({"x": s}, [pl.EinSum("a", "ij,jk->ik", "x", "x")])
    with pytest.raises(ValueError):
        pl.optimize(prog, pl.Costs.mi355x())


def test_planner_picks_scalar_adjacency_for_the_large_gcn():
    """The 1,048,576-vertex GNN chain (X 256 x n dense, Y n x n with 33.5M
    edges, Z 256 x 256) with a 256 MB cap on one kernel call: the cheapest
    plan promotes both vertex labels of E1 (the adjacency as scalar tuples,
    the features as per-vertex vectors, the paper's GCN schema), and E2
    keeps the vertex label promoted."""
    from paper_2603_08957_amd import planner as pl

    n, emb = 1 << 20, 256
    X = pl.Stats("ij", {"i": emb, "j": n}, float(emb * n), {"i": emb, "j": n}, 2)
    Y = pl.Stats("jk", {"j": n, "k": n}, 33.5e6, {"j": n, "k": n}, 2)
    Z = pl.Stats("im", {"i": emb, "m": emb}, float(emb * emb), {"i": emb, "m": emb}, 2)
    prog = pl.Program({"X": X, "Y": Y, "Z": Z},
                      [pl.EinSum("E1", "ij,jk->ki", "X", "Y"), pl.EinSum("E2", "ki,im->km", "E1", "Z")])
    best = pl.optimize(prog, pl.Costs.mi355x("bf16", max_call_bytes=256 << 20), k=3)
    cost, plan = best[0]
    assert plan["E1"] == {"j": 1, "k": 1}
    assert "k" in plan["E2"]
    assert all(c >= cost for c, _ in best)


def test_planner_prefers_scalar_adjacency_to_128_tiles():
    """The 262,144-vertex chain with 128x128 tiles allowed for the vertex
    labels (Y's 128-slices all non-empty): the cheapest plan still stores the
    adjacency as scalar tuples, and the 128-tiled split the workload fixes
    costs more than ten times as much under the model."""
    from paper_2603_08957_amd import planner as pl

    n, emb, nb = 1 << 18, 128, (1 << 18) // 128
    X = pl.Stats("ij", {"i": emb, "j": n}, float(emb * n), {"i": emb, "j": n}, 2, {"j": {128: nb}})
    Y = pl.Stats("jk", {"j": n, "k": n}, 4194304.0, {"j": n, "k": n}, 2, {"j": {128: nb}, "k": {128: nb}})
    Z = pl.Stats("im", {"i": emb, "m": emb}, float(emb * emb), {"i": emb, "m": emb}, 2)
    prog = pl.Program({"X": X, "Y": Y, "Z": Z},
                      [pl.EinSum("E1", "ij,jk->ki", "X", "Y"), pl.EinSum("E2", "ki,im->km", "E1", "Z")])
    costs = pl.Costs.mi355x("bf16", max_call_bytes=256 << 20, c_call=1.2e-4)
    cost, plan = pl.optimize(prog, costs, k=1)[0]
    assert plan["E1"] == {"j": 1, "k": 1}
    literal = pl.plan_cost(prog, costs, {"E1": {"j": 128, "k": 128}, "E2": {"k": 128}})
    assert literal > 10 * cost
