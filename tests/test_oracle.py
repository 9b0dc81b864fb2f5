"""Pins for the CPU oracle (no GPU).

Each test ties the oracle to something other than itself: the paper's worked
example (printed values), dense numpy.einsum on brute-force random plans,
SQLite running the paper's join / GROUP BY form, split invariance, closed-form
counts, the three-operand contraction evaluated directly, and torch's bf16
rounding.  A plausible mistake in the oracle (a dropped term, a wrong index or
sign, a transposed operand, a wrong tile offset or key order) fails at least
one of them.
"""
import itertools
import json
import os
import sqlite3

import numpy as np
import pytest

import workloads

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "worked_example.json")


# ------------------------------------------------------------------ helpers
# Dense assembly written independently of the oracle (numpy slicing).

def tile_shape(labels, upper, extents, tiles):
    return [tiles[c] if c in upper else extents[c] for c in labels]


def dense_of(labels, upper, extents, tiles, keys, tile_vals):
    """Full tensor from a relation: tuple with key K puts its tile at
    [K_l*t_l : (K_l+1)*t_l] along every promoted label l."""
    full = np.zeros([extents[c] for c in labels], dtype=np.float64)
    shp = tile_shape(labels, upper, extents, tiles)
    kl = [c for c in labels if c in upper]
    for n in range(len(keys)):
        sl = []
        for c in labels:
            if c in upper:
                K = int(keys[n][kl.index(c)])
                sl.append(slice(K * tiles[c], (K + 1) * tiles[c]))
            else:
                sl.append(slice(0, extents[c]))
        full[tuple(sl)] += np.asarray(tile_vals[n], dtype=np.float64).reshape(shp)
    return full


def vals_f64(rel):
    if rel["dtype"] == "bf16":
        return workloads.bf16_bits_to_f32(rel["tiles"]).astype(np.float64)
    return np.asarray(rel["tiles"], dtype=np.float64)


def plan_of(orc, s):
    return orc.Plan(s["einsum"], s["upper"], s["extents"], s["tiles"])


def split_einsum(e):
    lhs, w = e.split("->")
    u, v = lhs.split(",")
    return u, v, w


def brute_pairs(u_lab, v_lab, w_lab, upper, ukeys, vkeys):
    """Nested-loop join on the shared promoted labels; GROUP BY key of each pair."""
    uk = [c for c in u_lab if c in upper]
    vk = [c for c in v_lab if c in upper]
    wk = [c for c in w_lab if c in upper]
    join = [c for c in uk if c in vk]
    out = []
    for u in range(len(ukeys)):
        for v in range(len(vkeys)):
            if all(ukeys[u][uk.index(c)] == vkeys[v][vk.index(c)] for c in join):
                w = tuple(int(ukeys[u][uk.index(c)]) if c in uk else int(vkeys[v][vk.index(c)]) for c in wk)
                out.append((w, u, v))
    out.sort()
    return [(u, v) for _, u, v in out], sorted({w for w, _, _ in out})


# ---------------------------------------------------------- worked example

@pytest.mark.parametrize("name", ["a_rows_times_cols", "b_columns_times_scalars", "c_outer_products"])
def test_worked_example(orc, name):
    g = json.load(open(GOLDEN))
    d = g["decompositions"][name]
    plan = orc.Plan(d["einsum"], d["upper"], {"i": 4, "j": 4, "k": 4}, d["tiles"])
    U = {"keys": np.array(d["U_keys"], dtype=np.int32).reshape(len(d["U_keys"]), -1),
         "tiles": np.array(d["U_tiles"]), "dtype": "f64"}
    V = {"keys": np.array(d["V_keys"], dtype=np.int32).reshape(len(d["V_keys"]), -1),
         "tiles": np.array(d["V_tiles"]), "dtype": "f64"}
    r = orc.run(plan, U, V)
    assert r.pairs.tolist() == d["pairs"]
    assert r.wkeys.tolist() == d["W_keys"]
    np.testing.assert_allclose(r.acc, np.array(d["W_tiles"]), rtol=0, atol=1e-12)
    assert r.n_outside == 0
    if "scalar_multiplies" in d:
        # every (U entry, V entry) pair that shares j is one multiply when all
        # stored entries (zeros included) are counted: 4 pairs x 4 = 16
        te_u = plan.tile_elems[0]
        assert len(r.pairs) * te_u == d["scalar_multiplies"]
    # the full W of the example
    W = np.array(g["U"]) @ np.array(g["V"])
    for i, k, val in g["W_nonzero"]:
        assert abs(W[i, k] - val) < 1e-12
    assert np.count_nonzero(np.abs(W) > 1e-12) == len(g["W_nonzero"])


# --------------------------------------------------- brute force vs numpy

def random_plan(rng):
    letters = list(rng.choice(list("abcdefghijklmnopqrstuvwxyz"), size=rng.integers(1, 6), replace=False))
    while True:
        u = [c for c in letters if rng.random() < 0.6]
        v = [c for c in letters if rng.random() < 0.6]
        if set(u) | set(v) == set(letters):
            break
    rng.shuffle(u)
    rng.shuffle(v)
    w = [c for c in letters if rng.random() < 0.5]
    rng.shuffle(w)
    ext, til = {}, {}
    upper = ""
    for c in letters:
        ext[c] = int(rng.choice([1, 2, 3, 4, 6]))
        if rng.random() < 0.55:
            upper += c
            divs = [d for d in range(1, ext[c] + 1) if ext[c] % d == 0]
            til[c] = int(rng.choice(divs))
    return "".join(u) + "," + "".join(v) + "->" + "".join(w), upper, ext, til


@pytest.mark.parametrize("seed", range(60))
def test_bruteforce_random_plans(orc, seed):
    rng = np.random.default_rng(1000 + seed)
    e, upper, ext, til = random_plan(rng)
    u_lab, v_lab, w_lab = split_einsum(e)
    plan = orc.Plan(e, upper, ext, til)
    dtype = "bf16" if seed % 3 == 0 else "f32"
    U = workloads.random_relation(rng, u_lab, upper, ext, til, dtype, keep=0.6, zero_frac=0.3)
    V = workloads.random_relation(rng, v_lab, upper, ext, til, dtype, keep=0.6, zero_frac=0.3)
    r = orc.run(plan, U, V)
    # key level against the nested loop
    bp, bk = brute_pairs(u_lab, v_lab, w_lab, upper, U["keys"], V["keys"])
    assert [tuple(p) for p in r.pairs.tolist()] == bp
    assert [tuple(k) for k in r.wkeys.tolist()] == bk
    assert r.n_outside == 0
    # value level against numpy.einsum on the dense tensors
    Ud = dense_of(u_lab, upper, ext, til, U["keys"], vals_f64(U))
    Vd = dense_of(v_lab, upper, ext, til, V["keys"], vals_f64(V))
    ref = np.einsum(f"{u_lab},{v_lab}->{w_lab}", Ud, Vd)
    got = dense_of(w_lab, upper, ext, til, r.wkeys, r.acc)
    np.testing.assert_allclose(got, ref, rtol=1e-12, atol=1e-12)
    # magnitudes: sum of |products| = einsum of |U|, |V|
    magref = np.einsum(f"{u_lab},{v_lab}->{w_lab}", np.abs(Ud), np.abs(Vd))
    np.testing.assert_allclose(dense_of(w_lab, upper, ext, til, r.wkeys, r.mag), magref, rtol=1e-12, atol=1e-12)


def test_batch_matmul_with_transposes(orc):
    """Sec. 3: W_{i,k} = sum_{b,j} U_{i,j,b} V_{j,b,k} with bounds [10,100,20] and
    [100,20,2000] (scaled down 10x along the big labels); labels b and j are both
    aggregated."""
    rng = np.random.default_rng(7)
    ext = {"i": 10, "j": 10, "b": 20, "k": 200}
    for upper, til in [("", {}), ("j", {"j": 5}), ("bk", {"b": 4, "k": 50}), ("ijbk", {"i": 5, "j": 2, "b": 10, "k": 40})]:
        plan = orc.Plan("ijb,jbk->ik", upper, ext, til)
        U = workloads.random_relation(rng, "ijb", upper, ext, til, "f32", keep=0.7)
        V = workloads.random_relation(rng, "jbk", upper, ext, til, "f32", keep=0.7)
        r = orc.run(plan, U, V)
        Ud = dense_of("ijb", upper, ext, til, U["keys"], vals_f64(U))
        Vd = dense_of("jbk", upper, ext, til, V["keys"], vals_f64(V))
        got = dense_of("ik", upper, ext, til, r.wkeys, r.acc)
        np.testing.assert_allclose(got, np.einsum("ijb,jbk->ik", Ud, Vd), rtol=1e-12, atol=1e-12)


# --------------------------------------------------------------- sqlite

@pytest.mark.parametrize("seed", range(12))
def test_sqlite_purely_relational(orc, seed):
    """All labels promoted with tile 1: the oracle must equal the plain SQL
    join / GROUP BY / SUM of Sec. 1 and Sec. 5 run by SQLite."""
    rng = np.random.default_rng(500 + seed)
    e, _, ext, _ = random_plan(rng)
    u_lab, v_lab, w_lab = split_einsum(e)
    used = sorted(set(u_lab) | set(v_lab))
    upper = "".join(used)
    til = {c: 1 for c in used}
    plan = orc.Plan(e, upper, ext, til)
    U = workloads.random_relation(rng, u_lab, upper, ext, til, "f32", keep=0.5)
    V = workloads.random_relation(rng, v_lab, upper, ext, til, "f32", keep=0.5)
    r = orc.run(plan, U, V)
    con = sqlite3.connect(":memory:")
    ucols = [f"{c}_" for c in u_lab]
    vcols = [f"{c}_" for c in v_lab]
    con.execute(f"CREATE TABLE U ({', '.join(c + ' INT' for c in ucols)}{', ' if ucols else ''}uid INT, valU REAL)")
    con.execute(f"CREATE TABLE V ({', '.join(c + ' INT' for c in vcols)}{', ' if vcols else ''}vid INT, valV REAL)")
    for n, (k, t) in enumerate(zip(U["keys"].tolist(), U["tiles"].tolist())):
        con.execute(f"INSERT INTO U VALUES ({', '.join(['?'] * (len(ucols) + 2))})", (*k, n, t[0]))
    for n, (k, t) in enumerate(zip(V["keys"].tolist(), V["tiles"].tolist())):
        con.execute(f"INSERT INTO V VALUES ({', '.join(['?'] * (len(vcols) + 2))})", (*k, n, t[0]))
    wcols = [f"{c}_" for c in w_lab]
    sel = ", ".join(wcols)
    grp = f"GROUP BY {sel}" if wcols else ""
    order = ", ".join(wcols + ["uid", "vid"])
    rows = con.execute(f"SELECT uid, vid FROM U NATURAL JOIN V ORDER BY {order}").fetchall()
    assert [tuple(p) for p in r.pairs.tolist()] == rows
    agg = con.execute(f"SELECT {sel + ', ' if sel else ''}SUM(valU * valV) FROM U NATURAL JOIN V {grp} "
                      f"{'ORDER BY ' + sel if sel else ''}").fetchall()
    if not rows:
        assert len(r.wkeys) == 0
        return
    assert [tuple(x[:-1]) for x in agg] == [tuple(k) for k in r.wkeys.tolist()]
    np.testing.assert_allclose(r.acc[:, 0], [x[-1] for x in agg], rtol=1e-12, atol=1e-12)


@pytest.mark.parametrize("seed", range(8))
def test_sqlite_tile_join(orc, seed):
    """Tile relations: the pair list and key set equal SQLite's natural join of
    the key attributes (tiles replaced by tuple ids), ordered by W's keys."""
    rng = np.random.default_rng(700 + seed)
    e, upper, ext, til = random_plan(rng)
    u_lab, v_lab, w_lab = split_einsum(e)
    plan = orc.Plan(e, upper, ext, til)
    U = workloads.random_relation(rng, u_lab, upper, ext, til, "f32", keep=0.6)
    V = workloads.random_relation(rng, v_lab, upper, ext, til, "f32", keep=0.6)
    pairs, wkeys = orc.join(plan, U["keys"], V["keys"])
    con = sqlite3.connect(":memory:")
    uk = [c for c in u_lab if c in upper]
    vk = [c for c in v_lab if c in upper]
    wk = [c for c in w_lab if c in upper]
    con.execute(f"CREATE TABLE U ({''.join(c + '_ INT, ' for c in uk)}uid INT)")
    con.execute(f"CREATE TABLE V ({''.join(c + '_ INT, ' for c in vk)}vid INT)")
    for n, k in enumerate(U["keys"].tolist()):
        con.execute(f"INSERT INTO U VALUES ({', '.join(['?'] * (len(uk) + 1))})", (*k, n))
    for n, k in enumerate(V["keys"].tolist()):
        con.execute(f"INSERT INTO V VALUES ({', '.join(['?'] * (len(vk) + 1))})", (*k, n))
    order = ", ".join([c + "_" for c in wk] + ["uid", "vid"])
    rows = con.execute(f"SELECT uid, vid FROM U NATURAL JOIN V ORDER BY {order}").fetchall()
    assert [tuple(p) for p in pairs.tolist()] == rows
    if wk:
        ks = con.execute(f"SELECT DISTINCT {', '.join(c + '_' for c in wk)} FROM U NATURAL JOIN V "
                         f"ORDER BY {', '.join(c + '_' for c in wk)}").fetchall()
    else:
        ks = [()] if rows else []
    assert [tuple(k) for k in wkeys.tolist()] == ks


# ------------------------------------------------------ split invariance

def test_split_invariance(orc):
    """Every decomposition of the same tensors denotes the same function
    (Sec. 4.2), so every split and tile size yields the same dense W."""
    rng = np.random.default_rng(3)
    ext = {"i": 8, "j": 12, "k": 6}
    Ud = rng.standard_normal((8, 12)) * (rng.random((8, 12)) < 0.3)
    Vd = rng.standard_normal((12, 6)) * (rng.random((12, 6)) < 0.3)
    ref = Ud @ Vd
    for upper in ["", "i", "j", "k", "ij", "jk", "ik", "ijk"]:
        for tsel in itertools.product([1, 2], [1, 3], [2, 6]):
            til = {c: t for c, t in zip("ijk", tsel) if c in upper}

            def rel(labels, D):
                kl = [c for c in labels if c in upper]
                radix = [ext[c] // til[c] for c in kl]
                keys, tiles = [], []
                for K in itertools.product(*[range(x) for x in radix]):
                    sl = []
                    for c in labels:
                        if c in upper:
                            a = K[kl.index(c)]
                            sl.append(slice(a * til[c], (a + 1) * til[c]))
                        else:
                            sl.append(slice(None))
                    blk = D[tuple(sl)]
                    if np.any(blk != 0):
                        keys.append(K)
                        tiles.append(blk.reshape(-1))
                return {"keys": np.array(keys, dtype=np.int32).reshape(len(keys), len(kl)),
                        "tiles": np.array(tiles).reshape(len(keys), -1), "dtype": "f64"}

            plan = orc.Plan("ij,jk->ik", upper, ext, til)
            r = orc.run(plan, rel("ij", Ud), rel("jk", Vd))
            got = dense_of("ik", upper, ext, til, r.wkeys, r.acc)
            np.testing.assert_allclose(got, ref, rtol=1e-12, atol=1e-12)


# ------------------------------------------ chains and the 3-way path

def test_three_way_path_small(orc):
    """A[i,r] = sum_jk T[i,j,k] B[j,r] C[k,r] evaluated as E1 (join on j) then
    E2 (join on k) equals the three-operand einsum evaluated directly."""
    w = workloads.sparse_3way(64, 8, 8, 0.05, 0.1, seed=11)
    p1, p2 = plan_of(orc, w["E1"]), plan_of(orc, w["E2"])
    r1 = orc.run(p1, w["T"], w["B"])
    W = {"keys": r1.wkeys, "tiles": r1.acc, "dtype": "f64"}
    r2 = orc.run(p2, W, w["C"])
    s1, s2 = w["E1"], w["E2"]
    Td = dense_of("ijk", s1["upper"], s1["extents"], s1["tiles"], w["T"]["keys"], vals_f64(w["T"]))
    Bd = dense_of("jr", s1["upper"], s1["extents"], s1["tiles"], w["B"]["keys"], vals_f64(w["B"]))
    Cd = dense_of("kr", s2["upper"], s2["extents"], s2["tiles"], w["C"]["keys"], vals_f64(w["C"]))
    ref = np.einsum("ijk,jr,kr->ir", Td, Bd, Cd)
    got = dense_of("ir", s2["upper"], s2["extents"], s2["tiles"], r2.wkeys, r2.acc)
    np.testing.assert_allclose(got, ref, rtol=1e-11, atol=1e-11)
    # closed form: each T block (I,J,K) meets exactly one B tuple (J)
    assert len(r1.pairs) == len(w["T"]["keys"])


@pytest.mark.parametrize("c,layout", [(1, "jk"), (2, "jk"), (5, "kj"), (5, "jk")])
def test_gnn_chain_small(orc, c, layout):
    """(X.Y)^T.Z through E1 and E2 equals the dense product; the per-vertex
    form (tile 1) is re-stacked into 256-row tiles between the two EinSums.
    The adjacency keyed (J, K) ("ij,jk->ki") or (K, J) ("ij,kj->ki")."""
    w = workloads.config(c, "small", y_layout=layout)
    assert w["y_layout"] == layout
    p1, p2 = plan_of(orc, w["E1"]), plan_of(orc, w["E2"])
    r1 = orc.run(p1, w["X"], {"keys": w["Y"]["keys"], "coo": w["Y"]["coo"]})
    assert r1.n_outside == 0
    # closed form: each Y tile (J,K) meets exactly one X tuple (J)
    assert len(r1.pairs) == len(w["Y"]["keys"])
    keys, tiles = r1.wkeys, r1.acc
    if w["tile_e1"] != w["tile_e2"]:
        keys, tiles = orc.stack_rows(keys, tiles, w["tile_e2"] // w["tile_e1"])
    r2 = orc.run(p2, {"keys": keys, "tiles": tiles, "dtype": "f64"}, w["Z"])
    assert len(r2.pairs) == len(keys)  # cross product with the one Z tuple
    n, emb, zo = w["n"], w["emb"], w["z_out"]
    X = vals_f64(w["X"]).reshape(n // w["tile_e1"], emb, w["tile_e1"]).transpose(1, 0, 2).reshape(emb, n)
    import scipy.sparse as sp

    c0, c1 = w["Y"]["coo"][0].T  # coordinates in the operand's label order
    src, dst = (c0, c1) if layout == "jk" else (c1, c0)
    Y = sp.csr_matrix((w["Y"]["coo"][1], (src, dst)), shape=(n, n))
    Z = vals_f64(w["Z"]).reshape(emb, zo)
    ref = np.asarray((Y.T @ X.T)) @ Z
    s2 = w["E2"]
    got = dense_of("km", s2["upper"], s2["extents"], s2["tiles"], r2.wkeys, r2.acc)
    np.testing.assert_allclose(got, ref, rtol=1e-10, atol=1e-10)


def test_block_sparse_small(orc):
    w = workloads.config(3, "small")
    p = plan_of(orc, w["E"])
    r = orc.run(p, w["A"], w["B"])
    assert len(r.pairs) == len(w["A"]["keys"])  # each A block meets one B tuple
    s = w["E"]
    Ad = dense_of("ik", s["upper"], s["extents"], s["tiles"], w["A"]["keys"], vals_f64(w["A"]))
    Bd = dense_of("kn", s["upper"], s["extents"], s["tiles"], w["B"]["keys"], vals_f64(w["B"]))
    got = dense_of("in", s["upper"], s["extents"], s["tiles"], r.wkeys, r.acc)
    np.testing.assert_allclose(got, Ad @ Bd, rtol=1e-10, atol=1e-10)
    assert len(r.wkeys) == len(np.unique(w["A"]["keys"][:, 0]))


def test_tuple_count_estimator_c1():
    """Generator sanity (approximate): Eq. "eqn-count" predicts the number of
    stored 64x64 adjacency tiles for 8 uniform out-edges per vertex."""
    w = workloads.config(1)
    nposs = (4096 // 64) ** 2
    pred = nposs * (1 - np.exp(-w["n_edges"] / nposs))
    assert abs(len(w["Y"]["keys"]) - pred) < 8
    assert w["n_edges"] == 8 * 4096


# -------------------------------------------------------------- errors

@pytest.mark.parametrize("e,upper,ext,til,cat", [
    ("ij,jk", "", {"i": 2, "j": 2, "k": 2}, {}, "PARSE"),
    ("iij,jk->ik", "", {"i": 2, "j": 2, "k": 2}, {}, "PARSE"),
    ("ij,jk->iz", "", {"i": 2, "j": 2, "k": 2, "z": 2}, {}, "PARSE"),
    ("ij,jk,kl->il", "", {"i": 2, "j": 2, "k": 2, "l": 2}, {}, "PARSE"),
    ("iJ,Jk->ik", "", {"i": 2, "j": 2, "k": 2}, {}, "PARSE"),
    ("ij,jk->ik", "z", {"i": 2, "j": 2, "k": 2}, {}, "SPLIT"),
    ("ij,jk->ik", "j", {"i": 2, "j": 6, "k": 2}, {"j": 4}, "SHAPE"),
    ("ij,jk->ik", "j", {"i": 2, "j": 6, "k": 2}, {"j": 0}, "SHAPE"),
    ("ij,jk->ik", "", {"i": 2, "j": 0, "k": 2}, {}, "SHAPE"),
])
def test_plan_errors(orc, e, upper, ext, til, cat):
    with pytest.raises(orc.OracleError) as ei:
        orc.Plan(e, upper, ext, til)
    assert ei.value.category == cat


def test_key_checks(orc):
    plan = orc.Plan("ij,jk->ik", "jk", {"i": 4, "j": 8, "k": 8}, {"j": 2, "k": 2})
    ok = np.array([[0, 1], [0, 3], [2, 0]], dtype=np.int32)
    assert orc.check_keys(plan, 1, ok) == "OK"
    assert orc.check_keys(plan, 1, ok[[0, 2, 1]]) == "UNSORTED"
    assert orc.check_keys(plan, 1, ok[[0, 0, 1]]) == "DUPKEY"
    assert orc.check_keys(plan, 1, np.array([[0, 1], [0, 4]], dtype=np.int32)) == "KEYRANGE"
    assert orc.check_keys(plan, 1, np.array([[-1, 1]], dtype=np.int32)) == "KEYRANGE"


def test_empty_inputs(orc):
    plan = orc.Plan("ij,jk->ik", "j", {"i": 4, "j": 4, "k": 4}, {"j": 2})
    U = {"keys": np.zeros((0, 1), np.int32), "tiles": np.zeros((0, 8), np.float32), "dtype": "f32"}
    V = {"keys": np.array([[0]], np.int32), "tiles": np.ones((1, 8), np.float32), "dtype": "f32"}
    r = orc.run(plan, U, V)
    assert r.pairs.shape == (0, 2) and r.wkeys.shape[0] == 0


# ---------------------------------------------------------------- bf16

def test_bf16_rne_matches_torch(orc):
    import torch

    rng = np.random.default_rng(0)
    x = np.concatenate([rng.standard_normal(100000).astype(np.float32) * 10.0 ** rng.integers(-30, 30, 100000),
                        np.array([0.0, -0.0, np.inf, -np.inf, 1e-40, -1e-40, 3.3895314e38], np.float32)])
    # exact ties: low half 0x8000 with even and odd kept bit
    ties = (np.arange(1000, dtype=np.uint32) << 16 | 0x8000).view(np.float32) + np.float32(0)
    x = np.concatenate([x, ties.astype(np.float32)])
    ours = orc.f32_to_bf16(x)
    ref = torch.from_numpy(x).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    assert np.array_equal(ours, ref)
    # tie cases by hand: 1 + 2^-8 rounds down to 1, (1 + 3*2^-8) rounds up
    assert orc.f32_to_bf16(np.array([1 + 2 ** -8], np.float32))[0] == 0x3F80
    assert orc.f32_to_bf16(np.array([1 + 3 * 2 ** -8], np.float32))[0] == 0x3F82
    nan = orc.f32_to_bf16(np.array([np.nan], np.float32))[0]
    assert (nan & 0x7F80) == 0x7F80 and (nan & 0x7F) != 0


# ------------------------------------------------ restriction to samples

def test_restrict_matches_full(orc):
    w = workloads.config(2, "small")
    p1 = plan_of(orc, w["E1"])
    Y = {"keys": w["Y"]["keys"], "coo": w["Y"]["coo"]}
    full = orc.run(p1, w["X"], Y)
    rng = np.random.default_rng(1)
    pick = np.sort(rng.choice(len(full.wkeys), size=5, replace=False))
    S = full.wkeys[pick]
    mu, mv = orc.restrict(p1, w["X"]["keys"], w["Y"]["keys"], S)
    assert mv.sum() < len(mv)
    sub_u = {"keys": w["X"]["keys"][mu], "tiles": w["X"]["tiles"][mu], "dtype": "bf16"}
    ykeep = mv[w["Y"]["slot"]]
    sub_v = {"keys": w["Y"]["keys"][mv], "coo": (w["Y"]["coo"][0][ykeep], w["Y"]["coo"][1][ykeep])}
    uc, uv = orc._coo_of(p1, 0, sub_u)
    acc, mag, _ = orc.evaluate(p1, uc, uv, sub_v["coo"][0], sub_v["coo"][1], S)
    np.testing.assert_array_equal(acc, full.acc[pick])
    np.testing.assert_array_equal(mag, full.mag[pick])


def test_expand_roundtrip(orc):
    """Tiles built from the adjacency COO expand back to the same COO."""
    w = workloads.config(1, "small")
    p1 = plan_of(orc, w["E1"])
    c, v, _ = orc.expand(p1, 1, w["Y"]["keys"], w["Y"]["tiles"], "f32")
    got = sorted(zip(map(tuple, c.tolist()), v.tolist()))
    ref = sorted(zip(map(tuple, w["Y"]["coo"][0].tolist()), w["Y"]["coo"][1].tolist()))
    assert got == ref
    assert np.array_equal(orc.keys_from_coo(p1, 1, w["Y"]["coo"][0]), w["Y"]["keys"])


# ------------------------------------------------------------ repartition

def _dense(labels, up, ext, til, keys, tiles):
    """Place every tuple's tile into a dense array (written independently of
    the oracle: numpy slicing of each tuple's index box)."""
    shape = [ext[c] for c in labels]
    out = np.zeros(shape)
    tshape = [til[c] if c in up else ext[c] for c in labels]
    for key, tile in zip(np.asarray(keys).reshape(len(tiles), -1), tiles):
        box, ka = [], 0
        for c, t in zip(labels, tshape):
            if c in up:
                box.append(slice(int(key[ka]) * t, (int(key[ka]) + 1) * t))
                ka += 1
            else:
                box.append(slice(0, t))
        out[tuple(box)] = np.asarray(tile).reshape(tshape)
    return out


def _covered_keys(labels, up_in, up_out, ext, tin, tout, keys):
    """Target keys whose tile meets at least one source tile (brute force over
    the source tiles' index ranges)."""
    import itertools

    got = set()
    for key in np.asarray(keys).reshape(len(keys), -1):
        ranges, ka = {}, 0
        for c in labels:
            t = tin[c] if c in up_in else ext[c]
            lo = int(key[ka]) * t if c in up_in else 0
            ka += c in up_in
            ranges[c] = (lo, lo + t)
        axes = [range(ranges[c][0] // tout[c], (ranges[c][1] - 1) // tout[c] + 1) for c in labels if c in up_out]
        got.update(itertools.product(*axes))
    return sorted(got)


def test_repartition_paper_example(orc):
    """Sec. 6: T keyed by its row label (row vectors) re-partitioned to be
    keyed by its column label (column vectors)."""
    keys = np.array([[0], [1], [2]], np.int32)
    tiles = np.array([[1.0, 2.0], [3.0, 4.0], [5.0, 6.0]])
    k2, t2 = orc.repartition("ki", "k", "i", {"k": 3, "i": 2}, {"k": 1}, {"i": 1}, keys, tiles)
    assert k2.tolist() == [[0], [1]]
    assert t2.tolist() == [[1.0, 3.0, 5.0], [2.0, 4.0, 6.0]]


def test_repartition_identity(orc):
    rng = np.random.default_rng(3)
    keys = np.array([[0, 1], [1, 0], [2, 2]], np.int32)
    tiles = rng.standard_normal((3, 2 * 3 * 4))
    k2, t2 = orc.repartition("abc", "ab", "ab", {"a": 6, "b": 9, "c": 4}, {"a": 2, "b": 3}, {"a": 2, "b": 3},
                             keys, tiles)
    assert np.array_equal(k2, keys) and np.array_equal(t2, tiles)


@pytest.mark.parametrize("seed", range(16))
def test_repartition_random_dense_and_keys(orc, seed):
    """Random decompositions of random sparse tensors: the dense tensor is
    unchanged and the target key set is exactly the target tiles met by the
    source tiles (zero tiles included)."""
    rng = np.random.default_rng(300 + seed)
    nl = int(rng.integers(1, 4))
    labels = "".join(rng.choice(list("abcdefgh"), nl, replace=False))
    divs = {c: int(rng.choice([2, 3, 4, 6])) for c in labels}
    ext = {c: divs[c] * int(rng.integers(2, 5)) for c in labels}
    up_in = "".join(c for c in labels if rng.random() < 0.7)
    up_out = "".join(c for c in labels if rng.random() < 0.7)
    # tile sizes: divisors of the extent, possibly not dividing each other
    def pick(c):
        ds = [d for d in range(1, ext[c] + 1) if ext[c] % d == 0]
        return int(rng.choice(ds))
    tin = {c: pick(c) for c in up_in}
    tout = {c: pick(c) for c in up_out}
    axes = [range(ext[c] // tin[c]) for c in up_in]
    import itertools
    all_keys = list(itertools.product(*axes)) if up_in else [()]
    keep = [k for k in all_keys if rng.random() < 0.5] or all_keys[:1]
    keys = np.array(keep, np.int32).reshape(len(keep), len(up_in))
    te = int(np.prod([tin[c] if c in up_in else ext[c] for c in labels]))
    tiles = rng.standard_normal((len(keep), te)) * (rng.random((len(keep), te)) < 0.6)
    k2, t2 = orc.repartition(labels, up_in, up_out, ext, tin, tout, keys, tiles)
    np.testing.assert_array_equal(_dense(labels, up_out, ext, tout, k2, t2),
                                  _dense(labels, up_in, ext, tin, keys, tiles))
    assert [tuple(r) for r in k2.tolist()] == _covered_keys(labels, up_in, up_out, ext, tin, tout, keys)


def test_repartition_round_trip(orc):
    rng = np.random.default_rng(8)
    ext = {"i": 12, "j": 8}
    keys = np.array([[0, 1], [2, 0], [3, 3]], np.int32)
    tiles = rng.standard_normal((3, 3 * 2))
    k2, t2 = orc.repartition("ij", "ij", "j", ext, {"i": 3, "j": 2}, {"j": 4}, keys, tiles)
    k3, t3 = orc.repartition("ij", "j", "ij", ext, {"j": 4}, {"i": 3, "j": 2}, k2, t2)
    # the source tuples come back unchanged; every extra tuple is all zeros
    back = {tuple(k): t for k, t in zip(k3.tolist(), t3)}
    for k, t in zip(keys.tolist(), tiles):
        np.testing.assert_array_equal(back.pop(tuple(k)), t)
    assert all(not np.any(t) for t in back.values())


def test_repartition_stack_special_case(orc):
    """Grouping one promoted label from tile 1 to tile g is the stack of rows."""
    rng = np.random.default_rng(5)
    keys = np.sort(rng.choice(64, 20, replace=False)).astype(np.int32).reshape(-1, 1)
    rows = rng.standard_normal((20, 8))
    k2, t2 = orc.repartition("ki", "k", "k", {"k": 64, "i": 8}, {"k": 1}, {"k": 16}, keys, rows)
    k3, t3 = orc.stack_rows(keys, rows, 16)
    assert np.array_equal(k2, k3) and np.array_equal(t2, t3)


def test_repartition_errors(orc):
    with pytest.raises(orc.OracleError):
        orc.repartition("ij", "ij", "i", {"i": 4, "j": 4}, {"i": 3, "j": 1}, {"i": 2}, np.zeros((0, 2), np.int32),
                        np.zeros((0, 3)))
    with pytest.raises(orc.OracleError):
        orc.repartition("ij", "ik", "i", {"i": 4, "j": 4}, {"i": 1}, {"i": 2}, np.zeros((0, 2), np.int32),
                        np.zeros((0, 4)))


# ------------------------------------------ the three-operand EinSum (eval3)

_E3 = "ijk,jr,kr->ir"


def _three_way_case(seed, n=32, r=6, block=4, density=0.08, fill=0.3, drop=0.25):
    """A small sparse 3-way case whose B and C miss some blocks (so the
    triple join drops tuples)."""
    w = workloads.sparse_3way(n, r, block, density, fill, seed=seed)
    rng = np.random.default_rng(seed + 1)
    for name in ("B", "C"):
        keep = rng.random(len(w[name]["keys"])) >= drop
        keep[0] = True
        w[name] = {"keys": w[name]["keys"][keep], "tiles": w[name]["tiles"][keep], "dtype": "f32"}
    ext = {"i": n, "j": n, "k": n, "r": r}
    til = {"i": block, "j": block, "k": block}
    return w, ext, til


def test_eval3_matches_binary_path(orc):
    """The triple evaluation equals the two-EinSum path through the C oracle
    (E1 = T join B on j, E2 = W join C on k): same keys, same values."""
    for seed in (3, 4):
        w, ext, til = _three_way_case(seed)
        wk, acc, mag, tri = orc.eval3(_E3, "ijk", ext, til, w["T"], w["B"], w["C"])
        p1 = orc.Plan("ijk,jr->ikr", "ijk", ext, til)
        p2 = orc.Plan("ikr,kr->ir", "ik", {"i": ext["i"], "k": ext["k"], "r": ext["r"]},
                      {"i": til["i"], "k": til["k"]})
        r1 = orc.run(p1, w["T"], w["B"])
        r2 = orc.run(p2, {"keys": r1.wkeys, "tiles": r1.acc, "dtype": "f64"}, w["C"])
        assert np.array_equal(wk, r2.wkeys)
        np.testing.assert_allclose(acc, r2.acc, rtol=1e-12, atol=1e-12)
        assert (mag >= np.abs(acc) - 1e-12).all()
        assert len(tri) < len(w["T"]["keys"])  # some T blocks lost their B or C partner


def test_eval3_brute_force(orc):
    """Pure-Python loops over every global coordinate of the dense tensors
    (absent tuples are zero) give the same values; the output keys are the
    I blocks of T tuples whose J block is in B and K block in C."""
    w, ext, til = _three_way_case(7, n=16, r=3, block=4, density=0.2, fill=0.5)
    wk, acc, mag, tri = orc.eval3(_E3, "ijk", ext, til, w["T"], w["B"], w["C"])
    T = dense_of("ijk", "ijk", ext, til, w["T"]["keys"], vals_f64(w["T"]))
    B = dense_of("jr", "j", ext, til, w["B"]["keys"], vals_f64(w["B"]))
    C = dense_of("kr", "k", ext, til, w["C"]["keys"], vals_f64(w["C"]))
    n, r = ext["i"], ext["r"]
    A = [[0.0] * r for _ in range(n)]
    for i in range(n):
        for j in range(n):
            for k in range(n):
                t = T[i, j, k]
                if t == 0.0:
                    continue
                for q in range(r):
                    A[i][q] += t * B[j, q] * C[k, q]
    bj = {int(k[0]) for k in w["B"]["keys"]}
    ck = {int(k[0]) for k in w["C"]["keys"]}
    want_keys = sorted({int(I) for I, J, K in w["T"]["keys"] if int(J) in bj and int(K) in ck})
    assert wk.reshape(-1).tolist() == want_keys
    got = dense_of("ir", "i", ext, til, wk, acc)
    np.testing.assert_allclose(got, np.array(A), rtol=1e-12, atol=1e-12)
    # blocks outside the key set hold nothing
    mask = np.zeros(n, bool)
    for I in want_keys:
        mask[I * til["i"]:(I + 1) * til["i"]] = True
    assert np.all(np.array(A)[~mask] == 0.0)


def test_eval3_label_order_invariance(orc):
    """Renaming the roles and transposing every operand (U as "ikj", the two
    small operands swapped and one stored transposed, W as "ri") gives the
    transposed result."""
    w, ext, til = _three_way_case(5)
    wk, acc, _, _ = orc.eval3(_E3, "ijk", ext, til, w["T"], w["B"], w["C"])
    bt = til["i"]
    T2 = w["T"]["tiles"].reshape(-1, bt, bt, bt).transpose(0, 1, 3, 2).reshape(len(w["T"]["keys"]), -1)
    order = np.lexsort((w["T"]["keys"][:, 1], w["T"]["keys"][:, 2], w["T"]["keys"][:, 0]))
    U2 = {"keys": np.ascontiguousarray(w["T"]["keys"][order][:, [0, 2, 1]]), "tiles": T2[order], "dtype": "f32"}
    r = ext["r"]
    B2 = {"keys": w["B"]["keys"], "tiles": w["B"]["tiles"].reshape(-1, bt, r).transpose(0, 2, 1).reshape(
        len(w["B"]["keys"]), -1), "dtype": "f32"}
    wk2, acc2, _, _ = orc.eval3("ikj,kr,rj->ri", "ijk", ext, til, U2, w["C"], B2)
    assert np.array_equal(wk2, wk)
    np.testing.assert_allclose(acc2.reshape(-1, r, bt).transpose(0, 2, 1).reshape(acc.shape), acc,
                               rtol=1e-12, atol=1e-12)


def test_eval3_magnitude_positive_inputs(orc):
    """With non-negative inputs the magnitude sum equals the sum itself."""
    w, ext, til = _three_way_case(9)
    for name in ("T", "B", "C"):
        w[name]["tiles"] = np.abs(w[name]["tiles"])
    _, acc, mag, _ = orc.eval3(_E3, "ijk", ext, til, w["T"], w["B"], w["C"])
    np.testing.assert_allclose(mag, acc, rtol=1e-13, atol=0)


@pytest.mark.parametrize("einsum,upper,cat", [
    ("ijk,jr->ir", "ijk", "PARSE"),
    ("ijk,jr,kq->ir", "ijk", "SPLIT"),      # small operands share no label
    ("ijk,jr,jr->ir", "ijk", "SPLIT"),      # both meet U on j
    ("ijk,jr,kr->ikr", "ijk", "SPLIT"),     # W keeps a joined label
    ("jik,jr,kr->ir", "ijk", "SPLIT"),      # joined labels not U's last two
    ("ijk,jr,kr->ir", "ik", "SPLIT"),       # joined label demoted
    ("ijk,jr,kr->ir", "ijkr", "SPLIT"),     # shared label promoted
])
def test_eval3_structure_errors(orc, einsum, upper, cat):
    ext = {c: 8 for c in "ijkrq"}
    til = {c: 4 for c in "ijkrq"}
    with pytest.raises(orc.Spec3Error) as e:
        orc.parse3(einsum, upper, ext, til)
    assert e.value.category == cat


def test_eval3_key_errors(orc):
    w, ext, til = _three_way_case(3)
    bad = dict(w["T"])
    bad["keys"] = w["T"]["keys"][::-1].copy()
    with pytest.raises(orc.Spec3Error) as e:
        orc.eval3(_E3, "ijk", ext, til, bad, w["B"], w["C"])
    assert e.value.category == "UNSORTED"
    bad["keys"] = w["T"]["keys"].copy()
    bad["keys"][0, 0] = ext["i"]
    with pytest.raises(orc.Spec3Error) as e:
        orc.eval3(_E3, "ijk", ext, til, bad, w["B"], w["C"])
    assert e.value.category == "KEYRANGE"


# ------------------------- the masked three-operand form (attention scores)

_EM = "ij,ik,jk->ij"


def _masked_case(seed, n=24, r=7, ti=1, tj=1, keep=0.3, drop=0.25):
    """A random masked case: U over (I, J) blocks, V keyed I and X keyed J
    with some keys missing, so the triple join drops U tuples."""
    rng = np.random.default_rng(seed)
    ext = {"i": n, "j": n, "k": r}
    til = {"i": ti, "j": tj}
    U = workloads.random_relation(rng, "ij", "ij", ext, til, "f32", keep=keep)
    V = workloads.random_relation(rng, "ik", "i", ext, til, "f32", keep=1 - drop)
    X = workloads.random_relation(rng, "jk", "j", ext, til, "f32", keep=1 - drop)
    return U, V, X, ext, til


@pytest.mark.parametrize("ti,tj", [(1, 1), (2, 3), (4, 1)])
def test_masked_matches_binary_path(orc, ti, tj):
    """The masked triple evaluation equals the two binary EinSums of Table
    gt-schema through the C oracle: T2 = V join U on i with no aggregation
    ("ik,ij->ijk"), then T3 = T2 join X on j summing k ("ijk,jk->ij")."""
    for seed in (11, 12):
        U, V, X, ext, til = _masked_case(seed, ti=ti, tj=tj)
        wk, acc, mag, tri = orc.eval3(_EM, "ij", ext, til, U, V, X)
        r3 = orc.run(orc.Plan("ik,ij->ijk", "ij", ext, til), V, U)
        r4 = orc.run(orc.Plan("ijk,jk->ij", "ij", ext, til), {"keys": r3.wkeys, "tiles": r3.acc, "dtype": "f64"}, X)
        assert np.array_equal(wk, r4.wkeys)
        np.testing.assert_allclose(acc, r4.acc, rtol=1e-12, atol=1e-12)
        assert (mag >= np.abs(acc) - 1e-12).all()
        assert 0 < len(tri) < len(U["keys"])  # some U tuples lost a partner
        # every output key is a U key and the triples come in U order
        assert np.array_equal(wk, U["keys"][tri[:, 0]])
        assert np.all(np.diff(tri[:, 0]) > 0)


def test_masked_brute_force(orc):
    """Pure-Python loops over every global coordinate of the dense tensors
    (absent tuples are zero): S[i, j] = sum_k U[i, j] V[i, k] X[j, k]; the
    output keys are the U keys whose I block is in V and J block in X."""
    U, V, X, ext, til = _masked_case(21, n=12, r=5, ti=2, tj=3, keep=0.5)
    wk, acc, _, _ = orc.eval3(_EM, "ij", ext, til, U, V, X)
    Ud = dense_of("ij", "ij", ext, til, U["keys"], vals_f64(U))
    Vd = dense_of("ik", "i", ext, til, V["keys"], vals_f64(V))
    Xd = dense_of("jk", "j", ext, til, X["keys"], vals_f64(X))
    n, r = ext["i"], ext["k"]
    S = [[0.0] * n for _ in range(n)]
    for i in range(n):
        for j in range(n):
            for k in range(r):
                S[i][j] += Ud[i, j] * Vd[i, k] * Xd[j, k]
    vi = {int(k[0]) for k in V["keys"]}
    xj = {int(k[0]) for k in X["keys"]}
    want = [(int(I), int(J)) for I, J in U["keys"] if int(I) in vi and int(J) in xj]
    assert [tuple(k) for k in wk.tolist()] == want
    got = dense_of("ij", "ij", ext, til, wk, acc)
    np.testing.assert_allclose(got, np.array(S), rtol=1e-12, atol=1e-12)


def test_masked_sqlite_purely_relational(orc):
    """All labels promoted with tiles of 1 is the purely relational form
    (Sec. 2): SQLite's SUM(u.v * q.v * x.v) over the three-way join, grouped
    by (i, j), gives the same keys and values."""
    n, r = 20, 6
    rng = np.random.default_rng(31)
    ext = {"i": n, "j": n, "k": r}
    til = {"i": 1, "j": 1}
    U = workloads.random_relation(rng, "ij", "ij", ext, til, "f32", keep=0.25)
    V = workloads.random_relation(rng, "ik", "i", ext, til, "f32", keep=0.8)
    X = workloads.random_relation(rng, "jk", "j", ext, til, "f32", keep=0.8)
    wk, acc, _, _ = orc.eval3(_EM, "ij", ext, til, U, V, X)
    db = sqlite3.connect(":memory:")
    db.execute("CREATE TABLE u (i INT, j INT, v DOUBLE)")
    db.execute("CREATE TABLE q (i INT, k INT, v DOUBLE)")
    db.execute("CREATE TABLE x (j INT, k INT, v DOUBLE)")
    db.executemany("INSERT INTO u VALUES (?,?,?)",
                   [(int(a), int(b), float(v)) for (a, b), v in zip(U["keys"], U["tiles"][:, 0])])
    db.executemany("INSERT INTO q VALUES (?,?,?)",
                   [(int(a[0]), k, float(t[k])) for a, t in zip(V["keys"], V["tiles"]) for k in range(r)])
    db.executemany("INSERT INTO x VALUES (?,?,?)",
                   [(int(a[0]), k, float(t[k])) for a, t in zip(X["keys"], X["tiles"]) for k in range(r)])
    rows = db.execute("SELECT u.i, u.j, SUM(u.v * q.v * x.v) FROM u JOIN q ON q.i = u.i "
                      "JOIN x ON x.j = u.j AND x.k = q.k GROUP BY u.i, u.j ORDER BY u.i, u.j").fetchall()
    assert [tuple(k) for k in wk.tolist()] == [(a, b) for a, b, _ in rows]
    np.testing.assert_allclose(acc[:, 0], [s for _, _, s in rows], rtol=1e-12, atol=1e-12)


def test_masked_label_order_invariance(orc):
    """V and X stored with the shared label first ("ki", "kj", transposed
    tiles) give the same result."""
    U, V, X, ext, til = _masked_case(41, ti=2, tj=2)
    wk, acc, _, _ = orc.eval3(_EM, "ij", ext, til, U, V, X)
    r = ext["k"]

    def tr(rel, t):
        return {"keys": rel["keys"], "dtype": "f32",
                "tiles": rel["tiles"].reshape(-1, t, r).transpose(0, 2, 1).reshape(len(rel["keys"]), -1)}

    wk2, acc2, _, _ = orc.eval3("ij,ki,kj->ij", "ij", ext, til, U, tr(V, til["i"]), tr(X, til["j"]))
    assert np.array_equal(wk2, wk)
    np.testing.assert_allclose(acc2, acc, rtol=1e-12, atol=1e-12)


def test_masked_magnitude_positive_inputs(orc):
    U, V, X, ext, til = _masked_case(51)
    for rel in (U, V, X):
        rel["tiles"] = np.abs(rel["tiles"])
    _, acc, mag, _ = orc.eval3(_EM, "ij", ext, til, U, V, X)
    np.testing.assert_allclose(mag, acc, rtol=1e-13, atol=0)


@pytest.mark.parametrize("einsum,upper,cat", [
    ("ij,ik,jk->ji", "ij", "SPLIT"),     # W neither U's labels nor U's others plus k
    ("ij,ik,jk->ijk", "ij", "SPLIT"),    # W keeps the shared label and the joined ones
    ("ij,ik,jk->ij", "ijk", "SPLIT"),    # shared label promoted
    ("ij,ik,jk->ij", "i", "SPLIT"),      # joined label demoted
])
def test_masked_structure_errors(orc, einsum, upper, cat):
    ext = {c: 8 for c in "ijk"}
    til = {c: 4 for c in "ijk"}
    with pytest.raises(orc.Spec3Error) as e:
        orc.parse3(einsum, upper, ext, til)
    assert e.value.category == cat


def test_graph_attention_small_chain(orc):
    """The attention workload (scaled down) through the oracle -- E1 and E2
    with the C oracle, the masked EinSum with eval3, times 1/sqrt(d_k) --
    equals dense attention scores written with numpy matrix products:
    S = A * (F WQ)(F WK)^T / sqrt(d_k) on the edges, F the dense features."""
    w = workloads.config(6, "small")
    n, nf, dk = w["n"], w["n_feat"], w["d_k"]
    e1, e2 = w["E1"], w["E2"]
    r1 = orc.run(orc.Plan(e1["einsum"], e1["upper"], e1["extents"], e1["tiles"]), w["X"], w["WQ"])
    r2 = orc.run(orc.Plan(e2["einsum"], e2["upper"], e2["extents"], e2["tiles"]), w["X"], w["WK"])
    T0 = {"keys": r1.wkeys, "tiles": r1.acc, "dtype": "f64"}
    T1 = {"keys": r2.wkeys, "tiles": r2.acc, "dtype": "f64"}
    e = w["E34"]
    wk, acc, mag, _ = orc.eval3(e["einsum"], e["upper"], e["extents"], e["tiles"], w["A"], T0, T1)
    S = acc[:, 0] * w["scale"]
    F = np.zeros((n, nf))
    F[w["X"]["keys"][:, 0], w["X"]["keys"][:, 1]] = 1.0
    Q = F @ w["WQ"]["tiles"].astype(np.float64)
    K = F @ w["WK"]["tiles"].astype(np.float64)
    ai, aj = w["A"]["keys"][:, 0], w["A"]["keys"][:, 1]
    assert np.array_equal(wk, w["A"]["keys"])  # every node has a feature, so every edge is matched
    np.testing.assert_allclose(S, (Q[ai] * K[aj]).sum(axis=1) / np.sqrt(dk), rtol=1e-10, atol=1e-10)
    assert w["n_edges"] == len(ai) and len(np.unique(ai * n + aj)) == len(ai)
