"""GPU parity of the three-operand EinSum (tre_execute3) against the oracle's
plain per-triple evaluation (oracle.eval3): output keys and triple count
bit-exact, values within the mag-relative tolerance (1e-4, fp32)."""
import sys

import numpy as np
import pytest

import workloads
from _parity import assert_values, to_dev

pytestmark = pytest.mark.gpu


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    import torch

    assert torch.cuda.is_available(), "GPU test needs a GPU"
    import paper_2603_08957_amd as tre

    tre.lib()


def _relation(rng, labels, upper, ext, til, keep):
    kl = [c for c in labels if c in upper]
    radix = [ext[c] // til[c] for c in kl]
    grid = np.stack(np.meshgrid(*[np.arange(x) for x in radix], indexing="ij"), axis=-1).reshape(-1, len(kl))
    mask = rng.random(len(grid)) < keep
    mask[rng.integers(len(grid))] = True
    keys = np.ascontiguousarray(grid[mask].astype(np.int32))
    te = int(np.prod([til[c] if c in upper else ext[c] for c in labels]))
    tiles = rng.standard_normal((len(keys), te)).astype(np.float32)
    return {"keys": keys, "tiles": tiles, "dtype": "f32"}


def _case3(rng):
    """Random structure: 0-2 row labels (promoted or not), the joined pair in
    either order, the small operands stored either way round, W in any
    order; tile and extent sizes that leave ragged 32-row and 64-column
    blocks and ragged 128-element chunks."""
    letters = list("abcdefghlmnopst")
    rng.shuffle(letters)
    nm = int(rng.integers(0, 3))
    rows = letters[:nm]
    a, b, r = letters[nm:nm + 3]
    p, q = (a, b) if rng.random() < 0.5 else (b, a)
    u = "".join(rows) + p + q
    v = a + r if rng.random() < 0.5 else r + a
    x = b + r if rng.random() < 0.5 else r + b
    wl = rows + [r]
    rng.shuffle(wl)
    w = "".join(wl)
    upper = a + b + "".join(c for c in rows if rng.random() < 0.5)
    til, ext = {}, {}
    til[p] = int(rng.choice([1, 2, 3, 5, 8, 16, 32]))
    til[q] = int(rng.choice([4, 8, 12, 16, 32, 64]))
    for c in (p, q):
        ext[c] = til[c] * int(rng.integers(2, 6))
    for c in rows:
        if c in upper:
            til[c] = int(rng.choice([1, 4, 7, 16, 40]))
            ext[c] = til[c] * int(rng.integers(1, 4))
        else:
            ext[c] = int(rng.choice([1, 5, 33]))
    ext[r] = int(rng.choice([1, 3, 17, 64, 70, 130]))
    e = f"{u},{v},{x}->{w}"
    U = _relation(rng, u, upper, ext, til, 0.6)
    V = _relation(rng, v, upper, ext, til, 0.8)
    X = _relation(rng, x, upper, ext, til, 0.8)
    return e, upper, ext, til, U, V, X


def _run_and_check(orc, e, upper, ext, til, U, V, X):
    import paper_2603_08957_amd as tre

    uk, ut = to_dev(U)
    vk, vt = to_dev(V)
    xk, xt = to_dev(X)
    wk, wt, nt = tre.execute3(e, upper, ext, til, uk, ut, vk, vt, xk, xt)
    rk, acc, mag, tri = orc.eval3(e, upper, ext, til, U, V, X)
    assert nt == len(tri)
    assert int(wk.shape[0]) == len(rk)
    assert np.array_equal(wk.cpu().numpy().reshape(rk.shape), rk), "output key set differs"
    return assert_values(wt.cpu().numpy(), acc, mag, "f32")["mag_rel"]


@pytest.mark.parametrize("seed", range(40))
def test_execute3_random_gpu(orc, seed):
    rng = np.random.default_rng(4200 + seed)
    e, upper, ext, til, U, V, X = _case3(rng)
    say("execute3 random", seed, e, upper, ext, til, len(U["keys"]), len(V["keys"]), len(X["keys"]))
    _run_and_check(orc, e, upper, ext, til, U, V, X)


def test_execute3_three_way_small_gpu(orc):
    """The sparse 3-way workload at its small size (512^3, 32^3 blocks)."""
    w = workloads.config(4, "small")
    ext = {"i": w["n"], "j": w["n"], "k": w["n"], "r": w["r"]}
    til = {c: w["block"] for c in "ijk"}
    say("execute3 three-way small", len(w["T"]["keys"]))
    _run_and_check(orc, "ijk,jr,kr->ir", "ijk", ext, til, w["T"], w["B"], w["C"])


def test_execute3_many_triples_per_key_gpu(orc):
    """One output key with many triples (split over many units and summed by
    the reduction) next to keys with one triple each."""
    rng = np.random.default_rng(77)
    ext = {"i": 64, "j": 256, "k": 64, "r": 64}
    til = {"i": 32, "j": 8, "k": 16}
    U = _relation(rng, "ijk", "ijk", ext, til, 1.0)
    keep = (U["keys"][:, 0] == 0) | ((U["keys"][:, 1] == 3) & (U["keys"][:, 2] == 1))
    U = {"keys": np.ascontiguousarray(U["keys"][keep]), "tiles": U["tiles"][keep], "dtype": "f32"}
    V = _relation(rng, "jr", "ijk", ext, til, 1.0)
    X = _relation(rng, "kr", "ijk", ext, til, 1.0)
    say("execute3 long segment", len(U["keys"]))
    _run_and_check(orc, "ijk,jr,kr->ir", "ijk", ext, til, U, V, X)


def test_execute3_edge_cases_gpu(orc):
    import torch

    import paper_2603_08957_amd as tre

    rng = np.random.default_rng(5)
    ext = {"i": 8, "j": 8, "k": 8, "r": 5}
    til = {"i": 4, "j": 4, "k": 4}
    U = _relation(rng, "ijk", "ijk", ext, til, 1.0)
    V = _relation(rng, "jr", "ijk", ext, til, 1.0)
    X = _relation(rng, "kr", "ijk", ext, til, 1.0)
    uk, ut = to_dev(U)
    vk, vt = to_dev(V)
    xk, xt = to_dev(X)
    # empty U
    wk, wt, nt = tre.execute3("ijk,jr,kr->ir", "ijk", ext, til, uk[:0], ut[:0], vk, vt, xk, xt)
    assert nt == 0 and wk.shape[0] == 0
    # no U tuple meets a V tuple
    vk2 = torch.tensor([[1]], dtype=torch.int32, device="cuda")
    sel = (U["keys"][:, 1] == 0)
    wk, wt, nt = tre.execute3("ijk,jr,kr->ir", "ijk", ext, til, uk[torch.from_numpy(sel).cuda()].contiguous(),
                              ut[torch.from_numpy(sel).cuda()].contiguous(), vk2, vt[:1].contiguous(), xk, xt)
    assert nt == 0 and wk.shape[0] == 0
    # timing fields
    _, _, _, tm = tre.execute3("ijk,jr,kr->ir", "ijk", ext, til, uk, ut, vk, vt, xk, xt, timing=True)
    assert tm["contract_ms"] > 0 and tm["join_ms"] > 0
    # errors
    with pytest.raises(tre.TreError) as e:
        tre.execute3("ijk,jr,kr->ir", "ijk", ext, til, uk.flip(0).contiguous(), ut, vk, vt, xk, xt)
    assert e.value.status == "TRE_E_UNSORTED"
    with pytest.raises(tre.TreError) as e:
        tre.execute3("ijk,jr,jr->ir", "ijk", ext, til, uk, ut, vk, vt, xk, xt)
    assert e.value.status == "TRE_E_SPLIT"
    with pytest.raises(tre.TreError) as e:
        tre.execute3("ijk,jr,kr->ir", "ijk", ext, {"i": 4, "j": 4, "k": 2}, uk, ut, vk, vt, xk, xt)
    assert e.value.status == "TRE_E_SHAPE"


# --------------------------------------------------------- masked form

def _case_masked(rng):
    """Random masked case "rows p q, (a r), (b r) -> rows p q": p, q promoted
    with tiles of 1, row labels promoted or not, the small operands stored
    either way round, R both below and above the 256 elements one wavefront
    covers per step, multiples of 4 (16-byte loads) and not."""
    letters = list("abcdefghlmnopst")
    rng.shuffle(letters)
    nm = int(rng.integers(0, 3))
    rows = letters[:nm]
    a, b, r = letters[nm:nm + 3]
    p, q = (a, b) if rng.random() < 0.5 else (b, a)
    u = "".join(rows) + p + q
    v = a + r if rng.random() < 0.5 else r + a
    x = b + r if rng.random() < 0.5 else r + b
    upper = a + b + "".join(c for c in rows if rng.random() < 0.5)
    til, ext = {p: 1, q: 1}, {}
    for c in (p, q):
        ext[c] = int(rng.integers(2, 40))
    for c in rows:
        if c in upper:
            til[c] = int(rng.choice([1, 3, 8]))
            ext[c] = til[c] * int(rng.integers(1, 4))
        else:
            ext[c] = int(rng.choice([1, 5, 33, 70]))
    ext[r] = int(rng.choice([1, 3, 4, 17, 64, 256, 260, 1000, 1024]))
    e = f"{u},{v},{x}->{u}"
    U = _relation(rng, u, upper, ext, til, 0.4)
    V = _relation(rng, v, upper, ext, til, 0.8)
    X = _relation(rng, x, upper, ext, til, 0.8)
    return e, upper, ext, til, U, V, X


@pytest.mark.parametrize("seed", range(30))
def test_masked_random_gpu(orc, seed):
    rng = np.random.default_rng(5300 + seed)
    e, upper, ext, til, U, V, X = _case_masked(rng)
    say("masked random", seed, e, upper, ext, til, len(U["keys"]), len(V["keys"]), len(X["keys"]))
    _run_and_check(orc, e, upper, ext, til, U, V, X)


def _attention_inputs(w):
    dev = {}
    for name in ("X", "WQ", "WK", "A"):
        dev[name] = to_dev(w[name])
    return dev


def test_masked_attention_small_gpu(orc):
    """The graph-attention workload at its small size: E1 and E2 (scale +
    segmented sum) and the fused masked EinSum on the GPU, each checked
    against the oracle on the GPU's own inputs; the binary path (E3 with no
    aggregation, then E4) gives the same keys and values; the unary
    1/sqrt(d_k) matches an fp32 multiply bit for bit."""
    import torch

    import paper_2603_08957_amd as tre

    w = workloads.config(6, "small")
    d = _attention_inputs(w)
    T = {}
    for name, wname in (("E1", "WQ"), ("E2", "WK")):
        s = w[name]
        out = tre.einsum(tre.Plan.from_spec(s), d["X"][0], d["X"][1], d[wname][0], d[wname][1])
        ref = orc.run(orc.Plan(s["einsum"], s["upper"], s["extents"], s["tiles"]), w["X"], w[wname])
        assert np.array_equal(out.w_keys.cpu().numpy().reshape(ref.wkeys.shape), ref.wkeys)
        assert_values(out.w_tiles.cpu().numpy(), ref.acc, ref.mag, "f32", name)
        T[name] = (out.w_keys.reshape(-1, 1).contiguous(), out.w_tiles)
    host = {k: {"keys": v[0].cpu().numpy(), "tiles": v[1].cpu().numpy(), "dtype": "f32"} for k, v in T.items()}
    e = w["E34"]
    wk, wt, nt = tre.execute3(e["einsum"], e["upper"], e["extents"], e["tiles"], d["A"][0], d["A"][1],
                              T["E1"][0], T["E1"][1], T["E2"][0], T["E2"][1])
    rk, acc, mag, tri = orc.eval3(e["einsum"], e["upper"], e["extents"], e["tiles"], w["A"], host["E1"],
                                  host["E2"])
    assert nt == len(tri) == len(rk) == w["n_edges"]
    assert np.array_equal(wk.cpu().numpy(), rk)
    assert_values(wt.cpu().numpy(), acc, mag, "f32", "masked")
    S = tre.scale_f32(wt, w["scale"])
    np.testing.assert_array_equal(S.cpu().numpy(), (wt.cpu().numpy() * np.float32(w["scale"])).astype(np.float32))
    # binary path of Table gt-schema on the device
    s3, s4 = w["E3"], w["E4"]
    o3 = tre.einsum(tre.Plan.from_spec(s3), T["E1"][0], T["E1"][1], d["A"][0], d["A"][1])
    o4 = tre.einsum(tre.Plan.from_spec(s4), o3.w_keys, o3.w_tiles, T["E2"][0], T["E2"][1])
    assert torch.equal(o4.w_keys.reshape(wk.shape), wk)
    assert_values(o4.w_tiles.cpu().numpy(), acc, mag, "f32", "binary")


def test_masked_edge_cases_gpu(orc):
    import torch

    import paper_2603_08957_amd as tre

    rng = np.random.default_rng(8)
    ext = {"i": 16, "j": 16, "k": 33}
    til = {"i": 1, "j": 1}
    U = _relation(rng, "ij", "ij", ext, til, 0.5)
    V = _relation(rng, "ik", "ij", ext, til, 1.0)
    X = _relation(rng, "jk", "ij", ext, til, 1.0)
    uk, ut = to_dev(U)
    vk, vt = to_dev(V)
    xk, xt = to_dev(X)
    e = "ij,ik,jk->ij"
    wk, wt, nt = tre.execute3(e, "ij", ext, til, uk[:0], ut[:0], vk, vt, xk, xt)
    assert nt == 0 and wk.shape[0] == 0
    # no V tuple for any U row
    wk, wt, nt = tre.execute3(e, "ij", ext, til, uk, ut, vk[:0], vt[:0], xk, xt)
    assert nt == 0 and wk.shape[0] == 0
    _, _, _, tm = tre.execute3(e, "ij", ext, til, uk, ut, vk, vt, xk, xt, timing=True)
    assert tm["contract_ms"] > 0 and tm["join_ms"] > 0
    with pytest.raises(tre.TreError) as err:
        tre.execute3(e, "ij", ext, {"i": 2, "j": 1}, uk, ut, vk, vt, xk, xt)
    assert err.value.status == "TRE_E_SHAPE"
    with pytest.raises(tre.TreError) as err:
        tre.execute3("ij,ik,jk->ji", "ij", ext, til, uk, ut, vk, vt, xk, xt)
    assert err.value.status == "TRE_E_SPLIT"
    with pytest.raises(tre.TreError) as err:
        tre.execute3(e, "ij", ext, til, uk.flip(0).contiguous(), ut, vk, vt, xk, xt)
    assert err.value.status == "TRE_E_UNSORTED"
    # the scale glue: odd lengths, in place, a scale that rounds
    x = torch.randn(1003, device="cuda")
    y = tre.scale_f32(x, 0.1)
    np.testing.assert_array_equal(y.cpu().numpy(), x.cpu().numpy() * np.float32(0.1))
    z = x.clone()
    tre.scale_f32(z, 3.0, out=z)
    np.testing.assert_array_equal(z.cpu().numpy(), x.cpu().numpy() * np.float32(3.0))


# ------------------------------------------- small operands holding every key

def _complete(rng, case, keep_u):
    """The case with V and X refilled to hold every key of their label (the
    dense path: each U tuple is a triple, partners indexed by key value)
    and U thinned to `keep_u`."""
    e, upper, ext, til, U, V, X = case
    u, v, x = e.split("->")[0].split(",")
    U = _relation(rng, u, upper, ext, til, keep_u)
    V = _relation(rng, v, upper, ext, til, 1.0)
    X = _relation(rng, x, upper, ext, til, 1.0)
    return e, upper, ext, til, U, V, X


def _run_dense(orc, case):
    import paper_2603_08957_amd as tre

    e, upper, ext, til, U, V, X = case
    _run_and_check(orc, e, upper, ext, til, U, V, X)
    uk, ut = to_dev(U)
    vk, vt = to_dev(V)
    xk, xt = to_dev(X)
    _, _, nt, tm = tre.execute3(e, upper, ext, til, uk, ut, vk, vt, xk, xt, timing=True)
    assert tm["join_path"] == "u_driven_dense" and nt == len(U["keys"])
    # one V tuple fewer: the searching path, same triples minus those of the dropped key
    _, _, _, tm = tre.execute3(e, upper, ext, til, uk, ut, vk[1:].contiguous(), vt[1:].contiguous(), xk, xt,
                               timing=True)
    assert tm["join_path"] == "u_driven"


@pytest.mark.parametrize("seed", range(12))
def test_execute3_dense_gpu(orc, seed):
    rng = np.random.default_rng(6100 + seed)
    case = _complete(rng, _case3(rng), [1.0, 0.5, 0.05][seed % 3])
    say("execute3 dense", seed, case[0], case[1], case[2], case[3], len(case[4]["keys"]))
    _run_dense(orc, case)


@pytest.mark.parametrize("seed", range(12))
def test_masked_dense_gpu(orc, seed):
    rng = np.random.default_rng(6200 + seed)
    case = _complete(rng, _case_masked(rng), [1.0, 0.4, 0.05][seed % 3])
    say("masked dense", seed, case[0], case[1], case[2], case[3], len(case[4]["keys"]))
    _run_dense(orc, case)


@pytest.mark.parametrize("masked", [False, True])
def test_dense_key_errors_gpu(masked):
    """Key errors on the dense path: out-of-range U values (clamped on the
    device, reported by the key checks), unsorted U, a repeated key in a
    complete-sized V, and too small an output capacity after a good key set
    (capacity) versus after a bad one (the key error wins)."""
    import torch

    import paper_2603_08957_amd as tre

    rng = np.random.default_rng(91)
    if masked:
        e, upper, ext, til = "ij,ik,jk->ij", "ij", {"i": 12, "j": 9, "k": 33}, {"i": 1, "j": 1}
    else:
        e, upper, ext, til = "ijk,jr,kr->ir", "ijk", {"i": 8, "j": 12, "k": 16, "r": 5}, {"i": 4, "j": 4, "k": 4}
    u, v, x = e.split("->")[0].split(",")
    U = _relation(rng, u, upper, ext, til, 0.7)
    V = _relation(rng, v, upper, ext, til, 1.0)
    X = _relation(rng, x, upper, ext, til, 1.0)
    uk, ut = to_dev(U)
    vk, vt = to_dev(V)
    xk, xt = to_dev(X)
    op = tre.Einsum3(e, upper, ext, til, len(U["keys"]))
    op(uk, ut, vk, vt, xk, xt)
    bad = uk.clone()
    bad[-1, -1] = ext[u[-1]] // til[u[-1]]  # one past the last tile along U's last label
    with pytest.raises(tre.TreError) as err:
        op(bad, ut, vk, vt, xk, xt)
    assert err.value.status == "TRE_E_KEYRANGE"
    with pytest.raises(tre.TreError) as err:
        op(uk.flip(0).contiguous(), ut, vk, vt, xk, xt)
    assert err.value.status == "TRE_E_UNSORTED"
    vdup = vk.clone()
    vdup[1] = vdup[0]
    with pytest.raises(tre.TreError) as err:
        op(uk, ut, vdup, vt, xk, xt)
    assert err.value.status == "TRE_E_DUPKEY"
    small = (torch.empty((1, op.w_arity), dtype=torch.int32, device="cuda"),
             torch.empty((1, op.w_tile_elems), dtype=torch.float32, device="cuda"))
    with pytest.raises(tre.TreError) as err:
        op(uk, ut, vk, vt, xk, xt, out=small)
    assert err.value.status == "TRE_E_CAPACITY"
    with pytest.raises(tre.TreError) as err:
        op(bad, ut, vk, vt, xk, xt, out=small)
    assert err.value.status == "TRE_E_KEYRANGE"
