"""GPU parity of the three-operand EinSum (tre_execute3) against the oracle's
plain per-triple evaluation (oracle.eval3): output keys and triple count
bit-exact, values within the mag-relative tolerance (1e-4, fp32)."""
import sys

import numpy as np
import pytest

import workloads
from _parity import TOL, to_dev, value_error

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
    worst, zeros_ok = value_error(wt.cpu().numpy(), acc, mag)
    assert zeros_ok, "non-zero value where every product is zero"
    assert worst <= TOL["f32"], f"max mag-relative error {worst:.3e}"
    return worst


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
