"""Shared test helpers: move seeded relations to the device, run the HIP path
through the C ABI, run the oracle on the same inputs, compare.

Comparison rules
* pair list and output key set: bit-exact, as sequences in canonical order;
* values: err = |gpu - oracle| / mag, mag = sum of |products| (fp64), the
  componentwise bound of a floating-point sum of products; where mag == 0 the
  GPU value must be exactly 0.  Tolerances: 1e-4 for fp32 inputs, 1e-2 for
  bf16 inputs with fp32 accumulation.
* plain relative figures, on the same tolerances:
  - normwise: max|g - r| / max|r| over the compared tiles;
  - elementwise: |g - r| / |r| over the entries with |r| >= 1e-3 max|r|,
    asserted on those among them whose condition number kappa = mag / |r|
    lets the arithmetic meet the tolerance at all, kappa <= 0.1 tol / u
    with u = 2^-24 for an fp32 sum (the plain error is at most kappa times
    the mag-relative error, which is a few u), and u = 2^-8 where the GPU
    and the oracle each round a chain's intermediate to bf16 (a one-ulp
    difference in an input then moves the sum by about kappa u, so no
    entry qualifies at 1e-2 and the figures are reported only).  Entries
    with more cancellation are reported, not asserted: for sums of ~800
    N(0,1) products a plain fp32 sum of exact products already exceeds 1e-4
    on some of them.
"""
from __future__ import annotations

import numpy as np

TOL = {"f32": 1e-4, "bf16": 1e-2}


def to_dev(rel: dict):
    """(keys, tiles) as torch tensors on cuda:0."""
    import torch

    keys = torch.from_numpy(np.ascontiguousarray(rel["keys"], dtype=np.int32)).cuda()
    t = np.ascontiguousarray(rel["tiles"])
    if rel["dtype"] == "bf16":
        tiles = torch.from_numpy(t.view(np.int16)).cuda().view(torch.bfloat16)
    else:
        tiles = torch.from_numpy(t.astype(np.float32, copy=False)).cuda()
    return keys, tiles


def gpu_run(spec: dict, U: dict, V: dict, want_pairs=True, **plan_kw):
    import paper_2603_08957_amd as tre

    plan = tre.Plan.from_spec(spec, **plan_kw)
    uk, ut = to_dev(U)
    vk, vt = to_dev(V)
    out = tre.einsum(plan, uk, ut, vk, vt, want_pairs=want_pairs)
    return plan, out


def value_error(got: np.ndarray, acc: np.ndarray, mag: np.ndarray):
    """Max of |got - acc| / mag over mag > 0, and whether every mag == 0
    entry is exactly zero."""
    got = np.asarray(got, dtype=np.float64)
    nz = mag > 0
    err = np.abs(got - acc)
    worst = float((err[nz] / mag[nz]).max()) if nz.any() else 0.0
    zeros_ok = bool(np.all(got[~nz] == 0.0))
    return worst, zeros_ok


U_ACC = 2.0 ** -24  # unit roundoff of the fp32 accumulator


U_BF16 = 2.0 ** -8  # unit roundoff of bf16 (8-bit significand), for intermediates rounded on both sides


def value_figures(got: np.ndarray, acc: np.ndarray, mag: np.ndarray, tol: float, u: float = U_ACC):
    """All value figures of a comparison: mag-relative max, normwise plain
    relative, elementwise plain relative on |r| >= 1e-3 max|r| (all of them,
    and those with kappa <= 0.1 tol / u), whether mag == 0 entries are 0.
    ``u`` is the unit roundoff that separates the two sides' inputs to the
    final sum: the fp32 accumulator's, or bf16's when both sides round an
    intermediate to bf16 on their own (a chain compared end to end)."""
    got = np.asarray(got, dtype=np.float64).reshape(acc.shape)
    worst, zeros_ok = value_error(got, acc, mag)
    d = np.abs(got - acc)
    ra = np.abs(acc)
    rmax = float(ra.max()) if ra.size else 0.0
    normwise = float(d.max() / rmax) if rmax > 0 else float(d.max(initial=0.0))
    big = ra >= 1e-3 * rmax if rmax > 0 else np.zeros(ra.shape, bool)
    kappa = np.where(ra > 0, mag / np.where(ra > 0, ra, 1.0), np.inf)
    wc = big & (kappa <= 0.1 * tol / u)
    rel = lambda m: float((d[m] / ra[m]).max()) if m.any() else 0.0  # noqa: E731
    return {"mag_rel": worst, "normwise_rel": normwise, "plain_rel_big": rel(big), "n_big": int(big.sum()),
            "plain_rel_wc": rel(wc), "n_wc": int(wc.sum()), "zeros_ok": zeros_ok}


def assert_values(got, acc, mag, dtype: str, where: str = "", u: float = U_ACC):
    """Assert the value rules at the dtype's tolerance; returns the figures."""
    tol = TOL[dtype]
    f = value_figures(got, acc, mag, tol, u)
    tag = f"{where}: " if where else ""
    assert f["zeros_ok"], tag + "non-zero value where every product is zero"
    assert f["mag_rel"] <= tol, tag + f"max mag-relative error {f['mag_rel']:.3e} > {tol}"
    assert f["normwise_rel"] <= tol, tag + f"max|g-r|/max|r| {f['normwise_rel']:.3e} > {tol}"
    assert f["plain_rel_wc"] <= tol, tag + f"plain relative error {f['plain_rel_wc']:.3e} > {tol} on " \
                                           f"{f['n_wc']} well-conditioned entries"
    return f


def check(out, ref, dtype: str, check_pairs=True):
    """Assert GPU output == oracle result under the comparison rules."""
    wk = out.w_keys.cpu().numpy()
    assert out.n_w == len(ref.wkeys), (out.n_w, len(ref.wkeys))
    if out.n_w:
        assert np.array_equal(wk.reshape(out.n_w, -1), ref.wkeys.reshape(out.n_w, -1)), "output key set differs"
    if check_pairs:
        assert out.n_pairs == len(ref.pairs), (out.n_pairs, len(ref.pairs))
        assert np.array_equal(out.pairs.cpu().numpy(), ref.pairs), "pair list differs"
    got = out.w_tiles.float().cpu().numpy()
    return assert_values(got, ref.acc, ref.mag, dtype)["mag_rel"]
