"""Shared test helpers: move seeded relations to the device, run the HIP path
through the C ABI, run the oracle on the same inputs, compare.

Comparison rules
* pair list and output key set: bit-exact, as sequences in canonical order;
* values: err = |gpu - oracle| / mag, mag = sum of |products| (fp64), the
  componentwise bound of a floating-point sum of products; where mag == 0 the
  GPU value must be exactly 0.  Tolerances: 1e-4 for fp32 inputs, 1e-2 for
  bf16 inputs with fp32 accumulation.
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


def check(out, ref, dtype: str, check_pairs=True):
    """Assert GPU output == oracle result under the comparison rules."""
    wk = out.w_keys.cpu().numpy()
    assert out.n_w == len(ref.wkeys), (out.n_w, len(ref.wkeys))
    if out.n_w:
        assert np.array_equal(wk.reshape(out.n_w, -1), ref.wkeys.reshape(out.n_w, -1)), "output key set differs"
    if check_pairs:
        assert out.n_pairs == len(ref.pairs), (out.n_pairs, len(ref.pairs))
        assert np.array_equal(out.pairs.cpu().numpy(), ref.pairs), "pair list differs"
    got = out.w_tiles.cpu().numpy()
    worst, zeros_ok = value_error(got, ref.acc, ref.mag)
    assert zeros_ok, "non-zero value where every product is zero"
    assert worst <= TOL[dtype], f"max mag-relative error {worst:.3e} > {TOL[dtype]}"
    return worst
