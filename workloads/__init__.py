"""Seeded synthetic workloads shaped like the paper's (GNN message passing,
block-sparse products, a sparse 3-way contraction).

This module only draws random inputs and lays them out as tensor relations
(keys + dense tiles, Sec. 4.2): it holds none of the join / contraction /
aggregation arithmetic.  Both the HIP library's tests and the CPU oracle take
their inputs from here; neither is imported by this module.

Conventions
-----------
* RNG: ``numpy.random.default_rng(seed)`` (PCG64); draw order is fixed per
  generator.  Workload ``c`` (1-based) uses seed ``SEED_BASE + c``.
* bf16 inputs are drawn in fp32 and rounded to nearest even by torch's CPU
  conversion; arrays hold the raw bf16 bits as ``uint16``.
* A relation is a dict:
    ``keys``  [n, r] int32, sorted strictly increasing (lexicographic),
    ``tiles`` [n, tile_elems] float32 or uint16 (bf16 bits), row-major over
              the operand's labels in EinSum-string order,
    ``dtype`` "f32" | "bf16".
  A relation too large to hold as dense tiles on the host (the 128x128-tiled
  adjacency of the 262,144-vertex graph) instead carries ``coo`` = (coords
  [nnz, 2] int64 global, vals float64) plus ``slot``/``offset`` per entry
  (tuple index and in-tile offset) so tiles can be materialised on the device.
"""
from __future__ import annotations

import numpy as np

SEED_BASE = 20260308


def to_bf16_bits(x: np.ndarray) -> np.ndarray:
    import torch

    t = torch.from_numpy(np.ascontiguousarray(x, dtype=np.float32)).to(torch.bfloat16)
    return t.view(torch.int16).numpy().view(np.uint16).copy()


def bf16_bits_to_f32(b: np.ndarray) -> np.ndarray:
    return (np.asarray(b, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32)


def spec(einsum: str, upper: str, extents: dict, tiles: dict, dtype: str) -> dict:
    return {"einsum": einsum, "upper": upper, "extents": dict(extents), "tiles": dict(tiles), "dtype": dtype}


# ----------------------------------------------------------------- graphs

def powerlaw_degrees(rng, n: int, alpha: float, mean: float) -> np.ndarray:
    """Out-degrees with pmf ~ d^-alpha: d = clip(floor(x_min * u^(-1/(alpha-1))), 1, n-1),
    u ~ U(0,1], x_min bisected so the sample mean is ``mean``."""
    u = 1.0 - rng.random(n)
    p = -1.0 / (alpha - 1.0)
    base = u ** p

    def degs(xmin):
        return np.clip(np.floor(xmin * base), 1, n - 1)

    lo, hi = 1e-3, float(mean)
    for _ in range(80):
        mid = 0.5 * (lo + hi)
        if degs(mid).mean() < mean:
            lo = mid
        else:
            hi = mid
    return degs(hi).astype(np.int64)


def distinct_targets(rng, n: int, deg: np.ndarray):
    """For each source s, deg[s] distinct targets uniform over [0, n).
    Returns (src, dst) sorted by (src, dst)."""
    deg = np.asarray(deg, dtype=np.int64)
    hub = deg > n // 8
    src_parts, dst_parts = [], []
    # ordinary sources: draw with replacement, redraw duplicates until none
    s_ord = np.repeat(np.nonzero(~hub)[0], deg[~hub])
    d_ord = rng.integers(0, n, size=s_ord.size)
    while True:
        code = s_ord * n + d_ord
        order = np.argsort(code, kind="stable")
        cs = code[order]
        dup = np.zeros(cs.size, dtype=bool)
        dup[1:] = cs[1:] == cs[:-1]
        if not dup.any():
            break
        idx = order[dup]
        d_ord[idx] = rng.integers(0, n, size=idx.size)
    src_parts.append(s_ord)
    dst_parts.append(d_ord)
    # hubs (more than n/8 targets): sample without replacement directly
    for s in np.nonzero(hub)[0]:
        t = rng.choice(n, size=int(deg[s]), replace=False)
        src_parts.append(np.full(t.size, s, dtype=np.int64))
        dst_parts.append(t.astype(np.int64))
    src = np.concatenate(src_parts)
    dst = np.concatenate(dst_parts)
    order = np.lexsort((dst, src))
    return src[order], dst[order]


def _block_relation_from_coo(rows, cols, vals, t_r: int, t_c: int, n_cols: int):
    """Relation keyed (R, C) = (row // t_r, col // t_c) holding the blocks with
    at least one entry; per-entry slot and row-major in-tile offset."""
    nbc = n_cols // t_c
    code = (rows // t_r) * nbc + (cols // t_c)
    ucode, slot = np.unique(code, return_inverse=True)
    keys = np.stack([ucode // nbc, ucode % nbc], axis=1).astype(np.int32)
    offset = (rows % t_r) * t_c + (cols % t_c)
    return keys, slot.astype(np.int64), offset.astype(np.int64)


def gnn_chain(n: int, emb: int, z_out: int, tile_e1: int, tile_e2: int, degree: dict, dtype: str,
              seed: int, dense_y_tiles: bool = True, y_layout: str = "jk") -> dict:
    """GNN message passing (X.Y)^T.Z as two binary EinSums (Sec. 1, Sec. 4.3).

    X [emb x n] holds one embedding column per vertex, Y [n x n] the directed
    edges (Y[j, k] != 0 for an edge j -> k), Z [emb x z_out].
      E1  T[k, i] = sum_j X[i, j] Y[j, k]   "ij,jk->ki", promoted {j, k}
      E2  U[k, m] = sum_i T[k, i] Z[i, m]   "ki,im->km", promoted {k}
    ``degree``: {"kind": "fixed", "d": 8, "values": "ones"} or
                {"kind": "powerlaw", "alpha": 2.1, "mean": 16, "values": "normal"}.
    ``y_layout``: "jk" stores the adjacency keyed (J, K) (source-major) and
    E1 reads it as "ij,jk->ki"; "kj" stores the same tuples keyed (K, J)
    (destination-major, the transposed tiles) and E1 is "ij,kj->ki".  The
    tensor and every drawn value are the same either way.
    Draw order: degrees, targets, edge values, X, Z."""
    rng = np.random.default_rng(seed)
    if degree["kind"] == "fixed":
        deg = np.full(n, degree["d"], dtype=np.int64)
    else:
        deg = powerlaw_degrees(rng, n, degree["alpha"], degree["mean"])
    src, dst = distinct_targets(rng, n, deg)
    if degree.get("values", "normal") == "ones":
        ev = np.ones(src.size, dtype=np.float32)
    else:
        ev = rng.standard_normal(src.size, dtype=np.float32)
    X = rng.standard_normal((emb, n), dtype=np.float32)
    Z = rng.standard_normal((emb, z_out), dtype=np.float32)
    if dtype == "bf16":
        ev_s, X_s, Z_s = to_bf16_bits(ev), to_bf16_bits(X), to_bf16_bits(Z)
        ev_v = bf16_bits_to_f32(ev_s).astype(np.float64)
    else:
        ev_s, X_s, Z_s = ev, X, Z
        ev_v = ev.astype(np.float64)
    t = tile_e1
    nb = n // t
    # X keyed J: tile [i][j'] = X[:, J*t:(J+1)*t]
    x_tiles = np.ascontiguousarray(X_s.reshape(emb, nb, t).transpose(1, 0, 2)).reshape(nb, emb * t)
    x_rel = {"keys": np.arange(nb, dtype=np.int32).reshape(nb, 1), "tiles": x_tiles, "dtype": dtype}
    if y_layout == "kj":
        order = np.lexsort((src, dst))  # destination-major
        rows, cols, ev_s, ev_v = dst[order], src[order], ev_s[order], ev_v[order]
    elif y_layout == "jk":
        rows, cols = src, dst
    else:
        raise ValueError(y_layout)
    ykeys, slot, off = _block_relation_from_coo(rows, cols, None, t, t, n)
    y_rel = {"keys": ykeys, "dtype": dtype, "coo": (np.stack([rows, cols], axis=1), ev_v),
             "slot": slot, "offset": off, "values": ev_s, "tile_elems": t * t}
    if dense_y_tiles:
        yt = np.zeros((len(ykeys), t * t), dtype=ev_s.dtype)
        yt[slot, off] = ev_s
        y_rel["tiles"] = yt
    z_rel = {"keys": np.zeros((1, 0), dtype=np.int32), "tiles": np.ascontiguousarray(Z_s).reshape(1, -1),
             "dtype": dtype}
    e1 = spec("ij,jk->ki" if y_layout == "jk" else "ij,kj->ki", "jk", {"i": emb, "j": n, "k": n}, {"j": t, "k": t},
              dtype)
    e2 = spec("ki,im->km", "k", {"k": n, "i": emb, "m": z_out}, {"k": tile_e2}, dtype)
    return {"E1": e1, "E2": e2, "X": x_rel, "Y": y_rel, "Z": z_rel, "n_edges": int(src.size),
            "n": n, "emb": emb, "z_out": z_out, "tile_e1": t, "tile_e2": tile_e2, "dtype": dtype,
            "y_layout": y_layout, "y_k_col": 1 if y_layout == "jk" else 0}


# ----------------------------------------------------------- block sparse

def block_sparse(n: int, n_cols: int, block: int, density: float, seed: int) -> dict:
    """Block-sparse A [n x n] times dense B [n x n_cols], fp32.
    A keeps round(density * (n/block)^2) blocks chosen uniformly without
    replacement, N(0,1) inside; "ik,kn->in" with i, k promoted (tile block),
    n demoted.  Draw order: block ids, A values, B."""
    rng = np.random.default_rng(seed)
    nb = n // block
    nblk = int(round(density * nb * nb))
    ids = np.sort(rng.choice(nb * nb, size=nblk, replace=False))
    a_tiles = rng.standard_normal((nblk, block * block), dtype=np.float32)
    B = rng.standard_normal((n, n_cols), dtype=np.float32)
    a_keys = np.stack([ids // nb, ids % nb], axis=1).astype(np.int32)
    a_rel = {"keys": a_keys, "tiles": a_tiles, "dtype": "f32"}
    b_rel = {"keys": np.arange(nb, dtype=np.int32).reshape(nb, 1), "tiles": B.reshape(nb, block * n_cols),
             "dtype": "f32"}
    e = spec("ik,kn->in", "ik", {"i": n, "k": n, "n": n_cols}, {"i": block, "k": block}, "f32")
    return {"E": e, "A": a_rel, "B": b_rel, "n": n, "n_cols": n_cols, "block": block}


# -------------------------------------------------------- sparse 3-way

def sparse_3way(n: int, r: int, block: int, block_density: float, fill: float, seed: int) -> dict:
    """A[i, r] = sum_jk T[i, j, k] B[j, r] C[k, r], fp32, as two binary EinSums
    along the path E1 = T join B on j, E2 = W join C on k (Sec. 8, non-binary
    EinSum split into binary ones):
      E1  W[i, k, r] = sum_j T[i, j, k] B[j, r]   "ijk,jr->ikr", promoted {i, j, k}
      E2  A[i, r]    = sum_k W[i, k, r] C[k, r]   "ikr,kr->ir",  promoted {i, k}
    T keeps round(block_density * (n/block)^3) blocks uniformly, each with
    round(fill * block^3) non-zeros at uniform positions, N(0,1).
    Draw order: block ids, per-block positions, values, B, C."""
    rng = np.random.default_rng(seed)
    nb = n // block
    be = block ** 3
    nblk = int(round(block_density * nb ** 3))
    nnz = int(round(fill * be))
    ids = np.sort(rng.choice(nb ** 3, size=nblk, replace=False))
    t_tiles = np.zeros((nblk, be), dtype=np.float32)
    pos = np.empty((nblk, nnz), dtype=np.int64)
    for b in range(nblk):
        pos[b] = rng.choice(be, size=nnz, replace=False)
    vals = rng.standard_normal((nblk, nnz), dtype=np.float32)
    np.put_along_axis(t_tiles, pos, vals, axis=1)
    B = rng.standard_normal((n, r), dtype=np.float32)
    C = rng.standard_normal((n, r), dtype=np.float32)
    t_keys = np.stack([ids // (nb * nb), (ids // nb) % nb, ids % nb], axis=1).astype(np.int32)
    t_rel = {"keys": t_keys, "tiles": t_tiles, "dtype": "f32"}
    b_rel = {"keys": np.arange(nb, dtype=np.int32).reshape(nb, 1), "tiles": B.reshape(nb, block * r), "dtype": "f32"}
    c_rel = {"keys": np.arange(nb, dtype=np.int32).reshape(nb, 1), "tiles": C.reshape(nb, block * r), "dtype": "f32"}
    e1 = spec("ijk,jr->ikr", "ijk", {"i": n, "j": n, "k": n, "r": r}, {"i": block, "j": block, "k": block}, "f32")
    e2 = spec("ikr,kr->ir", "ik", {"i": n, "k": n, "r": r}, {"i": block, "k": block}, "f32")
    return {"E1": e1, "E2": e2, "T": t_rel, "B": b_rel, "C": c_rel, "n": n, "r": r, "block": block}


# ------------------------------------------------------- graph attention

def graph_attention(n: int, n_feat: int, feat_density: float, d_k: int, degree: dict, seed: int) -> dict:
    """Attention scores of a graph transformer before normalisation (Sec. 9,
    the plan of Table gt-schema), fp32:
      E1  T0[i, k] = sum_m X[i, m] WQ[m, k]    "im,mk->ik",  promoted {i, m}
      E2  T1[j, k] = sum_n X[j, n] WK[n, k]    "jn,nk->jk",  promoted {j, n}
      E3  T2[i, j, k] = T0[i, k] A[i, j]       "ik,ij->ijk", promoted {i, j}, no aggregation
      E4  T3[i, j] = sum_k T2[i, j, k] T1[j, k] "ijk,jk->ij", promoted {i, j}
      E5  S[i, j] = T3[i, j] / sqrt(d_k)       (unary)
    E3 and E4 together are the masked three-operand EinSum "ij,ik,jk->ij"
    (U = A, V = T0, X = T1).
    X: binary bag-of-words features, each (node, feature) present with
    probability ``feat_density`` (a node with none gets one uniform feature),
    stored as scalar tuples keyed (i, m); WQ, WK: n_feat x d_k N(0,1), stored
    as d_k-vectors keyed by the feature; A: directed edges with the out-degree
    law of ``degree`` and distinct uniform targets, value 1, stored as scalar
    tuples keyed (i, j).  Draw order: features, the fix-up features, WQ, WK,
    degrees, targets."""
    rng = np.random.default_rng(seed)
    F = rng.random((n, n_feat)) < feat_density
    empty = np.nonzero(~F.any(axis=1))[0]
    F[empty, rng.integers(0, n_feat, size=empty.size)] = True
    fi, fm = np.nonzero(F)
    WQ = rng.standard_normal((n_feat, d_k), dtype=np.float32)
    WK = rng.standard_normal((n_feat, d_k), dtype=np.float32)
    if degree["kind"] == "fixed":
        deg = np.full(n, degree["d"], dtype=np.int64)
    else:
        deg = powerlaw_degrees(rng, n, degree["alpha"], degree["mean"])
    src, dst = distinct_targets(rng, n, deg)
    x_rel = {"keys": np.stack([fi, fm], axis=1).astype(np.int32), "tiles": np.ones((fi.size, 1), np.float32),
             "dtype": "f32"}
    fkeys = np.arange(n_feat, dtype=np.int32).reshape(n_feat, 1)
    wq_rel = {"keys": fkeys, "tiles": WQ, "dtype": "f32"}
    wk_rel = {"keys": fkeys.copy(), "tiles": WK, "dtype": "f32"}
    a_rel = {"keys": np.stack([src, dst], axis=1).astype(np.int32), "tiles": np.ones((src.size, 1), np.float32),
             "dtype": "f32"}
    one = {"i": 1, "j": 1, "m": 1, "n": 1}
    e1 = spec("im,mk->ik", "im", {"i": n, "m": n_feat, "k": d_k}, one, "f32")
    e2 = spec("jn,nk->jk", "jn", {"j": n, "n": n_feat, "k": d_k}, one, "f32")
    e3 = spec("ik,ij->ijk", "ij", {"i": n, "j": n, "k": d_k}, one, "f32")
    e4 = spec("ijk,jk->ij", "ij", {"i": n, "j": n, "k": d_k}, one, "f32")
    e34 = spec("ij,ik,jk->ij", "ij", {"i": n, "j": n, "k": d_k}, one, "f32")
    return {"E1": e1, "E2": e2, "E3": e3, "E4": e4, "E34": e34, "X": x_rel, "WQ": wq_rel, "WK": wk_rel,
            "A": a_rel, "scale": float(1.0 / np.sqrt(d_k)), "n": n, "n_feat": n_feat, "d_k": d_k,
            "n_edges": int(src.size), "n_feat_entries": int(fi.size)}


# ------------------------------------------------------- random small plans

def random_relation(rng, labels: str, upper: str, extents: dict, tiles: dict, dtype: str, keep: float,
                    zero_frac: float = 0.0) -> dict:
    """A relation over ``labels``: every key tuple of the promoted labels is
    kept with probability ``keep``; tile entries N(0,1) with a fraction
    ``zero_frac`` set to exactly zero."""
    kl = [c for c in labels if c in upper]
    radix = [extents[c] // tiles[c] for c in kl]
    shape = [tiles[c] if c in upper else extents[c] for c in labels]
    te = int(np.prod(shape)) if shape else 1
    if kl:
        grid = np.stack(np.meshgrid(*[np.arange(x) for x in radix], indexing="ij"), axis=-1).reshape(-1, len(kl))
        mask = rng.random(len(grid)) < keep
        keys = grid[mask].astype(np.int32)
    else:
        keys = np.zeros((1 if rng.random() < max(keep, 0.5) else 0, 0), dtype=np.int32)
    vals = rng.standard_normal((len(keys), te), dtype=np.float32)
    if zero_frac > 0:
        vals[rng.random(vals.shape) < zero_frac] = 0.0
    tiles_arr = to_bf16_bits(vals) if dtype == "bf16" else vals
    return {"keys": keys, "tiles": tiles_arr, "dtype": dtype}


# --------------------------------------------------------- named configs

def config(c: int, scale: str = "full", **kw) -> dict:
    """The workloads (1-based; 6 is the graph-attention workload).  ``scale="small"`` gives a scaled-down twin
    with the same structure that the oracle finishes in seconds."""
    seed = SEED_BASE + c
    small = scale == "small"
    if c == 1:
        # the adjacency stored destination-major (keyed (K, J)), as for workload 5
        n = 1024 if small else 4096
        kw.setdefault("y_layout", "kj")
        return gnn_chain(n, 64, 32, 64, 64, {"kind": "fixed", "d": 8, "values": "ones"}, "f32", seed, **kw)
    if c == 2:
        # source-major (keyed (J, K)): its 128x128 MFMA path streams the tiles
        # with their rows contiguous
        n = 4096 if small else 262144
        return gnn_chain(n, 128, 128, 128, 128, {"kind": "powerlaw", "alpha": 2.1, "mean": 16, "values": "normal"},
                         "bf16", seed, dense_y_tiles=small, **kw)
    if c == 3:
        n = 2048 if small else 16384
        return block_sparse(n, 256 if small else 1024, 128, 0.05, seed)
    if c == 4:
        n = 512 if small else 4096
        return sparse_3way(n, 64, 32, 0.005 if not small else 0.05, 0.1, seed)
    if c == 5:
        # the adjacency as scalar tuples, stored destination-major (keyed (K, J))
        n = 4096 if small else 1048576
        kw.setdefault("y_layout", "kj")
        return gnn_chain(n, 256, 256, 1, 256, {"kind": "powerlaw", "alpha": 2.1, "mean": 32, "values": "normal"},
                         "bf16", seed, dense_y_tiles=True, **kw)
    if c == 6:
        # Amazon.Computers-shaped graph (13,752 nodes, ~0.4M edges, 767
        # features), key dimension 1024 as in Table gt-schema
        if small:
            return graph_attention(512, 64, 0.1, 128, {"kind": "powerlaw", "alpha": 2.1, "mean": 8}, seed)
        return graph_attention(13752, 767, 0.05, 1024, {"kind": "powerlaw", "alpha": 2.1, "mean": 29}, seed)
    raise ValueError(c)
