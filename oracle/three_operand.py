"""Oracle for one three-operand EinSum whose two small operands meet the large
one on different promoted labels and share one demoted label r, in one of two
forms:

* r is kept in the output and the joined labels are summed (the non-binary
  EinSum of Sec. 8, e.g. A[i,r] = sum_jk T[i,j,k] B[j,r] C[k,r]);
* the output has exactly U's labels and r is summed ("masked" form, e.g. the
  attention scores S[i,j] = sum_k A[i,j] T0[i,k] T1[j,k] of the graph
  transformer in Sec. 9, which Table gt-schema computes as two binary
  EinSums: T2[i,j,k] = T0[i,k] A[i,j] with no aggregation, then
  T3[i,j] = sum_k T2[i,j,k] T1[j,k]).

TEST INFRASTRUCTURE, NOT PART OF THE PRODUCT (see the package docstring).

Written as the plain definition, in numpy, fp64:

* key level (Sec. 5, the join and GROUP BY of Eq. "eqn-TRA" extended to three
  relations): a U tuple is matched when V holds a tuple with U's key on the
  label V shares with U, and X one with U's key on the label X shares with U;
  the output keys are the distinct projections of matched U keys onto W's
  promoted labels, sorted lexicographically in W's promoted-label order;
* value level: every matched triple contributes the kernel function K of
  Sec. 5 -- the EinSum restricted to the tile labels -- applied to its three
  tiles (numpy.einsum on one triple of tiles, the library routine serving as
  that step), and the contributions are summed per output key in U order;
  ``mag`` sums the same einsum over absolute values (the componentwise bound
  used by the parity tolerance).
"""
from __future__ import annotations

from dataclasses import dataclass

import numpy as np


class Spec3Error(ValueError):
    def __init__(self, category: str, msg: str):
        self.category = category
        super().__init__(f"{category}: {msg}")


@dataclass
class Spec3:
    u: str
    v: str
    x: str
    w: str
    upper: str
    a: str  # label V shares with U
    b: str  # label X shares with U
    r: str  # label V and X share (kept in W, or summed in the masked form)
    extents: dict
    tiles: dict
    masked: bool = False  # W has exactly U's labels and r is summed

    def tile_ext(self, c: str) -> int:
        return int(self.tiles[c]) if c in self.upper else int(self.extents[c])

    def key_labels(self, op: str) -> str:
        return "".join(c for c in op if c in self.upper)

    def tile_shape(self, op: str):
        return tuple(self.tile_ext(c) for c in op)


def parse3(einsum: str, upper: str, extents: dict, tiles: dict) -> Spec3:
    """Read "U,V,X->W" and check the structure this evaluation covers."""
    if "->" not in einsum:
        raise Spec3Error("PARSE", "missing ->")
    lhs, w = einsum.split("->")
    ops = lhs.split(",")
    if len(ops) != 3:
        raise Spec3Error("PARSE", "three inputs expected")
    u, v, x = ops
    for op in (u, v, x, w):
        if not op.isalpha() or not op.islower() or len(set(op)) != len(op):
            raise Spec3Error("PARSE", f"bad operand {op!r}")
    if len(v) != 2 or len(x) != 2:
        raise Spec3Error("SPLIT", "the two small operands have two labels each")
    shared = set(v) & set(x)
    if len(shared) != 1:
        raise Spec3Error("SPLIT", "the small operands share exactly one label")
    r = shared.pop()
    a = (set(v) - {r}).pop()
    b = (set(x) - {r}).pop()
    if r in u or a not in u or b not in u or a == b:
        raise Spec3Error("SPLIT", "each small operand meets U on its own label")
    masked = w == u
    if not masked and set(w) != (set(u) - {a, b}) | {r}:
        raise Spec3Error("SPLIT", "W holds U's other labels and the shared label, or exactly U's labels")
    if set(u[-2:]) != {a, b}:
        raise Spec3Error("SPLIT", "the two joined labels are U's last two")
    for c in upper:
        if c not in set(u) | {r}:
            raise Spec3Error("SPLIT", f"promoted label {c!r} not in the expression")
    if a not in upper or b not in upper or r in upper:
        raise Spec3Error("SPLIT", "joined labels promoted, shared label demoted")
    for c in set(u) | {r}:
        e = int(extents[c])
        t = int(tiles[c]) if c in upper else e
        if e < 1 or t < 1 or e % t:
            raise Spec3Error("SHAPE", f"tile of {c!r} does not divide its extent")
    return Spec3(u, v, x, w, upper, a, b, r, dict(extents), dict(tiles), masked)


def _check_keys(keys: np.ndarray, radix: list, what: str):
    if len(keys) == 0:
        return
    if keys.min(initial=0) < 0 or any((keys[:, i] >= radix[i]).any() for i in range(len(radix))):
        raise Spec3Error("KEYRANGE", what)
    for s in range(1, len(keys)):
        a, b = tuple(keys[s - 1]), tuple(keys[s])
        if a == b:
            raise Spec3Error("DUPKEY", what)
        if a > b:
            raise Spec3Error("UNSORTED", what)


def eval3(einsum: str, upper: str, extents: dict, tiles: dict, U: dict, V: dict, X: dict):
    """Returns (wkeys int32 [n_w x r_W], acc float64 [n_w x tile_elems(W)],
    mag float64 [same], triples int64 [n_t x 3] (u, v, x) in U order).
    Relations are dicts with "keys" int32 [n x r] and "tiles" float arrays
    (float32 / float64 values, or uint16 bf16 bits with "dtype": "bf16")."""
    sp = parse3(einsum, upper, extents, tiles)

    def vals(rel, op):
        t = np.asarray(rel["tiles"])
        if rel.get("dtype") == "bf16":
            t = (t.astype(np.uint16).astype(np.uint32) << 16).view(np.float32)
        n = len(rel["keys"])
        return t.astype(np.float64).reshape((n,) + sp.tile_shape(op))

    rels = {}
    for name, op, rel in (("U", sp.u, U), ("V", sp.v, V), ("X", sp.x, X)):
        kl = sp.key_labels(op)
        keys = np.asarray(rel["keys"], dtype=np.int64).reshape(len(rel["keys"]), len(kl))
        if not kl and len(keys) > 1:
            raise Spec3Error("DUPKEY", f"{name} has no promoted labels but several tuples")
        _check_keys(keys, [int(extents[c]) // int(tiles[c]) for c in kl], name)
        rels[name] = (kl, keys, vals(rel, op))
    ukl, ukeys, ut = rels["U"]
    vkl, vkeys, vt = rels["V"]
    xkl, xkeys, xt = rels["X"]
    # V is keyed by its one promoted label a, X by b
    v_of = {int(k[0]): i for i, k in enumerate(vkeys)}
    x_of = {int(k[0]): i for i, k in enumerate(xkeys)}
    wkl = sp.key_labels(sp.w)
    triples, wk = [], []
    for s in range(len(ukeys)):
        key = dict(zip(ukl, (int(q) for q in ukeys[s])))
        iv, ix = v_of.get(key[sp.a]), x_of.get(key[sp.b])
        if iv is None or ix is None:
            continue
        triples.append((s, iv, ix))
        wk.append(tuple(key[c] for c in wkl))
    out_keys = sorted(set(wk))
    pos = {k: i for i, k in enumerate(out_keys)}
    w_shape = sp.tile_shape(sp.w)
    acc = np.zeros((len(out_keys),) + w_shape)
    mag = np.zeros_like(acc)
    expr = f"{sp.u},{sp.v},{sp.x}->{sp.w}"
    for (s, iv, ix), k in zip(triples, wk):
        q = pos[k]
        acc[q] += np.einsum(expr, ut[s], vt[iv], xt[ix], optimize=True)
        mag[q] += np.einsum(expr, np.abs(ut[s]), np.abs(vt[iv]), np.abs(xt[ix]), optimize=True)
    n_w = len(out_keys)
    wkeys = np.array(out_keys, dtype=np.int32).reshape(n_w, len(wkl))
    return (wkeys, acc.reshape(n_w, -1), mag.reshape(n_w, -1),
            np.array(triples, dtype=np.int64).reshape(len(triples), 3))
