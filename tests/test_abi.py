"""C-ABI checks that need no GPU: the library loads, exports every function
include/tre.h declares, and its host planner agrees with the oracle's reading
of the same EinSums (key arity, tile sizes, errors)."""
import ctypes
import os
import re

import numpy as np
import pytest

from test_oracle import random_plan, split_einsum

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.fixture(scope="module")
def tre():
    import paper_2603_08957_amd as t

    t.lib()
    return t


def declared_functions():
    hdr = open(os.path.join(ROOT, "include", "tre.h")).read()
    hdr = re.sub(r"/\*.*?\*/", "", hdr, flags=re.S)
    return sorted(set(re.findall(r"\b(tre_[a-z0-9_]+)\s*\(", hdr)))


def test_exports_every_declared_symbol(tre):
    names = declared_functions()
    assert len(names) >= 15
    L = ctypes.CDLL(tre.tre.LIB_PATH)
    for n in names:
        assert hasattr(L, n), f"libtre.so does not export {n}"
    assert sorted(tre.EXPORTS) == names


def test_version_and_status_strings(tre):
    L = tre.lib()
    assert b"gfx950" in L.tre_version()
    for code, name in tre.tre.STATUS.items():
        assert L.tre_status_str(code).decode() == name


@pytest.mark.parametrize("seed", range(40))
def test_plan_matches_oracle_reading(orc, tre, seed):
    rng = np.random.default_rng(1000 + seed)
    e, upper, ext, til = random_plan(rng)
    p = tre.Plan(e, upper, ext, til, "f32")
    o = orc.Plan(e, upper, ext, til)
    assert p.key_arity == o.key_arity
    assert p.tile_elems == o.tile_elems
    assert p.key_labels == o.key_labels
    u, v, w = split_einsum(e)
    B, M, N, K = p.bmnk
    # per-pair flops: every label of U or V taken once at its tile extent
    sz = {c: (til[c] if c in upper else ext[c]) for c in set(u) | set(v)}
    prod = int(np.prod([sz[c] for c in set(u) | set(v)])) if (set(u) | set(v)) else 1
    assert B * M * N * K == prod
    assert p.flops_per_pair == 2 * prod


def test_roles_of_the_paper_examples(tre):
    # batch matmul with transposes (Sec. 3): b and j aggregated
    p = tre.Plan("ijb,jbk->ik", "", {"i": 10, "j": 100, "b": 20, "k": 2000}, {}, "f32")
    assert p.roles[ord("i") - 97] == "m" and p.roles[ord("k") - 97] == "n"
    assert p.roles[ord("j") - 97] == "k" and p.roles[ord("b") - 97] == "k"
    assert p.bmnk == (1, 10, 2000, 2000)
    # GNN chain E1 with vertex labels promoted (Sec. 4.3)
    p = tre.Plan("ij,jk->ki", "jk", {"i": 64, "j": 4096, "k": 4096}, {"j": 64, "k": 64}, "f32")
    assert p.key_labels == ["j", "jk", "k"] and p.n_join == 1 and p.group_needs_sort and not p.v_needs_sort
    assert p.kernel_class == "gemm" and p.bmnk == (1, 64, 64, 64)
    # per-vertex vectors and scalar edges: a scale kernel
    p = tre.Plan("ij,jk->ki", "jk", {"i": 256, "j": 1 << 20, "k": 1 << 20}, {"j": 1, "k": 1}, "bf16")
    assert p.kernel_class == "vec" and p.bmnk == (1, 256, 1, 1)
    # V keyed (K, J) with W keyed K: the join walks V and the pairs come out
    # grouped by K, nothing is sorted
    p = tre.Plan("ij,kj->ik", "jk", {"i": 8, "j": 8, "k": 8}, {"j": 2, "k": 2}, "f32")
    assert p.join_outer == "v" and not p.v_needs_sort and not p.group_needs_sort
    # V keyed (K, J) with K summed: V is sorted by its join key on the device
    p = tre.Plan("ij,kj->i", "jk", {"i": 8, "j": 8, "k": 8}, {"j": 2, "k": 2}, "f32")
    assert p.join_outer == "u" and p.v_needs_sort
    # V keyed (J, K): the join walks U and the pairs are sorted by K
    p = tre.Plan("ij,jk->ki", "jk", {"i": 8, "j": 8, "k": 8}, {"j": 2, "k": 2}, "f32")
    assert p.join_outer == "u" and p.group_needs_sort and not p.v_needs_sort


@pytest.mark.parametrize("e,upper,outer", [
    ("ij,kj->ki", "jk", "v"),      # adjacency keyed by destination, then source
    ("ja,kj->k", "jka", "v"),      # U keyed (J, A): each V tuple meets a run of U tuples
    ("jlx,kjl->kx", "jlk", "v"),   # two join labels, in the same order in U and V
    ("jx,kmj->kmx", "jkm", "v"),   # W keyed by two of V's labels
    ("jlx,klj->kx", "jlk", "u"),   # join labels in another order in V than in U
    ("ix,kj->ki", "ijk", "u"),     # W takes a label from U
    ("jx,jk->kx", "jk", "u"),      # V keyed (J, K): W's label is not V's prefix
])
def test_join_direction(tre, e, upper, outer):
    ext = {c: 8 for c in set(e) if c.isalpha()}
    p = tre.Plan(e, upper, ext, {c: 2 for c in upper}, "f32")
    assert p.join_outer == outer, (e, p.join_outer)
    if outer == "v":
        assert not p.group_needs_sort and not p.v_needs_sort


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
def test_plan_errors_match_oracle(orc, tre, e, upper, ext, til, cat):
    with pytest.raises(orc.OracleError) as eo:
        orc.Plan(e, upper, ext, til)
    with pytest.raises(tre.TreError) as et:
        tre.Plan(e, upper, ext, til, "f32")
    assert eo.value.category == cat
    assert et.value.status == "TRE_E_" + cat


def test_bad_dtype_and_options(tre):
    L = tre.lib()
    ext = np.full(26, 4, dtype=np.int64)
    til = np.ones(26, dtype=np.int32)
    h = ctypes.c_void_p()
    rc = L.tre_plan(b"ij,jk->ik", b"", ext.ctypes.data_as(ctypes.c_void_p), til.ctypes.data_as(ctypes.c_void_p), 7,
                    None, ctypes.byref(h))
    assert tre.tre.STATUS[rc] == "TRE_E_DTYPE"
    opt = tre.tre.Options(1, -1)
    rc = L.tre_plan(b"ij,jk->ik", b"", ext.ctypes.data_as(ctypes.c_void_p), til.ctypes.data_as(ctypes.c_void_p), 0,
                    ctypes.byref(opt), ctypes.byref(h))
    assert tre.tre.STATUS[rc] == "TRE_E_ARG"


def test_workspace_sizing(tre):
    p = tre.Plan("ij,jk->ki", "jk", {"i": 128, "j": 262144, "k": 262144}, {"j": 128, "k": 128}, "bf16")
    prev = 0
    for mp in [0, 1, 10, 1000, 10 ** 5, 3 * 10 ** 6]:
        b = p.workspace_bytes(2048, 2_300_000, mp)
        assert b % 256 == 0 and b >= prev
        prev = b
    L = tre.lib()
    ws = p.workspace_bytes(2048, 2_300_000, 2_300_000)
    mp = L.tre_workspace_max_pairs(p.handle, 2048, 2_300_000, ws)
    assert mp >= 2_300_000
    assert p.workspace_bytes(2048, 2_300_000, mp + 1) > ws
    assert L.tre_workspace_max_pairs(p.handle, 2048, 2_300_000, 16) == -1


def test_null_arguments_rejected_without_device(tre):
    """Argument errors are caught on the host before any device call."""
    L = tre.lib()
    p = tre.Plan("ij,jk->ik", "j", {"i": 4, "j": 4, "k": 4}, {"j": 2}, "f32")
    jr = tre.JoinResult()
    assert tre.tre.STATUS[L.tre_join(p.handle, None, 1, None, 1, None, 0, None, ctypes.byref(jr), None)] == "TRE_E_ARG"
    assert tre.tre.STATUS[L.tre_contract(p.handle, ctypes.byref(jr), None, None, None, 0, None, None, 0, None,
                                         None)] == "TRE_E_STATE"
    assert tre.tre.STATUS[L.tre_cast_f32_bf16(None, None, -1, None)] == "TRE_E_ARG"


def test_binding_structs_match_the_header(tre, tmp_path):
    """Every struct the binding mirrors has the header's size and field
    offsets (a C program built with gcc against include/tre.h prints them)."""
    import subprocess

    structs = {"tre_options": tre.tre.Options, "tre_plan_info": tre.tre.PlanInfo,
               "tre_join_result": tre.tre.JoinResult, "tre_timing": tre.Timing}
    lines = ['#include <stdio.h>', '#include <stddef.h>', '#include "tre.h"', "int main(void) {"]
    for cname, cls in structs.items():
        lines.append(f'printf("{cname} size %zu\\n", sizeof({cname}));')
        for f, _ in cls._fields_:
            lines.append(f'printf("{cname} {f} %zu\\n", offsetof({cname}, {f}));')
    lines += ["return 0;", "}"]
    src = tmp_path / "layout.c"
    src.write_text("\n".join(lines))
    exe = tmp_path / "layout"
    subprocess.run(["gcc", "-std=c11", "-I", os.path.join(ROOT, "include"), str(src), "-o", str(exe)], check=True)
    out = subprocess.run([str(exe)], check=True, capture_output=True, text=True).stdout.split("\n")
    got = {tuple(l.split()[:2]): int(l.split()[2]) for l in out if l.strip()}
    for cname, cls in structs.items():
        assert got[(cname, "size")] == ctypes.sizeof(cls), cname
        for f, _ in cls._fields_:
            assert got[(cname, f)] == getattr(cls, f).offset, (cname, f)


def test_output_bounds_closed_forms(tre):
    """tre_output_bounds (host only) against the bounds it promises: one pair
    per V tuple when U's key is the join labels, the cross product
    otherwise, the pair capacity of the workspace, W's key space, n_u for a
    keyless one-tuple V with W keyed by U, zero pairs for an empty side, and
    TRE_E_WORKSPACE below the smallest workspace."""
    ws_of = lambda p, n_u, n_v, mp: p.workspace_bytes(n_u, n_v, mp)  # noqa: E731
    # U keyed (J) = the join labels: a V tuple meets at most one U tuple
    a = tre.Plan("ij,jk->ki", "jk", {"i": 64, "j": 64 * 8, "k": 64 * 16}, {"j": 64, "k": 64})
    assert tre.output_bounds(a, 8, 50, ws_of(a, 8, 50, 1000)) == (50, 16, True)  # keys: 16 K blocks
    # a workspace sized for 20 pairs caps the pair bound at its capacity
    ws20 = ws_of(a, 8, 50, 20)
    pb, kb, ok = tre.output_bounds(a, 8, 50, ws20)
    assert 20 <= pb <= 50 and kb == min(pb, 16) and ok
    assert pb == 50 or ws_of(a, 8, 50, pb + 1) > ws20
    # neither key is made of join labels only: the cross product
    b = tre.Plan("ij,jk->ik", "ijk", {"i": 64 * 3, "j": 64 * 4, "k": 64 * 5}, {"i": 64, "j": 64, "k": 64})
    assert tre.output_bounds(b, 5, 7, ws_of(b, 5, 7, 1000)) == (35, 15, True)  # keys: 3 x 5 (I, K) blocks
    assert tre.output_bounds(b, 5, 2, ws_of(b, 5, 2, 1000)) == (10, 10, True)
    # keyless one-tuple V, W keyed by U: one pair and one key per U tuple
    c = tre.Plan("ij,jk->ik", "i", {"i": 64 * 100, "j": 32, "k": 16}, {"i": 64})
    assert tre.output_bounds(c, 37, 1, ws_of(c, 37, 1, 37)) == (37, 37, True)
    # an empty side: nothing to bound
    assert tre.output_bounds(a, 0, 50, ws_of(a, 0, 50, 0)) == (0, 0, True)
    assert tre.output_bounds(b, 5, 0, ws_of(b, 5, 0, 0)) == (0, 0, True)
    with pytest.raises(tre.TreError) as e:
        tre.output_bounds(a, 8, 50, ws_of(a, 8, 50, 0) - 1)
    assert e.value.status == "TRE_E_WORKSPACE"
