"""GPU parity: the HIP path (through the C ABI) against the CPU oracle on the
same seeded inputs.  Pair lists and key sets bit-exact; values within the
mag-relative tolerance (1e-4 fp32, 1e-2 bf16 in / fp32 accumulate)."""
import json
import os
import sys

import numpy as np
import pytest

import workloads
from _parity import assert_values, check, gpu_run, to_dev
from test_oracle import random_plan, split_einsum

pytestmark = pytest.mark.gpu

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "worked_example.json")


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    import torch

    assert torch.cuda.is_available(), "GPU test needs a GPU"
    import paper_2603_08957_amd as tre

    tre.lib()


def orc_plan(orc, s):
    return orc.Plan(s["einsum"], s["upper"], s["extents"], s["tiles"])


@pytest.mark.parametrize("name", ["a_rows_times_cols", "b_columns_times_scalars", "c_outer_products"])
def test_worked_example_gpu(orc, name):
    g = json.load(open(GOLDEN))
    d = g["decompositions"][name]
    spec = workloads.spec(d["einsum"], d["upper"], {"i": 4, "j": 4, "k": 4}, d["tiles"], "f32")
    U = {"keys": np.array(d["U_keys"], np.int32).reshape(len(d["U_keys"]), -1),
         "tiles": np.array(d["U_tiles"], np.float32), "dtype": "f32"}
    V = {"keys": np.array(d["V_keys"], np.int32).reshape(len(d["V_keys"]), -1),
         "tiles": np.array(d["V_tiles"], np.float32), "dtype": "f32"}
    say("worked example", name)
    _, out = gpu_run(spec, U, V)
    ref = orc.run(orc_plan(orc, spec), U, V)
    check(out, ref, "f32")
    assert out.pairs.cpu().numpy().tolist() == d["pairs"]
    np.testing.assert_allclose(out.w_tiles.cpu().numpy(), np.array(d["W_tiles"]), rtol=1e-6, atol=1e-6)


@pytest.mark.parametrize("seed", range(60))
@pytest.mark.parametrize("small_join", [0, -1])
def test_random_plans_gpu(orc, seed, small_join):
    """Random small EinSums against the oracle, with the one-workgroup join
    allowed (most of these inputs take it) and switched off (the multi-kernel
    join on the same inputs)."""
    rng = np.random.default_rng(1000 + seed)
    e, upper, ext, til = random_plan(rng)
    u_lab, v_lab, _ = split_einsum(e)
    dtype = "bf16" if seed % 3 == 0 else "f32"
    U = workloads.random_relation(rng, u_lab, upper, ext, til, dtype, keep=0.6, zero_frac=0.3)
    V = workloads.random_relation(rng, v_lab, upper, ext, til, dtype, keep=0.6, zero_frac=0.3)
    spec = workloads.spec(e, upper, ext, til, dtype)
    say("random plan", seed, e, upper, til, len(U["keys"]), len(V["keys"]))
    if len(U["keys"]) == 0 or len(V["keys"]) == 0:
        _, out = gpu_run(spec, U, V, small_join=small_join)
        assert out.n_pairs == 0 and out.n_w == 0
        return
    _, out = gpu_run(spec, U, V, small_join=small_join)
    ref = orc.run(orc_plan(orc, spec), U, V)
    check(out, ref, dtype)


def _wider_plans():
    """Plans with larger tiles so the MFMA class and ragged blocks are hit."""
    return [
        ("ij,jk->ik", "j", {"i": 100, "j": 96, "k": 70}, {"j": 32}),          # GEMM, ragged M/N
        ("ij,jk->ki", "jk", {"i": 64, "j": 256, "k": 256}, {"j": 64, "k": 64}),  # GNN E1 form
        ("ki,im->km", "k", {"k": 512, "i": 64, "m": 32}, {"k": 64}),            # GNN E2 form
        ("ik,kn->in", "ik", {"i": 512, "k": 512, "n": 160}, {"i": 128, "k": 128}),
        ("ijk,jr->ikr", "ijk", {"i": 64, "j": 64, "k": 64, "r": 24}, {"i": 16, "j": 16, "k": 16}),
        ("ikr,kr->ir", "ik", {"i": 64, "k": 64, "r": 24}, {"i": 16, "k": 16}),
        ("bij,bjk->bik", "j", {"b": 3, "i": 40, "j": 48, "k": 36}, {"j": 16}),  # batch role in a GEMM
        ("ija,jkc->ik", "j", {"i": 33, "j": 40, "a": 3, "k": 20, "c": 2}, {"j": 8}),  # pre-sum labels
        ("ij,kj->ik", "ik", {"i": 96, "j": 80, "k": 96}, {"i": 32, "k": 32}),   # K-fast B, cross product
        ("ji,jk->ik", "", {"i": 70, "j": 90, "k": 50}, {}),                    # all demoted: one tuple each
    ]


@pytest.mark.parametrize("idx", range(10))
@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_wider_plans_gpu(orc, idx, dtype):
    e, upper, ext, til = _wider_plans()[idx]
    rng = np.random.default_rng(42 + idx)
    u_lab, v_lab, _ = split_einsum(e)
    keep = 1.0 if not upper else 0.7
    U = workloads.random_relation(rng, u_lab, upper, ext, til, dtype, keep=keep, zero_frac=0.1)
    V = workloads.random_relation(rng, v_lab, upper, ext, til, dtype, keep=keep, zero_frac=0.1)
    spec = workloads.spec(e, upper, ext, til, dtype)
    say("wider plan", idx, dtype, e)
    _, out = gpu_run(spec, U, V)
    ref = orc.run(orc_plan(orc, spec), U, V)
    check(out, ref, dtype)


FAST_PLANS = [
    # (einsum, upper, extents, tiles): each hits one operand-layout variant of
    # the 128x128 kernel (A row- or k-contiguous, B row- or k-contiguous), in
    # bf16 and in fp32
    ("ij,jk->ki", "jk", {"i": 128, "j": 1024, "k": 1024}, {"j": 128, "k": 128}),
    ("ki,im->km", "k", {"k": 2048, "i": 128, "m": 256}, {"k": 128}),
    ("ik,jk->ij", "ij", {"i": 512, "j": 384, "k": 192}, {"i": 128, "j": 128}),
    ("ki,kj->ij", "ij", {"i": 256, "j": 512, "k": 64}, {"i": 256, "j": 128}),
]


@pytest.mark.parametrize("idx", range(len(FAST_PLANS)))
@pytest.mark.parametrize("pmax,ur", [(0, -1), (3, -1), (0, 3), (0, 64)])
@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_fast_path_gpu(orc, idx, pmax, ur, dtype):
    """128x128 MFMA path (bf16 and fp32), including U-range units (ur > 0:
    every key's pairs cut into ur ranges of U index, empty ranges included,
    partials summed after)."""
    import paper_2603_08957_amd as tre

    e, upper, ext, til = FAST_PLANS[idx]
    assert tre.Plan(e, upper, ext, til, dtype).kernel_class == "gemm128"
    rng = np.random.default_rng(77 + idx)
    u_lab, v_lab, _ = split_einsum(e)
    U = workloads.random_relation(rng, u_lab, upper, ext, til, dtype, keep=0.6, zero_frac=0.05)
    V = workloads.random_relation(rng, v_lab, upper, ext, til, dtype, keep=0.6, zero_frac=0.05)
    spec = workloads.spec(e, upper, ext, til, dtype)
    say("fast path", idx, dtype, pmax, ur, e, len(U["keys"]), len(V["keys"]))
    _, out = gpu_run(spec, U, V, max_pairs_per_unit=pmax, u_ranges=ur)
    check(out, orc.run(orc_plan(orc, spec), U, V), dtype)


@pytest.mark.parametrize("idx", [0, 2])
@pytest.mark.parametrize("windows", [1, 3, 64])
@pytest.mark.parametrize("dtype,w_bf16", [("bf16", False), ("f32", False), ("bf16", True)])
def test_paced_path_gpu(orc, idx, windows, dtype, w_bf16):
    """Persistent paced kernel (one 128x128 block per W tile): whole keys per
    workgroup, rounds of units, pacing over windows of U index; the result
    must not depend on the window count.  With w_bf16 the paced kernel
    stores W as bf16 (the launch the benchmark times for its default
    workload); the upcast values are compared with the oracle at the bf16
    tolerance."""
    import paper_2603_08957_amd as tre

    e, upper, ext, til = FAST_PLANS[idx]
    rng = np.random.default_rng(177 + idx)
    u_lab, v_lab, _ = split_einsum(e)
    # every U tile present: the paced grid needs at least two U tuples
    U = workloads.random_relation(rng, u_lab, upper, ext, til, dtype, keep=1.0, zero_frac=0.05)
    V = workloads.random_relation(rng, v_lab, upper, ext, til, dtype, keep=0.6 if idx == 0 else 1.0, zero_frac=0.05)
    spec = workloads.spec(e, upper, ext, til, dtype)
    assert tre.Plan(e, upper, ext, til, dtype).kernel_class == "gemm128"
    say("paced path", idx, dtype, windows, w_bf16, e, len(U["keys"]), len(V["keys"]))
    plan = tre.Plan.from_spec(spec, pace_windows=windows, w_bf16=w_bf16)
    out = tre.einsum(plan, *to_dev(U), *to_dev(V), want_pairs=True, timing=True)
    assert out.timing["contract_path"] == "gemm128_paced", out.timing
    assert out.w_tiles.dtype == (torch_bf16() if w_bf16 else torch_f32())
    check(out, orc.run(orc_plan(orc, spec), U, V), dtype)


def torch_bf16():
    import torch

    return torch.bfloat16


def torch_f32():
    import torch

    return torch.float32


@pytest.mark.parametrize("dtype,w_bf16", [("bf16", False), ("bf16", True), ("f32", False)])
def test_paced_rounds_gpu(orc, dtype, w_bf16):
    """More keys than resident workgroups (512 on 256 CUs): the paced kernel
    deals whole keys in rounds, the last one partial; bf16 and fp32 inputs,
    and bf16 output.  Each key is still summed by one workgroup in pair
    order, so the result equals the one-unit-per-key launch bit for bit, and
    sampled keys match the oracle."""
    import torch

    from test_gpu_fullsize import sampled_check

    e, upper = "ij,jk->ki", "jk"
    nk = 512 * 3 + 77
    ext, til = {"i": 128, "j": 128 * 3, "k": 128 * nk}, {"j": 128, "k": 128}
    rng = np.random.default_rng(4242)
    U = workloads.random_relation(rng, "ij", upper, ext, til, dtype, keep=1.0)
    V = workloads.random_relation(rng, "jk", upper, ext, til, dtype, keep=0.7)
    spec = workloads.spec(e, upper, ext, til, dtype)
    say("paced rounds", dtype, w_bf16, len(U["keys"]), len(V["keys"]))
    _, paced = gpu_run(spec, U, V, pace_windows=2, w_bf16=w_bf16)
    _, whole = gpu_run(spec, U, V, pace_windows=-1, u_ranges=-1, max_pairs_per_unit=1 << 20, w_bf16=w_bf16)
    torch.cuda.synchronize()
    assert 3 * 512 < paced.n_w < 4 * 512, paced.n_w
    assert paced.n_w == whole.n_w and torch.equal(paced.w_keys, whole.w_keys)
    assert torch.equal(paced.pairs, whole.pairs)
    assert torch.equal(paced.w_tiles.view(torch.int16 if w_bf16 else torch.int32),
                       whole.w_tiles.view(torch.int16 if w_bf16 else torch.int32)), "paced result differs"
    wk = paced.w_keys.cpu().numpy().reshape(paced.n_w, -1)
    S = wk[np.sort(rng.choice(paced.n_w, 12, replace=False))]
    sampled_check(orc, spec, U, V, paced, S, pairs=paced.pairs.cpu().numpy())


@pytest.mark.parametrize("pmax", [1, 2, 3, 7])
def test_split_segments_gpu(orc, pmax):
    """Forcing short work units splits every key's pairs; the segmented sum of
    the partial tiles must give the same result."""
    e, upper, ext, til = "ij,jk->ki", "jk", {"i": 64, "j": 512, "k": 256}, {"j": 64, "k": 64}
    rng = np.random.default_rng(9)
    U = workloads.random_relation(rng, "ij", upper, ext, til, "f32", keep=0.9)
    V = workloads.random_relation(rng, "jk", upper, ext, til, "f32", keep=0.8)
    spec = workloads.spec(e, upper, ext, til, "f32")
    say("split", pmax)
    _, out = gpu_run(spec, U, V, max_pairs_per_unit=pmax)
    assert out.timing is None
    ref = orc.run(orc_plan(orc, spec), U, V)
    check(out, ref, "f32")


W_BF16_SPLIT = [
    # (einsum, upper, extents, tiles, plan options): bf16 inputs, keys cut
    # into several units, W written in bf16 by the segmented sum
    ("ik,kj->ij", "ijk", {"i": 256, "j": 256, "k": 1024}, {"i": 128, "j": 128, "k": 128}, {"max_pairs_per_unit": 3}),
    ("ik,kj->ij", "ijk", {"i": 256, "j": 256, "k": 1024}, {"i": 128, "j": 128, "k": 128}, {"u_ranges": 2}),
    ("ij,jk->ki", "jk", {"i": 64, "j": 300, "k": 40}, {"j": 1, "k": 1}, {"max_pairs_per_unit": 3}),  # 64-element W tiles
    ("ij,jk->ki", "jk", {"i": 6, "j": 300, "k": 40}, {"j": 1, "k": 1}, {"max_pairs_per_unit": 3}),   # 6-element W tiles
]


@pytest.mark.parametrize("idx", range(len(W_BF16_SPLIT)))
def test_split_segments_bf16_w_gpu(orc, idx):
    """Keys cut into several units with W written in bf16: the partial tiles
    (fp32) are summed in unit order and rounded once, four elements per lane
    when a W tile holds a multiple of 4 elements and one otherwise; keys,
    pairs and the upcast values against the oracle (Sec. 5, the GROUP BY
    sum of the matched tile products)."""
    import torch

    import paper_2603_08957_amd as tre

    e, upper, ext, til, opts = W_BF16_SPLIT[idx]
    rng = np.random.default_rng(940 + idx)
    u_lab, v_lab, _ = split_einsum(e)
    U = workloads.random_relation(rng, u_lab, upper, ext, til, "bf16", keep=0.9)
    V = workloads.random_relation(rng, v_lab, upper, ext, til, "bf16", keep=0.9)
    spec = workloads.spec(e, upper, ext, til, "bf16")
    plan = tre.Plan.from_spec(spec, w_bf16=True, **opts)
    say("split bf16 W", idx, e, opts, plan.kernel_class, len(U["keys"]), len(V["keys"]))
    out = tre.einsum(plan, *to_dev(U), *to_dev(V), want_pairs=True, timing=True)
    assert out.w_tiles.dtype == torch.bfloat16
    assert out.timing["n_split_segments"] > 0, out.timing
    check(out, orc.run(orc_plan(orc, spec), U, V), "bf16")


@pytest.mark.parametrize("c", [1, 2, 3, 4, 5])
def test_small_configs_gpu(orc, c):
    """Scaled-down twins of the five workloads, every EinSum of each."""
    w = workloads.config(c, "small")
    say("small config", c)
    if c in (1, 2, 5):
        Y = w["Y"]
        _, o1 = gpu_run(w["E1"], w["X"], Y)
        r1 = orc.run(orc_plan(orc, w["E1"]), w["X"], {"keys": Y["keys"], "coo": Y["coo"]})
        check(o1, r1, w["dtype"])
        # E2 on its own, with a seeded T of the shape E1 produces
        rng = np.random.default_rng(5)
        t2 = w["tile_e2"]
        nT = w["n"] // t2
        T = {"keys": np.arange(nT, dtype=np.int32).reshape(-1, 1),
             "tiles": rng.standard_normal((nT, t2 * w["emb"]), dtype=np.float32), "dtype": w["dtype"]}
        if w["dtype"] == "bf16":
            T["tiles"] = workloads.to_bf16_bits(T["tiles"])
        _, o2 = gpu_run(w["E2"], T, w["Z"])
        r2 = orc.run(orc_plan(orc, w["E2"]), T, w["Z"])
        check(o2, r2, w["dtype"])
    elif c == 3:
        _, o = gpu_run(w["E"], w["A"], w["B"])
        check(o, orc.run(orc_plan(orc, w["E"]), w["A"], w["B"]), "f32")
    else:
        _, o1 = gpu_run(w["E1"], w["T"], w["B"])
        r1 = orc.run(orc_plan(orc, w["E1"]), w["T"], w["B"])
        check(o1, r1, "f32")
        rng = np.random.default_rng(6)
        Wr = {"keys": r1.wkeys, "tiles": rng.standard_normal(r1.acc.shape, dtype=np.float32), "dtype": "f32"}
        _, o2 = gpu_run(w["E2"], Wr, w["C"])
        check(o2, orc.run(orc_plan(orc, w["E2"]), Wr, w["C"]), "f32")


def test_determinism_gpu(orc):
    """Atomic-free path: two runs give bit-identical tiles and pair lists."""
    w = workloads.config(2, "small")
    _, a = gpu_run(w["E1"], w["X"], w["Y"], max_pairs_per_unit=3)
    _, b = gpu_run(w["E1"], w["X"], w["Y"], max_pairs_per_unit=3)
    assert np.array_equal(a.pairs.cpu().numpy(), b.pairs.cpu().numpy())
    assert np.array_equal(a.w_tiles.cpu().numpy().view(np.uint32), b.w_tiles.cpu().numpy().view(np.uint32))


def test_key_errors_gpu():
    import paper_2603_08957_amd as tre
    import torch

    plan = tre.Plan("ij,jk->ik", "jk", {"i": 4, "j": 8, "k": 8}, {"j": 2, "k": 2}, "f32")
    uk = torch.arange(4, dtype=torch.int32).reshape(4, 1).cuda()
    ut = torch.ones((4, 8), dtype=torch.float32).cuda()
    good = np.array([[0, 1], [0, 3], [2, 0]], np.int32)
    cases = {"TRE_E_UNSORTED": good[[0, 2, 1]], "TRE_E_DUPKEY": good[[0, 0, 1]],
             "TRE_E_KEYRANGE": np.array([[0, 1], [0, 4]], np.int32)}
    for status, vk in cases.items():
        vkt = torch.from_numpy(vk).cuda()
        vt = torch.ones((len(vk), 4), dtype=torch.float32).cuda()
        with pytest.raises(tre.TreError) as ei:
            tre.einsum(plan, uk, ut, vkt, vt)
        assert ei.value.status == status
    # validation off: a valid input still works and the call does not fault
    plan2 = tre.Plan("ij,jk->ik", "jk", {"i": 4, "j": 8, "k": 8}, {"j": 2, "k": 2}, "f32", validate=False)
    out = tre.einsum(plan2, uk, ut, torch.from_numpy(good).cuda(), torch.ones((3, 4)).cuda())
    assert out.n_pairs == 3


def test_capacity_and_workspace_errors_gpu():
    import paper_2603_08957_amd as tre
    import torch

    plan = tre.Plan("ij,jk->ik", "j", {"i": 8, "j": 8, "k": 8}, {"j": 1}, "f32")
    uk = torch.arange(8, dtype=torch.int32).reshape(8, 1).cuda()
    ut = torch.ones((8, 8)).cuda()
    # workspace for 0 pairs: join reports the required count
    ws = tre.alloc_workspace(plan.workspace_bytes(8, 8, 0))
    with pytest.raises(tre.TreError) as ei:
        tre.join(plan, uk, 8, uk, 8, ws)
    assert ei.value.status == "TRE_E_WORKSPACE" and ei.value.join_result.n_pairs == 8
    ws = tre.alloc_workspace(plan.workspace_bytes(8, 8, 8))
    jr = tre.join(plan, uk, 8, uk, 8, ws)
    assert jr.n_pairs == 8 and jr.n_w == 1
    small = torch.empty((0, 64)).cuda()
    with pytest.raises(tre.TreError) as ei:
        tre.contract(plan, jr, ut, ut, None, small)
    assert ei.value.status == "TRE_E_CAPACITY"


def test_empty_inputs_gpu():
    import paper_2603_08957_amd as tre
    import torch

    plan = tre.Plan("ij,jk->ik", "j", {"i": 4, "j": 4, "k": 4}, {"j": 2}, "f32")
    out = tre.einsum(plan, torch.zeros((0, 1), dtype=torch.int32).cuda(), torch.zeros((0, 8)).cuda(),
                     torch.zeros((1, 1), dtype=torch.int32).cuda(), torch.ones((1, 8)).cuda(), want_pairs=True)
    assert out.n_pairs == 0 and out.n_w == 0


def test_cast_bf16_gpu(orc):
    import paper_2603_08957_amd as tre
    import torch

    rng = np.random.default_rng(0)
    x = (rng.standard_normal(100003) * 10.0 ** rng.integers(-20, 20, 100003)).astype(np.float32)
    x[:6] = [0.0, -0.0, np.inf, -np.inf, np.nan, 1 + 2 ** -8]
    y = tre.cast_f32_bf16(torch.from_numpy(x).cuda())
    got = y.view(torch.int16).cpu().numpy().view(np.uint16)
    ref = orc.f32_to_bf16(x)
    assert np.array_equal(got[5:], ref[5:])
    assert (got[4] & 0x7F80) == 0x7F80 and (got[4] & 0x7F)  # NaN stays NaN


def test_stack_rows_gpu(orc):
    import paper_2603_08957_amd as tre
    import torch

    rng = np.random.default_rng(3)
    keys = np.sort(rng.choice(1000, size=300, replace=False)).astype(np.int32)
    rows = rng.standard_normal((300, 12)).astype(np.float32)
    k, t = tre.stack_rows(torch.from_numpy(keys).cuda(), torch.from_numpy(rows).cuda(), 16)
    rk, rt = orc.stack_rows(keys, rows, 16)
    assert np.array_equal(k.cpu().numpy(), rk)
    assert np.array_equal(t.cpu().numpy(), rt)


def test_tiles_from_entries_gpu(orc):
    import paper_2603_08957_amd as tre
    import torch

    w = workloads.config(2, "small")
    Y = w["Y"]
    vals = torch.from_numpy(Y["values"].view(np.int16)).cuda().view(torch.bfloat16)
    tiles = tre.tiles_from_entries(torch.from_numpy(Y["slot"]).cuda(), torch.from_numpy(Y["offset"]).cuda(), vals,
                                   len(Y["keys"]), Y["tile_elems"])
    assert np.array_equal(tiles.view(torch.int16).cpu().numpy().view(np.uint16), Y["tiles"])
    p1 = orc_plan(orc, w["E1"])
    c, v, _ = orc.expand(p1, 1, Y["keys"], tiles.view(torch.int16).cpu().numpy().view(np.uint16), "bf16")
    got = sorted(zip(map(tuple, c.tolist()), v.tolist()))
    ref = sorted(zip(map(tuple, Y["coo"][0].tolist()), Y["coo"][1].tolist()))
    assert got == ref


# ------------------------------------------------------------ repartition

def _rp_case(rng, nl_max=3, ext_mult=(2, 6)):
    import itertools

    nl = int(rng.integers(1, nl_max + 1))
    labels = "".join(rng.choice(list("abcdefgh"), nl, replace=False))
    base = {c: int(rng.choice([2, 3, 4, 8])) for c in labels}
    ext = {c: base[c] * int(rng.integers(*ext_mult)) for c in labels}
    up_in = "".join(c for c in labels if rng.random() < 0.75)
    up_out = "".join(c for c in labels if rng.random() < 0.75)

    def pick(c):
        ds = [d for d in range(1, ext[c] + 1) if ext[c] % d == 0]
        return int(rng.choice(ds))

    tin = {c: pick(c) for c in up_in}
    tout = {c: pick(c) for c in up_out}
    axes = [range(ext[c] // tin[c]) for c in up_in]
    all_keys = list(itertools.product(*axes)) if up_in else [()]
    keep = [k for k in all_keys if rng.random() < 0.4] or all_keys[:1]
    keys = np.array(keep, np.int32).reshape(len(keep), len(up_in))
    te = int(np.prod([tin[c] if c in up_in else ext[c] for c in labels]))
    return labels, up_in, up_out, ext, tin, tout, keys, te


@pytest.mark.parametrize("seed", range(24))
def test_repartition_gpu(orc, seed):
    """Random decompositions: target keys and every target element bit-exact
    against the oracle (fp32 and bf16 bit patterns)."""
    import torch

    import paper_2603_08957_amd as tre

    rng = np.random.default_rng(900 + seed)
    labels, up_in, up_out, ext, tin, tout, keys, te = _rp_case(rng)
    dtype = "bf16" if seed % 2 else "f32"
    vals = (rng.standard_normal((len(keys), te)) * (rng.random((len(keys), te)) < 0.7)).astype(np.float32)
    if dtype == "bf16":
        bits = orc.f32_to_bf16(vals)
        dev_tiles = torch.from_numpy(bits.view(np.int16)).cuda()
        ref_vals = orc.bf16_to_f64(bits)
    else:
        dev_tiles = torch.from_numpy(vals).cuda()
        ref_vals = vals.astype(np.float64)
    say("repartition", seed, labels, up_in, up_out, tin, tout, len(keys), dtype)
    k2, t2 = tre.repartition(labels, up_in, up_out, ext, tin, tout, torch.from_numpy(keys).cuda(), dev_tiles)
    rk, rt = orc.repartition(labels, up_in, up_out, ext, tin, tout, keys, ref_vals)
    assert np.array_equal(k2.cpu().numpy().reshape(rk.shape), rk)
    got = t2.cpu().numpy()
    got = orc.bf16_to_f64(got.view(np.uint16)) if dtype == "bf16" else got.astype(np.float64)
    assert np.array_equal(got.reshape(rt.shape), rt)


# Larger decompositions, each chosen for one path of the device copy: whole
# rows stacked (target order already sorted, 16-byte chunks, one run per
# pair), rows unstacked, row blocks to column blocks (sorted, many 16-byte
# runs per pair), ragged boxes of unequal size (element chunks, binary
# search over the pair prefix), a demoted inner label, and more pairs than
# the copy grid holds workgroups (the batch loop).
_RP_LARGE = [
    ("ki", "k", "k", {"k": 8192, "i": 256}, {"k": 1}, {"k": 256}, "bf16", 1.0),
    ("ki", "k", "k", {"k": 8192, "i": 256}, {"k": 256}, {"k": 1}, "bf16", 1.0),
    ("ij", "i", "j", {"i": 512, "j": 512}, {"i": 64}, {"j": 64}, "f32", 1.0),
    ("ij", "ij", "ij", {"i": 960, "j": 900}, {"i": 32, "j": 30}, {"i": 24, "j": 45}, "f32", 0.6),
    ("ij", "ij", "ij", {"i": 1200, "j": 960}, {"i": 40, "j": 12}, {"i": 24, "j": 32}, "bf16", 0.5),
    ("abc", "ab", "ab", {"a": 256, "b": 512, "c": 16}, {"a": 4, "b": 8}, {"a": 8, "b": 2}, "f32", 0.3),
    ("k", "k", "k", {"k": 1 << 21}, {"k": 1}, {"k": 8}, "f32", 1.0),
]


@pytest.mark.parametrize("case", range(len(_RP_LARGE)))
def test_repartition_gpu_large(orc, case):
    """Bit-exact keys and tiles against the oracle on the cases above."""
    import itertools

    import torch

    import paper_2603_08957_amd as tre

    labels, up_in, up_out, ext, tin, tout, dtype, keep = _RP_LARGE[case]
    rng = np.random.default_rng(1700 + case)
    axes = [range(ext[c] // tin[c]) for c in up_in]
    if keep < 1.0:
        all_keys = np.array(list(itertools.product(*axes)), np.int32)
        keys = all_keys[rng.random(len(all_keys)) < keep]
    else:
        grids = np.meshgrid(*[np.arange(len(a), dtype=np.int32) for a in axes], indexing="ij")
        keys = np.stack([g.reshape(-1) for g in grids], axis=1)
    keys = np.ascontiguousarray(keys.reshape(-1, len(up_in)))
    te = int(np.prod([tin[c] if c in up_in else ext[c] for c in labels]))
    vals = rng.standard_normal((len(keys), te)).astype(np.float32)
    if dtype == "bf16":
        bits = orc.f32_to_bf16(vals)
        dev_tiles = torch.from_numpy(bits.view(np.int16)).cuda()
        ref_vals = orc.bf16_to_f64(bits)
    else:
        dev_tiles = torch.from_numpy(vals).cuda()
        ref_vals = vals.astype(np.float64)
    say("repartition large", case, labels, up_in, up_out, tin, tout, len(keys), dtype)
    k2, t2 = tre.repartition(labels, up_in, up_out, ext, tin, tout, torch.from_numpy(keys).cuda(), dev_tiles)
    rk, rt = orc.repartition(labels, up_in, up_out, ext, tin, tout, keys, ref_vals)
    assert np.array_equal(k2.cpu().numpy().reshape(rk.shape), rk)
    got = t2.cpu().numpy()
    got = orc.bf16_to_f64(got.view(np.uint16)) if dtype == "bf16" else got.astype(np.float64)
    assert np.array_equal(got.reshape(rt.shape), rt)


def test_repartition_gpu_paper_example_and_stack(orc):
    import torch

    import paper_2603_08957_amd as tre

    keys = torch.tensor([[0], [1], [2]], dtype=torch.int32).cuda()
    tiles = torch.tensor([[1.0, 2.0], [3.0, 4.0], [5.0, 6.0]]).cuda()
    k2, t2 = tre.repartition("ki", "k", "i", {"k": 3, "i": 2}, {"k": 1}, {"i": 1}, keys, tiles)
    assert k2.cpu().tolist() == [[0], [1]]
    assert t2.cpu().tolist() == [[1.0, 3.0, 5.0], [2.0, 4.0, 6.0]]
    # stack of per-vertex rows into 256-row tiles (the chain's re-composition)
    rng = np.random.default_rng(4)
    n, emb = 4096, 256
    present = np.sort(rng.choice(n, 3000, replace=False)).astype(np.int32).reshape(-1, 1)
    rows = rng.standard_normal((len(present), emb)).astype(np.float32)
    k2, t2 = tre.repartition("ki", "k", "k", {"k": n, "i": emb}, {"k": 1}, {"k": 256},
                             torch.from_numpy(present).cuda(), torch.from_numpy(rows).cuda())
    k3, t3 = tre.stack_rows(torch.from_numpy(present).cuda(), torch.from_numpy(rows).cuda(), 256)
    assert torch.equal(k2, k3) and torch.equal(t2, t3)


def test_repartition_gpu_errors_and_empty(orc):
    import torch

    import paper_2603_08957_amd as tre

    t = torch.zeros((2, 4)).cuda()
    with pytest.raises(tre.TreError) as ei:
        tre.repartition("ij", "i", "j", {"i": 4, "j": 4}, {"i": 1}, {"j": 2},
                        torch.tensor([[1], [0]], dtype=torch.int32).cuda(), t)
    assert ei.value.status == "TRE_E_UNSORTED"
    with pytest.raises(tre.TreError) as ei:
        tre.repartition("ij", "i", "j", {"i": 4, "j": 4}, {"i": 1}, {"j": 2},
                        torch.tensor([[0], [9]], dtype=torch.int32).cuda(), t)
    assert ei.value.status == "TRE_E_KEYRANGE"
    with pytest.raises(tre.TreError) as ei:
        tre.repartition("ij", "i", "j", {"i": 4, "j": 4}, {"i": 3}, {"j": 2},
                        torch.tensor([[0]], dtype=torch.int32).cuda(), t[:1])
    assert ei.value.status == "TRE_E_SHAPE"
    k2, t2 = tre.repartition("ij", "i", "j", {"i": 4, "j": 4}, {"i": 1}, {"j": 2},
                             torch.zeros((0, 1), dtype=torch.int32).cuda(), torch.zeros((0, 4)).cuda())
    assert k2.shape[0] == 0 and t2.shape[0] == 0


def test_repartition_gpu_in_place(orc):
    """In place (tiles_out is tiles_in): stacking complete per-vertex rows
    into row blocks leaves every byte where it is and only writes the keys;
    a missing row, a column stack or a split is refused with the tiles
    untouched.  Random full-coverage cases: whenever in place is accepted,
    keys and tiles equal the oracle's copy."""
    import torch

    import paper_2603_08957_amd as tre

    rng = np.random.default_rng(77)
    n, emb = 4096, 64
    keys = torch.arange(n, dtype=torch.int32).reshape(-1, 1).cuda()
    for dtype in (torch.float32, torch.bfloat16):
        rows = torch.from_numpy(rng.standard_normal((n, emb)).astype(np.float32)).cuda().to(dtype)
        before = rows.clone()
        k2, t2 = tre.repartition("ki", "k", "k", {"k": n, "i": emb}, {"k": 1}, {"k": 256}, keys, rows,
                                 in_place=True)
        assert t2.data_ptr() == rows.data_ptr() and tuple(t2.shape) == (n // 256, 256 * emb)
        k3, t3 = tre.repartition("ki", "k", "k", {"k": n, "i": emb}, {"k": 1}, {"k": 256}, keys, before)
        assert torch.equal(k2, k3) and torch.equal(t2, t3)
    rows = torch.from_numpy(rng.standard_normal((n, emb)).astype(np.float32)).cuda()
    refused = [
        ("ki", "k", "k", {"k": n, "i": emb}, {"k": 1}, {"k": 256}, keys[1:], rows[1:]),  # row 0 missing
        ("ki", "ki", "ki", {"k": n, "i": emb}, {"k": 1, "i": 8}, {"k": 4, "i": 8},  # source order is not target order
         torch.stack(torch.meshgrid(torch.arange(n), torch.arange(emb // 8), indexing="ij"), -1).reshape(-1, 2)
         .to(torch.int32).contiguous().cuda(), rows.reshape(-1, 8)),
        ("ki", "k", "k", {"k": n, "i": emb}, {"k": 4}, {"k": 1}, keys[:n // 4], rows.reshape(n // 4, -1)),  # split
    ]
    for labels, ui, uo, ext, ti, to, kk, tt in refused:
        before = tt.clone()
        with pytest.raises(tre.TreError) as ei:
            tre.repartition(labels, ui, uo, ext, ti, to, kk, tt, in_place=True)
        assert ei.value.status == "TRE_E_ARG"
        assert torch.equal(tt, before)
    accepted = 0
    for seed in range(40):
        r = np.random.default_rng(5000 + seed)
        labels, up_in, up_out, ext, tin, tout, _, te = _rp_case(r)
        import itertools

        axes = [range(ext[c] // tin[c]) for c in up_in]
        combos = list(itertools.product(*axes)) if up_in else [()]
        keys_all = np.array(combos, np.int32).reshape(len(combos), len(up_in))
        vals = r.standard_normal((len(keys_all), te)).astype(np.float32)
        dev = torch.from_numpy(vals).cuda()
        say("repartition in place", seed, labels, up_in, up_out, tin, tout, len(keys_all))
        try:
            k2, t2 = tre.repartition(labels, up_in, up_out, ext, tin, tout, torch.from_numpy(keys_all).cuda(), dev,
                                     in_place=True)
        except tre.TreError as e:
            assert e.status == "TRE_E_ARG"
            assert np.array_equal(dev.cpu().numpy(), vals)
            continue
        accepted += 1
        rk, rt = orc.repartition(labels, up_in, up_out, ext, tin, tout, keys_all, vals.astype(np.float64))
        assert np.array_equal(k2.cpu().numpy().reshape(rk.shape), rk)
        assert np.array_equal(t2.cpu().numpy().astype(np.float64).reshape(rt.shape), rt)
    assert accepted > 0


def test_join_keys_gpu(orc):
    """tre_join_keys writes, before any contraction, the keys tre_contract
    writes; a short buffer is TRE_E_CAPACITY."""
    import torch

    import paper_2603_08957_amd as tre

    rng = np.random.default_rng(31)
    plan = tre.Plan("ij,jk->ik", "ijk", {"i": 64, "j": 64, "k": 64}, {"i": 8, "j": 8, "k": 8})
    def rel(n_keys):
        import itertools
        allk = np.array(list(itertools.product(range(8), range(8))), np.int32)
        keep = np.sort(rng.choice(len(allk), n_keys, replace=False))
        return torch.from_numpy(allk[keep]).cuda(), torch.from_numpy(rng.standard_normal((n_keys, 64)).astype(np.float32)).cuda()
    uk, ut = rel(40)
    vk, vt = rel(30)
    ws = tre.alloc_workspace(plan.workspace_bytes(40, 30, 40 * 30))
    jr = tre.join(plan, uk, 40, vk, 30, ws)
    early = torch.full((jr.n_w, 2), -1, dtype=torch.int32, device="cuda")
    tre.join_keys(plan, jr, early)
    wk = torch.empty((jr.n_w, 2), dtype=torch.int32, device="cuda")
    wt = torch.empty((jr.n_w, 64), dtype=torch.float32, device="cuda")
    tre.contract(plan, jr, ut, vt, wk, wt)
    torch.cuda.synchronize()
    assert jr.n_w > 1 and torch.equal(early, wk)
    with pytest.raises(tre.TreError) as ei:
        tre.join_keys(plan, jr, early[:jr.n_w - 1])
    assert ei.value.status == "TRE_E_CAPACITY"


@pytest.mark.parametrize("validate", [True, False])
def test_join_keyed_by_u_gpu(orc, validate):
    """A keyless one-tuple V with W keyed by U's key (the chains' E2,
    T keyed k times the whole Z): pairs are (u, 0) in U order and W's keys
    are U's; values against the oracle.  With validation, a repeated U key is
    still reported."""
    import torch

    import paper_2603_08957_amd as tre

    rng = np.random.default_rng(8)
    ext = {"k": 4096, "i": 64, "m": 32}
    til = {"k": 64}
    keys = np.sort(rng.choice(64, 40, replace=False)).astype(np.int32).reshape(-1, 1)
    ut = rng.standard_normal((40, 64 * 64)).astype(np.float32)
    vt = rng.standard_normal((1, 64 * 32)).astype(np.float32)
    plan = tre.Plan("ki,im->km", "k", ext, til, validate=validate)
    out = tre.einsum(plan, torch.from_numpy(keys).cuda(), torch.from_numpy(ut).cuda(),
                     torch.zeros((1, 0), dtype=torch.int32).cuda(), torch.from_numpy(vt).cuda(), want_pairs=True)
    assert out.n_pairs == 40 and out.n_w == 40
    assert np.array_equal(out.w_keys.cpu().numpy(), keys)
    pairs = out.pairs.cpu().numpy()
    assert np.array_equal(pairs[:, 0], np.arange(40)) and not pairs[:, 1].any()
    op = orc.Plan("ki,im->km", "k", ext, til)
    uc, uv, _ = orc.expand(op, 0, keys, ut, "f32")
    vc, vv, _ = orc.expand(op, 1, np.zeros((1, 0), np.int32), vt, "f32")
    acc, mag, _ = orc.evaluate(op, uc, uv, vc, vv, keys)
    assert_values(out.w_tiles.cpu().numpy().reshape(acc.shape), acc, mag, "f32")
    if validate:
        bad = keys.copy()
        bad[5] = bad[4]
        with pytest.raises(tre.TreError) as ei:
            tre.einsum(plan, torch.from_numpy(bad).cuda(), torch.from_numpy(ut).cuda(),
                       torch.zeros((1, 0), dtype=torch.int32).cuda(), torch.from_numpy(vt).cuda())
        assert ei.value.status == "TRE_E_DUPKEY"


def _rand_rel(rng, grid, tile_elems, keep, dtype):
    import itertools

    import torch

    allk = np.array(list(itertools.product(*[range(g) for g in grid])), np.int32).reshape(-1, len(grid))
    keys = allk[rng.random(len(allk)) < keep]
    vals = torch.from_numpy(rng.standard_normal((len(keys), tile_elems)).astype(np.float32))
    return torch.from_numpy(np.ascontiguousarray(keys)).cuda(), vals.to(dtype).cuda()


@pytest.mark.parametrize("case", ["vec", "vec_split", "fast", "fast_split", "fast_ranges"])
def test_w_bf16_gpu(case):
    """W written as bf16 by the vector class, the 128x128 path, and the
    partial-tile sum of split keys is bit for bit the bf16 cast of the fp32
    result of the same plan; the generic GEMM class refuses the option."""
    import torch

    import paper_2603_08957_amd as tre

    rng = np.random.default_rng(["vec", "vec_split", "fast", "fast_split", "fast_ranges"].index(case) + 60)
    if case.startswith("vec"):
        spec = ("ij,jk->ki", "jk", {"i": 64, "j": 300, "k": 300}, {"j": 1, "k": 1})
        uk, ut = _rand_rel(rng, [300], 64, 1.0, torch.bfloat16)
        vk, vt = _rand_rel(rng, [300, 300], 1, 0.05, torch.bfloat16)
    else:
        spec = ("ik,kj->ij", "ijk", {"i": 512, "j": 512, "k": 2048}, {"i": 128, "j": 128, "k": 128})
        uk, ut = _rand_rel(rng, [4, 16], 128 * 128, 0.5, torch.bfloat16)
        vk, vt = _rand_rel(rng, [16, 4], 128 * 128, 0.5, torch.bfloat16)
    opts = {"max_pairs_per_unit": 3} if case.endswith("split") else {"u_ranges": 2} if case.endswith("ranges") else {}
    say("w_bf16", case, opts)
    p32 = tre.Plan(*spec, dtype="bf16", **opts)
    p16 = tre.Plan(*spec, dtype="bf16", w_bf16=True, **opts)
    assert p16.kernel_class == ("vec" if case.startswith("vec") else "gemm128")
    o32 = tre.einsum(p32, uk, ut, vk, vt)
    o16 = tre.einsum(p16, uk, ut, vk, vt)
    torch.cuda.synchronize()
    assert o16.w_tiles.dtype == torch.bfloat16 and o16.n_w == o32.n_w and o32.n_w > 1
    assert torch.equal(o16.w_keys, o32.w_keys)
    ref = tre.cast_f32_bf16(o32.w_tiles)
    assert torch.equal(o16.w_tiles.view(torch.int16), ref.view(torch.int16))
    generic = ("ij,jk->ki", "jk", {"i": 64, "j": 4096, "k": 4096}, {"j": 64, "k": 64})
    assert tre.Plan(*generic).kernel_class == "gemm"
    with pytest.raises(tre.TreError) as ei:
        tre.Plan(*generic, w_bf16=True)
    assert ei.value.status == "TRE_E_DTYPE"


V_OUTER_PLANS = [
    # (einsum, upper, extents, tiles, dtype, keep of V): joins the plan drives
    # from V (W's key is V's key prefix, then the join labels, which U's key
    # starts with); pairs come out grouped with no sort
    ("ij,kj->ki", "jk", {"i": 64, "j": 300, "k": 300}, {"j": 1, "k": 1}, "bf16", 0.05),
    ("ij,kj->ki", "jk", {"i": 64, "j": 512, "k": 512}, {"j": 64, "k": 64}, "f32", 0.5),
    ("ij,kj->ki", "jk", {"i": 128, "j": 1024, "k": 512}, {"j": 128, "k": 128}, "bf16", 0.6),
    ("ja,kj->k", "jka", {"j": 40, "a": 12, "k": 40}, {"j": 4, "a": 3, "k": 4}, "f32", 0.5),
    ("jlx,kjl->kx", "jlk", {"j": 16, "l": 12, "x": 8, "k": 20}, {"j": 2, "l": 3, "k": 4}, "f32", 0.4),
    ("jx,kmj->kmx", "jkm", {"j": 24, "x": 16, "k": 12, "m": 8}, {"j": 3, "k": 2, "m": 2}, "bf16", 0.5),
]


@pytest.mark.parametrize("idx", range(len(V_OUTER_PLANS)))
@pytest.mark.parametrize("validate,keep_u", [(True, 0.8), (False, 0.8), (True, 1.0), (False, 1.0)])
def test_v_outer_join_gpu(orc, idx, validate, keep_u):
    """Joins driven by V: pair list, keys and values against the oracle, with
    U missing some join keys (unmatched V tuples) or holding all of them (U
    indexed by the key itself where U's key is the join labels), and key
    validation on or off."""
    import paper_2603_08957_amd as tre

    e, upper, ext, til, dtype, keep_v = V_OUTER_PLANS[idx]
    rng = np.random.default_rng(500 + idx)
    u_lab, v_lab, _ = split_einsum(e)
    U = workloads.random_relation(rng, u_lab, upper, ext, til, dtype, keep=keep_u, zero_frac=0.05)
    V = workloads.random_relation(rng, v_lab, upper, ext, til, dtype, keep=keep_v, zero_frac=0.05)
    spec = workloads.spec(e, upper, ext, til, dtype)
    plan = tre.Plan.from_spec(spec, validate=validate)
    assert plan.join_outer == "v" and not plan.group_needs_sort
    say("v outer", idx, validate, e, len(U["keys"]), len(V["keys"]))
    out = tre.einsum(plan, *to_dev(U), *to_dev(V), want_pairs=True)
    check(out, orc.run(orc_plan(orc, spec), U, V), dtype)


def test_v_outer_key_errors_gpu():
    """Key validation in a V-driven join: unsorted, duplicate and
    out-of-range keys of V are reported, as for a U-driven one."""
    import torch

    import paper_2603_08957_amd as tre

    plan = tre.Plan("ij,kj->ki", "jk", {"i": 8, "j": 16, "k": 16}, {"j": 1, "k": 1}, "f32")
    assert plan.join_outer == "v"
    uk = torch.arange(16, dtype=torch.int32, device="cuda").reshape(-1, 1)
    ut = torch.ones((16, 8), dtype=torch.float32, device="cuda")
    good = np.array([[0, 1], [0, 5], [3, 2], [7, 7]], np.int32)
    for bad, status in ((good[[1, 0, 2, 3]], "TRE_E_UNSORTED"), (good[[0, 0, 2, 3]], "TRE_E_DUPKEY"),
                        (np.array([[0, 1], [0, 5], [3, 2], [7, 16]], np.int32), "TRE_E_KEYRANGE")):
        vk = torch.from_numpy(np.ascontiguousarray(bad)).cuda()
        vt = torch.ones((4, 1), dtype=torch.float32, device="cuda")
        with pytest.raises(tre.TreError) as ei:
            tre.einsum(plan, uk, ut, vk, vt)
        assert ei.value.status == status


def test_v_dense_workspace_gpu(orc):
    """A V-driven join over a U that holds every key: with room for no pair
    the join reports TRE_E_WORKSPACE and the pair count (one per V tuple)
    before any device work; with room it matches the oracle."""
    import paper_2603_08957_amd as tre

    spec = workloads.spec("ij,kj->ki", "jk", {"i": 16, "j": 64, "k": 64}, {"j": 1, "k": 1}, "f32")
    rng = np.random.default_rng(77)
    U = workloads.random_relation(rng, "ij", "jk", spec["extents"], spec["tiles"], "f32", keep=1.0)
    V = workloads.random_relation(rng, "kj", "jk", spec["extents"], spec["tiles"], "f32", keep=0.2)
    plan = tre.Plan.from_spec(spec)
    assert plan.join_outer == "v" and len(U["keys"]) == 64
    uk, ut = to_dev(U)
    vk, vt = to_dev(V)
    ws = tre.alloc_workspace(plan.workspace_bytes(64, len(V["keys"]), 0))
    with pytest.raises(tre.TreError) as ei:
        tre.join(plan, uk, 64, vk, len(V["keys"]), ws)
    assert ei.value.status == "TRE_E_WORKSPACE" and ei.value.join_result.n_pairs == len(V["keys"])
    out = tre.einsum(plan, uk, ut, vk, vt, want_pairs=True, pair_hint=1)
    check(out, orc.run(orc_plan(orc, spec), U, V), "f32")


SMALL_JOINS = [
    # (einsum, upper, extents, tiles, keep U, keep V): small joins of every
    # join direction and GROUP BY order; those whose pairs come out grouped
    # take the one-workgroup path, the others (sorted by W key) must not
    ("ij,jk->ki", "jk", {"i": 8, "j": 64, "k": 64}, {"j": 1, "k": 1}, 0.9, 0.3),       # driven by U, sorted by K
    ("ik,kn->in", "ik", {"i": 64, "k": 64, "n": 8}, {"i": 4, "k": 4}, 0.3, 1.0),       # driven by U, in order
    ("ij,kj->ki", "jk", {"i": 8, "j": 64, "k": 64}, {"j": 1, "k": 1}, 0.7, 0.3),       # driven by V, one match
    ("ja,kj->k", "jka", {"j": 40, "a": 12, "k": 40}, {"j": 4, "a": 3, "k": 4}, 0.5, 0.5),  # driven by V, runs
    ("i,j->ij", "ij", {"i": 60, "j": 50}, {"i": 1, "j": 1}, 0.8, 0.8),                 # cross product
    ("ij,jk->ik", "ijk", {"i": 12, "j": 12, "k": 12}, {"i": 1, "j": 1, "k": 1}, 0.5, 0.5),  # sorted by (I, K)
    ("ij,jk->ki", "jk", {"i": 8, "j": 64, "k": 64}, {"j": 1, "k": 1}, 0.9, 0.0),       # no V tuples
]


@pytest.mark.parametrize("idx", range(len(SMALL_JOINS)))
def test_small_join_gpu(orc, idx):
    """The one-workgroup join: pairs, keys and values against the oracle,
    the path reported by tre_timing, and the multi-kernel join's pair list,
    keys and bits on the same inputs."""
    import torch

    import paper_2603_08957_amd as tre

    e, upper, ext, til, ku, kv = SMALL_JOINS[idx]
    rng = np.random.default_rng(600 + idx)
    u_lab, v_lab, _ = split_einsum(e)
    U = workloads.random_relation(rng, u_lab, upper, ext, til, "f32", keep=ku, zero_frac=0.1)
    V = workloads.random_relation(rng, v_lab, upper, ext, til, "f32", keep=kv, zero_frac=0.1)
    spec = workloads.spec(e, upper, ext, til, "f32")
    say("small join", idx, e, len(U["keys"]), len(V["keys"]))
    uk, ut = to_dev(U)
    vk, vt = to_dev(V)
    small = tre.einsum(tre.Plan.from_spec(spec), uk, ut, vk, vt, want_pairs=True, timing=True)
    multi = tre.einsum(tre.Plan.from_spec(spec, small_join=-1), uk, ut, vk, vt, want_pairs=True, timing=True)
    torch.cuda.synchronize()
    plan = tre.Plan.from_spec(spec)
    if len(V["keys"]) and len(U["keys"]) and not plan.group_needs_sort:
        assert small.timing["join_path"] == "one_workgroup", small.timing
    assert multi.timing["join_path"] != "one_workgroup"
    assert small.n_pairs == multi.n_pairs and small.n_w == multi.n_w
    if small.n_pairs:
        assert torch.equal(small.pairs, multi.pairs) and torch.equal(small.w_keys, multi.w_keys)
        assert torch.equal(small.w_tiles.view(torch.int32), multi.w_tiles.view(torch.int32))
        check(small, orc.run(orc_plan(orc, spec), U, V), "f32")
    else:
        assert small.n_w == 0


def test_small_join_workspace_gpu():
    """The one-workgroup join with room for fewer pairs than the join makes:
    TRE_E_WORKSPACE with the full pair count."""
    import paper_2603_08957_amd as tre
    import torch

    plan = tre.Plan("i,j->ij", "ij", {"i": 40, "j": 30}, {"i": 1, "j": 1}, "f32")
    k40 = torch.arange(40, dtype=torch.int32, device="cuda").reshape(-1, 1)
    k30 = torch.arange(30, dtype=torch.int32, device="cuda").reshape(-1, 1)
    ws = tre.alloc_workspace(plan.workspace_bytes(40, 30, 100))
    tm = tre.Timing()
    with pytest.raises(tre.TreError) as ei:
        tre.join(plan, k40, 40, k30, 30, ws, timing=tm)
    assert ei.value.status == "TRE_E_WORKSPACE" and ei.value.join_result.n_pairs == 1200


U_DENSE_PLANS = [
    # (einsum, upper, extents, tiles, dtype): joins driven by U over a V that
    # holds every key of its key space (V's key is the join labels), with and
    # without the GROUP BY sort
    ("im,mk->ik", "im", {"i": 300, "m": 40, "k": 16}, {"i": 1, "m": 1}, "f32"),   # attention projection form
    ("ik,kn->in", "ik", {"i": 64, "k": 64, "n": 8}, {"i": 4, "k": 4}, "f32"),     # block-sparse form
    ("mi,mk->ik", "im", {"i": 50, "m": 30, "k": 16}, {"i": 1, "m": 1}, "bf16"),   # W key not U's prefix: sorted
    ("iab,ab->i", "iab", {"i": 40, "a": 6, "b": 5}, {"i": 1, "a": 2, "b": 1}, "f32"),  # two join labels
]


@pytest.mark.parametrize("idx", range(len(U_DENSE_PLANS)))
@pytest.mark.parametrize("validate", [True, False])
def test_u_dense_join_gpu(orc, idx, validate):
    """U-driven joins over a complete V (V's index is the join key itself),
    with the one-workgroup join switched off so the dense pass runs: pairs,
    keys and values against the oracle."""
    import paper_2603_08957_amd as tre

    e, upper, ext, til, dtype = U_DENSE_PLANS[idx]
    rng = np.random.default_rng(700 + idx)
    u_lab, v_lab, _ = split_einsum(e)
    U = workloads.random_relation(rng, u_lab, upper, ext, til, dtype, keep=0.4, zero_frac=0.05)
    V = workloads.random_relation(rng, v_lab, upper, ext, til, dtype, keep=1.0, zero_frac=0.05)
    spec = workloads.spec(e, upper, ext, til, dtype)
    plan = tre.Plan.from_spec(spec, validate=validate, small_join=-1)
    say("u dense", idx, validate, e, len(U["keys"]), len(V["keys"]))
    out = tre.einsum(plan, *to_dev(U), *to_dev(V), want_pairs=True, timing=True)
    assert out.timing["join_path"] == "u_driven_dense", out.timing
    check(out, orc.run(orc_plan(orc, spec), U, V), dtype)


V_DENSE_PLANS = [
    # (einsum, upper, extents, tiles, dtype): joins over a U that holds every
    # key of its key space (U's key is the join labels) driven by V, also for
    # plans whose join U drives but whose V key starts with the join labels
    # (V's order is then (u, v) order), with and without the GROUP BY sort
    ("ij,jk->ki", "jk", {"i": 16, "j": 32, "k": 24}, {"j": 4, "k": 4}, "f32"),     # the bf16 chain's E1 form: sorted
    ("ij,jk->ki", "jk", {"i": 8, "j": 24, "k": 40}, {"j": 4, "k": 4}, "bf16"),
    ("ij,kj->ki", "jk", {"i": 16, "j": 32, "k": 24}, {"j": 4, "k": 4}, "f32"),     # V keyed (K, J): V drives
    ("j,jk->jk", "jk", {"j": 30, "k": 20}, {"j": 1, "k": 1}, "f32"),               # W keyed as V: no sort
]


@pytest.mark.parametrize("idx", range(len(V_DENSE_PLANS)))
@pytest.mark.parametrize("validate", [True, False])
def test_v_dense_join_gpu(orc, idx, validate):
    """V-driven joins over a complete U (U's index is the join key itself),
    with the one-workgroup join switched off so the dense pass runs: pairs,
    keys and values against the oracle."""
    import paper_2603_08957_amd as tre

    e, upper, ext, til, dtype = V_DENSE_PLANS[idx]
    rng = np.random.default_rng(760 + idx)
    u_lab, v_lab, _ = split_einsum(e)
    U = workloads.random_relation(rng, u_lab, upper, ext, til, dtype, keep=1.0, zero_frac=0.05)
    V = workloads.random_relation(rng, v_lab, upper, ext, til, dtype, keep=0.4, zero_frac=0.05)
    spec = workloads.spec(e, upper, ext, til, dtype)
    plan = tre.Plan.from_spec(spec, validate=validate, small_join=-1)
    say("v dense", idx, validate, e, plan.join_outer, len(U["keys"]), len(V["keys"]))
    out = tre.einsum(plan, *to_dev(U), *to_dev(V), want_pairs=True, timing=True)
    assert out.timing["join_path"] == "v_driven_dense", out.timing
    check(out, orc.run(orc_plan(orc, spec), U, V), dtype)


# ------------------------------------------------------------ tre_execute

def _execute(spec, U, V, w_cap=None, max_pairs=None, **plan_kw):
    """tre_execute into caller buffers; returns (output namespace, timing dict)."""
    import types

    import torch

    import paper_2603_08957_amd as tre

    plan = tre.Plan.from_spec(spec, **plan_kw)
    uk, ut = to_dev(U)
    vk, vt = to_dev(V)
    n_u, n_v = len(U["keys"]), len(V["keys"])
    cross = max(n_u * n_v, 1)
    w_space = 1
    for c in plan.key_labels[2]:
        w_space *= spec["extents"][c] // spec["tiles"][c]
    cap = min(cross, w_space) if w_cap is None else w_cap
    mp = cross if max_pairs is None else max_pairs
    ws = tre.alloc_workspace(plan.workspace_bytes(n_u, n_v, mp))
    wk = torch.empty((max(cap, 1), max(plan.key_arity[2], 1)), dtype=torch.int32, device="cuda")
    wt = torch.empty((max(cap, 1), plan.tile_elems[2]), dtype=torch.float32, device="cuda")
    pairs = torch.empty((cross, 2), dtype=torch.int32, device="cuda")
    tm = tre.Timing()
    n_w, n_p = tre.execute(plan, uk, ut, vk, vt, wk if plan.key_arity[2] else None, wt, ws, pairs_out=pairs,
                           timing=tm)
    keys = wk[:n_w] if plan.key_arity[2] else wk[:n_w, :0]
    out = types.SimpleNamespace(w_keys=keys, w_tiles=wt[:n_w], n_w=n_w, n_pairs=n_p, pairs=pairs[:n_p])
    return out, tm.as_dict()


@pytest.mark.parametrize("seed", range(40))
def test_execute_random_plans_gpu(orc, seed):
    """tre_execute (join and contraction in one call, into caller buffers)
    on random plans against the oracle: pair lists and key sets bit for bit,
    values within the tolerance."""
    rng = np.random.default_rng(7100 + seed)
    e, upper, ext, til = random_plan(rng)
    u_lab, v_lab, _ = split_einsum(e)
    U = workloads.random_relation(rng, u_lab, upper, ext, til, "f32", keep=0.6, zero_frac=0.3)
    V = workloads.random_relation(rng, v_lab, upper, ext, til, "f32", keep=0.6, zero_frac=0.3)
    spec = workloads.spec(e, upper, ext, til, "f32")
    say("execute", seed, e, upper, til, len(U["keys"]), len(V["keys"]))
    if len(U["keys"]) == 0 or len(V["keys"]) == 0:
        return
    out, tm = _execute(spec, U, V, validate=bool(seed % 2))
    say("  ", tm["join_path"], tm["contract_path"], out.n_pairs, out.n_w)
    ref = orc.run(orc_plan(orc, spec), U, V)
    check(out, ref, "f32")


def test_execute_errors_gpu():
    """tre_execute's errors: key errors (validation on), pairs beyond the
    workspace and an output capacity below the key count, each with the
    counts reported."""
    import paper_2603_08957_amd as tre

    rng = np.random.default_rng(5)
    e, upper, ext, til = "ij,jk->ik", "ijk", {"i": 64, "j": 64, "k": 64}, {"i": 8, "j": 8, "k": 8}
    U = workloads.random_relation(rng, "ij", upper, ext, til, "f32", keep=0.3, zero_frac=0.0)
    V = workloads.random_relation(rng, "jk", upper, ext, til, "f32", keep=0.3, zero_frac=0.0)
    spec = workloads.spec(e, upper, ext, til, "f32")
    out, _ = _execute(spec, U, V)
    n_pairs, n_w = out.n_pairs, out.n_w
    assert 0 < n_w < 64
    bad = dict(U)
    bad["keys"] = np.ascontiguousarray(U["keys"][::-1])
    bad["tiles"] = np.ascontiguousarray(U["tiles"][::-1])
    with pytest.raises(tre.TreError) as err:
        _execute(spec, bad, V)
    assert err.value.status == "TRE_E_UNSORTED"
    with pytest.raises(tre.TreError) as err:
        _execute(spec, U, V, max_pairs=n_pairs // 2)
    assert err.value.status == "TRE_E_WORKSPACE" and err.value.n_pairs == n_pairs
    with pytest.raises(tre.TreError) as err:
        _execute(spec, U, V, w_cap=n_w - 1)
    assert err.value.status == "TRE_E_CAPACITY" and err.value.n_w == n_w and err.value.n_pairs == n_pairs


def test_deferred_timing_gpu():
    """Deferred timing records the contraction kernel's own start and end
    (no wait in the call): read later, contract_ms is positive and close to
    the synchronous phase timing's; with no pairs nothing is pending; the
    three-operand call does the same."""
    import torch

    import paper_2603_08957_amd as tre

    rng = np.random.default_rng(11)
    e, upper, ext, til = "ij,jk->ik", "ijk", {"i": 512, "j": 512, "k": 512}, {"i": 64, "j": 64, "k": 64}
    U = workloads.random_relation(rng, "ij", upper, ext, til, "f32", keep=0.8, zero_frac=0.0)
    V = workloads.random_relation(rng, "jk", upper, ext, til, "f32", keep=0.8, zero_frac=0.0)
    plan = tre.Plan.from_spec(workloads.spec(e, upper, ext, til, "f32"), validate=False)
    uk, ut = to_dev(U)
    vk, vt = to_dev(V)
    ws = tre.alloc_workspace(plan.workspace_bytes(len(uk), len(vk), len(uk) * len(vk)))
    wk = torch.empty((64, 2), dtype=torch.int32, device="cuda")
    wt = torch.empty((64, 64 * 64), dtype=torch.float32, device="cuda")
    sync = tre.Timing()
    tre.execute(plan, uk, ut, vk, vt, wk, wt, ws, timing=sync)
    ref = wt.clone()
    ms = []
    for _ in range(3):
        tm = tre.Timing()
        tm.deferred = 1
        tre.execute(plan, uk, ut, vk, vt, wk, wt, ws, timing=tm)
        assert tm.pending == 1 and tm.join_ms == 0.0
        tm.read()
        assert tm.pending == 0 and tm.contract_ms > 0 and tm.units_ms == 0.0
        ms.append(tm.contract_ms)
    torch.cuda.synchronize()
    assert torch.equal(wt, ref)
    say("deferred", ms, "synchronous", sync.contract_ms)
    assert min(ms) <= 1.5 * sync.contract_ms + 0.05
    # no pairs: no kernel, nothing pending
    tm = tre.Timing()
    tm.deferred = 1
    n_w, n_p = tre.execute(plan, uk[:0], ut[:0], vk, vt, wk, wt, ws, timing=tm)
    assert n_p == 0 and tm.pending == 0
    # three operands (masked form)
    ext3, til3 = {"i": 16, "j": 16, "k": 33}, {"i": 1, "j": 1}
    A = workloads.random_relation(rng, "ij", "ij", ext3, til3, "f32", keep=0.5, zero_frac=0.0)
    B = workloads.random_relation(rng, "ik", "ij", ext3, til3, "f32", keep=1.0, zero_frac=0.0)
    C = workloads.random_relation(rng, "jk", "ij", ext3, til3, "f32", keep=1.0, zero_frac=0.0)
    ak, at = to_dev(A)
    bk, bt = to_dev(B)
    ck, ct = to_dev(C)
    op = tre.Einsum3("ij,ik,jk->ij", "ij", ext3, til3, len(A["keys"]))
    tm = tre.Timing()
    tm.deferred = 1
    op(ak, at, bk, bt, ck, ct, timing=tm)
    assert tm.pending == 1
    tm.read()
    assert tm.contract_ms > 0 and tm.pending == 0


# ------------------------------------------------ size boundaries of the paths

def _rel(rng, keys, tile_elems):
    keys = np.ascontiguousarray(np.asarray(keys, dtype=np.int32).reshape(len(keys), -1))
    return {"keys": keys, "tiles": rng.standard_normal((len(keys), tile_elems)).astype(np.float32), "dtype": "f32"}


@pytest.mark.parametrize("n_u,n_v", [(64, 64), (64, 65), (181, 181), (182, 181), (300, 300)])
def test_cross_product_sizes_gpu(orc, n_u, n_v):
    """A cross product (no join label) whose pairs and output keys number
    4,096 / 4,160 / 32,761 / 32,942 / 90,000: the pair-head scan in one tile,
    in one workgroup and in three passes; the unit table in one workgroup
    (4,096 keys) and over several launches; compared with the oracle, and
    through tre_execute as well."""
    rng = np.random.default_rng(n_u * 1000 + n_v)
    ext, til = {"i": 1 << 14, "k": 1 << 14, "a": 3}, {"i": 1, "k": 1}
    e, upper = "ia,ka->ik", "ik"
    U = _rel(rng, np.sort(rng.choice(1 << 14, n_u, replace=False)), 3)
    V = _rel(rng, np.sort(rng.choice(1 << 14, n_v, replace=False)), 3)
    spec = workloads.spec(e, upper, ext, til, "f32")
    say("cross product", n_u, n_v)
    _, out = gpu_run(spec, U, V, validate=True)
    ref = orc.run(orc_plan(orc, spec), U, V)
    check(out, ref, "f32")
    out2, _ = _execute(spec, U, V, validate=False, max_pairs=n_u * n_v)
    check(out2, ref, "f32")


@pytest.mark.parametrize("radix_k", [32768, 32769])
def test_key_space_segments_sizes_gpu(orc, radix_k):
    """The segments over a dense W key space: 32,768 keys (one workgroup) and
    65,536 (a radix of 32,769 takes 16 key bits: flags, scan, compaction),
    with about a third of the keys absent; the join driven by V over a U that
    holds every key."""
    rng = np.random.default_rng(radix_k)
    n_j = 512
    ext, til = {"i": 4, "j": n_j, "k": radix_k}, {"j": 1, "k": 1}
    e, upper = "ij,kj->ki", "jk"
    X = _rel(rng, np.arange(n_j), 4)
    ks = np.sort(rng.choice(radix_k, (2 * radix_k) // 3, replace=False))
    pairs = [(k, j) for k in ks for j in np.sort(rng.choice(n_j, 3, replace=False))]
    Y = _rel(rng, pairs, 1)
    spec = workloads.spec(e, upper, ext, til, "f32")
    say("key space", radix_k, len(pairs))
    plan, out = gpu_run(spec, X, Y, validate=True)
    ref = orc.run(orc_plan(orc, spec), X, Y)
    check(out, ref, "f32")


@pytest.mark.parametrize("n", [4096, 4097])
def test_small_join_limit_gpu(orc, n):
    """A one-to-one join of n keys (W keyed by the join label): 4,096 pairs
    take the one-workgroup join at its limit, 4,097 the multi-kernel join;
    both against the oracle, and the path taken as reported."""
    rng = np.random.default_rng(n)
    ext, til = {"j": 1 << 20, "a": 5, "b": 4}, {"j": 1}
    e, upper = "ja,jb->jab", "j"
    keys = np.sort(rng.choice(1 << 20, n, replace=False))
    U = _rel(rng, keys, 5)
    V = _rel(rng, keys, 4)
    spec = workloads.spec(e, upper, ext, til, "f32")
    out, tm = _execute(spec, U, V, validate=True)
    say("small join limit", n, tm["join_path"])
    assert (tm["join_path"] == "one_workgroup") == (n <= 4096)
    ref = orc.run(orc_plan(orc, spec), U, V)
    check(out, ref, "f32")
    assert out.n_pairs == n


# ------------------------------------------------- tre_execute_async

def _execute_async(spec, U, V, w_cap=None, pair_cap=None, max_pairs=None, **plan_kw):
    """tre_execute_async into buffers sized by tre_output_bounds; returns
    (output namespace built from the device counts, counts, async_ok)."""
    import types

    import torch

    import paper_2603_08957_amd as tre

    plan = tre.Plan.from_spec(spec, **plan_kw)
    uk, ut = to_dev(U)
    vk, vt = to_dev(V)
    n_u, n_v = len(U["keys"]), len(V["keys"])
    mp = max(n_u * n_v, 1) if max_pairs is None else max_pairs
    ws = tre.alloc_workspace(plan.workspace_bytes(n_u, n_v, mp))
    pb, kb, ok = tre.output_bounds(plan, n_u, n_v, ws.numel())
    kc = kb if w_cap is None else w_cap
    pc = pb if pair_cap is None else pair_cap
    wk = torch.empty((max(kc, 1), max(plan.key_arity[2], 1)), dtype=torch.int32, device="cuda")
    wt = torch.empty((max(kc, 1), plan.tile_elems[2]), dtype=torch.float32, device="cuda")
    pairs = torch.empty((max(pc, 1), 2), dtype=torch.int32, device="cuda")
    counts = torch.full((4,), -1, dtype=torch.int64, device="cuda")
    tre.execute_async(plan, uk, ut, vk, vt, wk if plan.key_arity[2] else None, wt, ws, counts, pairs_out=pairs)
    c = counts.cpu().tolist()
    n_p, n_w = int(c[0]), int(c[1])
    keys = wk[:n_w] if plan.key_arity[2] else wk[:n_w, :0]
    out = types.SimpleNamespace(w_keys=keys, w_tiles=wt[:n_w], n_w=n_w, n_pairs=n_p, pairs=pairs[:n_p])
    return out, c, ok


@pytest.mark.parametrize("seed", range(40))
def test_execute_async_random_plans_gpu(orc, seed):
    """tre_execute_async on random plans (most sizes run with no read-back;
    the others through tre_execute): counts from device memory, pair lists
    and key sets bit for bit against the oracle, values within the
    tolerance."""
    rng = np.random.default_rng(8100 + seed)
    e, upper, ext, til = random_plan(rng)
    u_lab, v_lab, _ = split_einsum(e)
    U = workloads.random_relation(rng, u_lab, upper, ext, til, "f32", keep=0.6, zero_frac=0.3)
    V = workloads.random_relation(rng, v_lab, upper, ext, til, "f32", keep=0.6, zero_frac=0.3)
    spec = workloads.spec(e, upper, ext, til, "f32")
    if len(U["keys"]) == 0 or len(V["keys"]) == 0:
        return
    out, c, ok = _execute_async(spec, U, V, validate=bool(seed % 2))
    say("execute async", seed, e, upper, til, len(U["keys"]), len(V["keys"]), c, ok)
    assert c[2] == 0 and c[3] == 0
    ref = orc.run(orc_plan(orc, spec), U, V)
    check(out, ref, "f32")


def test_execute_async_chain_gpu(orc):
    """The 4096-vertex chain with no host wait: E1 asynchronously, then E2 on
    E1's output buffers with U's count taken from E1's device counts; both
    against the synchronous calls (bit for bit: the bounds are the counts
    here) and E2 against the oracle on E1's output."""
    import torch

    import paper_2603_08957_amd as tre

    w = workloads.config(1, "small")
    p1 = tre.Plan.from_spec(w["E1"], validate=False)
    p2 = tre.Plan.from_spec(w["E2"], validate=False)
    xk, xt = to_dev(w["X"])
    yk, yt = to_dev(w["Y"])
    zk, zt = to_dev(w["Z"])
    n_x, n_y = len(w["X"]["keys"]), len(w["Y"]["keys"])
    ws1 = tre.alloc_workspace(p1.workspace_bytes(n_x, n_y, n_y))
    pb1, kb1, ok1 = tre.output_bounds(p1, n_x, n_y, ws1.numel())
    assert ok1
    t_k = torch.empty((kb1, p1.key_arity[2]), dtype=torch.int32, device="cuda")
    t_t = torch.empty((kb1, p1.tile_elems[2]), dtype=torch.float32, device="cuda")
    c1 = torch.zeros(4, dtype=torch.int64, device="cuda")
    ws2 = tre.alloc_workspace(p2.workspace_bytes(kb1, 1, kb1))
    pb2, kb2, ok2 = tre.output_bounds(p2, kb1, 1, ws2.numel())
    assert ok2 and kb2 == kb1
    o_k = torch.empty((kb2, p2.key_arity[2]), dtype=torch.int32, device="cuda")
    o_t = torch.empty((kb2, p2.tile_elems[2]), dtype=torch.float32, device="cuda")
    c2 = torch.zeros(4, dtype=torch.int64, device="cuda")
    for _ in range(3):  # back to back, no host wait
        tre.execute_async(p1, xk, xt, yk, yt, t_k, t_t, ws1, c1)
        tre.execute_async(p2, t_k, t_t, zk, zt, o_k, o_t, ws2, c2, n_u=kb1, n_u_dev=c1[1:2])
    torch.cuda.synchronize()
    cc1, cc2 = c1.cpu().tolist(), c2.cpu().tolist()
    say("chain counts", cc1, cc2)
    assert cc1[2] == 0 and cc2[2] == 0 and cc2[0] == cc2[1] == cc1[1]
    n_t = cc1[1]
    # synchronous reference on the same inputs
    s1 = tre.einsum(p1, xk, xt, yk, yt)
    assert torch.equal(s1.w_keys, t_k[:n_t]) and torch.equal(s1.w_tiles, t_t[:n_t])
    s2 = tre.einsum(p2, s1.w_keys, s1.w_tiles, zk, zt)
    assert torch.equal(s2.w_keys, o_k[:n_t]) and torch.equal(s2.w_tiles, o_t[:n_t])
    T = {"keys": s1.w_keys.cpu().numpy(), "tiles": s1.w_tiles.cpu().numpy(), "dtype": "f32"}
    ref = orc.run(orc_plan(orc, w["E2"]), T, w["Z"])
    assert np.array_equal(o_k[:n_t].cpu().numpy().reshape(ref.wkeys.shape), ref.wkeys)
    assert_values(o_t[:n_t].cpu().numpy(), ref.acc, ref.mag, "f32", "E2 async")


def test_execute_async_errors_gpu():
    """Errors of the asynchronous call: key errors and pairs beyond the
    workspace come back in the device counts ([2]; [0] the pairs needed);
    output capacity below the bounds and a device-side U count on a plan
    that cannot take one are host errors; sizes beyond the device-count
    launches run synchronously and still fill the counts."""
    import torch

    import paper_2603_08957_amd as tre

    rng = np.random.default_rng(6)
    e, upper, ext, til = "ij,jk->ik", "ijk", {"i": 64, "j": 64, "k": 64}, {"i": 8, "j": 8, "k": 8}
    U = workloads.random_relation(rng, "ij", upper, ext, til, "f32", keep=0.3, zero_frac=0.0)
    V = workloads.random_relation(rng, "jk", upper, ext, til, "f32", keep=0.3, zero_frac=0.0)
    spec = workloads.spec(e, upper, ext, til, "f32")
    out, c, ok = _execute_async(spec, U, V)
    assert ok and c[2] == 0
    n_pairs = c[0]
    bad = dict(U)
    bad["keys"] = np.ascontiguousarray(U["keys"][::-1])
    bad["tiles"] = np.ascontiguousarray(U["tiles"][::-1])
    _, c2, _ = _execute_async(spec, bad, V)
    assert c2[2] == tre.tre.STATUS_CODE["TRE_E_UNSORTED"]
    _, c3, _ = _execute_async(spec, U, V, max_pairs=n_pairs // 2)
    assert c3[2] == tre.tre.STATUS_CODE["TRE_E_WORKSPACE"] and c3[0] == n_pairs
    with pytest.raises(tre.TreError) as err:
        _execute_async(spec, U, V, w_cap=1)
    assert err.value.status == "TRE_E_CAPACITY"
    plan = tre.Plan.from_spec(spec)
    uk, ut = to_dev(U)
    vk, vt = to_dev(V)
    ws = tre.alloc_workspace(plan.workspace_bytes(len(uk), len(vk), len(uk) * len(vk)))
    n_dev = torch.tensor([len(uk)], dtype=torch.int64, device="cuda")
    counts = torch.zeros(4, dtype=torch.int64, device="cuda")
    big = torch.empty((4096, 64), dtype=torch.float32, device="cuda")
    bigk = torch.empty((4096, 2), dtype=torch.int32, device="cuda")
    with pytest.raises(tre.TreError) as err:
        tre.execute_async(plan, uk, ut, vk, vt, bigk, big, ws, counts, n_u_dev=n_dev)
    assert err.value.status == "TRE_E_ARG"
    # more than 4,096 output keys cut into units: synchronous, counts filled
    ext2, til2 = {"i": 1 << 14, "k": 1 << 14, "a": 3}, {"i": 1, "k": 1}
    U2 = _rel(rng, np.sort(rng.choice(1 << 14, 100, replace=False)), 3)
    V2 = _rel(rng, np.sort(rng.choice(1 << 14, 100, replace=False)), 3)
    spec2 = workloads.spec("ia,ka->ik", "ik", ext2, til2, "f32")
    out2, c4, ok2 = _execute_async(spec2, U2, V2)
    assert not ok2 and c4[2] == 0 and c4[0] == 10000 and c4[1] == 10000


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("keep,pmax", [(0.01, 1000), (0.2, 1000), (0.2, 0)])
def test_vec_staged_span_gpu(orc, dtype, keep, pmax):
    """Vector class with many units per workgroup (16-element W tiles: 64
    units per workgroup in fp32, 128 in bf16): a workgroup stages its units'
    pair indices (and, V being scalar tiles, each pair's factor) in LDS when
    their span holds at most 512 pairs, and reads them from memory when it
    does not.  One unit per key (pmax 1000) with about 3 pairs per key
    (keep 0.01) stages; with about 60 (keep 0.2) it does not; the default
    unit length (pmax 0) cuts those keys into short units, staged, with
    partial tiles summed afterwards.  All against the oracle."""
    import paper_2603_08957_amd as tre

    e, upper = "ij,kj->ki", "jk"
    ext, til = {"i": 16, "j": 300, "k": 900}, {"j": 1, "k": 1}
    rng = np.random.default_rng(7100 + int(keep * 100) + 7 * (dtype == "bf16") + (pmax > 0))
    U = workloads.random_relation(rng, "ij", upper, ext, til, dtype, keep=1.0, zero_frac=0.05)
    V = workloads.random_relation(rng, "kj", upper, ext, til, dtype, keep=keep, zero_frac=0.05)
    spec = workloads.spec(e, upper, ext, til, dtype)
    plan = tre.Plan.from_spec(spec, max_pairs_per_unit=pmax)
    assert plan.kernel_class == "vec"
    say("vec staged span", dtype, keep, pmax, len(U["keys"]), len(V["keys"]))
    out = tre.einsum(plan, *to_dev(U), *to_dev(V), want_pairs=True, timing=True)
    assert out.timing["contract_path"] == "vec", out.timing
    check(out, orc.run(orc_plan(orc, spec), U, V), dtype)
