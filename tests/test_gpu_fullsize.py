"""GPU parity at the full sizes of the five workloads, in the launch
configuration the benchmark times.

The oracle cannot evaluate every output at these sizes, so each test samples
output keys (seeded), restricts the input relations to the tuples that feed
them (selection on the promoted labels, Sec. 5) and compares:
  * the pair list restricted to the sampled keys: bit-exact,
  * the output key set: bit-exact against the oracle's key-level join where
    that is cheap, else against closed forms,
  * the sampled output tiles: mag-relative error within 1e-4 (fp32) / 1e-2
    (bf16 inputs, fp32 accumulation).
Chains are also checked end to end on sampled keys, each side computing its
own intermediate (the GPU in fp32 then bf16 via its cast kernel, the oracle in
fp64 rounded to fp32 then bf16)."""
import gc
import sys
import types

import numpy as np
import pytest

import workloads
from _parity import U_ACC, U_BF16, assert_values

pytestmark = [pytest.mark.gpu, pytest.mark.slow]


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


@pytest.fixture(autouse=True)
def _free_gpu():
    yield
    import torch

    gc.collect()
    torch.cuda.empty_cache()


def orc_plan(orc, s):
    return orc.Plan(s["einsum"], s["upper"], s["extents"], s["tiles"])


def split_einsum(e):
    lhs, w = e.split("->")
    u, v = lhs.split(",")
    return u, v, w


def w_keys_of_pairs(spec, ukeys, vkeys, pairs):
    """Output key of every pair: W's promoted labels taken from U's key when U
    has the label, else from V's."""
    u, v, w = split_einsum(spec["einsum"])
    up = spec["upper"]
    uk = [c for c in u if c in up]
    vk = [c for c in v if c in up]
    cols = []
    for c in [c for c in w if c in up]:
        if c in uk:
            cols.append(ukeys[pairs[:, 0], uk.index(c)])
        else:
            cols.append(vkeys[pairs[:, 1], vk.index(c)])
    return np.stack(cols, axis=1) if cols else np.zeros((len(pairs), 0), np.int32)


def rows_in(a, b):
    """Boolean mask: rows of a that occur in b."""
    if a.shape[1] == 0:
        return np.ones(len(a), bool)
    base = int(max(a.max(initial=0), b.max(initial=0))) + 1
    enc = lambda x: (x.astype(np.int64) * (base ** np.arange(x.shape[1] - 1, -1, -1))).sum(axis=1)  # noqa: E731
    return np.isin(enc(a), enc(b))


def dev(a, bf16=False):
    import torch

    a = np.ascontiguousarray(a)
    if bf16:
        return torch.from_numpy(a.view(np.int16)).cuda().view(torch.bfloat16)
    return torch.from_numpy(a).cuda()


def sampled_check(orc, spec, U, V, out, S, u_tiles_host=True, pairs=None):
    """Restrict U and V to the tuples feeding the sampled keys S, run the
    oracle there and compare pairs and tiles of S."""
    p = orc_plan(orc, spec)
    mu, mv = orc.restrict(p, U["keys"], V["keys"], S)
    iu, iv = np.nonzero(mu)[0], np.nonzero(mv)[0]

    def sub(rel, idx, m):
        r = {"keys": rel["keys"][idx]}
        if "tiles" in rel:
            r.update(tiles=rel["tiles"][idx], dtype=rel["dtype"])
        else:  # scalar entries: keep those of kept tuples
            keep = m[rel["slot"]]
            r["coo"] = (rel["coo"][0][keep], rel["coo"][1][keep])
        return r

    su, sv = sub(U, iu, mu), sub(V, iv, mv)
    ref_pairs, ref_keys = orc.join(p, su["keys"], sv["keys"])
    ref_pairs = np.stack([iu[ref_pairs[:, 0]], iv[ref_pairs[:, 1]]], axis=1) if len(ref_pairs) else ref_pairs
    in_s = rows_in(ref_keys, S)
    assert in_s.sum() == len(S), "a sampled key has no pairs"
    if pairs is not None:
        wk = w_keys_of_pairs(spec, U["keys"], V["keys"], pairs)
        got = pairs[rows_in(wk, S)]
        rwk = w_keys_of_pairs(spec, U["keys"], V["keys"], ref_pairs)
        assert np.array_equal(got, ref_pairs[rows_in(rwk, S)]), "pair list differs on the sampled keys"
    uc, uv = orc._coo_of(p, 0, su)
    vc, vv = orc._coo_of(p, 1, sv)
    acc, mag, _ = orc.evaluate(p, uc, uv, vc, vv, S)
    gk = out.w_keys.cpu().numpy().reshape(out.n_w, -1)
    index = {tuple(r): i for i, r in enumerate(gk.tolist())}
    rows = [index[tuple(r)] for r in S.tolist()]
    got = out.w_tiles[rows].float().cpu().numpy()  # (bf16 outputs upcast exactly)
    f = assert_values(got, acc, mag, spec["dtype"], "sampled keys")
    say(f"sampled keys: {f}")
    return f["mag_rel"]


def pick(rng, keys, n):
    idx = np.sort(rng.choice(len(keys), size=min(n, len(keys)), replace=False))
    return np.ascontiguousarray(keys[idx])


# ----------------------------------------------------------------- GNN

def run_gnn(orc, c):
    import paper_2603_08957_amd as tre
    import torch

    w = workloads.config(c)
    Y = w["Y"]
    bf = w["dtype"] == "bf16"
    say(f"workload {c}: {w['n']} vertices, {w['n_edges']} edges, {len(Y['keys'])} Y tuples")
    xk, xt = dev(w["X"]["keys"]), dev(w["X"]["tiles"], bf)
    yk = dev(Y["keys"])
    if "tiles" in Y:
        yt = dev(Y["tiles"], bf)
    else:
        yt = tre.tiles_from_entries(dev(Y["slot"]), dev(Y["offset"]), dev(Y["values"], bf), len(Y["keys"]),
                                    Y["tile_elems"])
    p1 = tre.Plan.from_spec(w["E1"])
    o1 = tre.einsum(p1, xk, xt, yk, yt, want_pairs=True, pair_hint=len(Y["keys"]) if w["tile_e1"] > 1 else w["n_edges"])
    torch.cuda.synchronize()
    del yt
    torch.cuda.empty_cache()
    # closed forms: one pair per Y tuple (X holds every J); keys = distinct K
    assert o1.n_pairs == len(Y["keys"])
    assert np.array_equal(o1.w_keys.cpu().numpy()[:, 0], np.unique(Y["keys"][:, w["y_k_col"]]))
    pairs = o1.pairs.cpu().numpy()
    rng = np.random.default_rng(100 + c)
    S1 = pick(rng, o1.w_keys.cpu().numpy(), 6)
    say("E1 sampled", S1.ravel().tolist())
    sampled_check(orc, w["E1"], w["X"], Y if "tiles" not in Y else {**Y, "tiles": Y["tiles"]}, o1, S1,
                  pairs=pairs)
    # glue and E2 on the GPU
    tk, tt = o1.w_keys, o1.w_tiles
    stack = w["tile_e2"] // w["tile_e1"]
    if stack > 1:  # re-partition T (Sec. 6) from per-vertex rows to E2's tiles
        tk, tt = tre.repartition("ki", "k", "k", {"k": w["n"], "i": w["emb"]}, {"k": 1}, {"k": stack}, tk, tt)
    tb = tre.cast_f32_bf16(tt).view(tt.shape) if bf else tt
    p2 = tre.Plan.from_spec(w["E2"])
    o2 = tre.einsum(p2, tk, tb, dev(w["Z"]["keys"]), dev(w["Z"]["tiles"], bf), want_pairs=True)
    assert o2.n_pairs == tk.shape[0] and o2.n_w == tk.shape[0]
    assert np.array_equal(o2.pairs.cpu().numpy(), np.stack([np.arange(o2.n_pairs), np.zeros(o2.n_pairs)], 1))
    # end to end on sampled E2 keys
    chain_end_to_end(orc, w, o2.w_keys.cpu().numpy(), o2.w_tiles, rng, 4)


def chain_end_to_end(orc, w, e2_keys, e2_tiles, rng, n_keys):
    """End to end on sampled E2 keys: the oracle computes the T rows they need
    itself (E1 restricted to those vertices), rounds fp64 -> fp32 -> bf16,
    stacks, and runs E2; the GPU's E2 tiles of those keys must match."""
    Y = w["Y"]
    bf = w["dtype"] == "bf16"
    stack = w["tile_e2"] // w["tile_e1"]
    S2 = pick(rng, e2_keys, n_keys)
    t2, t1 = w["tile_e2"], w["tile_e1"]
    need = np.unique(np.concatenate([np.arange(k * t2 // t1, (k + 1) * t2 // t1) for k in S2[:, 0]]))
    have = set(np.unique(Y["keys"][:, w["y_k_col"]]).tolist())
    need = np.array([k for k in need if k in have], dtype=np.int32).reshape(-1, 1)
    op1 = orc_plan(orc, w["E1"])
    mu, mv = orc.restrict(op1, w["X"]["keys"], Y["keys"], need)
    keep = mv[Y["slot"]]
    uc, uv, _ = orc.expand(op1, 0, w["X"]["keys"][mu], w["X"]["tiles"][mu], w["dtype"])
    acc1, _, _ = orc.evaluate(op1, uc, uv, Y["coo"][0][keep], Y["coo"][1][keep], need)
    t32 = acc1.astype(np.float32)
    kk, tiles = need, t32
    if stack > 1:
        kk, tiles = orc.repartition("ki", "k", "k", {"k": w["n"], "i": w["emb"]}, {"k": 1}, {"k": stack}, need, t32)
        tiles = tiles.astype(np.float32)
    op2 = orc_plan(orc, w["E2"])
    if bf:
        Tin = {"keys": kk, "tiles": orc.f32_to_bf16(tiles), "dtype": "bf16"}
    else:
        Tin = {"keys": kk, "tiles": tiles, "dtype": "f32"}
    r2 = orc.run(op2, Tin, w["Z"])
    index = {int(k): i for i, k in enumerate(np.asarray(e2_keys).reshape(-1))}
    rk = {int(k): i for i, k in enumerate(r2.wkeys[:, 0])}
    got = e2_tiles[[index[int(k)] for k in S2[:, 0]]].float().cpu().numpy()
    acc = r2.acc[[rk[int(k)] for k in S2[:, 0]]]
    mag = r2.mag[[rk[int(k)] for k in S2[:, 0]]]
    # a bf16 chain's intermediate is rounded to bf16 by each side on its own
    f = assert_values(got, acc, mag, w["dtype"], "chain end to end", u=U_BF16 if bf else U_ACC)
    say(f"chain end-to-end on {len(S2)} keys: {f}")


def test_gnn_chain_fp32_full(orc):
    run_gnn(orc, 1)


def test_gnn_chain_bf16_262k_full(orc):
    run_gnn(orc, 2)


def test_gnn_chain_bf16_1m_full(orc):
    run_gnn(orc, 5)


# --------------------------------------------------------- block sparse

def test_block_sparse_full(orc):
    import paper_2603_08957_amd as tre

    w = workloads.config(3)
    p = tre.Plan.from_spec(w["E"])
    o = tre.einsum(p, dev(w["A"]["keys"]), dev(w["A"]["tiles"]), dev(w["B"]["keys"]), dev(w["B"]["tiles"]),
                   want_pairs=True)
    ref_pairs, ref_keys = orc.join(orc_plan(orc, w["E"]), w["A"]["keys"], w["B"]["keys"])
    assert np.array_equal(o.pairs.cpu().numpy(), ref_pairs) and len(ref_pairs) == 819
    assert np.array_equal(o.w_keys.cpu().numpy(), ref_keys)
    rng = np.random.default_rng(103)
    sampled_check(orc, w["E"], w["A"], w["B"], o, pick(rng, ref_keys, 4))


# ------------------------------------------------------------ 3-way

def test_sparse_three_way_full(orc):
    import paper_2603_08957_amd as tre
    import torch

    w = workloads.config(4)
    p1 = tre.Plan.from_spec(w["E1"])
    o1 = tre.einsum(p1, dev(w["T"]["keys"]), dev(w["T"]["tiles"]), dev(w["B"]["keys"]), dev(w["B"]["tiles"]),
                    want_pairs=True)
    op1 = orc_plan(orc, w["E1"])
    ref_pairs, ref_keys = orc.join(op1, w["T"]["keys"], w["B"]["keys"])
    assert np.array_equal(o1.pairs.cpu().numpy(), ref_pairs) and len(ref_pairs) == len(w["T"]["keys"])
    assert np.array_equal(o1.w_keys.cpu().numpy(), ref_keys)
    rng = np.random.default_rng(104)
    sampled_check(orc, w["E1"], w["T"], w["B"], o1, pick(rng, ref_keys, 24))
    # E2 on the GPU's W, then end to end on sampled output rows I
    p2 = tre.Plan.from_spec(w["E2"])
    o2 = tre.einsum(p2, o1.w_keys, o1.w_tiles, dev(w["C"]["keys"]), dev(w["C"]["tiles"]), want_pairs=True)
    torch.cuda.synchronize()
    ref2_pairs, ref2_keys = orc.join(orc_plan(orc, w["E2"]), ref_keys, w["C"]["keys"])
    assert np.array_equal(o2.pairs.cpu().numpy(), ref2_pairs)
    assert np.array_equal(o2.w_keys.cpu().numpy(), ref2_keys)
    S = pick(rng, ref2_keys, 3)
    need = ref_keys[np.isin(ref_keys[:, 0], S[:, 0])]
    mu, mv = orc.restrict(op1, w["T"]["keys"], w["B"]["keys"], need)
    uc, uv, _ = orc.expand(op1, 0, w["T"]["keys"][mu], w["T"]["tiles"][mu], "f32")
    vc, vv, _ = orc.expand(op1, 1, w["B"]["keys"][mv], w["B"]["tiles"][mv], "f32")
    acc1, _, _ = orc.evaluate(op1, uc, uv, vc, vv, need)
    r2 = orc.run(orc_plan(orc, w["E2"]), {"keys": need, "tiles": acc1, "dtype": "f64"}, w["C"])
    gk = o2.w_keys.cpu().numpy()[:, 0]
    rows = [int(np.nonzero(gk == k)[0][0]) for k in S[:, 0]]
    rr = [int(np.nonzero(r2.wkeys[:, 0] == k)[0][0]) for k in S[:, 0]]
    f = assert_values(o2.w_tiles[rows].cpu().numpy(), r2.acc[rr], r2.mag[rr], "f32", "3-way end to end")
    say(f"3-way end-to-end on {len(S)} rows: {f}")


def test_sparse_three_way_fused_full(orc):
    """The same contraction through the fused three-operand path
    (tre_execute3, the launch the benchmark times for this workload): triple
    count = T blocks (B and C hold every block), output keys = distinct I
    blocks of T, sampled output tiles against the oracle's per-triple
    evaluation of the T tuples that feed them."""
    import paper_2603_08957_amd as tre

    w = workloads.config(4)
    ext = {"i": w["n"], "j": w["n"], "k": w["n"], "r": w["r"]}
    til = {c: w["block"] for c in "ijk"}
    wk, wt, nt = tre.execute3("ijk,jr,kr->ir", "ijk", ext, til, dev(w["T"]["keys"]), dev(w["T"]["tiles"]),
                              dev(w["B"]["keys"]), dev(w["B"]["tiles"]), dev(w["C"]["keys"]), dev(w["C"]["tiles"]))
    tk = w["T"]["keys"]
    assert nt == len(tk)
    want = np.unique(tk[:, 0]).astype(np.int32).reshape(-1, 1)
    gk = wk.cpu().numpy()
    assert np.array_equal(gk, want)
    rng = np.random.default_rng(105)
    S = pick(rng, want, 4)[:, 0]
    sel = np.isin(tk[:, 0], S)
    T = {"keys": np.ascontiguousarray(tk[sel]), "tiles": w["T"]["tiles"][sel], "dtype": "f32"}
    rk, acc, mag, _ = orc.eval3("ijk,jr,kr->ir", "ijk", ext, til, T, w["B"], w["C"])
    rows = [int(np.nonzero(gk[:, 0] == k)[0][0]) for k in rk[:, 0]]
    f = assert_values(wt[rows].cpu().numpy(), acc, mag, "f32", "fused 3-way")
    say(f"fused 3-way on {len(S)} output keys ({int(sel.sum())} triples): {f}")


def test_graph_attention_full(orc):
    """The graph-attention workload at full size (13,752 nodes, ~0.4M edges,
    767 features, d_k 1024) in the benchmark's launch configuration: E1 and
    E2 on sampled output keys against the C oracle; the masked EinSum's keys
    on every edge (bit-exact: every node has a feature, so every edge is
    matched) and its values on sampled edges against the oracle's per-triple
    evaluation fed the GPU's own T0 and T1; the binary path of Table
    gt-schema (E3 with no aggregation, then E4) gives the same keys and, on
    the sampled edges, values within the tolerance."""
    import torch

    import paper_2603_08957_amd as tre

    w = workloads.config(6)
    rng = np.random.default_rng(66)
    d = {name: (dev(w[name]["keys"]), dev(w[name]["tiles"])) for name in ("X", "WQ", "WK", "A")}
    T, host = {}, {}
    for name, wname in (("E1", "WQ"), ("E2", "WK")):
        s = w[name]
        out = tre.einsum(tre.Plan.from_spec(s, validate=False), d["X"][0], d["X"][1], d[wname][0], d[wname][1])
        torch.cuda.synchronize()
        assert out.n_w == w["n"]
        S = np.sort(rng.choice(w["n"], 48, replace=False)).reshape(-1, 1).astype(np.int32)
        say("attention", name, out.n_pairs, out.n_w)
        sampled_check(orc, s, w["X"], w[wname], out, S)
        T[name] = (out.w_keys.reshape(-1, 1).contiguous(), out.w_tiles)
        host[name] = {"keys": out.w_keys.cpu().numpy().reshape(-1, 1), "tiles": out.w_tiles.cpu().numpy(),
                      "dtype": "f32"}
    e = w["E34"]
    wk, wt, nt = tre.execute3(e["einsum"], e["upper"], e["extents"], e["tiles"], d["A"][0], d["A"][1],
                              T["E1"][0], T["E1"][1], T["E2"][0], T["E2"][1])
    torch.cuda.synchronize()
    assert nt == w["n_edges"] == int(wk.shape[0])
    assert np.array_equal(wk.cpu().numpy(), w["A"]["keys"])
    sel = np.sort(rng.choice(w["n_edges"], 3000, replace=False))
    A_s = {"keys": np.ascontiguousarray(w["A"]["keys"][sel]), "tiles": w["A"]["tiles"][sel], "dtype": "f32"}
    rk, acc, mag, _ = orc.eval3(e["einsum"], e["upper"], e["extents"], e["tiles"], A_s, host["E1"], host["E2"])
    assert np.array_equal(rk, A_s["keys"])
    f = assert_values(wt.cpu().numpy()[sel], acc, mag, "f32", "attention fused")
    say("attention fused", nt, f)
    o3 = tre.einsum(tre.Plan.from_spec(w["E3"], validate=False), T["E1"][0], T["E1"][1], d["A"][0], d["A"][1])
    o4 = tre.einsum(tre.Plan.from_spec(w["E4"], validate=False), o3.w_keys, o3.w_tiles, T["E2"][0], T["E2"][1])
    torch.cuda.synchronize()
    assert torch.equal(o4.w_keys.reshape(wk.shape), wk)
    f = assert_values(o4.w_tiles.cpu().numpy()[sel], acc, mag, "f32", "attention binary")
    say("attention binary", o3.n_w, f)


@pytest.mark.parametrize("config", [1, 5])
def test_bench_chain_overlap_matches_serial(config):
    """The benchmark's chain step -- for the 4096-vertex chain both EinSums
    through tre_execute_async with no host wait (E2's U count from E1's
    device counts), for the 1,048,576-vertex chain E2's join and the key-only
    stack on a second stream while E1's contraction runs -- must equal the
    serial order's result bit for bit, on every repeat."""
    import torch

    import bench
    import paper_2603_08957_amd as tre

    print(f"[chain overlap] config {config}", flush=True)
    W = bench.GnnChain(config, tre, torch)
    assert W.async_ok == (config in (1, 2))
    k_ref, t_ref = (x.clone() for x in W._step_serial())
    for _ in range(3):
        k, t = W.step()
        torch.cuda.synchronize()
        if W.async_ok:
            W.check_async()
            n = W.e2.check_async()[1]
            k, t = k[:n], t[:n]
        assert torch.equal(k, k_ref)
        assert torch.equal(t, t_ref)
    del W
    gc.collect()
    torch.cuda.empty_cache()


@pytest.mark.parametrize("path", ["fused", "binary"])
def test_bench_attention_overlap_matches_serial(path):
    """The attention step contracts its two projections on two streams at
    once; the scores must equal the serial order's bit for bit."""
    import torch

    import bench
    import paper_2603_08957_amd as tre

    print(f"[attention overlap] {path}", flush=True)
    W = bench.Attention(6, tre, torch, path=path)
    k_ref, t_ref = (x.clone() for x in W.step(overlap=False))
    for _ in range(3):
        k, t = W.step()
        torch.cuda.synchronize()
        assert torch.equal(k, k_ref)
        assert torch.equal(t, t_ref)
    del W
    gc.collect()
    torch.cuda.empty_cache()


@pytest.mark.parametrize("config", [2, 5])
def test_bench_timed_launch_matches_oracle(orc, config):
    """Exactly what the benchmark times for the bf16 chains: its own Stage
    objects (key validation off, E1 writing W as bf16 from its fp32 sums,
    the paced persistent 128x128 grid for the 262,144-vertex chain, the
    vector class for the 1,048,576-vertex one) and its own step.  Checked
    against the oracle:
      * E1's whole pair list and output key set, bit for bit against the
        oracle's join (2,248,311 and 33,554,432 pairs);
      * sampled E1 output tiles, upcast from bf16, within the bf16 tolerance;
      * the chain end to end on sampled E2 keys."""
    import torch

    import bench
    import paper_2603_08957_amd as tre

    print(f"[bench launch] config {config}", flush=True)
    W = bench.GnnChain(config, tre, torch)
    e1 = W.e1
    assert e1.plan.w_dtype == "bf16" and e1.plan.kernel_class == ("gemm128" if config == 2 else "vec")
    e1.pairs_out = torch.empty((e1.n_v, 2), dtype=torch.int32, device="cuda")  # one pair per Y tuple at most
    W.step()
    torch.cuda.synchronize()
    if W.async_ok:  # the timed step runs tre_execute_async: outputs and counts stay on the device
        W.check_async()
        n_p, n_w = e1.check_async()
        k1_buf, t1_buf = e1.a_keys, e1.a_tiles
        n_w2 = W.e2.check_async()[1]
        k2, t2 = W.e2.a_keys[:n_w2].cpu().numpy(), W.e2.a_tiles[:n_w2].clone()
    else:
        n_p, n_w = e1.n_pairs, e1.n_w
        k1_buf, t1_buf = e1.w_keys, e1.w_tiles
        k2, t2 = W.e2.w_keys[:W.e2.n_w].cpu().numpy(), W.e2.w_tiles[:W.e2.n_w].clone()
    got_pairs = e1.pairs_out[:n_p].cpu().numpy()
    got_keys = k1_buf[:n_w].cpu().numpy()
    t1 = t1_buf[:n_w].clone()
    # which contraction launch the timed step used
    tm = tre.Timing()
    e1.record = tm
    e1.pairs_out = None
    W.step()
    torch.cuda.synchronize()
    e1.record = None
    say(f"E1 launch: {tm.as_dict()}")
    assert tm.as_dict()["contract_path"] == ("gemm128_paced" if config == 2 else "vec")
    w = W.w
    del W
    gc.collect()
    torch.cuda.empty_cache()
    ref_pairs, ref_keys = orc.join(orc_plan(orc, w["E1"]), w["X"]["keys"], w["Y"]["keys"])
    say(f"E1: {n_p} pairs, {n_w} keys; oracle {len(ref_pairs)} pairs, {len(ref_keys)} keys")
    assert np.array_equal(got_pairs, ref_pairs), "pair list differs from the oracle's join"
    assert np.array_equal(got_keys, ref_keys), "output key set differs from the oracle's"
    del ref_pairs
    rng = np.random.default_rng(200 + config)
    S1 = pick(rng, ref_keys, 8)
    out = types.SimpleNamespace(w_keys=torch.from_numpy(got_keys), w_tiles=t1.float(), n_w=n_w)
    sampled_check(orc, w["E1"], w["X"], w["Y"], out, S1)
    chain_end_to_end(orc, w, k2, t2, rng, 4)
