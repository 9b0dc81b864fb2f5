"""The allocation-free entry point tre_execute_noalloc (static device scratch
instead of a workspace argument) against tre_execute on the same inputs:
two calls in a row, the second on a smaller input, so the second call runs on
scratch the first one left behind.  Keys and pairs bit for bit; values within
the oracle's tolerance (the launch may differ from tre_execute's when the
workspace sizes differ, so the summation order of split keys may too)."""
import numpy as np
import pytest

import workloads
from _parity import assert_values

pytestmark = pytest.mark.gpu


def _case(rng, n_k, dtype):
    e, upper = "ij,jk->ki", "jk"
    ext, til = {"i": 64, "j": 64 * 24, "k": 64 * n_k}, {"j": 64, "k": 64}
    U = workloads.random_relation(rng, "ij", upper, ext, til, dtype, keep=0.9)
    V = workloads.random_relation(rng, "jk", upper, ext, til, dtype, keep=0.5)
    return workloads.spec(e, upper, ext, til, dtype), U, V


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_noalloc_matches_execute(orc, dtype):
    import torch

    import paper_2603_08957_amd as tre
    from _parity import to_dev

    assert tre.noalloc_scratch_bytes() == 256 << 20
    rng = np.random.default_rng(31 if dtype == "f32" else 32)
    for n_k in (40, 9):  # the second call is smaller
        spec, U, V = _case(rng, n_k, dtype)
        print(f"[noalloc] {dtype} n_k={n_k} U={len(U['keys'])} V={len(V['keys'])}", flush=True)
        plan = tre.Plan.from_spec(spec)
        uk, ut = to_dev(U)
        vk, vt = to_dev(V)
        ref = tre.einsum(plan, uk, ut, vk, vt, want_pairs=True)
        # outputs allocated before the call: the entry point itself allocates nothing
        cap_w, cap_p = ref.n_w + 5, ref.n_pairs + 7
        wk = torch.full((cap_w, plan.key_arity[2]), -1, dtype=torch.int32, device="cuda")
        wt = torch.full((cap_w, plan.tile_elems[2]), float("nan"), dtype=torch.float32, device="cuda")
        pr = torch.full((cap_p, 2), -1, dtype=torch.int32, device="cuda")
        n_w, n_p = tre.execute_noalloc(plan, uk, ut, vk, vt, wk, wt, pr)
        torch.cuda.synchronize()
        assert (n_w, n_p) == (ref.n_w, ref.n_pairs)
        assert torch.equal(wk[:n_w], ref.w_keys) and torch.equal(pr[:n_p], ref.pairs)
        assert torch.all(wk[n_w:] == -1) and torch.all(pr[n_p:] == -1)  # nothing past the counts
        oref = orc.run(orc.Plan(spec["einsum"], spec["upper"], spec["extents"], spec["tiles"]), U, V)
        assert np.array_equal(pr[:n_p].cpu().numpy(), oref.pairs)
        assert_values(wt[:n_w].cpu().numpy(), oref.acc, oref.mag, dtype, "noalloc")
        assert_values(ref.w_tiles.cpu().numpy(), oref.acc, oref.mag, dtype, "execute")


def test_noalloc_rejects_inputs_beyond_the_scratch():
    """More tuples than the 256 MiB scratch can index: TRE_E_WORKSPACE with a
    message naming the limit, before any device work."""
    import torch

    import paper_2603_08957_amd as tre

    plan = tre.Plan("i,i->i", "i", {"i": 1 << 30}, {"i": 1}, validate=False)
    n = 40 << 20  # about 1 GiB of join bookkeeping for 40 M tuples
    k = torch.arange(4, dtype=torch.int32, device="cuda").reshape(-1, 1)
    t = torch.ones((4, 1), dtype=torch.float32, device="cuda")
    big_k = k[:1].expand(n, 1)  # n rows on paper (stride 0): rejected before any device access
    big_t = t[:1].expand(n, 1)
    with pytest.raises(tre.TreError) as ei:
        tre.execute_noalloc(plan, big_k, big_t, big_k, big_t, k, t)
    assert ei.value.status == "TRE_E_WORKSPACE" and "MiB" in str(ei.value)
