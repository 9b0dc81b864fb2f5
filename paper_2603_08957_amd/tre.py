"""ctypes binding of ``libtre.so`` (the C ABI declared in ``include/tre.h``).

Argument marshalling only: torch supplies device memory and the stream, and
every step of the path runs in the library's HIP kernels.  There is no CPU
fallback; a missing library raises at load time.
"""
from __future__ import annotations

import ctypes
import os
from dataclasses import dataclass

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
# TRE_HOST_SANITIZED=1 loads the host-only AddressSanitizer / UBSan build
# (no device code) for the CPU tests; see build.build_host_sanitized
SANITIZED = os.environ.get("TRE_HOST_SANITIZED") == "1"
LIB_PATH = os.path.join(_HERE, "libtre_host_san.so" if SANITIZED else "libtre.so")

STATUS = {
    0: "TRE_OK", 1: "TRE_E_ARG", 2: "TRE_E_PARSE", 3: "TRE_E_SPLIT", 4: "TRE_E_SHAPE", 5: "TRE_E_DTYPE",
    6: "TRE_E_UNSORTED", 7: "TRE_E_DUPKEY", 8: "TRE_E_KEYRANGE", 9: "TRE_E_CAPACITY", 10: "TRE_E_WORKSPACE",
    11: "TRE_E_DEVICE", 12: "TRE_E_STATE",
}
STATUS_CODE = {v: k for k, v in STATUS.items()}
DTYPE = {"f32": 0, "bf16": 1}

# every symbol include/tre.h declares
EXPORTS = [
    "tre_plan", "tre_plan_get_info", "tre_plan_destroy", "tre_workspace_bytes", "tre_workspace_max_pairs",
    "tre_join", "tre_join_keys", "tre_contract", "tre_execute", "tre_timing_read", "tre_cast_f32_bf16", "tre_scale_f32",
    "tre_stack_workspace_bytes", "tre_stack_rows",
    "tre_tiles_from_entries", "tre_status_str", "tre_last_error", "tre_version",
    "tre_repartition_workspace_bytes", "tre_repartition", "tre_execute3_workspace_bytes", "tre_execute3",
    "tre_noalloc_scratch_bytes", "tre_execute_noalloc", "tre_output_bounds", "tre_execute_async",
]


class TreError(RuntimeError):
    def __init__(self, code: int, where: str, detail: str = ""):
        self.code = code
        self.status = STATUS.get(code, str(code))
        super().__init__(f"{where}: {self.status}" + (f" ({detail})" if detail else ""))


class Options(ctypes.Structure):
    _fields_ = [("validate_keys", ctypes.c_int32), ("max_pairs_per_unit", ctypes.c_int32),
                ("u_ranges", ctypes.c_int32), ("pace_windows", ctypes.c_int32), ("w_bf16", ctypes.c_int32),
                ("small_join", ctypes.c_int32), ("reserved", ctypes.c_int32 * 2)]


class PlanInfo(ctypes.Structure):
    _fields_ = [("key_arity", ctypes.c_int32 * 3), ("tile_elems", ctypes.c_int64 * 3), ("n_join", ctypes.c_int32),
                ("kernel_class", ctypes.c_int32), ("batch", ctypes.c_int64), ("m", ctypes.c_int64),
                ("n", ctypes.c_int64), ("k", ctypes.c_int64), ("flops_per_pair", ctypes.c_int64),
                ("key_labels", (ctypes.c_char * 27) * 3), ("roles", ctypes.c_char * 27),
                ("group_needs_sort", ctypes.c_int32), ("v_needs_sort", ctypes.c_int32), ("w_dtype", ctypes.c_int32),
                ("join_outer", ctypes.c_int32)]


class JoinResult(ctypes.Structure):
    _fields_ = [("n_u", ctypes.c_int64), ("n_v", ctypes.c_int64), ("n_pairs", ctypes.c_int64), ("n_w", ctypes.c_int64),
                ("internal", ctypes.c_uint64 * 16)]


class Timing(ctypes.Structure):
    _fields_ = [("join_ms", ctypes.c_float), ("units_ms", ctypes.c_float), ("contract_ms", ctypes.c_float),
                ("reduce_ms", ctypes.c_float), ("total_ms", ctypes.c_float), ("deferred", ctypes.c_int32),
                ("pending", ctypes.c_int32), ("n_units", ctypes.c_int64), ("n_split_segments", ctypes.c_int64),
                ("n_partials", ctypes.c_int64), ("events", ctypes.c_void_p * 4), ("contract_path", ctypes.c_int32),
                ("join_path", ctypes.c_int32)]

    PATHS = {0: "gemm", 1: "vec", 2: "gemm128", 3: "gemm128_paced", 4: "gemm128_u_ranges"}
    JOIN_PATHS = {0: "u_driven", 1: "v_driven", 2: "v_driven_one_match", 3: "v_driven_dense", 4: "keyed_by_u",
                  5: "one_workgroup", 6: "u_driven_dense"}

    def read(self):
        """Wait for deferred events and fill the millisecond fields."""
        _check(lib().tre_timing_read(ctypes.byref(self)), "tre_timing_read")
        return self

    def as_dict(self):
        d = {k: getattr(self, k) for k, _ in self._fields_ if k not in ("events", "deferred", "pending")}
        d["contract_path"] = self.PATHS.get(self.contract_path, self.contract_path)
        d["join_path"] = self.JOIN_PATHS.get(self.join_path, self.join_path)
        return d


_lib = None


def lib():
    """Load libtre.so; raises if it has not been built (no fallback path)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing: build it with `python -m paper_2603_08957_amd.build`")
        L = ctypes.CDLL(LIB_PATH)
        P, i64, i32, sz = ctypes.c_void_p, ctypes.c_int64, ctypes.c_int32, ctypes.c_size_t
        L.tre_plan.argtypes = [ctypes.c_char_p, ctypes.c_char_p, P, P, ctypes.c_int, P, P]
        L.tre_plan_get_info.argtypes = [P, P]
        L.tre_plan_destroy.argtypes = [P]
        L.tre_plan_destroy.restype = None
        L.tre_workspace_bytes.argtypes = [P, i64, i64, i64]
        L.tre_workspace_bytes.restype = sz
        L.tre_workspace_max_pairs.argtypes = [P, i64, i64, sz]
        L.tre_workspace_max_pairs.restype = i64
        L.tre_join.argtypes = [P, P, i64, P, i64, P, sz, P, P, P]
        L.tre_join_keys.argtypes = [P, P, P, i64, P]
        L.tre_contract.argtypes = [P, P, P, P, P, i64, P, P, i64, P, P]
        L.tre_execute.argtypes = [P, P, i64, P, P, i64, P, P, P, i64, P, P, i64, P, P, sz, P, P]
        L.tre_output_bounds.argtypes = [P, i64, i64, sz, P, P, P]
        L.tre_execute_async.argtypes = [P, P, i64, P, P, P, i64, P, P, P, i64, P, i64, P, P, sz, P, P]
        L.tre_timing_read.argtypes = [P]
        L.tre_cast_f32_bf16.argtypes = [P, P, i64, P]
        L.tre_scale_f32.argtypes = [P, P, i64, ctypes.c_float, P]
        L.tre_stack_workspace_bytes.argtypes = [i64]
        L.tre_stack_workspace_bytes.restype = sz
        L.tre_stack_rows.argtypes = [P, i64, P, i64, i32, i32, P, P, i64, P, P, sz, P]
        L.tre_tiles_from_entries.argtypes = [P, P, P, i64, i32, P, i64, i64, P]
        cs = ctypes.c_char_p
        L.tre_repartition_workspace_bytes.argtypes = [cs, cs, cs, P, P, P, i64]
        L.tre_repartition_workspace_bytes.restype = sz
        L.tre_repartition.argtypes = [cs, cs, cs, P, P, P, i32, P, i64, P, P, P, i64, P, P, sz, P]
        L.tre_execute3_workspace_bytes.argtypes = [cs, cs, P, P, i64]
        L.tre_execute3_workspace_bytes.restype = sz
        L.tre_execute3.argtypes = [cs, cs, P, P, ctypes.c_int, P, i64, P, P, i64, P, P, i64, P, P, P, i64, P, P, P, sz,
                                   P, P]
        L.tre_noalloc_scratch_bytes.argtypes = []
        L.tre_noalloc_scratch_bytes.restype = sz
        L.tre_execute_noalloc.argtypes = [P, P, i64, P, P, i64, P, P, P, i64, P, P, i64, P, P]
        L.tre_status_str.restype = ctypes.c_char_p
        L.tre_last_error.restype = ctypes.c_char_p
        L.tre_version.restype = ctypes.c_char_p
        _lib = L
    return _lib


def _check(rc: int, where: str):
    if rc != 0:
        raise TreError(rc, where, lib().tre_last_error().decode())


def _ptr(t):
    """Device pointer of a torch tensor (or None)."""
    if t is None:
        return None
    return ctypes.c_void_p(t.data_ptr())


def _stream(stream=None):
    import torch

    s = stream if stream is not None else torch.cuda.current_stream()
    return ctypes.c_void_p(s.cuda_stream)


class Plan:
    """A parsed, classified binary EinSum (host object, see tre_plan)."""

    def __init__(self, einsum: str, upper: str, extents: dict, tiles: dict, dtype: str = "f32",
                 validate: bool = True, max_pairs_per_unit: int = 0, u_ranges: int = 0, pace_windows: int = 0,
                 w_bf16: bool = False, small_join: int = 0):
        L = lib()
        ext = np.zeros(26, dtype=np.int64)
        til = np.ones(26, dtype=np.int32)
        for k, v in extents.items():
            ext[ord(k) - 97] = v
        for k, v in (tiles or {}).items():
            til[ord(k) - 97] = v
        opt = Options(int(validate), int(max_pairs_per_unit), int(u_ranges), int(pace_windows), int(w_bf16),
                      int(small_join))
        self.w_bf16 = bool(w_bf16)
        h = ctypes.c_void_p(0)
        rc = L.tre_plan(einsum.encode(), upper.encode(), ext.ctypes.data_as(ctypes.c_void_p),
                        til.ctypes.data_as(ctypes.c_void_p), DTYPE[dtype], ctypes.byref(opt), ctypes.byref(h))
        _check(rc, "tre_plan")
        self._h = h
        self.einsum, self.upper, self.dtype = einsum, upper, dtype
        info = PlanInfo()
        _check(L.tre_plan_get_info(h, ctypes.byref(info)), "tre_plan_get_info")
        self.key_arity = list(info.key_arity)
        self.tile_elems = list(info.tile_elems)
        self.n_join = info.n_join
        self.kernel_class = {0: "gemm", 1: "vec", 2: "gemm128"}[info.kernel_class]
        self.bmnk = (info.batch, info.m, info.n, info.k)
        self.flops_per_pair = info.flops_per_pair
        self.key_labels = [bytes(info.key_labels[o]).split(b"\0")[0].decode() for o in range(3)]
        self.roles = bytes(info.roles).split(b"\0")[0].decode()
        self.group_needs_sort = bool(info.group_needs_sort)
        self.v_needs_sort = bool(info.v_needs_sort)
        self.w_dtype = {0: "f32", 1: "bf16"}[info.w_dtype]
        self.join_outer = "v" if info.join_outer else "u"

    @classmethod
    def from_spec(cls, spec: dict, **kw):
        return cls(spec["einsum"], spec["upper"], spec["extents"], spec["tiles"], spec["dtype"], **kw)

    @property
    def handle(self):
        return self._h

    def workspace_bytes(self, n_u: int, n_v: int, max_pairs: int) -> int:
        return int(lib().tre_workspace_bytes(self._h, n_u, n_v, max_pairs))

    def __del__(self):
        h = getattr(self, "_h", None)
        if h is not None and h.value and _lib is not None:
            _lib.tre_plan_destroy(h)
            self._h = None


def alloc_workspace(nbytes: int, device="cuda"):
    import torch

    ws = torch.empty(max(int(nbytes), 256), dtype=torch.uint8, device=device)
    assert ws.data_ptr() % 256 == 0
    return ws


def join(plan: Plan, u_keys, n_u: int, v_keys, n_v: int, ws, stream=None, timing: Timing | None = None) -> JoinResult:
    jr = JoinResult()
    rc = lib().tre_join(plan.handle, _ptr(u_keys), n_u, _ptr(v_keys), n_v, _ptr(ws), ws.numel(), _stream(stream),
                        ctypes.byref(jr), ctypes.byref(timing) if timing is not None else None)
    if rc != 0:
        err = TreError(rc, "tre_join", lib().tre_last_error().decode())
        err.join_result = jr
        raise err
    return jr


def contract(plan: Plan, jr: JoinResult, u_tiles, v_tiles, w_keys, w_tiles, pairs_out=None, stream=None,
             timing: Timing | None = None):
    w_cap = w_tiles.shape[0] if w_tiles is not None else 0
    pair_cap = pairs_out.shape[0] if pairs_out is not None else 0
    rc = lib().tre_contract(plan.handle, ctypes.byref(jr), _ptr(u_tiles), _ptr(v_tiles), _ptr(w_keys), w_cap,
                            _ptr(w_tiles), _ptr(pairs_out), pair_cap, _stream(stream),
                            ctypes.byref(timing) if timing is not None else None)
    _check(rc, "tre_contract")


def join_keys(plan: Plan, jr: JoinResult, w_keys, stream=None):
    """Write the join's output keys (tre_join_keys) into w_keys [>= n_w, r_W]."""
    w_cap = w_keys.shape[0] if w_keys is not None else 0
    _check(lib().tre_join_keys(plan.handle, ctypes.byref(jr), _ptr(w_keys), w_cap, _stream(stream)),
           "tre_join_keys")


def execute(plan: Plan, u_keys, u_tiles, v_keys, v_tiles, w_keys, w_tiles, ws, pairs_out=None, stream=None,
            timing: Timing | None = None):
    """tre_execute into caller-owned outputs and workspace (their row counts
    are the capacities): the join and the contraction in one call.  Returns
    (n_w, n_pairs); a TreError carries them when a capacity is short."""
    n_u, n_v = int(u_tiles.shape[0]), int(v_tiles.shape[0])
    n_w, n_p = ctypes.c_int64(0), ctypes.c_int64(0)
    rc = lib().tre_execute(plan.handle, _ptr(u_keys), n_u, _ptr(u_tiles), _ptr(v_keys), n_v, _ptr(v_tiles),
                           _ptr(w_keys), _ptr(w_tiles), int(w_tiles.shape[0]) if w_tiles is not None else 0,
                           ctypes.byref(n_w), _ptr(pairs_out), int(pairs_out.shape[0]) if pairs_out is not None else 0,
                           ctypes.byref(n_p), _ptr(ws), ws.numel(), _stream(stream),
                           ctypes.byref(timing) if timing is not None else None)
    if rc != 0:
        err = TreError(rc, "tre_execute", lib().tre_last_error().decode())
        err.n_w, err.n_pairs = int(n_w.value), int(n_p.value)
        raise err
    return int(n_w.value), int(n_p.value)


def output_bounds(plan: Plan, n_u: int, n_v: int, ws_bytes: int):
    """tre_output_bounds: (pair bound, key bound, whether tre_execute_async
    runs without a read-back for these sizes)."""
    pb, kb, ok = ctypes.c_int64(0), ctypes.c_int64(0), ctypes.c_int32(0)
    _check(lib().tre_output_bounds(plan.handle, int(n_u), int(n_v), int(ws_bytes), ctypes.byref(pb), ctypes.byref(kb),
                                   ctypes.byref(ok)), "tre_output_bounds")
    return int(pb.value), int(kb.value), bool(ok.value)


def execute_async(plan: Plan, u_keys, u_tiles, v_keys, v_tiles, w_keys, w_tiles, ws, counts, pairs_out=None,
                  n_u=None, n_u_dev=None, stream=None, timing: Timing | None = None):
    """tre_execute_async: join and contraction enqueued with no wait; the
    counts ([pairs, keys, status, 0]) land in ``counts`` (device int64 [4]).
    ``n_u`` defaults to u_tiles' rows; ``n_u_dev`` (a device int64 tensor)
    holds U's actual count when n_u is only a bound."""
    n_u = int(u_tiles.shape[0]) if n_u is None else int(n_u)
    n_v = int(v_tiles.shape[0])
    rc = lib().tre_execute_async(plan.handle, _ptr(u_keys), n_u, _ptr(n_u_dev), _ptr(u_tiles), _ptr(v_keys), n_v,
                                 _ptr(v_tiles), _ptr(w_keys), _ptr(w_tiles),
                                 int(w_tiles.shape[0]) if w_tiles is not None else 0, _ptr(pairs_out),
                                 int(pairs_out.shape[0]) if pairs_out is not None else 0, _ptr(counts), _ptr(ws),
                                 ws.numel(), _stream(stream), ctypes.byref(timing) if timing is not None else None)
    _check(rc, "tre_execute_async")


@dataclass
class Output:
    w_keys: object      # torch int32 [n_w, r_W]
    w_tiles: object     # torch float32 [n_w, tile_elems(W)]
    pairs: object       # torch int32 [n_pairs, 2] or None
    n_pairs: int
    n_w: int
    timing: dict | None
    ws: object


def einsum(plan: Plan, u_keys, u_tiles, v_keys, v_tiles, want_pairs: bool = False, ws=None, stream=None,
           timing: bool = False, pair_hint: int | None = None) -> Output:
    """Join + contract with output buffers allocated by torch.  The workspace
    is grown and the join repeated once if the pair list does not fit."""
    import torch

    n_u, n_v = int(u_tiles.shape[0]), int(v_tiles.shape[0])
    dev = u_tiles.device
    if ws is None:
        hint = pair_hint if pair_hint is not None else max(n_u, n_v, 1) * 2
        ws = alloc_workspace(plan.workspace_bytes(n_u, n_v, hint), dev)
    tm = Timing() if timing else None
    try:
        jr = join(plan, u_keys, n_u, v_keys, n_v, ws, stream, tm)
    except TreError as e:
        if e.code != 10 or e.join_result.n_pairs <= 0:
            raise
        ws = alloc_workspace(plan.workspace_bytes(n_u, n_v, int(e.join_result.n_pairs)), dev)
        jr = join(plan, u_keys, n_u, v_keys, n_v, ws, stream, tm)
    n_w, n_p = int(jr.n_w), int(jr.n_pairs)
    rw = plan.key_arity[2]
    w_keys = torch.empty((n_w, rw), dtype=torch.int32, device=dev)
    w_tiles = torch.empty((n_w, plan.tile_elems[2]), dtype=torch.bfloat16 if plan.w_bf16 else torch.float32,
                          device=dev)
    pairs = torch.empty((n_p, 2), dtype=torch.int32, device=dev) if want_pairs else None
    contract(plan, jr, u_tiles, v_tiles, w_keys if rw > 0 else None, w_tiles, pairs, stream, tm)
    return Output(w_keys, w_tiles, pairs, n_p, n_w, tm.as_dict() if tm is not None else None, ws)


def execute_noalloc(plan: Plan, u_keys, u_tiles, v_keys, v_tiles, w_keys, w_tiles, pairs_out=None, stream=None):
    """tre_execute_noalloc: join + contract with the library's static device
    scratch as workspace; every output buffer is the caller's (their row
    counts are the capacities).  Returns (n_w, n_pairs)."""
    n_u, n_v = int(u_tiles.shape[0]), int(v_tiles.shape[0])
    n_w, n_p = ctypes.c_int64(0), ctypes.c_int64(0)
    rc = lib().tre_execute_noalloc(plan.handle, _ptr(u_keys), n_u, _ptr(u_tiles), _ptr(v_keys), n_v, _ptr(v_tiles),
                                   _ptr(w_keys), _ptr(w_tiles), int(w_tiles.shape[0]), ctypes.byref(n_w),
                                   _ptr(pairs_out), int(pairs_out.shape[0]) if pairs_out is not None else 0,
                                   ctypes.byref(n_p), _stream(stream))
    if rc != 0:
        err = TreError(rc, "tre_execute_noalloc", lib().tre_last_error().decode())
        err.n_w, err.n_pairs = int(n_w.value), int(n_p.value)
        raise err
    return int(n_w.value), int(n_p.value)


def noalloc_scratch_bytes() -> int:
    return int(lib().tre_noalloc_scratch_bytes())


def cast_f32_bf16(x, out=None, stream=None):
    import torch

    y = out if out is not None else torch.empty(x.shape, dtype=torch.bfloat16, device=x.device)
    _check(lib().tre_cast_f32_bf16(_ptr(x), _ptr(y), x.numel(), _stream(stream)), "tre_cast_f32_bf16")
    return y


def scale_f32(x, scale: float, out=None, stream=None):
    """out = scale * x (fp32, elementwise; out may be x)."""
    import torch

    y = out if out is not None else torch.empty_like(x)
    _check(lib().tre_scale_f32(_ptr(x), _ptr(y), x.numel(), float(scale), _stream(stream)), "tre_scale_f32")
    return y


def stack_rows(keys, tiles, group: int, stream=None):
    """STACK re-composition (see tre_stack_rows); keys [n] or [n,1] int32."""
    import torch

    n = int(keys.shape[0])
    row = int(tiles.numel() // max(n, 1)) if n else int(tiles.shape[1])
    eb = tiles.element_size()
    ws = alloc_workspace(int(lib().tre_stack_workspace_bytes(n)), tiles.device)
    cap = n
    out_keys = torch.empty((cap, 1), dtype=torch.int32, device=tiles.device)
    out_tiles = torch.empty((cap, group * row), dtype=tiles.dtype, device=tiles.device)
    n_out = ctypes.c_int64(0)
    rc = lib().tre_stack_rows(_ptr(keys), n, _ptr(tiles), row, group, eb, _ptr(out_keys), _ptr(out_tiles), cap,
                              ctypes.byref(n_out), _ptr(ws), ws.numel(), _stream(stream))
    _check(rc, "tre_stack_rows")
    k = int(n_out.value)
    return out_keys[:k], out_tiles[:k]


def repartition(labels: str, upper_in: str, upper_out: str, extents: dict, tiles_in: dict, tiles_out: dict,
                keys, tiles, stream=None, in_place: bool = False):
    """The relation (keys, tiles) under the target decomposition (see
    tre_repartition).  Returns (keys_out [n_out, r_out] int32, tiles_out
    [n_out, tile_elems_out], same dtype as ``tiles``).  ``in_place``: the
    target tiles are a view of ``tiles`` (a regrouping of whole tiles in
    order, nothing missing; TreError otherwise)."""
    import numpy as _np
    import torch

    ext = _np.zeros(26, dtype=_np.int64)
    tin = _np.ones(26, dtype=_np.int32)
    tout = _np.ones(26, dtype=_np.int32)
    for k, v in extents.items():
        ext[ord(k) - 97] = v
    for k, v in (tiles_in or {}).items():
        tin[ord(k) - 97] = v
    for k, v in (tiles_out or {}).items():
        tout[ord(k) - 97] = v
    args = (labels.encode(), upper_in.encode(), upper_out.encode(), ext.ctypes.data_as(ctypes.c_void_p),
            tin.ctypes.data_as(ctypes.c_void_p), tout.ctypes.data_as(ctypes.c_void_p))
    n = int(keys.shape[0]) if keys is not None else int(tiles.shape[0])
    wsb = int(lib().tre_repartition_workspace_bytes(*args, n))
    n_out = ctypes.c_int64(0)
    if wsb == 0:  # bad arguments: let the call itself name the error
        rc = lib().tre_repartition(*args, tiles.element_size(), _ptr(keys), n, _ptr(tiles), None, None, 0,
                                   ctypes.byref(n_out), None, 0, _stream(stream))
        _check(rc if rc else STATUS_CODE["TRE_E_ARG"], "tre_repartition")
    ws = alloc_workspace(wsb, tiles.device)
    te_in = te_out = 1
    grid = cover = 1
    for c in labels:
        e, ti, to = int(ext[ord(c) - 97]), int(tin[ord(c) - 97]), int(tout[ord(c) - 97])
        ti = ti if c in upper_in else e
        te_in *= ti
        te_out *= to if c in upper_out else e
        if c in upper_out and to > 0:
            grid *= e // to
            cover *= min(e // to, (ti - 1) // to + 2)
    if in_place:
        cap = (n * te_in) // max(te_out, 1)
        out_keys = torch.empty((max(cap, 1), len(upper_out)), dtype=torch.int32, device=tiles.device)
        rc = lib().tre_repartition(*args, tiles.element_size(), _ptr(keys), n, _ptr(tiles), _ptr(out_keys),
                                   _ptr(tiles), cap, ctypes.byref(n_out), _ptr(ws), ws.numel(), _stream(stream))
        _check(rc, "tre_repartition")
        k = int(n_out.value)
        return out_keys[:k], tiles.reshape(-1)[:k * te_out].view(k, te_out)
    # first call with room for every target tile the sources can meet when
    # that costs little memory; otherwise the call reports the count first
    bound = min(grid, n * cover)
    esz = tiles.element_size()
    cap = bound if bound * te_out * esz <= max(2 * n * te_in * esz, 1 << 26) else 0
    while True:
        out_keys = torch.empty((max(cap, 1), len(upper_out)), dtype=torch.int32, device=tiles.device)
        out_tiles = torch.empty((max(cap, 1), te_out), dtype=tiles.dtype, device=tiles.device)
        rc = lib().tre_repartition(*args, tiles.element_size(), _ptr(keys), n, _ptr(tiles), _ptr(out_keys),
                                   _ptr(out_tiles), cap, ctypes.byref(n_out), _ptr(ws), ws.numel(), _stream(stream))
        if rc == STATUS_CODE["TRE_E_CAPACITY"] and n_out.value > cap:
            cap = int(n_out.value)
            continue
        _check(rc, "tre_repartition")
        k = int(n_out.value)
        return out_keys[:k], out_tiles[:k]


def tiles_from_entries(slot, offset, values, n_tiles: int, tile_elems: int, stream=None):
    """Dense tiles [n_tiles, tile_elems] (dtype of ``values``) from scalar entries."""
    import torch

    tiles = torch.empty((n_tiles, tile_elems), dtype=values.dtype, device=values.device)
    rc = lib().tre_tiles_from_entries(_ptr(slot), _ptr(offset), _ptr(values), int(values.numel()),
                                      values.element_size(), _ptr(tiles), n_tiles, tile_elems, _stream(stream))
    _check(rc, "tre_tiles_from_entries")
    return tiles


class Einsum3:
    """One three-operand EinSum "U,V,X->W" (see tre_execute3): U joined with V
    and X in one pass, one fused contraction per matched triple.  Holds the
    letter-indexed shape arrays and a workspace sized for ``n_u_max``."""

    def __init__(self, einsum: str, upper: str, extents: dict, tiles: dict, n_u_max: int, device="cuda"):
        import numpy as _np

        self.einsum, self.upper = einsum, upper
        self._ext = _np.zeros(26, dtype=_np.int64)
        self._tile = _np.ones(26, dtype=_np.int32)
        for k, v in extents.items():
            self._ext[ord(k) - 97] = v
        for k, v in (tiles or {}).items():
            self._tile[ord(k) - 97] = v
        w = einsum.split("->")[1]
        self.w_arity = sum(1 for c in w if c in upper)
        self.w_tile_elems = 1
        self.w_key_space = 1
        for c in w:
            e, t = int(self._ext[ord(c) - 97]), int(self._tile[ord(c) - 97])
            self.w_tile_elems *= t if c in upper else e
            if c in upper:
                self.w_key_space *= e // t
        self.n_u_max = int(n_u_max)
        wsb = int(lib().tre_execute3_workspace_bytes(*self._args(), self.n_u_max))
        if wsb == 0:  # bad arguments: let the call itself name the error
            n_w, n_t = ctypes.c_int64(0), ctypes.c_int64(0)
            rc = lib().tre_execute3(*self._args(), 0, None, 0, None, None, 0, None, None, 0, None, None, None, 0,
                                    ctypes.byref(n_w), ctypes.byref(n_t), None, 0, None, None)
            _check(rc if rc else STATUS_CODE["TRE_E_ARG"], "tre_execute3")
        self.ws = alloc_workspace(wsb, device)

    def _args(self):
        return (self.einsum.encode(), self.upper.encode(), self._ext.ctypes.data_as(ctypes.c_void_p),
                self._tile.ctypes.data_as(ctypes.c_void_p))

    def __call__(self, u_keys, u_tiles, v_keys, v_tiles, x_keys, x_tiles, stream=None, timing: Timing | None = None,
                 out=None):
        """Returns (w_keys int32 [n_w, r_W], w_tiles float32 [n_w, tile_elems(W)], n_triples).
        ``out`` = (w_keys, w_tiles) preallocated buffers (their row count is the capacity)."""
        import torch

        n_u, n_v, n_x = int(u_tiles.shape[0]), int(v_tiles.shape[0]), int(x_tiles.shape[0])
        if n_u > self.n_u_max:
            raise ValueError(f"n_u {n_u} above the workspace sizing {self.n_u_max}")
        dev = u_tiles.device
        if out is None:
            cap = min(n_u, self.w_key_space)
            out = (torch.empty((max(cap, 1), self.w_arity), dtype=torch.int32, device=dev),
                   torch.empty((max(cap, 1), self.w_tile_elems), dtype=torch.float32, device=dev))
            cap_given = cap
        else:
            cap_given = int(out[1].shape[0])
        n_w, n_t = ctypes.c_int64(0), ctypes.c_int64(0)
        rc = lib().tre_execute3(*self._args(), 0, _ptr(u_keys), n_u, _ptr(u_tiles), _ptr(v_keys), n_v, _ptr(v_tiles),
                                _ptr(x_keys), n_x, _ptr(x_tiles), _ptr(out[0]) if self.w_arity else None,
                                _ptr(out[1]), cap_given, ctypes.byref(n_w), ctypes.byref(n_t), _ptr(self.ws),
                                self.ws.numel(), _stream(stream), ctypes.byref(timing) if timing is not None else None)
        _check(rc, "tre_execute3")
        k = int(n_w.value)
        return out[0][:k], out[1][:k], int(n_t.value)


def execute3(einsum: str, upper: str, extents: dict, tiles: dict, u_keys, u_tiles, v_keys, v_tiles, x_keys, x_tiles,
             stream=None, timing: bool = False):
    """One-shot tre_execute3 with a fresh workspace; returns (w_keys, w_tiles,
    n_triples[, timing dict])."""
    op = Einsum3(einsum, upper, extents, tiles, int(u_tiles.shape[0]), u_tiles.device)
    tm = Timing() if timing else None
    wk, wt, nt = op(u_keys, u_tiles, v_keys, v_tiles, x_keys, x_tiles, stream, tm)
    return (wk, wt, nt, tm.as_dict()) if timing else (wk, wt, nt)
