"""MI355X-native shard of a pooled sparse embedding layer.

Thin ctypes binding over ``libemb.so`` (HIP kernels for gfx950, C ABI in
``include/emb.h``).  This module only marshals arguments: every step of the
layer runs in the library's kernels.  PyTorch provides device memory and
streams; tensors are passed by ``data_ptr()`` and the current HIP stream.

The layer is the one the paper's introduction names as the high data-access
part of a recommendation model, turning sparse ids into dense features
(Introduction; Section "Multi-mode Execution", heterogeneous pipeline).
"""
from __future__ import annotations

import array
import ctypes
import os
from dataclasses import dataclass
from typing import Optional, Sequence

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libemb.so")

EMB_OK, EMB_EINVAL, EMB_EWORKSPACE, EMB_EUNSUPPORTED, EMB_EHIP = range(5)
FP32, BF16 = 0, 1
POOL = {"sum": 0, "mean": 1}
OPT = {"sgd": 0, "adagrad": 1, "adagrad_ew": 2}
DTYPE = {"fp32": FP32, "bf16": BF16}

EXPORTED = ("emb_pool_fwd", "emb_workspace_size", "emb_workspace_init", "emb_unique_ids", "emb_unique_ids_concurrent",
            "emb_grad_reduce",
            "emb_sparse_update", "emb_validate_batch", "emb_workspace_error_offset", "emb_workspace_status",
            "emb_status_string", "emb_route_workspace_size", "emb_route_ids", "emb_route_ids_noalloc",
            "emb_pipeline_steps", "emb_unique_ids_batched")


class EmbError(RuntimeError):
    def __init__(self, fn: str, status: int):
        self.status = status
        super().__init__(f"{fn}: {_status_string(status)} (status {status})")


class StepFailed(RuntimeError):
    """A dedup (and the reduce after it) failed on the device: one of its
    bounded waits for a word another workgroup publishes ran out, or a sort
    pass found inconsistent digit totals.  No table or state row was written
    by that step."""

    SITES = {0x100: "sort pass {p}: tile waiting for its digit offsets",
             0x102: "sort pass {p}: prefix block waiting for its group's counts",
             0x103: "sort pass {p}: prefix block waiting for the group sums",
             0x104: "sort pass {p}: prefix block waiting for the later passes' counts",
             0x105: "sort pass {p}: range block waiting for its tiles' counts",
             0x200: "unique scan look-back", 0x300: "gradient combine"}

    def __init__(self, bits: int, site: int, block: int, timeouts: int):
        self.bits, self.site, self.block, self.timeouts = bits, site, block, timeouts
        what = []
        if bits & 1:
            what.append("a dedup wait ran out")
        if bits & 2:
            what.append("a sort pass found digit totals inconsistent with its keys (workspace not initialised?)")
        if bits & 4:
            what.append("a gradient-combine wait ran out")
        desc = self.SITES.get(site & ~0xf0, "none").format(p=(site >> 4) & 0xf) if site else "none"
        super().__init__(f"embedding step failed on the device: {'; '.join(what)} (error bits {bits}); first wait "
                         f"that ran out since the workspace was initialised: {desc}, workgroup {block}; "
                         f"{timeouts} waits ran out in all")


class CTables(ctypes.Structure):
    _fields_ = [("num_tables", ctypes.c_int32), ("row_offset", ctypes.POINTER(ctypes.c_int64)),
                ("dim", ctypes.c_int32), ("dtype", ctypes.c_int32), ("weights", ctypes.c_void_p)]


class CBatch(ctypes.Structure):
    _fields_ = [("bags_per_table", ctypes.c_int32), ("offsets", ctypes.c_void_p), ("indices", ctypes.c_void_p),
                ("num_indices", ctypes.c_int64), ("index_bytes", ctypes.c_int32)]


class CUpdate(ctypes.Structure):
    _fields_ = [("opt", ctypes.c_int32), ("lr", ctypes.c_float), ("eps", ctypes.c_float),
                ("state", ctypes.c_void_p), ("rounding", ctypes.c_int32), ("seed", ctypes.c_uint64)]


ROUNDING = {"nearest": 0, "stochastic": 1}


class CDedupSet(ctypes.Structure):
    _fields_ = [("unique_keys", ctypes.c_void_p), ("counts", ctypes.c_void_p), ("seg_offsets", ctypes.c_void_p),
                ("sort_perm", ctypes.c_void_p), ("num_unique", ctypes.c_void_p), ("ws", ctypes.c_void_p),
                ("ws_bytes", ctypes.c_size_t)]


_lib = None


def lib():
    """Load libemb.so; raises if it is not built (there is no fallback path)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing: build it with __graft_entry__.build() "
                               "(the embedding layer has no non-HIP implementation)")
        L = ctypes.CDLL(LIB_PATH)
        vp, i32, i64, sz = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_size_t
        T, B, Up = ctypes.POINTER(CTables), ctypes.POINTER(CBatch), ctypes.POINTER(CUpdate)
        L.emb_pool_fwd.restype = i32
        L.emb_pool_fwd.argtypes = [T, B, i32, vp, vp]
        L.emb_workspace_size.restype = sz
        L.emb_workspace_size.argtypes = [i64, i64, i32]
        L.emb_workspace_init.restype = i32
        L.emb_workspace_init.argtypes = [vp, sz, vp]
        L.emb_unique_ids.restype = i32
        L.emb_unique_ids.argtypes = [T, B, vp, vp, vp, vp, vp, vp, sz, vp]
        L.emb_unique_ids_concurrent.restype = i32
        L.emb_unique_ids_concurrent.argtypes = [T, B, vp, vp, vp, vp, vp, vp, sz, vp]
        L.emb_grad_reduce.restype = i32
        L.emb_grad_reduce.argtypes = [T, B, i32, vp, vp, vp, vp, vp, vp, Up, vp, sz, vp]
        L.emb_sparse_update.restype = i32
        L.emb_sparse_update.argtypes = [T, Up, vp, vp, i64, vp, vp]
        L.emb_route_workspace_size.restype = sz
        L.emb_route_workspace_size.argtypes = [i64, i64, i32]
        L.emb_route_ids.restype = i32
        L.emb_route_ids.argtypes = [T, B, i32, ctypes.POINTER(ctypes.c_int64), vp, vp, vp, vp, vp, sz, vp]
        PV = ctypes.POINTER(vp)
        L.emb_pipeline_steps.restype = i32
        L.emb_pipeline_steps.argtypes = [T, i32, Up, i32, B, PV, PV, i32, ctypes.POINTER(CDedupSet), vp, i32, PV, PV,
                                         vp, sz, i32, i32, i32, i32]
        L.emb_unique_ids_batched.restype = i32
        L.emb_unique_ids_batched.argtypes = [T, i32, B, ctypes.POINTER(CDedupSet), vp, sz, vp]
        L.emb_route_ids_noalloc.restype = i32
        L.emb_route_ids_noalloc.argtypes = [T, B, i32, ctypes.POINTER(ctypes.c_int64), vp, vp, vp, vp, vp]
        L.emb_validate_batch.restype = i32
        L.emb_validate_batch.argtypes = [T, B, vp, vp]
        L.emb_workspace_error_offset.restype = sz
        L.emb_workspace_error_offset.argtypes = []
        L.emb_workspace_status.restype = i32
        L.emb_workspace_status.argtypes = [vp, sz, vp, vp]
        L.emb_status_string.restype = ctypes.c_char_p
        L.emb_status_string.argtypes = [i32]
        _lib = L
    return _lib


def _status_string(st: int) -> str:
    try:
        return lib().emb_status_string(st).decode()
    except Exception:  # pragma: no cover - only while the library is unloadable
        return "unknown"


def _check(fn: str, st: int) -> None:
    if st != EMB_OK:
        raise EmbError(fn, st)


def _ptr(t) -> Optional[int]:
    if t is None:
        return None
    return int(t.data_ptr())


def _stream(stream) -> Optional[int]:
    if stream is None:
        import torch
        return int(torch.cuda.current_stream().cuda_stream)
    if isinstance(stream, int):
        return stream
    return int(stream.cuda_stream)


@dataclass
class Tables:
    """Stacked tables (device weights [R][D], host row offsets [T+1])."""
    weights: object                  # torch tensor float32 [R][D] or bfloat16 [R][D]
    row_offset: Sequence[int]

    def c(self) -> CTables:
        key = (_ptr(self.weights), tuple(self.weights.shape), self.weights.dtype)
        if getattr(self, "_ckey", None) != key:
            import torch
            ro = (ctypes.c_int64 * len(self.row_offset))(*[int(x) for x in self.row_offset])
            dt = BF16 if self.weights.dtype == torch.bfloat16 else FP32
            self._ro = ro  # kept alive with the struct
            self._c = CTables(len(self.row_offset) - 1, ro, int(self.weights.shape[1]), dt, _ptr(self.weights))
            self._ckey = key
        return self._c


@dataclass
class Batch:
    """A table-major batch in CSR form (device int32 offsets [M+1], int32 or
    int64 indices [N])."""
    offsets: object
    indices: object
    bags_per_table: int

    def __post_init__(self):
        # the C descriptor is built with the batch, not on its first use
        self.c()

    def __setattr__(self, name, value):
        # assigning a field drops the cached descriptor
        if name in ("offsets", "indices", "bags_per_table"):
            self.__dict__["_ckey"] = None
        object.__setattr__(self, name, value)

    def c(self) -> CBatch:
        """The C descriptor; rebuilt if a tensor was replaced or reallocated."""
        idx = self.indices
        key = (self.offsets.data_ptr(), idx.data_ptr(), idx.numel(), self.bags_per_table, idx.element_size())
        if getattr(self, "_ckey", None) != key:
            n = key[2]
            self._c = CBatch(self.bags_per_table, key[0], key[1] if n else None, n, key[4])
            self._cb = bytes(self._c)
            self._ckey = key
        return self._c

    def _c_bytes(self) -> bytes:
        """The descriptor's bytes, for arrays of descriptors: with the fields
        unassigned since it was built, only a reallocation of a tensor (its
        address or length) is checked for."""
        k = self.__dict__.get("_ckey")
        idx = self.indices
        if k is None or k[0] != self.offsets.data_ptr() or k[1] != idx.data_ptr() or k[2] != idx.numel():
            self.c()
        return self._cb


def workspace_size(num_indices: int, num_bags: int, dim: int) -> int:
    return int(lib().emb_workspace_size(num_indices, num_bags, dim))


def workspace_init(ws, stream=None) -> None:
    _check("emb_workspace_init", lib().emb_workspace_init(_ptr(ws), ws.numel() * ws.element_size(),
                                                          _stream(stream)))


def pool_fwd(tables: Tables, batch: Batch, pool: str, out, stream=None) -> None:
    _check("emb_pool_fwd", lib().emb_pool_fwd(ctypes.byref(tables.c()), ctypes.byref(batch.c()), POOL[pool],
                                              _ptr(out), _stream(stream)))


def unique_ids(tables: Tables, batch: Batch, unique_keys, counts, seg_offsets, sort_perm, num_unique, ws,
               stream=None, concurrent: bool = False) -> None:
    """The batch's dedup; ``concurrent`` selects emb_unique_ids_concurrent
    (no workgroup waits for another; any number may be in flight at once)."""
    fn = "emb_unique_ids_concurrent" if concurrent else "emb_unique_ids"
    _check(fn, getattr(lib(), fn)(
        ctypes.byref(tables.c()), ctypes.byref(batch.c()), _ptr(unique_keys), _ptr(counts), _ptr(seg_offsets),
        _ptr(sort_perm), _ptr(num_unique), _ptr(ws), ws.numel() * ws.element_size(), _stream(stream)))


def _dedup_set(b) -> "CDedupSet":
    return CDedupSet(_ptr(b.unique_keys), _ptr(b.counts), _ptr(b.seg_offsets), _ptr(b.sort_perm), _ptr(b.num_unique),
                     _ptr(b.ws), b.ws.numel() * b.ws.element_size())


def unique_ids_batched(tables: Tables, batches, sets, ws, stream=None) -> None:
    """The dedups of several batches as one sort (emb_unique_ids_batched):
    ``sets[i]`` (DedupBuffers) receives exactly what ``unique_ids`` of
    ``batches[i]`` would leave in it; ``ws`` is the group's own workspace."""
    batches, sets = list(batches), list(sets)
    if len(batches) != len(sets):
        raise ValueError("one buffer set per batch")
    n = len(batches)
    cb = (CBatch * max(n, 1))(*[b.c() for b in batches])
    cs = (CDedupSet * max(n, 1))(*[_dedup_set(b) for b in sets])
    _check("emb_unique_ids_batched", lib().emb_unique_ids_batched(
        ctypes.byref(tables.c()), n, cb, cs, _ptr(ws), ws.numel() * ws.element_size(), _stream(stream)))


def _update(opt: str, lr: float, eps: float, state, rounding: str = "nearest", seed: int = 0) -> CUpdate:
    return CUpdate(OPT[opt], lr, eps, _ptr(state), ROUNDING[rounding], seed)


def grad_reduce(tables: Tables, batch: Batch, pool: str, grad_out, sort_perm, seg_offsets, unique_keys,
                num_unique, ws, grad_rows=None, opt: Optional[str] = None, lr: float = 0.0, eps: float = 0.0,
                state=None, stream=None, rounding: str = "nearest", seed: int = 0) -> None:
    """Segment-reduce the upstream gradient; with ``opt`` also apply the fused optimizer step."""
    upd = ctypes.byref(_update(opt, lr, eps, state, rounding, seed)) if opt is not None else None
    _check("emb_grad_reduce", lib().emb_grad_reduce(
        ctypes.byref(tables.c()), ctypes.byref(batch.c()), POOL[pool], _ptr(grad_out), _ptr(sort_perm),
        _ptr(seg_offsets), _ptr(unique_keys), _ptr(num_unique), _ptr(grad_rows), upd, _ptr(ws),
        ws.numel() * ws.element_size(), _stream(stream)))


def sparse_update(tables: Tables, opt: str, lr: float, eps: float, state, unique_keys, num_unique,
                  max_unique: int, grad_rows, stream=None, rounding: str = "nearest", seed: int = 0) -> None:
    _check("emb_sparse_update", lib().emb_sparse_update(
        ctypes.byref(tables.c()), ctypes.byref(_update(opt, lr, eps, state, rounding, seed)), _ptr(unique_keys),
        _ptr(num_unique), max_unique, _ptr(grad_rows), _stream(stream)))


def validate_batch(tables: Tables, batch: Batch, flag, stream=None) -> None:
    _check("emb_validate_batch", lib().emb_validate_batch(ctypes.byref(tables.c()), ctypes.byref(batch.c()),
                                                          _ptr(flag), _stream(stream)))


def route_workspace_size(num_indices: int, num_bags: int, world_size: int) -> int:
    return int(lib().emb_route_workspace_size(num_indices, num_bags, world_size))


def route_ids(tables: Tables, batch: Batch, shard_start: Sequence[int], send_counts, send_ids, send_pos, send_bag,
              ws, stream=None) -> None:
    """Bucket the batch's ids by the owner rank of a row-range sharding
    (rank r owns global rows [shard_start[r], shard_start[r+1]))."""
    W = len(shard_start) - 1
    ss = (ctypes.c_int64 * len(shard_start))(*[int(x) for x in shard_start])
    _check("emb_route_ids", lib().emb_route_ids(
        ctypes.byref(tables.c()), ctypes.byref(batch.c()), W, ss, _ptr(send_counts), _ptr(send_ids), _ptr(send_pos),
        _ptr(send_bag), _ptr(ws), ws.numel() * ws.element_size() if ws is not None else 0, _stream(stream)))


def route_ids_noalloc(tables: Tables, batch: Batch, shard_start: Sequence[int], send_counts, send_ids, send_pos,
                      send_bag, stream=None) -> None:
    """route_ids without a workspace (the library's per-device scratch array
    holds the per-block counts); for callers that cannot allocate."""
    W = len(shard_start) - 1
    ss = (ctypes.c_int64 * len(shard_start))(*[int(x) for x in shard_start])
    _check("emb_route_ids_noalloc", lib().emb_route_ids_noalloc(
        ctypes.byref(tables.c()), ctypes.byref(batch.c()), W, ss, _ptr(send_counts), _ptr(send_ids), _ptr(send_pos),
        _ptr(send_bag), _stream(stream)))


ROUTE_SCRATCH_BYTES = 4 << 20


def workspace_error_offset() -> int:
    return int(lib().emb_workspace_error_offset())


def workspace_status(ws, status, stream=None) -> None:
    """Enqueue the write of the workspace's last-call status to ``status``
    (device int32 [4]): error bits, first timed-out wait's site, its
    workgroup, waits that ran out since the workspace was initialised."""
    _check("emb_workspace_status", lib().emb_workspace_status(_ptr(ws), ws.numel() * ws.element_size(),
                                                              _ptr(status), _stream(stream)))


def read_status(ws, stream=None):
    """The workspace's last-call status as host ints (synchronises)."""
    import torch
    st = torch.zeros(4, dtype=torch.int32, device=ws.device)
    workspace_status(ws, st, stream)
    return tuple(int(x) for x in st.cpu())


class Layer:
    """One GPU's shard of the layer with its buffers: forward, then the
    backward (dedup, segment-reduce, fused optimizer step) of the same batch.

    ``concurrent`` picks the schedule of a step.  False: forward, dedup and
    reduce one after another on the caller's stream.  True: the id dedup
    runs at the same time as the forward, which goes to a side stream after
    every earlier update on the caller's stream (the dedup reads only ids and
    offsets, never the table); the segment-reduce with the update waits for
    both.  The results are those of the serial order bit for bit.  "auto":
    concurrent for batches of at least AUTO_MIN_LOOKUPS lookups.  On MI355X
    the overlap pays for the large batches, whose sort is the look-back kind
    (26 tables x 8192 bags: 1101 us per step instead of 1160), but not for
    batches under about a million lookups, whose co-resident sort passes are
    latency-bound and slowed by the forward's traffic about as much as the
    overlap saves; each cross-stream wait also costs the host 15-25 us.

    ``step_stale`` is the asynchronous schedule with staleness one: the
    forward of the next batch reads the table before the current batch's
    update, as in the paper's asynchronous push-pull executor."""

    AUTO_MIN_LOOKUPS = 1_000_000

    def __init__(self, tables: Tables, pool: str, opt: str, lr: float, eps: float = 1e-8, state=None,
                 max_indices: int = 0, max_bags: int = 0, concurrent=False, rounding: str = "nearest",
                 seed: int = 0):
        import torch
        if concurrent not in (False, True, "auto"):
            raise ValueError("concurrent must be False, True or 'auto'")
        self.tables, self.pool, self.opt, self.lr, self.eps, self.state = tables, pool, opt, lr, eps, state
        dev = tables.weights.device
        n = max(1, max_indices)
        D = int(tables.weights.shape[1])
        wsb = workspace_size(n, max_bags, D)
        if wsb == 0:
            raise ValueError("batch too large for one call")
        self.ws = torch.empty(wsb, dtype=torch.uint8, device=dev)
        workspace_init(self.ws)
        i32 = dict(dtype=torch.int32, device=dev)
        self.unique_keys = torch.zeros(n, **i32)
        self.counts = torch.zeros(n, **i32)
        self.seg_offsets = torch.zeros(n + 1, **i32)
        self.sort_perm = torch.zeros(n, **i32)
        self.num_unique = torch.zeros(1, **i32)
        self._status = torch.zeros(4, **i32)
        self.max_indices = n
        self.concurrent = concurrent
        self._events = False
        if concurrent:
            self._side_stream = torch.cuda.Stream(device=dev)
            self._side = int(self._side_stream.cuda_stream)
            self._ev_ready = _Hip.event()
            self._ev_fwd = _Hip.event()
            self._events = True
        # argument values fixed for the layer's life, marshalled once
        self._ct = ctypes.byref(tables.c())
        # bf16 stochastic rounding draws fresh bits every step: seed, seed + 1, ...
        self.rounding, self.seed, self.steps_done = rounding, seed, 0
        self._updc = _update(opt, lr, eps, state, rounding, seed)
        self._upd = ctypes.byref(self._updc)
        self._dd = (_ptr(self.unique_keys), _ptr(self.counts), _ptr(self.seg_offsets), _ptr(self.sort_perm),
                    _ptr(self.num_unique), _ptr(self.ws), self.ws.numel() * self.ws.element_size())

    def __del__(self):
        if getattr(self, "_events", False):
            try:
                L = _Hip.lib()
                L.hipEventDestroy(self._ev_ready)
                L.hipEventDestroy(self._ev_fwd)
            except Exception:
                pass

    def status(self, stream=None):
        """Status of the last step (emb_workspace_status): (error bits,
        first timed-out wait's site, its workgroup, waits that ran out since
        the workspace was initialised); synchronises."""
        workspace_status(self.ws, self._status, stream)
        return tuple(int(x) for x in self._status.cpu())

    def check(self, stream=None) -> None:
        """Raise StepFailed if the last step failed on the device (it then
        wrote no table or state row)."""
        st = self.status(stream)
        if st[0]:
            raise StepFailed(*st)

    def forward(self, batch: Batch, out, stream=None) -> None:
        pool_fwd(self.tables, batch, self.pool, out, stream)

    def backward(self, batch: Batch, grad_out, grad_rows=None, stream=None) -> None:
        if int(batch.indices.numel()) > self.max_indices:
            raise ValueError("batch larger than the layer's buffers")
        unique_ids(self.tables, batch, self.unique_keys, self.counts, self.seg_offsets, self.sort_perm,
                   self.num_unique, self.ws, stream)
        grad_reduce(self.tables, batch, self.pool, grad_out, self.sort_perm, self.seg_offsets, self.unique_keys,
                    self.num_unique, self.ws, grad_rows=grad_rows, opt=self.opt, lr=self.lr, eps=self.eps,
                    state=self.state, stream=stream, rounding=self.rounding, seed=self.seed + self.steps_done)
        self.steps_done += 1

    def overlaps(self, num_indices: int) -> bool:
        """Whether a step of a batch of this many lookups runs concurrently."""
        if self.concurrent == "auto":
            return num_indices >= self.AUTO_MIN_LOOKUPS
        return bool(self.concurrent)

    def step(self, batch: Batch, out, grad_out, stream=None) -> None:
        """Forward of ``batch`` into ``out`` and its backward with ``grad_out``
        (fused optimizer step), enqueued on ``stream``; ``out`` is complete
        when ``stream`` reaches the end of the step."""
        self._enqueue(batch, out, batch, grad_out, stream)

    def step_stale(self, fwd_batch: Batch, out, bwd_batch: Batch, grad_out, stream=None) -> None:
        """One step of the asynchronous schedule with staleness one: the
        forward of ``fwd_batch`` (the next batch) into ``out`` reads the table
        as it is before the update of ``bwd_batch`` (the current batch, whose
        backward runs with ``grad_out``), i.e. it misses exactly that one
        update.  With a concurrent layer the forward overlaps the dedup."""
        self._enqueue(fwd_batch, out, bwd_batch, grad_out, stream)

    def _enqueue(self, fb: Batch, out, bb: Batch, grad_out, stream) -> None:
        n = int(bb.indices.numel())
        if n > self.max_indices:
            raise ValueError("batch larger than the layer's buffers")
        L = lib()
        main = _stream(stream)
        cf, cb = ctypes.byref(fb.c()), ctypes.byref(bb.c())
        uk, cnt, seg, perm, nu, ws, wsb = self._dd
        pool = POOL[self.pool]
        self._updc.seed = self.seed + self.steps_done
        self.steps_done += 1
        if not self.overlaps(max(n, int(fb.indices.numel()))):
            _check("emb_pool_fwd", L.emb_pool_fwd(self._ct, cf, pool, _ptr(out), main))
            _check("emb_unique_ids", L.emb_unique_ids(self._ct, cb, uk, cnt, seg, perm, nu, ws, wsb, main))
            _check("emb_grad_reduce", L.emb_grad_reduce(self._ct, cb, pool, _ptr(grad_out), perm, seg, uk, nu, None,
                                                        self._upd, ws, wsb, main))
            return
        # every earlier update on the caller's stream precedes this forward
        _Hip.record(self._ev_ready, main)
        _Hip.wait(self._side, self._ev_ready)
        _check("emb_pool_fwd", L.emb_pool_fwd(self._ct, cf, pool, _ptr(out), self._side))
        _Hip.record(self._ev_fwd, self._side)
        _check("emb_unique_ids", L.emb_unique_ids(self._ct, cb, uk, cnt, seg, perm, nu, ws, wsb, main))
        # the update must not overwrite rows before this forward has read them
        _Hip.wait(main, self._ev_fwd)
        _check("emb_grad_reduce", L.emb_grad_reduce(self._ct, cb, pool, _ptr(grad_out), perm, seg, uk, nu, None,
                                                    self._upd, ws, wsb, main))


class DedupBuffers:
    """Outputs and workspace of one emb_unique_ids call."""

    def __init__(self, device, max_indices: int, max_bags: int, dim: int):
        import torch
        n = max(1, max_indices)
        wsb = workspace_size(n, max_bags, dim)
        if wsb == 0:
            raise ValueError("batch too large for one call")
        self.ws = torch.empty(wsb, dtype=torch.uint8, device=device)
        workspace_init(self.ws)
        i32 = dict(dtype=torch.int32, device=device)
        self.unique_keys = torch.zeros(n, **i32)
        self.counts = torch.zeros(n, **i32)
        self.seg_offsets = torch.zeros(n + 1, **i32)
        self.sort_perm = torch.zeros(n, **i32)
        self.num_unique = torch.zeros(1, **i32)


class _Hip:
    """Direct HIP runtime calls for stream ordering (events), with cached
    handles: cheaper per call than the framework's wrappers."""
    _L = None

    @classmethod
    def lib(cls):
        if cls._L is None:
            L = ctypes.CDLL("libamdhip64.so")
            vp = ctypes.c_void_p
            L.hipEventCreateWithFlags.argtypes = [ctypes.POINTER(vp), ctypes.c_uint]
            L.hipEventCreateWithFlags.restype = ctypes.c_int
            L.hipEventDestroy.argtypes = [vp]
            L.hipEventDestroy.restype = ctypes.c_int
            L.hipEventRecord.argtypes = [vp, vp]
            L.hipEventRecord.restype = ctypes.c_int
            L.hipStreamWaitEvent.argtypes = [vp, vp, ctypes.c_uint]
            L.hipStreamWaitEvent.restype = ctypes.c_int
            cls._L = L
        return cls._L

    @classmethod
    def event(cls) -> int:
        ev = ctypes.c_void_p()
        rc = cls.lib().hipEventCreateWithFlags(ctypes.byref(ev), 0x2)  # hipEventDisableTiming
        if rc != 0:
            raise RuntimeError(f"hipEventCreateWithFlags: {rc}")
        return ev.value

    @classmethod
    def record(cls, ev: int, stream: int) -> None:
        rc = cls.lib().hipEventRecord(ev, stream)
        if rc != 0:
            raise RuntimeError(f"hipEventRecord: {rc}")

    @classmethod
    def wait(cls, stream: int, ev: int) -> None:
        rc = cls.lib().hipStreamWaitEvent(stream, ev, 0)
        if rc != 0:
            raise RuntimeError(f"hipStreamWaitEvent: {rc}")


def pipeline_group(max_indices: int) -> int:
    """Batches per group of the pipelined schedule for batches of up to
    ``max_indices`` ids: 8, whose one sort per group costs less per batch than
    a sort of 4 (MI355X, 20-step chains: c3 73.6 against 74.8 us per step, c2
    and c5 2-5 us less), or 4 when 8 batches would hold more than 2^25 ids
    (the 26-table bf16 workload, 5.5M ids a batch: 941 against 964 us)."""
    return 8 if 8 * max(1, int(max_indices)) <= (1 << 25) else 4


class Pipeline:
    """Training steps of the layer with the id dedups of the next group of
    batches running on side streams while the main stream runs the forward
    and the fused update of the current group.

    The dedup reads only a batch's ids and offsets, never the table, so
    running it ahead changes no result: every forward still follows the
    previous update on the main stream, and tables, state and pooled outputs
    equal those of serial steps bit for bit.  By default (``group_dedup``)
    the dedups of a group are one emb_unique_ids_batched call on one side
    stream: one sort of all the group's keys, each batch's share then split
    off into its own buffers (no workgroup waits for another; about 30 us of
    device time per c3 batch in a group of 8, 39 in a group of 4, against 55
    for emb_unique_ids alone).  The group's first forward runs before the
    wait for its dedups, which it does not read.  Without
    it, with one side stream the dedups run one after another with
    emb_unique_ids (whose sort may make the workgroups of a pass wait for one
    another, which is safe with one dedup in flight next to kernels that
    never wait); with several side streams the dedups of a group are dealt
    round-robin over them and run concurrently with
    emb_unique_ids_concurrent, in which no workgroup waits for another.
    ``depth`` sets of ``group`` dedup buffers rotate; the side streams
    overwrite a set only after the main stream's group that read it, so each
    group costs one cross-stream wait per stream and direction (each costs
    the host 15-25 us on ROCm while its event is pending, hence groups rather
    than single steps), and chained calls may look ahead up to ``depth - 1``
    groups.

    This is the paper's embedding stage run ahead of the dense stage
    (Section "Multi-mode Execution", heterogeneous pipeline) with no
    staleness: only the dedup, which the table never feeds, runs early."""

    def __init__(self, tables: Tables, pool: str, opt: str, lr: float, eps: float = 1e-8, state=None,
                 max_indices: int = 0, max_bags: int = 0, group: Optional[int] = None, side_streams: int = 3,
                 rounding: str = "nearest", seed: int = 0, group_dedup: bool = True, depth: int = 2):
        import torch
        if group is None:
            group = pipeline_group(max_indices)
        if group < 1 or not 1 <= side_streams <= 16 or not 2 <= depth <= 8:
            raise ValueError("group must be >= 1, side_streams in 1..16 and depth in 2..8")
        if group_dedup and group > 16:
            raise ValueError("a group dedup takes at most 16 batches")
        self.tables, self.pool, self.opt, self.lr, self.eps, self.state = tables, pool, opt, lr, eps, state
        dev = tables.weights.device
        D = int(tables.weights.shape[1])
        # group_dedup: each group's dedups are one emb_unique_ids_batched call
        # on one side stream, with a workspace of its own for a whole group
        self.K, self.S = group, 1 if group_dedup else min(side_streams, group)
        self.group_ws = None
        if group_dedup:
            gb = workspace_size(group * max(1, max_indices), group * max_bags, D)
            if gb == 0:
                raise ValueError("a group of batches too large for one dedup")
            self.group_ws = torch.empty(gb, dtype=torch.uint8, device=dev)
            workspace_init(self.group_ws)
        self.depth = depth
        self.sets = [DedupBuffers(dev, max_indices, max_bags, D) for _ in range(depth * group)]
        self.max_indices = max(1, max_indices)
        self._side_streams = [torch.cuda.Stream(device=dev) for _ in range(self.S)]
        self.sides = [int(x.cuda_stream) for x in self._side_streams]
        # events the native schedule records and waits on: the start, the main
        # stream's group done (per set parity), each side stream's group done
        # (per parity and stream)
        self._events = [_Hip.event() for _ in range(1 + depth + depth * self.S)]
        self._events_c = (ctypes.c_void_p * len(self._events))(*self._events)
        self._sides_c = (ctypes.c_void_p * self.S)(*self.sides)
        self._sets_c = (CDedupSet * len(self.sets))(*[
            CDedupSet(_ptr(b.unique_keys), _ptr(b.counts), _ptr(b.seg_offsets), _ptr(b.sort_perm),
                      _ptr(b.num_unique), _ptr(b.ws), b.ws.numel() * b.ws.element_size()) for b in self.sets])
        self._status = torch.zeros((len(self.sets), 4), dtype=torch.int32, device=dev)
        self._ct = ctypes.byref(tables.c())
        self.rounding, self.seed, self.steps_done = rounding, seed, 0
        self._updc = _update(opt, lr, eps, state, rounding, seed)
        self._pool = POOL[pool]
        # chained calls: groups numbered across calls, and the batches whose
        # dedups the last call enqueued for the next one
        self._group_base = 0
        self._primed = None

    def __del__(self):
        try:
            L = _Hip.lib()
            for e in self._events:
                L.hipEventDestroy(e)
        except Exception:
            pass

    def run(self, steps, stream=None, ahead=None) -> None:
        """Enqueue one training step per ``(batch, out, grad_out)`` of
        ``steps``, in order, on ``stream`` (the forward of each batch into its
        ``out``, then its backward with ``grad_out`` and the optimizer step),
        through one call of the native schedule (emb_pipeline_steps).  Every
        step's results are complete when ``stream`` reaches the end of the
        enqueued work; the side streams' work all precedes it.

        ``ahead``: the next call's first batches, ``A * group`` of them for
        A in 1..depth-1 (a training loop's look-ahead).  Their dedups are
        enqueued at the end of this call, beside its last groups' forwards and
        updates, and the next call, whose first steps must use exactly these
        batches (unchanged), starts with them done.  A call that starts with
        other batches raises; ``discard`` drops the look-ahead instead."""
        steps = list(steps)
        n = len(steps)
        n_ahead = 0
        if ahead is not None:
            ahead = list(ahead)
            n_ahead = len(ahead) // self.K
            if n == 0 or n_ahead < 1 or n_ahead >= self.depth or len(ahead) != n_ahead * self.K:
                raise ValueError(f"ahead takes the next call's first A * {self.K} batches, A in 1..{self.depth - 1}, "
                                 "after at least one step")
        if n == 0:
            return
        primed = 0
        if self._primed is not None:
            first = [b for b, _, _ in steps[:len(self._primed)]]
            if len(first) != len(self._primed) or any(x is not y for x, y in zip(first, self._primed)):
                raise ValueError("the first steps are not the batches deduplicated ahead by the last call "
                                 "(call discard() to drop them)")
            primed = len(self._primed) // self.K
        # the descriptors' bytes joined into one array (one copy)
        bl = [b for b, _, _ in steps] + (ahead if ahead else [])
        cbs = [b._c_bytes() for b in bl]
        if max(b._ckey[2] for b in bl) > self.max_indices:
            raise ValueError("batch larger than the pipeline's buffers")
        batches = (CBatch * len(cbs)).from_buffer_copy(b"".join(cbs))
        # pointer arrays built as 64-bit integers (0 for an absent tensor), the
        # output's address taken once while consecutive steps share it
        ol, gl = [], []
        last_o, last_p = None, 0
        for _, o, g in steps:
            if o is not last_o:
                last_o, last_p = o, (o.data_ptr() if o is not None else 0)
            ol.append(last_p)
            gl.append(g.data_ptr() if g is not None else 0)
        outs = (ctypes.c_void_p * n).from_buffer(array.array("Q", ol))
        grads = (ctypes.c_void_p * n).from_buffer(array.array("Q", gl))
        self._updc.seed = self.seed + self.steps_done
        gws = self.group_ws
        _check("emb_pipeline_steps", lib().emb_pipeline_steps(
            self._ct, self._pool, ctypes.byref(self._updc), n, batches, outs, grads, self.K, self._sets_c,
            _stream(stream), self.S, self._sides_c, self._events_c, _ptr(gws),
            gws.numel() if gws is not None else 0, self._group_base % self.depth, primed, n_ahead, self.depth))
        self.steps_done += n
        self._group_base += (n + self.K - 1) // self.K
        self._primed = ahead

    def discard(self) -> None:
        """Drop the look-ahead dedups of the last call: the next call starts
        with its own."""
        self._primed = None

    def status(self, stream=None):
        """Per buffer set, the status of its last step (emb_workspace_status);
        synchronises once: every set's status is written on the device, then
        copied back together."""
        import torch
        for i, b in enumerate(self.sets):
            workspace_status(b.ws, self._status[i], stream)
        torch.cuda.synchronize(self._status.device)
        return [tuple(int(x) for x in row) for row in self._status.cpu().tolist()]

    def check(self, stream=None) -> None:
        """Raise StepFailed if the last step of any buffer set failed on the
        device (that step wrote no table row)."""
        for st in self.status(stream):
            if st[0]:
                raise StepFailed(*st)
