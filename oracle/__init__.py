"""ORACLE -- test infrastructure only.

Python wrapper over ``oracle.c``: a plain CPU statement of one step of the
pooled sparse embedding layer (forward, dedup, gradient reduce, optimizer
step), accumulated in double; its bag and segment loops may run on several
threads with results that do not depend on the thread count.  Only ``tests/``, the smoke
check and the benchmark's CPU-baseline leg may import this package; the
product library never does.  It shares no code with the HIP path.

The paper (Introduction; Section "Multi-mode Execution") names the layer and
its data-access cost but states none of its arithmetic; the definitions used
are the plain ones written at the top of ``oracle.c``.
"""
from __future__ import annotations

import ctypes
import os
import subprocess
from dataclasses import dataclass
from typing import Optional

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SO = os.path.join(_HERE, "liboracle.so")

POOL = {"sum": 0, "mean": 1}
OPT = {"sgd": 0, "adagrad": 1, "adagrad_ew": 2}
DTYPE = {"fp32": 0, "bf16": 1}


def build() -> None:
    src = os.path.join(_HERE, "oracle.c")
    subprocess.check_call(["gcc", "-O2", "-fPIC", "-shared", "-fopenmp", "-ffp-contract=off", "-std=c11",
                           src, "-o", _SO + ".tmp", "-lm"])
    os.replace(_SO + ".tmp", _SO)


_L = None


def _lib():
    global _L
    if _L is None:
        if not os.path.exists(_SO):
            build()
        L = ctypes.CDLL(_SO)
        i32, i64, vp, f32 = ctypes.c_int32, ctypes.c_int64, ctypes.c_void_p, ctypes.c_float
        L.oracle_pool_fwd.restype = ctypes.c_int
        L.oracle_pool_fwd.argtypes = [i32, vp, i32, vp, vp, i32, i32, i64, vp, vp, i32, vp]
        L.oracle_unique_ids.restype = ctypes.c_int
        L.oracle_unique_ids.argtypes = [i32, vp, i32, vp, vp, vp, vp, vp, vp, vp]
        L.oracle_grad_reduce.restype = ctypes.c_int
        L.oracle_grad_reduce.argtypes = [i32, i32, vp, i32, i32, vp, vp, vp, i32, vp, vp]
        L.oracle_route_ids.restype = ctypes.c_int
        L.oracle_route_ids.argtypes = [i32, vp, i32, vp, vp, i32, vp, vp, vp, vp, vp]
        L.oracle_sparse_update.restype = ctypes.c_int
        L.oracle_sparse_update.argtypes = [i32, f32, f32, i32, i32, i64, vp, vp, vp, vp, i32, vp, i32,
                                           ctypes.c_uint64]
        L.oracle_sr_bits.restype = ctypes.c_uint32
        L.oracle_sr_bits.argtypes = [ctypes.c_uint64, ctypes.c_uint64]
        L.oracle_bf16_stochastic.restype = ctypes.c_uint16
        L.oracle_bf16_stochastic.argtypes = [f32, ctypes.c_uint32]
        L.oracle_set_threads.restype = None
        L.oracle_set_threads.argtypes = [i32]
        L.oracle_get_threads.restype = i32
        L.oracle_get_threads.argtypes = []
        _L = L
    return _L


def set_threads(n: int) -> None:
    """Threads of the oracle's parallel loops (n < 1: one per processor).
    Results do not depend on it: every output is computed by one thread."""
    _lib().oracle_set_threads(int(n))


def get_threads() -> int:
    return int(_lib().oracle_get_threads())


class OracleError(RuntimeError):
    pass


def _p(a: Optional[np.ndarray]):
    if a is None:
        return None
    assert a.flags["C_CONTIGUOUS"], "oracle inputs must be C-contiguous"
    return a.ctypes.data


def _check(rc: int, what: str) -> None:
    if rc != 0:
        raise OracleError(f"{what}: error {rc}")


@dataclass
class RowStore:
    """Table rows held by the oracle: dense (keys None, row r at slot r) or the
    listed global rows (sorted uint32 keys) with their values."""
    vals: np.ndarray                  # float32 [n][D] or uint16 bf16 bits [n][D]
    keys: Optional[np.ndarray] = None  # uint32 [n] sorted, or None
    state: Optional[np.ndarray] = None  # float32 [n] row-wise or [n][D] element-wise Adagrad accumulators

    @property
    def dtype(self) -> int:
        return 0 if self.vals.dtype == np.float32 else 1

    @property
    def n(self) -> int:
        return int(self.vals.shape[0])


def pool_fwd(num_tables: int, row_offset: np.ndarray, bags_per_table: int, offsets: np.ndarray,
             indices: np.ndarray, store: RowStore, pool: str) -> np.ndarray:
    D = store.vals.shape[1]
    M = num_tables * bags_per_table
    out = np.zeros((M, D), dtype=np.float32)
    rc = _lib().oracle_pool_fwd(num_tables, _p(row_offset), bags_per_table, _p(offsets), _p(indices), D,
                                store.dtype, store.n, _p(store.keys), _p(store.vals), POOL[pool], _p(out))
    _check(rc, "oracle_pool_fwd")
    return out


@dataclass
class Dedup:
    unique_keys: np.ndarray  # uint32 [U]
    counts: np.ndarray       # int32 [U]
    seg_offsets: np.ndarray  # int32 [U+1]
    perm: np.ndarray         # int32 [N]

    @property
    def num_unique(self) -> int:
        return int(self.unique_keys.shape[0])


def unique_ids(num_tables: int, row_offset: np.ndarray, bags_per_table: int, offsets: np.ndarray,
               indices: np.ndarray) -> Dedup:
    N = int(indices.shape[0])
    uk = np.zeros(max(N, 1), dtype=np.uint32)
    cnt = np.zeros(max(N, 1), dtype=np.int32)
    seg = np.zeros(N + 1, dtype=np.int32)
    perm = np.zeros(max(N, 1), dtype=np.int32)
    nu = np.zeros(1, dtype=np.int32)
    rc = _lib().oracle_unique_ids(num_tables, _p(row_offset), bags_per_table, _p(offsets), _p(indices), _p(uk),
                                  _p(cnt), _p(seg), _p(perm), _p(nu))
    _check(rc, "oracle_unique_ids")
    U = int(nu[0])
    return Dedup(uk[:U].copy(), cnt[:U].copy(), seg[:U + 1].copy(), perm[:N].copy())


def grad_reduce(num_tables: int, bags_per_table: int, offsets: np.ndarray, grad: np.ndarray, pool: str,
                dedup: Dedup):
    """Returns (grad_rows float32 [U][D], acc float64 [U][D])."""
    D = grad.shape[1]
    U = dedup.num_unique
    gr = np.zeros((max(U, 1), D), dtype=np.float32)
    acc = np.zeros((max(U, 1), D), dtype=np.float64)
    rc = _lib().oracle_grad_reduce(num_tables, bags_per_table, _p(offsets), D, POOL[pool], _p(grad),
                                   _p(dedup.perm), _p(dedup.seg_offsets), U, _p(gr), _p(acc))
    _check(rc, "oracle_grad_reduce")
    return gr[:U], acc[:U]


ROUNDING = {"nearest": 0, "stochastic": 1}


def sr_bits(seed: int, counter: int) -> int:
    """The 16 random bits of stochastic rounding for element counter row * D + column."""
    return int(_lib().oracle_sr_bits(seed, counter))


def bf16_stochastic(x: float, r16: int) -> int:
    """Stochastic rounding of an fp32 value to bf16 bits with 16 random bits."""
    return int(_lib().oracle_bf16_stochastic(x, r16))


def sparse_update(store: RowStore, unique_keys: np.ndarray, grad: np.ndarray, opt: str, lr: float,
                  eps: float, rounding: str = "nearest", seed: int = 0) -> None:
    """In-place optimizer step on ``store`` (grad: float64 [U][D] or float32, widened)."""
    D = store.vals.shape[1]
    g = np.ascontiguousarray(grad, dtype=np.float64)
    uk = np.ascontiguousarray(unique_keys, dtype=np.uint32)
    if OPT[opt] == 1 and store.state is None:
        store.state = np.zeros(store.n, dtype=np.float32)
    if OPT[opt] == 2 and store.state is None:
        store.state = np.zeros((store.n, D), dtype=np.float32)
    if OPT[opt] == 2:
        assert store.state.shape == (store.n, D) and store.state.flags["C_CONTIGUOUS"]
    rc = _lib().oracle_sparse_update(OPT[opt], lr, eps, D, store.dtype, store.n, _p(store.keys), _p(store.vals),
                                     _p(store.state), _p(uk), int(uk.shape[0]), _p(g), ROUNDING[rounding], seed)
    _check(rc, "oracle_sparse_update")


@dataclass
class Route:
    send_counts: np.ndarray  # int32 [W]
    send_ids: np.ndarray     # int32 [N], local row ids in send order
    send_pos: np.ndarray     # int32 [N], position of each sent id
    send_bag: np.ndarray     # int32 [N], bag of each sent id


def route_ids(num_tables: int, row_offset: np.ndarray, bags_per_table: int, offsets: np.ndarray,
              indices: np.ndarray, shard_start: np.ndarray) -> Route:
    """Ids of a batch bucketed by the owner rank of a row-range sharding
    (rank r owns global rows [shard_start[r], shard_start[r+1]))."""
    N = int(indices.shape[0])
    W = int(len(shard_start)) - 1
    ss = np.ascontiguousarray(shard_start, dtype=np.int64)
    cnt = np.zeros(max(W, 1), np.int32)
    ids, pos, bag = (np.zeros(max(N, 1), np.int32) for _ in range(3))
    rc = _lib().oracle_route_ids(num_tables, _p(row_offset), bags_per_table, _p(offsets), _p(indices), W, _p(ss),
                                 _p(cnt), _p(ids), _p(pos), _p(bag))
    _check(rc, "oracle_route_ids")
    return Route(cnt[:W].copy(), ids[:N].copy(), pos[:N].copy(), bag[:N].copy())


def step(num_tables: int, row_offset: np.ndarray, bags_per_table: int, offsets: np.ndarray, indices: np.ndarray,
         grad: np.ndarray, store: RowStore, pool: str, opt: str, lr: float, eps: float, rounding: str = "nearest",
         seed: int = 0):
    """One whole step in the layer's order: forward on the pre-update rows,
    dedup, gradient reduce, optimizer step (in place on ``store``).
    Returns (out, dedup, grad_rows)."""
    out = pool_fwd(num_tables, row_offset, bags_per_table, offsets, indices, store, pool)
    dd = unique_ids(num_tables, row_offset, bags_per_table, offsets, indices)
    gr, acc = grad_reduce(num_tables, bags_per_table, offsets, grad, pool, dd)
    sparse_update(store, dd.unique_keys, acc, opt, lr, eps, rounding, seed)
    return out, dd, gr
