"""Seeded synthetic workloads for the sparse embedding layer.

Holds none of the layer's arithmetic: only the draws of table sizes, table
initial values, bag lengths, ids and upstream gradients (``synth.c``), a
device fill of table initial values with the same counter-based draw
(``synth_dev.hip``), and the five workload definitions below.  The HIP path's
tests and benchmark and the CPU oracle both take their inputs from here.

The workloads stand in for the Criteo click logs of the paper's CTR
experiments (Section "Heterogeneous Pipeline Asynchronous Execution"), whose
table shapes the paper does not give: ids are bounded-Zipf skewed, tables are
stacked table-major, bags are table-major.
"""
from __future__ import annotations

import ctypes
import math
import os
import subprocess
from dataclasses import dataclass, field, replace
from typing import List, Optional, Tuple

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_HOST_SO = os.path.join(_HERE, "libsynth.so")
_DEV_SO = os.path.join(_HERE, "libsynth_dev.so")

HIP_FLAGS = ["--offload-arch=gfx950", "-O3", "-fPIC", "-shared", "-std=c++17",
             "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops"]


def build(device: bool = True) -> None:
    """Compile the host generator (gcc) and, if asked, the device fill (hipcc)."""
    src = os.path.join(_HERE, "synth.c")
    subprocess.check_call(["gcc", "-O2", "-fPIC", "-shared", "-ffp-contract=off", "-std=c11",
                           src, "-o", _HOST_SO + ".tmp", "-lm"])
    os.replace(_HOST_SO + ".tmp", _HOST_SO)
    if device:
        dsrc = os.path.join(_HERE, "synth_dev.hip")
        subprocess.check_call(["hipcc", *HIP_FLAGS, dsrc, "-o", _DEV_SO + ".tmp"])
        os.replace(_DEV_SO + ".tmp", _DEV_SO)


_host = None
_dev = None


def _lib():
    global _host
    if _host is None:
        if not os.path.exists(_HOST_SO):
            build(device=False)
        L = ctypes.CDLL(_HOST_SO)
        u64, i64, i32, dbl, vp = ctypes.c_uint64, ctypes.c_int64, ctypes.c_int32, ctypes.c_double, ctypes.c_void_p
        L.synth_stream.restype = u64
        L.synth_stream.argtypes = [u64, u64, u64, u64]
        L.synth_hash.restype = u64
        L.synth_hash.argtypes = [u64, u64]
        L.synth_weights_f32.argtypes = [u64, u64, u64, i32, vp]
        L.synth_weights_bf16.argtypes = [u64, u64, u64, i32, vp]
        L.synth_weight_rows_f32.argtypes = [u64, vp, i64, i32, vp]
        L.synth_weight_rows_bf16.argtypes = [u64, vp, i64, i32, vp]
        L.synth_loguniform_rows.argtypes = [u64, i32, dbl, dbl, vp]
        L.synth_scramble_params.argtypes = [u64, i32, i64, vp, vp]
        L.synth_bag_lengths.argtypes = [u64, i64, i32, i32, i32, dbl, i64, vp]
        L.synth_ids.argtypes = [u64, i64, i32, i32, dbl, i64, i64, vp]
        L.synth_rank_to_row.restype = i64
        L.synth_rank_to_row.argtypes = [u64, i32, i64, i64]
        L.synth_normal_f32.argtypes = [u64, i64, i64, i64, vp]
        for f in ("synth_weights_f32", "synth_weights_bf16", "synth_weight_rows_f32", "synth_weight_rows_bf16",
                  "synth_loguniform_rows", "synth_scramble_params", "synth_bag_lengths", "synth_ids",
                  "synth_normal_f32"):
            getattr(L, f).restype = None
        _host = L
    return _host


def _devlib():
    global _dev
    if _dev is None:
        if not os.path.exists(_DEV_SO):
            raise RuntimeError(f"{_DEV_SO} is not built; run __graft_entry__.build()")
        L = ctypes.CDLL(_DEV_SO)
        L.synth_dev_fill_weights.restype = ctypes.c_int
        L.synth_dev_fill_weights.argtypes = [ctypes.c_void_p, ctypes.c_int32, ctypes.c_uint64, ctypes.c_uint64,
                                             ctypes.c_uint64, ctypes.c_int32, ctypes.c_void_p]
        L.synth_dev_zero_f32.restype = ctypes.c_int
        L.synth_dev_zero_f32.argtypes = [ctypes.c_void_p, ctypes.c_uint64, ctypes.c_void_p]
        _dev = L
    return _dev


def _ptr(a: np.ndarray) -> int:
    assert a.flags["C_CONTIGUOUS"]
    return a.ctypes.data


# ------------------------------------------------------------------ workloads

@dataclass(frozen=True)
class TableSpec:
    rows: int
    len_kind: int      # 0 uniform 1..lmax, 1 clamp(Poisson(lam), 1, lmax), 2 one-hot
    lmax: int
    lam: float
    id_dist: int       # 0 uniform, 1 bounded Zipf(s) + affine scramble
    zipf_s: float


@dataclass(frozen=True)
class Workload:
    name: str
    seed: int
    tables: Tuple[TableSpec, ...]
    dim: int
    dtype: str         # "fp32" | "bf16"
    bags_per_table: int
    pool: str          # "sum" | "mean"
    opt: str           # "sgd" | "adagrad"
    lr: float = 0.01
    eps: float = 1e-8
    steps: int = 1
    description: str = ""

    @property
    def num_tables(self) -> int:
        return len(self.tables)

    @property
    def rows(self) -> List[int]:
        return [t.rows for t in self.tables]

    @property
    def row_offset(self) -> np.ndarray:
        ro = np.zeros(self.num_tables + 1, dtype=np.int64)
        ro[1:] = np.cumsum(self.rows)
        return ro

    @property
    def total_rows(self) -> int:
        return int(sum(self.rows))

    @property
    def num_bags(self) -> int:
        return self.num_tables * self.bags_per_table

    @property
    def weight_bytes(self) -> int:
        return self.total_rows * self.dim * (4 if self.dtype == "fp32" else 2)

    @property
    def key_bits(self) -> int:
        return max(1, int(math.ceil(math.log2(max(2, self.total_rows)))))


def _seed(c: int) -> int:
    return 0x5EED0000 + c


def _c4_tables(seed: int) -> Tuple[TableSpec, ...]:
    rows = np.zeros(26, dtype=np.int64)
    _lib().synth_loguniform_rows(seed, 26, 1e3, 4e7, _ptr(rows))
    out = []
    for t in range(26):
        r = int(rows[t])
        one_hot = t < 13
        zipf = r >= 200_000
        out.append(TableSpec(rows=r, len_kind=2 if one_hot else 0, lmax=1 if one_hot else 100, lam=0.0,
                             id_dist=1 if zipf else 0, zipf_s=1.05 if zipf else 0.0))
    return tuple(out)


def workload(name: str) -> Workload:
    """The five synthetic workloads of the embedding layer (c1..c5)."""
    if name == "c1":
        return Workload("c1", _seed(1), (TableSpec(100_000, 0, 20, 0.0, 1, 1.05),), 16, "fp32", 512, "sum", "sgd",
                        description="1 table 100k x 16 fp32, 512 bags, L~U{1..20}, Zipf(1.05), sum, SGD")
    if name == "c2":
        return Workload("c2", _seed(2), tuple(TableSpec(1_000_000, 0, 50, 0.0, 1, 1.1) for _ in range(8)), 64,
                        "fp32", 4096, "mean", "adagrad",
                        description="8 tables 1M x 64 fp32, 4096 bags/table, L~U{1..50}, Zipf(1.1), mean, "
                                    "row-wise Adagrad")
    if name == "c3":
        return Workload("c3", _seed(3), (TableSpec(50_000_000, 1, 200, 30.0, 1, 1.2),), 64, "fp32", 16384, "sum",
                        "adagrad",
                        description="1 table 50M x 64 fp32 (12.8 GB), 16384 bags, L=clamp(Poisson(30),1,200), "
                                    "Zipf(1.2), sum, row-wise Adagrad")
    if name == "c4":
        s = _seed(4)
        return Workload("c4", s, _c4_tables(s), 128, "bf16", 8192, "sum", "adagrad",
                        description="26 tables log-uniform 1e3..4e7 rows x 128 bf16, 8192 bags/table, half one-hot, "
                                    "half L~U{1..100}, uniform ids below 2e5 rows else Zipf(1.05), sum, "
                                    "row-wise Adagrad")
    if name == "c5":
        return Workload("c5", _seed(5), (TableSpec(200_000_000, 0, 100, 0.0, 1, 0.9),), 64, "fp32", 65536, "sum",
                        "sgd", steps=100,
                        description="1 table 200M x 64 fp32 (51.2 GB), 65536 bags, L~U{1..100}, Zipf(0.9), sum, "
                                    "SGD, 100 steps")
    raise KeyError(name)


WORKLOADS = ("c1", "c2", "c3", "c4", "c5")


def scaled(w: Workload, rows_div: int = 1, bags_div: int = 1, name: Optional[str] = None) -> Workload:
    """A smaller workload of the same shape family (rows and bags divided)."""
    tabs = tuple(replace(t, rows=max(1, t.rows // rows_div)) for t in w.tables)
    return replace(w, name=name or f"{w.name}/r{rows_div}b{bags_div}", tables=tabs,
                   bags_per_table=max(1, w.bags_per_table // bags_div))


# -------------------------------------------------------------------- batches

@dataclass
class Batch:
    offsets: np.ndarray   # int32 [M+1]
    indices: np.ndarray   # int32 [N], table-local ids
    grad: np.ndarray      # float32 [M][D], upstream gradient of the pooled output

    @property
    def num_indices(self) -> int:
        return int(self.indices.shape[0])


def bag_lengths(w: Workload, step: int) -> np.ndarray:
    L = _lib()
    out = np.zeros(w.num_bags, dtype=np.int32)
    B = w.bags_per_table
    for t, ts in enumerate(w.tables):
        part = np.zeros(B, dtype=np.int32)
        L.synth_bag_lengths(w.seed, step, t, ts.len_kind, ts.lmax, ts.lam, B, _ptr(part))
        out[t * B:(t + 1) * B] = part
    return out


def make_batch(w: Workload, step: int = 0, with_grad: bool = True) -> Batch:
    L = _lib()
    lens = bag_lengths(w, step)
    offsets = np.zeros(w.num_bags + 1, dtype=np.int32)
    np.cumsum(lens, out=offsets[1:])
    B = w.bags_per_table
    idx = np.zeros(int(offsets[-1]), dtype=np.int32)
    for t, ts in enumerate(w.tables):
        lo, hi = int(offsets[t * B]), int(offsets[(t + 1) * B])
        part = np.zeros(hi - lo, dtype=np.int32)
        L.synth_ids(w.seed, step, t, ts.id_dist, ts.zipf_s, ts.rows, hi - lo, _ptr(part))
        idx[lo:hi] = part
    grad = make_grad(w, step) if with_grad else np.zeros((0, w.dim), np.float32)
    return Batch(offsets, idx, grad)


def make_grad(w: Workload, step: int = 0) -> np.ndarray:
    g = np.zeros((w.num_bags, w.dim), dtype=np.float32)
    _lib().synth_normal_f32(w.seed, step, 0, g.size, _ptr(g))
    return g


def weight_rows(w: Workload, rows: np.ndarray) -> np.ndarray:
    """Initial values of the given global rows: fp32 [n][D] or bf16 bits uint16 [n][D]."""
    rows = np.ascontiguousarray(rows, dtype=np.uint32)
    n = rows.shape[0]
    if w.dtype == "fp32":
        out = np.zeros((n, w.dim), dtype=np.float32)
        _lib().synth_weight_rows_f32(w.seed, _ptr(rows), n, w.dim, _ptr(out))
    else:
        out = np.zeros((n, w.dim), dtype=np.uint16)
        _lib().synth_weight_rows_bf16(w.seed, _ptr(rows), n, w.dim, _ptr(out))
    return out


def dense_weights(w: Workload) -> np.ndarray:
    """The whole initial table (small workloads only)."""
    if w.dtype == "fp32":
        out = np.zeros((w.total_rows, w.dim), dtype=np.float32)
        _lib().synth_weights_f32(w.seed, 0, w.total_rows, w.dim, _ptr(out))
    else:
        out = np.zeros((w.total_rows, w.dim), dtype=np.uint16)
        _lib().synth_weights_bf16(w.seed, 0, w.total_rows, w.dim, _ptr(out))
    return out


def fill_device_weights(w: Workload, dev_ptr: int, stream: int = 0, row0: int = 0,
                        rows: Optional[int] = None) -> None:
    """Fill a device table with the workload's initial values (device draw)."""
    rows = w.total_rows - row0 if rows is None else rows
    rc = _devlib().synth_dev_fill_weights(ctypes.c_void_p(dev_ptr), 0 if w.dtype == "fp32" else 1, w.seed, row0,
                                          rows, w.dim, ctypes.c_void_p(stream))
    if rc != 0:
        raise RuntimeError(f"synth_dev_fill_weights failed: hipError {rc}")


def zero_device_f32(dev_ptr: int, n: int, stream: int = 0) -> None:
    rc = _devlib().synth_dev_zero_f32(ctypes.c_void_p(dev_ptr), n, ctypes.c_void_p(stream))
    if rc != 0:
        raise RuntimeError(f"synth_dev_zero_f32 failed: hipError {rc}")


def rank_to_row(w: Workload, table: int, rank1: int) -> int:
    return int(_lib().synth_rank_to_row(w.seed, table, w.tables[table].rows, rank1))


def bf16_bits_to_f32(b: np.ndarray) -> np.ndarray:
    return (b.astype(np.uint32) << 16).view(np.float32)
