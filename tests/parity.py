"""Shared helpers of the GPU parity tests: run one step of the layer through
the HIP library (C ABI via the binding) and through the CPU oracle on the
same seeded inputs, and compare.

Comparison rule (row-wise infinity-norm relative error, integer outputs
bit-exact):
  rel = max over rows of  max_d |x - y| / max_d |y|
fp32 results must meet rel <= 1e-5; bf16 table rows rel <= 1e-2 (one bf16
ulp is 2^-8 of the value); row-wise Adagrad state elementwise rel <= 1e-5,
element-wise Adagrad state rows by the row-norm rule.
"""
from __future__ import annotations

from dataclasses import dataclass, field
from typing import Dict, List, Optional

import numpy as np

import oracle
import synth
import paper_2112_02752_amd as emb

TOL_FP32 = 1e-5
TOL_BF16_ROWS = 1e-2


def rel_rownorm(x: np.ndarray, y: np.ndarray) -> float:
    x = np.asarray(x, dtype=np.float64)
    y = np.asarray(y, dtype=np.float64)
    assert x.shape == y.shape, (x.shape, y.shape)
    if x.size == 0:
        return 0.0
    x = x.reshape(len(x), -1)
    y = y.reshape(len(y), -1)
    den = np.maximum(np.abs(y).max(axis=1), 1e-30)
    return float((np.abs(x - y).max(axis=1) / den).max())


def as_f32(vals: np.ndarray) -> np.ndarray:
    return synth.bf16_bits_to_f32(vals) if vals.dtype == np.uint16 else vals


# --------------------------------------------------------------- device side

def torch_mod():
    import torch
    return torch


@dataclass
class DeviceLayer:
    """Device tables + optimizer state + the layer's buffers."""
    row_offset: List[int]
    D: int
    dtype: str
    W: object
    state: Optional[object]
    layer: Optional[emb.Layer] = None

    @property
    def tables(self) -> emb.Tables:
        return emb.Tables(self.W, self.row_offset)

    def rows(self, keys: np.ndarray) -> np.ndarray:
        torch = torch_mod()
        k = torch.from_numpy(np.asarray(keys, dtype=np.int64)).to(self.W.device)
        r = self.W.index_select(0, k)
        if self.dtype == "bf16":
            return r.view(torch.int16).cpu().numpy().view(np.uint16)
        return r.cpu().numpy()

    def state_rows(self, keys: np.ndarray) -> np.ndarray:
        torch = torch_mod()
        k = torch.from_numpy(np.asarray(keys, dtype=np.int64)).to(self.state.device)
        return self.state.index_select(0, k).cpu().numpy()


def device_layer_from_workload(w: synth.Workload, device="cuda", h0: float = 0.0) -> DeviceLayer:
    """Device table of a workload; Adagrad state filled with h0 ([R] row-wise,
    [R][D] element-wise)."""
    torch = torch_mod()
    tdt = torch.float32 if w.dtype == "fp32" else torch.bfloat16
    W = torch.empty((w.total_rows, w.dim), dtype=tdt, device=device)
    synth.fill_device_weights(w, W.data_ptr(), int(torch.cuda.current_stream().cuda_stream))
    state = None
    if w.opt == "adagrad":
        state = torch.full((w.total_rows,), h0, dtype=torch.float32, device=device)
    elif w.opt == "adagrad_ew":
        state = torch.full((w.total_rows, w.dim), h0, dtype=torch.float32, device=device)
    return DeviceLayer([int(x) for x in w.row_offset], w.dim, w.dtype, W, state)


def device_layer_from_host(row_offset, W_host: np.ndarray, state_host: Optional[np.ndarray], device="cuda"):
    torch = torch_mod()
    if W_host.dtype == np.uint16:
        W = torch.from_numpy(W_host.view(np.int16).copy()).to(device).view(torch.bfloat16)
        dt = "bf16"
    else:
        W = torch.from_numpy(W_host.copy()).to(device)
        dt = "fp32"
    st = torch.from_numpy(state_host.copy()).to(device) if state_host is not None else None
    return DeviceLayer([int(x) for x in row_offset], int(W_host.shape[1]), dt, W, st)


@dataclass
class StepResult:
    out: np.ndarray
    num_unique: int
    unique_keys: np.ndarray
    counts: np.ndarray
    seg_offsets: np.ndarray
    perm: np.ndarray
    grad_rows: Optional[np.ndarray]
    ws_error: int = 0


def gpu_step(dl: DeviceLayer, offsets: np.ndarray, indices: np.ndarray, grad: np.ndarray, B: int, pool: str,
             opt: str, lr: float, eps: float, fused: bool = True, want_grad_rows: bool = True,
             layer: Optional[emb.Layer] = None, idx64: bool = False, rounding: str = "nearest",
             seed: int = 0) -> StepResult:
    """One step (fwd on pre-update rows, dedup, reduce, optimizer) on the GPU.
    A layer built with concurrent=True runs the step through Layer.step (the
    forward on a side stream alongside the dedup; no unfused gradient rows)."""
    torch = torch_mod()
    dev = dl.W.device
    N = int(indices.shape[0])
    M = int(offsets.shape[0]) - 1
    off = torch.from_numpy(offsets.astype(np.int32)).to(dev)
    idx = torch.from_numpy(indices.astype(np.int64 if idx64 else np.int32)).to(dev)
    G = torch.from_numpy(np.ascontiguousarray(grad, dtype=np.float32)).to(dev)
    if layer is None:
        layer = emb.Layer(dl.tables, pool, opt, lr, eps, dl.state, max_indices=N, max_bags=M, concurrent=False)
    b = emb.Batch(off, idx, B)
    out = torch.empty((M, dl.D), dtype=torch.float32, device=dev)
    if layer.concurrent:
        assert fused
        grad_rows = None
        layer.step(b, out, G)
    else:
        grad_rows = _serial_step(dl, b, out, G, N, pool, opt, lr, eps, fused, want_grad_rows, layer, rounding, seed)
    torch.cuda.synchronize()
    U = int(layer.num_unique.cpu().item())
    ws_err = layer.status()[0]
    return StepResult(
        out=out.cpu().numpy(), num_unique=U,
        unique_keys=layer.unique_keys[:U].cpu().numpy().view(np.uint32),
        counts=layer.counts[:U].cpu().numpy(), seg_offsets=layer.seg_offsets[:U + 1].cpu().numpy(),
        perm=layer.sort_perm[:N].cpu().numpy(),
        grad_rows=grad_rows[:U].cpu().numpy() if grad_rows is not None else None, ws_error=ws_err)


def _serial_step(dl, b, out, G, N, pool, opt, lr, eps, fused, want_grad_rows, layer, rounding="nearest", seed=0):
    torch = torch_mod()
    dev = dl.W.device
    emb.pool_fwd(dl.tables, b, pool, out)
    emb.unique_ids(dl.tables, b, layer.unique_keys, layer.counts, layer.seg_offsets, layer.sort_perm,
                   layer.num_unique, layer.ws)
    grad_rows = torch.empty((max(N, 1), dl.D), dtype=torch.float32, device=dev) if want_grad_rows else None
    if fused:
        emb.grad_reduce(dl.tables, b, pool, G, layer.sort_perm, layer.seg_offsets, layer.unique_keys,
                        layer.num_unique, layer.ws, grad_rows=grad_rows, opt=opt, lr=lr, eps=eps, state=dl.state,
                        rounding=rounding, seed=seed)
    else:
        emb.grad_reduce(dl.tables, b, pool, G, layer.sort_perm, layer.seg_offsets, layer.unique_keys,
                        layer.num_unique, layer.ws, grad_rows=grad_rows)
        emb.sparse_update(dl.tables, opt, lr, eps, dl.state, layer.unique_keys, layer.num_unique, N, grad_rows,
                          rounding=rounding, seed=seed)
    return grad_rows


# --------------------------------------------------------------- oracle side

def global_keys(row_offset, B: int, offsets: np.ndarray, indices: np.ndarray) -> np.ndarray:
    M = len(offsets) - 1
    bag = np.repeat(np.arange(M), np.diff(offsets))
    return (np.asarray(row_offset, dtype=np.int64)[bag // B] + indices).astype(np.uint32)


def check_against_oracle(g: StepResult, o_out, o_dd: oracle.Dedup, o_gr, tol_out=TOL_FP32):
    """Integer outputs bit-exact, floats within tolerance."""
    assert g.ws_error == 0, f"the step failed on the device: error bits {g.ws_error}"
    r = rel_rownorm(g.out, o_out)
    assert r <= tol_out, f"forward rel err {r}"
    assert g.num_unique == o_dd.num_unique, (g.num_unique, o_dd.num_unique)
    np.testing.assert_array_equal(g.unique_keys, o_dd.unique_keys)
    np.testing.assert_array_equal(g.counts, o_dd.counts)
    np.testing.assert_array_equal(g.seg_offsets, o_dd.seg_offsets)
    np.testing.assert_array_equal(g.perm, o_dd.perm)
    if g.grad_rows is not None:
        r = rel_rownorm(g.grad_rows, o_gr)
        assert r <= TOL_FP32, f"grad_rows rel err {r}"


def check_sr_agreement(dl: DeviceLayer, store: oracle.RowStore, keys: np.ndarray, min_frac: float = 0.999):
    """Stochastically rounded bf16 rows: the device and the oracle draw the
    same bits for every element, so they store the same value except where
    their fp32 results (summed in different orders) straddle the random
    threshold, which happens for a tiny fraction of the elements."""
    slots = np.searchsorted(store.keys, keys) if store.keys is not None else keys.astype(np.int64)
    same = np.mean(dl.rows(keys) == store.vals[slots])
    assert same >= min_frac, f"only {same:.5f} of the stochastically rounded elements agree"


def check_rows(dl: DeviceLayer, store: oracle.RowStore, keys: np.ndarray, opt: str):
    """Updated rows (and Adagrad state) of `keys` on the device vs the oracle's store."""
    slots = np.searchsorted(store.keys, keys) if store.keys is not None else keys.astype(np.int64)
    dev_rows = dl.rows(keys)
    ref = store.vals[slots]
    tol = TOL_BF16_ROWS if dl.dtype == "bf16" else TOL_FP32
    r = rel_rownorm(as_f32(dev_rows), as_f32(ref))
    assert r <= tol, f"updated rows rel err {r}"
    if opt == "adagrad":
        h_dev = dl.state_rows(keys).astype(np.float64)
        h_ref = store.state[slots].astype(np.float64)
        rel = np.abs(h_dev - h_ref) / np.maximum(np.abs(h_ref), 1e-30)
        assert rel.max() <= TOL_FP32, f"adagrad state rel err {rel.max()}"
    elif opt == "adagrad_ew":
        r = rel_rownorm(dl.state_rows(keys), store.state[slots])
        assert r <= TOL_FP32, f"element-wise adagrad state rel err {r}"


def check_untouched(dl: DeviceLayer, w: synth.Workload, touched: np.ndarray, n: int = 10_000, seed: int = 0):
    """A seeded sample of rows no step touched, plus the last row, still hold their initial values."""
    rng = np.random.default_rng(seed)
    cand = np.unique(np.concatenate([rng.integers(0, w.total_rows, size=n), [w.total_rows - 1]]))
    cand = np.setdiff1d(cand, touched).astype(np.uint32)
    if cand.size == 0:
        return
    np.testing.assert_array_equal(dl.rows(cand), synth.weight_rows(w, cand))


def run_workload(w: synth.Workload, steps: int = 1, fused: bool = True, device="cuda", concurrent: bool = False,
                 h0: float = 0.0, idx64: bool = False, rounding: str = "nearest", seed: int = 0):
    """Full-size parity of `steps` consecutive steps of a workload (serial
    calls, or Layer.step's concurrent schedule); Adagrad state starts at h0."""
    dl = device_layer_from_workload(w, device, h0)
    batches = [synth.make_batch(w, s) for s in range(steps)]
    keys_all = [global_keys(w.row_offset, w.bags_per_table, b.offsets, b.indices) for b in batches]
    touched = np.unique(np.concatenate(keys_all)) if keys_all else np.zeros(0, np.uint32)
    state = None
    if w.opt == "adagrad":
        state = np.full(len(touched), h0, np.float32)
    elif w.opt == "adagrad_ew":
        state = np.full((len(touched), w.dim), h0, np.float32)
    store = oracle.RowStore(synth.weight_rows(w, touched), keys=touched.astype(np.uint32), state=state)
    nmax = max(len(b.indices) for b in batches)
    layer = emb.Layer(dl.tables, w.pool, w.opt, w.lr, w.eps, dl.state, max_indices=nmax, max_bags=w.num_bags,
                      concurrent=concurrent, rounding=rounding, seed=seed)
    for s, b in enumerate(batches):
        g = gpu_step(dl, b.offsets, b.indices, b.grad, w.bags_per_table, w.pool, w.opt, w.lr, w.eps, fused=fused,
                     layer=layer, idx64=idx64, rounding=rounding, seed=seed + s)
        o_out, o_dd, o_gr = oracle.step(w.num_tables, w.row_offset, w.bags_per_table, b.offsets, b.indices, b.grad,
                                        store, w.pool, w.opt, w.lr, w.eps, rounding, seed + s)
        check_against_oracle(g, o_out, o_dd, o_gr)
        check_rows(dl, store, o_dd.unique_keys, w.opt)
        if rounding == "stochastic" and w.dtype == "bf16":
            check_sr_agreement(dl, store, o_dd.unique_keys)
            # the few elements whose fp32 results straddled the random
            # threshold hold neighbouring bf16 values on the two sides; the
            # next step starts both from the device's rows
            slots = np.searchsorted(store.keys, o_dd.unique_keys)
            store.vals[slots] = dl.rows(o_dd.unique_keys)
    check_untouched(dl, w, touched)
    return dl, store


def run_case(row_offset, W_host: np.ndarray, offsets, indices, grad, B: int, pool: str, opt: str, lr: float,
             eps: float, state0=None, fused=True, device="cuda", exact=False, idx64=False, rounding="nearest",
             seed=0):
    """Parity of one step on explicit host inputs (dense tables)."""
    offsets = np.ascontiguousarray(offsets, dtype=np.int32)
    indices = np.ascontiguousarray(indices, dtype=np.int32)
    grad = np.ascontiguousarray(grad, dtype=np.float32)
    ro = np.asarray(row_offset, dtype=np.int64)
    if opt == "adagrad" and state0 is None:
        state0 = np.zeros(W_host.shape[0], np.float32)
    if opt == "adagrad_ew" and state0 is None:
        state0 = np.zeros(W_host.shape, np.float32)
    dl = device_layer_from_host(ro, W_host, state0 if opt != "sgd" else None, device)
    store = oracle.RowStore(W_host.copy(), state=state0.copy() if state0 is not None else None)
    g = gpu_step(dl, offsets, indices, grad, B, pool, opt, lr, eps, fused=fused, idx64=idx64, rounding=rounding,
                 seed=seed)
    o_out, o_dd, o_gr = oracle.step(len(ro) - 1, ro, B, offsets, indices, grad, store, pool, opt, lr, eps, rounding,
                                    seed)
    check_against_oracle(g, o_out, o_dd, o_gr)
    check_rows(dl, store, o_dd.unique_keys, opt)
    if rounding == "stochastic" and W_host.dtype == np.uint16:
        check_sr_agreement(dl, store, o_dd.unique_keys)
    if exact:
        np.testing.assert_array_equal(g.out, o_out)
        np.testing.assert_array_equal(g.grad_rows, o_gr)
        np.testing.assert_array_equal(dl.rows(o_dd.unique_keys), store.vals[o_dd.unique_keys])
    # rows outside the batch are untouched
    untouched = np.setdiff1d(np.arange(W_host.shape[0]), o_dd.unique_keys)
    if untouched.size:
        sample = untouched[:: max(1, untouched.size // 5000)]
        np.testing.assert_array_equal(dl.rows(sample), W_host[sample])
    return g, store, dl
