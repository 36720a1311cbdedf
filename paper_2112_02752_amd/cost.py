"""Cost model of the embedding layer's step on MI355X.

The paper's planner chooses placements and parallel strategies with a cost
model whose per-operator costs come from a database of measured costs
(Section "Cost Model").  This is that entry for the sparse embedding layer:
each phase's time is predicted from the batch's sizes through the byte
models of the phases and a small set of coefficients fitted (non-negative
least squares) to measured phase times, `cost_table.json`.

  forward        t = a0 + a1 * N*rowbytes + a2 * U*rowbytes
  dedup          t = b0 + b1 * passes + b2 * N (co-resident sort) + b3 * N (reduce-then-scan sort)
  reduce+update  t = c0 + c1 * N*D*4 + c2 * U*(2*rowbytes + 2*statebytes)

N lookups, U distinct rows, rowbytes = D * (4 fp32 | 2 bf16), passes = the
number of 10-bit radix passes for the table's key width, statebytes = 0
(SGD), 4 (row-wise Adagrad) or 4*D (element-wise).  The co-resident sort
holds every tile of a pass on the device at once (up to about a million
keys); larger batches take the reduce-then-scan sort.  Host logic only: nothing
here runs on the device.
"""
from __future__ import annotations

import json
import math
import os
from dataclasses import dataclass
from typing import Dict, List, Optional, Sequence

import numpy as np

TABLE = os.path.join(os.path.dirname(os.path.abspath(__file__)), "cost_table.json")
PHASES = ("fwd", "dedup", "bwd_update")
# keys one pass of the co-resident sort holds at most (256 blocks of 4096 keys, minus its prefix blocks)
CORESIDENT_KEYS = 240 * 4096


@dataclass(frozen=True)
class StepShape:
    """What the model needs of a batch and its tables."""
    lookups: float      # N
    unique: float       # U
    rows: int           # R, all tables together
    dim: int            # D
    dtype: str = "fp32"
    opt: str = "adagrad"

    @property
    def rowbytes(self) -> int:
        return self.dim * (2 if self.dtype == "bf16" else 4)

    @property
    def statebytes(self) -> int:
        return {"sgd": 0, "adagrad": 4, "adagrad_ew": 4 * self.dim}[self.opt]

    @property
    def passes(self) -> int:
        bits = max(1, math.ceil(math.log2(max(self.rows, 2))))
        return (bits + 9) // 10


def features(s: StepShape) -> Dict[str, np.ndarray]:
    N, U = float(s.lookups), float(s.unique)
    co = N <= CORESIDENT_KEYS
    return {
        "fwd": np.array([1.0, N * s.rowbytes, U * s.rowbytes]),
        "dedup": np.array([1.0, float(s.passes), N if co else 0.0, 0.0 if co else N]),
        "bwd_update": np.array([1.0, N * s.dim * 4.0, U * (2.0 * s.rowbytes + 2.0 * s.statebytes)]),
    }


def shape_of(row: dict) -> StepShape:
    return StepShape(row["lookups"], row["unique"], row["rows"], row["dim"], row["dtype"], row["opt"])


def load_table(path: str = TABLE) -> List[dict]:
    with open(path) as f:
        return json.load(f)["rows"]


def _nnls(A: np.ndarray, b: np.ndarray) -> np.ndarray:
    """Non-negative least squares by the Lawson-Hanson active-set method."""
    n = A.shape[1]
    x = np.zeros(n)
    passive = np.zeros(n, bool)
    for _ in range(10 * n):
        w = A.T @ (b - A @ x)
        if passive.all() or (w[~passive] <= 1e-12 * max(1.0, np.abs(w).max())).all():
            break
        j = int(np.argmax(np.where(passive, -np.inf, w)))
        passive[j] = True
        while True:
            z = np.zeros(n)
            z[passive] = np.linalg.lstsq(A[:, passive], b, rcond=None)[0]
            if (z[passive] > 0).all():
                x = z
                break
            neg = passive & (z <= 0)
            alpha = np.min(x[neg] / (x[neg] - z[neg]))
            x = x + alpha * (z - x)
            passive &= x > 1e-15
    return x


@dataclass
class Model:
    coef: Dict[str, np.ndarray]
    scale: Dict[str, np.ndarray]

    def predict(self, s: StepShape) -> Dict[str, float]:
        f = features(s)
        out = {p: float(f[p] @ self.coef[p]) for p in PHASES}
        out["step"] = sum(out[p] for p in PHASES)
        return out


def fit(rows: Sequence[dict]) -> Model:
    """Fit each phase's coefficients to measured rows (relative residuals, so
    small and large batches weigh alike)."""
    coef, scale = {}, {}
    for p in PHASES:
        F = np.array([features(shape_of(r))[p] for r in rows])
        t = np.array([r[f"{p}_us"] for r in rows])
        sc = np.maximum(np.abs(F).max(axis=0), 1e-30)
        A = (F / sc) / t[:, None]
        x = _nnls(A, np.ones(len(rows)))
        coef[p] = x / sc
        scale[p] = sc
    return Model(coef, scale)


_model: Optional[Model] = None


def model() -> Model:
    """The model fitted to the committed measurements."""
    global _model
    if _model is None:
        _model = fit(load_table())
    return _model


def predict(lookups: float, unique: float, rows: int, dim: int, dtype: str = "fp32",
            opt: str = "adagrad") -> Dict[str, float]:
    """Predicted microseconds of each phase and of the step on one MI355X."""
    return model().predict(StepShape(lookups, unique, rows, dim, dtype, opt))


def leave_one_out(rows: Optional[Sequence[dict]] = None) -> List[dict]:
    """Each measured row predicted by a model fitted to the others."""
    rows = list(rows if rows is not None else load_table())
    out = []
    for i, r in enumerate(rows):
        m = fit(rows[:i] + rows[i + 1:])
        pr = m.predict(shape_of(r))
        meas = {p: r[f"{p}_us"] for p in PHASES}
        meas["step"] = sum(meas.values())
        out.append({"args": r["args"], "predicted": pr, "measured": meas,
                    "rel_err": {k: (pr[k] - meas[k]) / meas[k] for k in meas}})
    return out
