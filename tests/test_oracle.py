"""Pins of the CPU oracle against things other than itself.

The paper states no formula or value for the embedding layer, so the pins
are: hand-worked examples (tests/golden), brute force with an explicit dense
bag-incidence matrix, dyadic inputs where every order of summation is exact,
closed forms of the two optimizers, library routines (numpy sort/unique,
torch CPU embedding_bag), and invariants (gradient mass, untouched rows).
"""
import json
import os

import numpy as np
import pytest

import oracle
from oracle import RowStore

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _golden(name):
    with open(os.path.join(GOLDEN, name)) as f:
        return json.load(f)


def _arr(x, dt):
    return np.ascontiguousarray(np.array(x, dtype=dt))


# ------------------------------------------------------------------ helpers

def random_case(rng, T=3, rows=(7, 5, 11), D=4, B=6, lmax=9, empty_frac=0.2, dyadic=True):
    row_offset = np.zeros(T + 1, np.int64)
    row_offset[1:] = np.cumsum(rows[:T])
    M = T * B
    lens = rng.integers(1, lmax + 1, size=M).astype(np.int32)
    lens[rng.random(M) < empty_frac] = 0
    offsets = np.zeros(M + 1, np.int32)
    offsets[1:] = np.cumsum(lens)
    idx = np.zeros(offsets[-1], np.int32)
    for m in range(M):
        t = m // B
        idx[offsets[m]:offsets[m + 1]] = rng.integers(0, rows[t], size=lens[m])
    R = int(row_offset[-1])
    if dyadic:  # small integers times 2^-4: all sums exact in fp32 and fp64
        W = (rng.integers(-64, 64, size=(R, D)) / 16.0).astype(np.float32)
        G = (rng.integers(-64, 64, size=(M, D)) / 16.0).astype(np.float32)
    else:
        W = rng.uniform(-1, 1, size=(R, D)).astype(np.float32)
        G = rng.standard_normal(size=(M, D)).astype(np.float32)
    return row_offset, B, offsets, idx, W, G


def incidence(row_offset, B, offsets, idx, pool):
    """Dense A[m][r] = scale_m * multiplicity, built with plain Python loops."""
    M = len(offsets) - 1
    R = int(row_offset[-1])
    A = np.zeros((M, R), np.float64)
    for m in range(M):
        t = m // B
        L = offsets[m + 1] - offsets[m]
        for j in range(offsets[m], offsets[m + 1]):
            A[m, row_offset[t] + idx[j]] += (1.0 / L) if pool == "mean" else 1.0
    return A


def keys_of(row_offset, B, offsets, idx):
    M = len(offsets) - 1
    bag = np.repeat(np.arange(M), np.diff(offsets))
    return (row_offset[bag // B] + idx).astype(np.uint32)


# ------------------------------------------------------------------ golden

@pytest.mark.parametrize("name", ["tiny_sum_step.json", "tiny_mean_step.json"])
def test_golden_forward_dedup_grad(name):
    g = _golden(name)
    T, B = g["num_tables"], g["bags_per_table"]
    ro = _arr(g["row_offset"], np.int64)
    off = _arr(g["offsets"], np.int32)
    idx = _arr(g["indices"], np.int32)
    W = _arr(g["weights"], np.float32)
    G = _arr(g["grad"], np.float32)
    out = oracle.pool_fwd(T, ro, B, off, idx, RowStore(W.copy()), g["pool"])
    np.testing.assert_array_equal(out, _arr(g["expect_out"], np.float32))
    dd = oracle.unique_ids(T, ro, B, off, idx)
    np.testing.assert_array_equal(dd.unique_keys, g["expect_unique_keys"])
    np.testing.assert_array_equal(dd.counts, g["expect_counts"])
    np.testing.assert_array_equal(dd.seg_offsets, g["expect_seg_offsets"])
    np.testing.assert_array_equal(dd.perm, g["expect_perm"])
    gr, acc = oracle.grad_reduce(T, B, off, G, g["pool"], dd)
    np.testing.assert_array_equal(gr, _arr(g["expect_grad_rows"], np.float32))
    np.testing.assert_array_equal(acc, _arr(g["expect_grad_rows"], np.float64))


@pytest.mark.parametrize("name", ["tiny_sum_step.json", "tiny_mean_step.json"])
def test_golden_sgd(name):
    g = _golden(name)
    T, B = g["num_tables"], g["bags_per_table"]
    ro, off, idx = _arr(g["row_offset"], np.int64), _arr(g["offsets"], np.int32), _arr(g["indices"], np.int32)
    st = RowStore(_arr(g["weights"], np.float32))
    oracle.step(T, ro, B, off, idx, _arr(g["grad"], np.float32), st, g["pool"], "sgd", g["sgd"]["lr"], 0.0)
    np.testing.assert_array_equal(st.vals, _arr(g["sgd"]["expect_weights"], np.float32))


def test_golden_adagrad():
    g = _golden("tiny_sum_step.json")
    T, B = g["num_tables"], g["bags_per_table"]
    ro, off, idx = _arr(g["row_offset"], np.int64), _arr(g["offsets"], np.int32), _arr(g["indices"], np.int32)
    st = RowStore(_arr(g["weights"], np.float32), state=np.zeros(5, np.float32))
    a = g["adagrad"]
    oracle.step(T, ro, B, off, idx, _arr(g["grad"], np.float32), st, "sum", "adagrad", a["lr"], a["eps"])
    np.testing.assert_array_equal(st.vals, _arr(a["expect_weights"], np.float32))
    np.testing.assert_array_equal(st.state, _arr(a["expect_state"], np.float32))


# ------------------------------------------------------ brute force (dense A)

@pytest.mark.parametrize("pool", ["sum", "mean"])
@pytest.mark.parametrize("seed", [0, 1, 2])
def test_forward_and_grad_equal_dense_incidence(pool, seed):
    rng = np.random.default_rng(seed)
    ro, B, off, idx, W, G = random_case(rng, dyadic=False)
    T = len(ro) - 1
    A = incidence(ro, B, off, idx, pool)
    out = oracle.pool_fwd(T, ro, B, off, idx, RowStore(W.copy()), pool)
    ref = (A @ W.astype(np.float64))
    np.testing.assert_allclose(out, ref, rtol=1e-6, atol=1e-7)
    dd = oracle.unique_ids(T, ro, B, off, idx)
    gr, acc = oracle.grad_reduce(T, B, off, G, pool, dd)
    dense_grad = A.T @ G.astype(np.float64)
    np.testing.assert_allclose(acc, dense_grad[dd.unique_keys], rtol=1e-12, atol=1e-12)
    # rows outside the unique set have zero gradient
    untouched = np.setdiff1d(np.arange(A.shape[1]), dd.unique_keys)
    assert np.all(dense_grad[untouched] == 0.0)
    assert np.all(A[:, untouched] == 0.0)


@pytest.mark.parametrize("pool", ["sum", "mean"])
def test_dyadic_forward_is_exact(pool):
    rng = np.random.default_rng(7)
    ro, B, off, idx, W, G = random_case(rng, dyadic=True, lmax=8)
    if pool == "mean":  # L in {1, 2, 4, 8} keeps 1/L dyadic
        lens = np.diff(off)
        lens = np.where(lens == 0, 0, 2 ** np.floor(np.log2(np.maximum(lens, 1)))).astype(np.int32)
        off = np.zeros_like(off)
        off[1:] = np.cumsum(lens)
        idx = idx[:off[-1]].copy()
        M = len(off) - 1
        for m in range(M):
            t = m // B
            idx[off[m]:off[m + 1]] %= (ro[t + 1] - ro[t])
    T = len(ro) - 1
    A = incidence(ro, B, off, idx, pool)
    out = oracle.pool_fwd(T, ro, B, off, idx, RowStore(W.copy()), pool)
    np.testing.assert_array_equal(out, (A @ W.astype(np.float64)).astype(np.float32))
    dd = oracle.unique_ids(T, ro, B, off, idx)
    gr, _ = oracle.grad_reduce(T, B, off, G, pool, dd)
    np.testing.assert_array_equal(gr, (A.T @ G.astype(np.float64))[dd.unique_keys].astype(np.float32))


@pytest.mark.parametrize("opt", ["sgd", "adagrad", "adagrad_ew"])
def test_sparse_step_equals_dense_step(opt):
    """A dense optimizer step over every row changes exactly the touched rows,
    by the same amounts as the sparse step."""
    rng = np.random.default_rng(11)
    ro, B, off, idx, W, G = random_case(rng, dyadic=False)
    T = len(ro) - 1
    R = W.shape[0]
    lr, eps = np.float32(0.05), np.float32(1e-8)
    state0 = rng.uniform(0, 2, size=(R, W.shape[1]) if opt == "adagrad_ew" else R).astype(np.float32)
    st = RowStore(W.copy(), state=state0.copy())
    oracle.step(T, ro, B, off, idx, G, st, "sum", opt, float(lr), float(eps))
    A = incidence(ro, B, off, idx, "sum")
    g = A.T @ G.astype(np.float64)  # dense gradient, every row
    W64 = W.astype(np.float64)
    if opt == "sgd":
        W_dense = W64 - np.float64(lr) * g
        h = state0.astype(np.float64)
    elif opt == "adagrad_ew":
        h = state0.astype(np.float64) + g * g
        W_dense = W64 - np.float64(lr) * g / (np.sqrt(h) + np.float64(eps))
    else:
        h = state0.astype(np.float64) + (g * g).sum(1) / W.shape[1]
        W_dense = W64 - np.float64(lr) * g / (np.sqrt(h)[:, None] + np.float64(eps))
    touched = np.unique(keys_of(ro, B, off, idx))
    untouched = np.setdiff1d(np.arange(R), touched)
    np.testing.assert_array_equal(st.vals[untouched], W[untouched])
    np.testing.assert_array_equal(st.state[untouched], state0[untouched])
    np.testing.assert_allclose(st.vals[touched], W_dense[touched], rtol=1e-6, atol=1e-7)
    if opt != "sgd":
        np.testing.assert_allclose(st.state[touched], h[touched], rtol=1e-6)


# ---------------------------------------------------------- special cases

def test_one_hot_bags_reproduce_rows_exactly():
    rng = np.random.default_rng(3)
    R, D, T, B = 50, 8, 2, 40
    ro = np.array([0, 20, 50], np.int64)
    W = rng.standard_normal((R, D)).astype(np.float32)
    off = np.arange(T * B + 1, dtype=np.int32)
    idx = np.concatenate([rng.integers(0, 20, B), rng.integers(0, 30, B)]).astype(np.int32)
    keys = keys_of(ro, B, off, idx)
    for pool in ("sum", "mean"):
        out = oracle.pool_fwd(T, ro, B, off, idx, RowStore(W.copy()), pool)
        np.testing.assert_array_equal(out, W[keys])


def test_empty_bags_give_zero_and_no_gradient():
    ro = np.array([0, 4], np.int64)
    W = np.arange(12, dtype=np.float32).reshape(4, 3) + 1
    off = np.array([0, 0, 2, 2, 2], np.int32)
    idx = np.array([1, 3], np.int32)
    G = np.full((4, 3), 1000.0, np.float32)
    G[1] = [1, 2, 3]
    out = oracle.pool_fwd(1, ro, 4, off, idx, RowStore(W.copy()), "sum")
    np.testing.assert_array_equal(out[[0, 2, 3]], 0)
    np.testing.assert_array_equal(out[1], W[1] + W[3])
    dd = oracle.unique_ids(1, ro, 4, off, idx)
    gr, _ = oracle.grad_reduce(1, 4, off, G, "sum", dd)
    np.testing.assert_array_equal(gr, [[1, 2, 3], [1, 2, 3]])


def test_all_empty_batch():
    ro = np.array([0, 4], np.int64)
    off = np.zeros(5, np.int32)
    idx = np.zeros(0, np.int32)
    out = oracle.pool_fwd(1, ro, 4, off, idx, RowStore(np.ones((4, 2), np.float32)), "mean")
    assert np.all(out == 0)
    dd = oracle.unique_ids(1, ro, 4, off, idx)
    assert dd.num_unique == 0 and list(dd.seg_offsets) == [0]


@pytest.mark.parametrize("seed", [0, 5])
def test_dedup_matches_numpy(seed):
    rng = np.random.default_rng(seed)
    ro, B, off, idx, W, G = random_case(rng, rows=(3, 1000, 2), lmax=30)
    T = len(ro) - 1
    dd = oracle.unique_ids(T, ro, B, off, idx)
    keys = keys_of(ro, B, off, idx)
    u, c = np.unique(keys, return_counts=True)
    np.testing.assert_array_equal(dd.unique_keys, u)
    np.testing.assert_array_equal(dd.counts, c)
    np.testing.assert_array_equal(dd.perm, np.argsort(keys, kind="stable"))
    np.testing.assert_array_equal(dd.seg_offsets, np.concatenate([[0], np.cumsum(c)]))
    assert dd.counts.sum() == len(idx)
    assert np.all(np.diff(dd.unique_keys.astype(np.int64)) > 0)


def test_dedup_key_boundaries():
    """ids 0 and rows-1 of every table, global keys above 2^31, N = 1."""
    big = 2 ** 31 - 1                      # rows of table 2: the largest int32 id is big - 1
    ro = np.array([0, 1, 4, 4 + big], np.int64)
    B = 2
    off = np.array([0, 3, 3, 5, 7, 8, 10], np.int32)
    idx = np.array([0, 0, 0, 2, 0, 2, 0, big - 1, 0, big - 1], np.int32)
    dd = oracle.unique_ids(3, ro, B, off, idx)
    keys = keys_of(ro, B, off, idx)
    assert keys.max() == 4 + big - 1 and keys.max() > 2 ** 31
    np.testing.assert_array_equal(dd.perm, np.argsort(keys, kind="stable"))
    np.testing.assert_array_equal(dd.unique_keys, np.unique(keys))
    one = oracle.unique_ids(1, np.array([0, 10], np.int64), 1, np.array([0, 1], np.int32),
                            np.array([9], np.int32))
    assert list(one.unique_keys) == [9] and list(one.perm) == [0] and list(one.seg_offsets) == [0, 1]


@pytest.mark.parametrize("pool", ["sum", "mean"])
def test_gradient_mass_invariant(pool):
    """sum_u grad_rows[u] = sum_m L_m * scale_m * G[m] (= sum_m G[m] over nonempty bags for mean)."""
    rng = np.random.default_rng(9)
    ro, B, off, idx, W, G = random_case(rng, dyadic=False, lmax=25)
    T = len(ro) - 1
    dd = oracle.unique_ids(T, ro, B, off, idx)
    _, acc = oracle.grad_reduce(T, B, off, G, pool, dd)
    L = np.diff(off).astype(np.float64)
    w = (L > 0).astype(np.float64) if pool == "mean" else L
    np.testing.assert_allclose(acc.sum(0), (w[:, None] * G.astype(np.float64)).sum(0), rtol=1e-12, atol=1e-10)


# ----------------------------------------------------------- closed forms

def test_sgd_closed_form():
    ro = np.array([0, 3], np.int64)
    W = np.array([[1.0, -2.0], [0.5, 0.25], [3.0, 3.0]], np.float32)
    st = RowStore(W.copy())
    g = np.array([[2.0, -4.0]])
    oracle.sparse_update(st, np.array([1], np.uint32), g, "sgd", 0.125, 0.0)
    np.testing.assert_array_equal(st.vals, [[1.0, -2.0], [0.25, 0.75], [3.0, 3.0]])


@pytest.mark.parametrize("c", [0.75, -3.0, 1e-3])
def test_rowwise_adagrad_closed_form_constant_row(c):
    """From zero state with g = c everywhere: h = c^2, W' = W - lr c / (|c| + eps)."""
    D = 16
    W = np.linspace(-1, 1, D, dtype=np.float32)[None, :]
    st = RowStore(W.copy(), state=np.zeros(1, np.float32))
    lr, eps = np.float32(0.01), np.float32(1e-8)
    oracle.sparse_update(st, np.array([0], np.uint32), np.full((1, D), c), "adagrad", float(lr), float(eps))
    h = c * c
    assert st.state[0] == np.float32(h)
    expect = (W.astype(np.float64) - np.float64(lr) * c / (abs(c) + np.float64(eps))).astype(np.float32)
    np.testing.assert_array_equal(st.vals, expect)


def test_adagrad_accumulates_across_steps():
    st = RowStore(np.zeros((1, 4), np.float32), state=np.zeros(1, np.float32))
    g = np.array([[1.0, 1.0, 1.0, 1.0]])
    oracle.sparse_update(st, np.array([0], np.uint32), g, "adagrad", 1.0, 0.0)
    oracle.sparse_update(st, np.array([0], np.uint32), g * 3, "adagrad", 1.0, 0.0)
    # h: 1 then 1 + 9 = 10; W: -1 then -1 - 3/sqrt(10)
    assert st.state[0] == np.float32(10.0)
    np.testing.assert_allclose(st.vals[0], -1 - 3 / np.sqrt(10.0), rtol=1e-7)


def test_bf16_store_rounds_once_to_nearest_even():
    # bf16 row 1.0; SGD with g chosen so the fp32 result sits between bf16 neighbours
    one = np.array([[0x3F80, 0x3F80]], np.uint16)  # 1.0, 1.0
    st = RowStore(one.copy())
    # 1 - 2^-9 is the midpoint of bf16 {1 - 2^-8, 1}: ties to even -> 1.0 (mantissa even)
    # 1 - 3*2^-10 is below the midpoint -> 1 - 2^-8 = 0x3F7F
    g = np.array([[2.0 ** -9, 3 * 2.0 ** -10]])
    oracle.sparse_update(st, np.array([0], np.uint32), g, "sgd", 1.0, 0.0)
    assert list(st.vals[0]) == [0x3F80, 0x3F7F]


# ------------------------------------------------- library cross-check (torch)

@pytest.mark.parametrize("pool", ["sum", "mean"])
def test_forward_and_grad_match_torch_embedding_bag(pool):
    torch = pytest.importorskip("torch")
    rng = np.random.default_rng(21)
    ro, B, off, idx, W, G = random_case(rng, T=1, rows=(37,), D=8, B=30, dyadic=False)
    Wt = torch.tensor(W.astype(np.float64), requires_grad=True)
    out_t = torch.nn.functional.embedding_bag(torch.tensor(idx.astype(np.int64)), Wt,
                                              torch.tensor(off[:-1].astype(np.int64)), mode=pool)
    out_t.backward(torch.tensor(G.astype(np.float64)))
    out = oracle.pool_fwd(1, ro, B, off, idx, RowStore(W.copy()), pool)
    np.testing.assert_allclose(out, out_t.detach().numpy(), rtol=1e-6, atol=1e-7)
    dd = oracle.unique_ids(1, ro, B, off, idx)
    _, acc = oracle.grad_reduce(1, B, off, G, pool, dd)
    np.testing.assert_allclose(acc, Wt.grad.numpy()[dd.unique_keys], rtol=1e-12, atol=1e-12)


@pytest.mark.parametrize("pool,h0", [("sum", 0.0), ("mean", 0.0), ("sum", 0.5)])
def test_elementwise_adagrad_matches_torch_optim(pool, h0):
    """Three steps of element-wise Adagrad against torch.optim.Adagrad (its
    update with lr_decay = weight_decay = 0 is the textbook one: eps outside the
    square root) on a dense float64 table whose gradient comes from torch's
    own embedding_bag backward; each step's batch is a fresh one."""
    torch = pytest.importorskip("torch")
    rng = np.random.default_rng(31)
    rows, D, B = 41, 8, 25
    ro = np.array([0, rows], np.int64)
    W0 = rng.uniform(-1, 1, size=(rows, D)).astype(np.float32)
    Wt = torch.tensor(W0.astype(np.float64), requires_grad=True)
    opt_t = torch.optim.Adagrad([Wt], lr=0.05, eps=1e-8, initial_accumulator_value=h0)
    st = RowStore(W0.copy(), state=np.full((rows, D), h0, np.float32))
    touched = set()
    for s in range(3):
        _, _, off, idx, _, G = random_case(rng, T=1, rows=(rows,), D=D, B=B, dyadic=False)
        touched |= set(int(k) for k in idx)
        oracle.step(1, ro, B, off, idx, G, st, pool, "adagrad_ew", 0.05, 1e-8)
        opt_t.zero_grad()
        out_t = torch.nn.functional.embedding_bag(torch.tensor(idx.astype(np.int64)), Wt,
                                                  torch.tensor(off[:-1].astype(np.int64)), mode=pool)
        out_t.backward(torch.tensor(G.astype(np.float64)))
        opt_t.step()
    # the oracle rounds W and h to fp32 after every step, torch keeps float64
    np.testing.assert_allclose(st.vals, Wt.detach().numpy(), rtol=1e-5, atol=1e-6)
    h_t = opt_t.state[Wt]["sum"].numpy()
    np.testing.assert_allclose(st.state, h_t, rtol=1e-5, atol=1e-6)
    untouched = sorted(set(range(rows)) - touched)
    np.testing.assert_array_equal(st.vals[untouched], W0[untouched])


# ------------------------------------------------------------ routing

def _shards(rng, R, W):
    """Row-range boundaries [W+1] over R rows, some ranges empty."""
    cuts = np.sort(rng.integers(0, R + 1, size=W - 1))
    return np.concatenate([[0], cuts, [R]]).astype(np.int64)


@pytest.mark.parametrize("W,seed", [(1, 0), (4, 1), (8, 2), (13, 3)])
def test_route_matches_numpy(W, seed):
    """Owners by np.searchsorted, the send order by a stable argsort of the
    owners, counts by np.bincount."""
    rng = np.random.default_rng(seed)
    ro, B, off, idx, _, _ = random_case(rng, dyadic=False)
    T = len(ro) - 1
    ss = _shards(rng, int(ro[-1]), W)
    r = oracle.route_ids(T, ro, B, off, idx, ss)
    key = keys_of(ro, B, off, idx).astype(np.int64)
    owner = np.searchsorted(ss, key, side="right") - 1
    order = np.argsort(owner, kind="stable")
    bag = np.repeat(np.arange(len(off) - 1), np.diff(off))
    np.testing.assert_array_equal(r.send_counts, np.bincount(owner, minlength=W))
    np.testing.assert_array_equal(r.send_pos, order)
    np.testing.assert_array_equal(r.send_ids, key[order] - ss[owner[order]])
    np.testing.assert_array_equal(r.send_bag, bag[order])


@pytest.mark.parametrize("pool,tablewise", [("sum", False), ("mean", False), ("sum", True)])
def test_route_fragments_reassemble_the_forward(pool, tablewise):
    """Every owner pools its fragments (runs of equal bag in its send range)
    from its own slice of the table; adding the fragments' rows by bag (then
    dividing by the bag length for mean pooling) gives the single-device
    forward exactly (dyadic inputs)."""
    rng = np.random.default_rng(5)
    ro, B, off, idx, W, _ = random_case(rng, T=3, rows=(40, 25, 60), D=4, B=12, lmax=9, empty_frac=0.2)
    T = len(ro) - 1
    M = len(off) - 1
    ss = ro.copy() if tablewise else _shards(rng, int(ro[-1]), 5)
    r = oracle.route_ids(T, ro, B, off, idx, ss)
    full = oracle.pool_fwd(T, ro, B, off, idx, RowStore(W.copy()), pool)
    acc = np.zeros((M, W.shape[1]), np.float64)
    k0 = 0
    for rank in range(len(ss) - 1):
        k1 = k0 + int(r.send_counts[rank])
        bags = r.send_bag[k0:k1]
        heads = np.concatenate([[True], bags[1:] != bags[:-1]]) if k1 > k0 else np.zeros(0, bool)
        frag_off = np.concatenate([np.nonzero(heads)[0], [k1 - k0]]).astype(np.int32)
        local = W[ss[rank]:ss[rank + 1]].copy()
        if len(frag_off) > 1:
            part = oracle.pool_fwd(1, np.array([0, local.shape[0]], np.int64), len(frag_off) - 1, frag_off,
                                   np.ascontiguousarray(r.send_ids[k0:k1]), RowStore(local), "sum")
            for f in range(len(frag_off) - 1):
                acc[bags[frag_off[f]]] += part[f]
        k0 = k1
    if pool == "mean":
        L = np.diff(off)
        acc[L > 0] /= L[L > 0, None]
    np.testing.assert_array_equal(acc.astype(np.float32), full)


def test_route_rejects_bad_shards():
    ro = np.array([0, 10], np.int64)
    off = np.array([0, 1], np.int32)
    idx = np.array([3], np.int32)
    for bad in ([0, 9], [1, 10], [0, 6, 4, 10]):
        with pytest.raises(oracle.OracleError):
            oracle.route_ids(1, ro, 1, off, idx, np.array(bad, np.int64))


# ------------------------------------------------- bf16 stochastic rounding

def test_sr_bits_match_the_input_generators_splitmix64():
    """The oracle's random bits are the top 16 bits of the counter hash the
    seeded input generator implements separately (splitmix64 of the seed xor
    splitmix64 of the counter)."""
    import synth
    L = synth._lib()
    for seed in (0, 1, 0x5EED0004, 2 ** 63 + 12345):
        for c in (0, 1, 63, 64, 10 ** 9, 2 ** 40 + 7):
            assert oracle.sr_bits(seed, c) == int(L.synth_hash(seed, c)) >> 48, (seed, c)


# splitmix64 (Steele, Lea and Flood 2014) started from state 0: its first
# four outputs, the published reference sequence (each output mixes the state
# after adding the golden-ratio increment 0x9e3779b97f4a7c15)
SPLITMIX64_SEED0 = (0xE220A8397B1DCDAF, 0x6E789E6AA1B965F4, 0x06C45D188009454F, 0xF88BB8A8724C81EC)
SPLITMIX_INCREMENT = 0x9E3779B97F4A7C15


def test_sr_bits_known_answers_of_splitmix64():
    """Pins the oracle's random bits to the published splitmix64 outputs:
    sr_bits(seed, c) is the top 16 bits of splitmix64's output for state
    seed ^ (its output for state c).  With c = 0 the inner output is the
    first published value; a seed of that value xor i * increment makes the
    outer state i * increment, whose output is the (i+1)-th published value."""
    inner = SPLITMIX64_SEED0[0]   # the output for state 0
    for i, expect in enumerate(SPLITMIX64_SEED0):
        seed = inner ^ ((i * SPLITMIX_INCREMENT) % 2 ** 64)
        assert oracle.sr_bits(seed, 0) == expect >> 48, (i, hex(expect))


def test_input_generator_hash_known_answers_of_splitmix64():
    """The input generator's counter hash pins to the same published outputs
    (synth_hash(seed, c) = splitmix64 output for state seed ^ output for state c)."""
    import synth
    L = synth._lib()
    inner = SPLITMIX64_SEED0[0]
    for i, expect in enumerate(SPLITMIX64_SEED0):
        assert int(L.synth_hash(inner ^ ((i * SPLITMIX_INCREMENT) % 2 ** 64), 0)) == expect, i


def _bf16_neighbours(x: np.float32):
    u = int(np.array([x], np.float32).view(np.uint32)[0])
    down = u >> 16
    return down, down + (1 if (u & 0xFFFF) else 0)


def test_bf16_stochastic_rounding_is_exactly_unbiased_over_all_random_bits():
    """Over all 2^16 values of the random bits, rounding up happens for
    exactly (dropped bits) of them, so the mean of the rounded values is the
    fp32 value exactly; every result is one of its two bf16 neighbours, and a
    value bf16 holds exactly never moves."""
    rng = np.random.default_rng(8)
    xs = np.concatenate([rng.uniform(-2, 2, 6), rng.standard_normal(3) * 1e-3, [1.5, -0.25, 3.0]]).astype(np.float32)
    for x in xs:
        down, up = _bf16_neighbours(x)
        outs = np.array([oracle.bf16_stochastic(float(x), r) for r in range(1 << 16)], np.uint32)
        assert set(np.unique(outs)) <= {down, up}
        vals = (outs << 16).view(np.float32).astype(np.float64)
        assert vals.mean() == np.float64(x), (x, vals.mean())


def test_stochastic_step_rounds_to_a_neighbour_with_the_elements_bits():
    """A bf16 step with stochastic rounding stores, for every element, one of
    the two bf16 neighbours of the fp32 result the nearest-even step would
    round, and it depends on the seed."""
    rng = np.random.default_rng(12)
    ro, B, off, idx, Wf, G = random_case(rng, T=2, rows=(30, 20), D=8, B=10, dyadic=False)
    T = len(ro) - 1
    Wb = ((Wf.view(np.uint32).astype(np.uint64) + 0x7FFF + ((Wf.view(np.uint32) >> 16) & 1)) >> 16).astype(np.uint16)
    ref = RowStore(Wf.copy())  # fp32 table with the same starting values
    ref.vals[:] = (Wb.astype(np.uint32) << 16).view(np.float32)
    oracle.step(T, ro, B, off, idx, G, ref, "sum", "sgd", 0.5, 0.0)
    stores = []
    for seed in (1, 2):
        st = RowStore(Wb.copy())
        oracle.step(T, ro, B, off, idx, G, st, "sum", "sgd", 0.5, 0.0, rounding="stochastic", seed=seed)
        stores.append(st.vals.copy())
        for r in np.unique(keys_of(ro, B, off, idx)):
            for d in range(8):
                down, up = _bf16_neighbours(ref.vals[r, d])
                assert int(st.vals[r, d]) in (down, up)
    assert (stores[0] != stores[1]).any()


# ------------------------------------------------------------ sparse store

def test_sparse_row_store_equals_dense():
    rng = np.random.default_rng(4)
    ro, B, off, idx, W, G = random_case(rng, dyadic=False)
    T = len(ro) - 1
    dense = RowStore(W.copy(), state=np.zeros(W.shape[0], np.float32))
    keys = np.unique(keys_of(ro, B, off, idx))
    sparse = RowStore(W[keys].copy(), keys=keys.astype(np.uint32), state=np.zeros(len(keys), np.float32))
    o1, _, g1 = oracle.step(T, ro, B, off, idx, G, dense, "mean", "adagrad", 0.01, 1e-8)
    o2, _, g2 = oracle.step(T, ro, B, off, idx, G, sparse, "mean", "adagrad", 0.01, 1e-8)
    np.testing.assert_array_equal(o1, o2)
    np.testing.assert_array_equal(g1, g2)
    np.testing.assert_array_equal(dense.vals[keys], sparse.vals)
    np.testing.assert_array_equal(dense.state[keys], sparse.state)


def test_invalid_inputs_are_rejected():
    ro = np.array([0, 4], np.int64)
    st = RowStore(np.zeros((4, 2), np.float32))
    with pytest.raises(oracle.OracleError):
        oracle.pool_fwd(1, ro, 2, np.array([0, 2, 1], np.int32), np.array([0], np.int32), st, "sum")
    with pytest.raises(oracle.OracleError):
        oracle.pool_fwd(1, ro, 1, np.array([0, 1], np.int32), np.array([4], np.int32), st, "sum")
    with pytest.raises(oracle.OracleError):
        oracle.unique_ids(1, ro, 1, np.array([0, 1], np.int32), np.array([-1], np.int32))


# ------------------------------------------------------- thread count

@pytest.mark.parametrize("name,rounding", [("c2", "nearest"), ("c4", "stochastic"), ("c5", "nearest")])
def test_results_do_not_depend_on_thread_count(name, rounding):
    """The oracle's parallel loops (bags, segments, rows) compute every
    output on one thread in a fixed order: one thread and eight give the
    same forward, dedup, gradient rows, rows and state bit for bit."""
    import synth
    w = synth.scaled(synth.workload(name), rows_div=200, bags_div=16, name=f"{name}-small")
    b = synth.make_batch(w, 3)
    keys = np.unique((w.row_offset[np.repeat(np.arange(w.num_bags), np.diff(b.offsets)) // w.bags_per_table]
                      + b.indices).astype(np.uint32))
    results = []
    try:
        for threads in (1, 8):
            oracle.set_threads(threads)
            assert oracle.get_threads() == threads
            store = oracle.RowStore(synth.weight_rows(w, keys), keys=keys,
                                    state=np.zeros(len(keys), np.float32) if w.opt == "adagrad" else None)
            out, dd, gr = oracle.step(w.num_tables, w.row_offset, w.bags_per_table, b.offsets, b.indices, b.grad,
                                      store, w.pool, w.opt, w.lr, w.eps, rounding, 11)
            results.append((out, dd, gr, store))
    finally:
        oracle.set_threads(0)
    (o1, d1, g1, s1), (o8, d8, g8, s8) = results
    np.testing.assert_array_equal(o1, o8)
    for f in ("unique_keys", "counts", "seg_offsets", "perm"):
        np.testing.assert_array_equal(getattr(d1, f), getattr(d8, f))
    np.testing.assert_array_equal(g1, g8)
    np.testing.assert_array_equal(s1.vals, s8.vals)
    if s1.state is not None:
        np.testing.assert_array_equal(s1.state, s8.state)
