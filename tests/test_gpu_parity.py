"""GPU parity of the HIP path (through the C ABI) against the CPU oracle.

Integer outputs (unique keys, counts, segment offsets, sort permutation,
number of unique ids) must be bit-exact; floating outputs must meet the
row-norm relative tolerance (1e-5 fp32, 1e-2 for bf16 table rows); dyadic
inputs must agree bit-exactly in any summation order.
"""
import sys

import numpy as np
import pytest

import synth
from tests import parity

pytestmark = pytest.mark.gpu


def _say(msg):
    print(msg, flush=True)
    sys.stdout.flush()


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    torch = pytest.importorskip("torch")
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    yield
    torch.cuda.synchronize()
    torch.cuda.empty_cache()


def _rand_batch(rng, rows, B, lmax, empty_frac=0.0, zipf=None):
    T = len(rows)
    M = T * B
    lens = rng.integers(1, lmax + 1, size=M).astype(np.int32)
    if empty_frac:
        lens[rng.random(M) < empty_frac] = 0
    offsets = np.zeros(M + 1, np.int32)
    offsets[1:] = np.cumsum(lens)
    idx = np.zeros(int(offsets[-1]), np.int32)
    for m in range(M):
        t = m // B
        n = int(lens[m])
        if zipf:
            ids = (rng.zipf(zipf, size=n) - 1) % rows[t]
        else:
            ids = rng.integers(0, rows[t], size=n)
        idx[offsets[m]:offsets[m + 1]] = ids
    return offsets, idx


def _row_offset(rows):
    ro = np.zeros(len(rows) + 1, np.int64)
    ro[1:] = np.cumsum(rows)
    return ro


# ------------------------------------------------------------- small cases

@pytest.mark.parametrize("pool", ["sum", "mean"])
@pytest.mark.parametrize("opt", ["sgd", "adagrad"])
def test_small_random_multi_table(pool, opt):
    _say(f"case small_random pool={pool} opt={opt}")
    rng = np.random.default_rng(1)
    rows = [1000, 37, 5000]
    B, D = 300, 64
    off, idx = _rand_batch(rng, rows, B, 40, empty_frac=0.05, zipf=1.3)
    W = rng.uniform(-0.5, 0.5, size=(sum(rows), D)).astype(np.float32)
    G = rng.standard_normal(size=(len(off) - 1, D)).astype(np.float32)
    parity.run_case(_row_offset(rows), W, off, idx, G, B, pool, opt, 0.01, 1e-8)


@pytest.mark.parametrize("pool", ["sum", "mean"])
def test_dyadic_inputs_bit_exact(pool):
    """Dyadic W and G: every fp32 sum is exact, so GPU == oracle bit for bit."""
    _say(f"case dyadic pool={pool}")
    rng = np.random.default_rng(2)
    rows = [3000, 700]
    B, D = 500, 32
    lmax = 8
    off, idx = _rand_batch(rng, rows, B, lmax, empty_frac=0.1, zipf=1.5)
    if pool == "mean":  # bag lengths in {0, 1, 2, 4, 8} keep 1/L dyadic
        lens = np.diff(off)
        lens = np.where(lens == 0, 0, 2 ** np.floor(np.log2(np.maximum(lens, 1)))).astype(np.int32)
        off = np.zeros_like(off)
        off[1:] = np.cumsum(lens)
        idx = np.concatenate([idx[:0]] + [rng.integers(0, rows[m // B], size=lens[m]) for m in range(len(lens))])
    W = (rng.integers(-512, 512, size=(sum(rows), D)) / 1024.0).astype(np.float32)
    G = (rng.integers(-64, 64, size=(len(off) - 1, D)) / 64.0).astype(np.float32)
    parity.run_case(_row_offset(rows), W, off, idx.astype(np.int32), G, B, pool, "sgd", 0.5, 0.0, exact=True)


def test_empty_bags_and_empty_batch():
    _say("case empty bags")
    rng = np.random.default_rng(3)
    rows = [100]
    B, D = 64, 16
    lens = np.zeros(B, np.int32)
    lens[[1, 5, 6, 63]] = [3, 1, 70, 2]
    off = np.zeros(B + 1, np.int32)
    off[1:] = np.cumsum(lens)
    idx = rng.integers(0, 100, size=int(off[-1])).astype(np.int32)
    W = rng.standard_normal((100, D)).astype(np.float32)
    G = rng.standard_normal((B, D)).astype(np.float32)
    g, _, _ = parity.run_case(_row_offset(rows), W, off, idx, G, B, "mean", "adagrad", 0.05, 1e-8)
    assert np.all(g.out[lens == 0] == 0)
    # the whole batch empty
    off0 = np.zeros(B + 1, np.int32)
    g0, _, _ = parity.run_case(_row_offset(rows), W, off0, np.zeros(0, np.int32), G, B, "sum", "sgd", 0.1, 0.0)
    assert g0.num_unique == 0 and np.all(g0.out == 0)


def test_single_id():
    _say("case N=1")
    W = np.arange(64, dtype=np.float32).reshape(4, 16)
    off = np.array([0, 0, 1], np.int32)
    g, _, _ = parity.run_case([0, 4], W, off, np.array([3], np.int32), np.ones((2, 16), np.float32), 2, "sum",
                              "sgd", 0.25, 0.0, exact=True)
    assert g.num_unique == 1 and list(g.perm) == [0]


def test_all_same_id_one_heavy_segment():
    """100k lookups of one row: a single segment spanning ~1600 reduce chunks."""
    _say("case all same id")
    rng = np.random.default_rng(4)
    B, D = 2000, 64
    off, _ = _rand_batch(rng, [10], B, 100)
    idx = np.full(int(off[-1]), 7, np.int32)
    W = rng.uniform(-1, 1, size=(10, D)).astype(np.float32)
    G = rng.standard_normal((B, D)).astype(np.float32)
    g, _, _ = parity.run_case([0, 10], W, off, idx, G, B, "sum", "adagrad", 0.01, 1e-8)
    assert g.num_unique == 1 and g.counts[0] == len(idx)


@pytest.mark.parametrize("n", [63, 64, 65, 2047, 2048, 2049, 4097, 10_000])
def test_tile_and_chunk_boundaries(n):
    _say(f"case N={n}")
    rng = np.random.default_rng(n)
    rows = 5000
    B = max(1, n // 7)
    # exactly n ids over B bags
    cuts = np.sort(rng.integers(0, n + 1, size=B - 1))
    off = np.concatenate([[0], cuts, [n]]).astype(np.int32)
    idx = ((rng.zipf(1.2, size=n) - 1) % rows).astype(np.int32)
    W = rng.uniform(-1, 1, size=(rows, 16)).astype(np.float32)
    G = rng.standard_normal((B, 16)).astype(np.float32)
    parity.run_case([0, rows], W, off, idx, G, B, "sum", "adagrad", 0.01, 1e-8)


@pytest.mark.parametrize("rows", [2, 1024, 1025, 1 << 20, (1 << 20) + 1])
def test_key_bit_boundaries(rows):
    """Key widths that change the number of radix passes; ids 0 and rows-1 present."""
    _say(f"case rows={rows}")
    rng = np.random.default_rng(rows)
    B, D = 700, 8
    off, idx = _rand_batch(rng, [rows], B, 30)
    idx[:5] = 0
    idx[-5:] = rows - 1
    W = rng.uniform(-1, 1, size=(rows, D)).astype(np.float32)
    G = rng.standard_normal((B, D)).astype(np.float32)
    parity.run_case([0, rows], W, off, idx, G, B, "sum", "sgd", 0.01, 0.0)


@pytest.mark.parametrize("dtype,D", [("fp32", 4), ("fp32", 16), ("fp32", 48), ("fp32", 128), ("fp32", 256),
                                     ("fp32", 512), ("fp32", 1024), ("bf16", 8), ("bf16", 64), ("bf16", 128),
                                     ("bf16", 200), ("bf16", 1024)])
def test_row_widths(dtype, D):
    _say(f"case dtype={dtype} D={D}")
    rng = np.random.default_rng(D)
    rows = [3000, 2000]
    B = 200
    off, idx = _rand_batch(rng, rows, B, 60, zipf=1.2)
    Wf = rng.uniform(-0.5, 0.5, size=(sum(rows), D)).astype(np.float32)
    if dtype == "bf16":
        u = Wf.view(np.uint32).astype(np.uint64)
        W = ((u + 0x7FFF + ((u >> 16) & 1)) >> 16).astype(np.uint16)
    else:
        W = Wf
    G = rng.standard_normal((len(off) - 1, D)).astype(np.float32)
    parity.run_case(_row_offset(rows), W, off, idx, G, B, "mean", "adagrad", 0.01, 1e-8)


def test_unfused_equals_fused():
    _say("case unfused vs fused")
    rng = np.random.default_rng(5)
    rows = [20000]
    B, D = 1000, 64
    off, idx = _rand_batch(rng, rows, B, 50, zipf=1.1)
    W = rng.uniform(-0.1, 0.1, size=(rows[0], D)).astype(np.float32)
    G = rng.standard_normal((B, D)).astype(np.float32)
    g1, s1, d1 = parity.run_case([0, rows[0]], W, off, idx, G, B, "sum", "adagrad", 0.01, 1e-8, fused=True)
    g2, s2, d2 = parity.run_case([0, rows[0]], W, off, idx, G, B, "sum", "adagrad", 0.01, 1e-8, fused=False)
    np.testing.assert_array_equal(g1.grad_rows, g2.grad_rows)
    keys = g1.unique_keys
    np.testing.assert_array_equal(d1.rows(keys), d2.rows(keys))
    np.testing.assert_array_equal(d1.state_rows(keys), d2.state_rows(keys))


def test_run_to_run_bitwise_identical():
    _say("case determinism")
    import torch
    rng = np.random.default_rng(6)
    rows = [200000]
    B, D = 4000, 64
    off, idx = _rand_batch(rng, rows, B, 60, zipf=1.2)
    W = rng.uniform(-0.1, 0.1, size=(rows[0], D)).astype(np.float32)
    G = rng.standard_normal((B, D)).astype(np.float32)
    outs = []
    for rep in range(3):
        dl = parity.device_layer_from_host([0, rows[0]], W, np.zeros(rows[0], np.float32))
        g = parity.gpu_step(dl, off, idx, G, B, "sum", "adagrad", 0.01, 1e-8)
        outs.append((g, dl.rows(g.unique_keys), dl.state_rows(g.unique_keys)))
        torch.cuda.synchronize()
    for g, r, h in outs[1:]:
        np.testing.assert_array_equal(g.out, outs[0][0].out)
        np.testing.assert_array_equal(g.grad_rows, outs[0][0].grad_rows)
        np.testing.assert_array_equal(g.perm, outs[0][0].perm)
        np.testing.assert_array_equal(r, outs[0][1])
        np.testing.assert_array_equal(h, outs[0][2])


@pytest.mark.parametrize("concurrent", [False, True])
def test_workspace_reuse_with_varying_batch_sizes(concurrent):
    """One workspace, batches of very different N in a row (big, small, big),
    through serial calls and through Layer.step's concurrent schedule."""
    _say(f"case workspace reuse concurrent={concurrent}")
    import oracle
    import paper_2112_02752_amd as emb
    rng = np.random.default_rng(7)
    rows = 100000
    D = 16
    W = rng.uniform(-1, 1, size=(rows, D)).astype(np.float32)
    dl = parity.device_layer_from_host([0, rows], W, None)
    layer = emb.Layer(dl.tables, "sum", "sgd", 0.01, 0.0, None, max_indices=200_000, max_bags=5000,
                      concurrent=concurrent)
    store = oracle.RowStore(W.copy())
    for B, lmax in [(4000, 80), (3, 2), (1, 1), (5000, 60), (50, 10)]:
        off, idx = _rand_batch(rng, [rows], B, lmax, zipf=1.3)
        G = rng.standard_normal((B, D)).astype(np.float32)
        g = parity.gpu_step(dl, off, idx, G, B, "sum", "sgd", 0.01, 0.0, layer=layer)
        o_out, o_dd, o_gr = oracle.step(1, np.array([0, rows], np.int64), B, off, idx, G, store, "sum", "sgd",
                                        0.01, 0.0)
        parity.check_against_oracle(g, o_out, o_dd, o_gr)
        parity.check_rows(dl, store, o_dd.unique_keys, "sgd")


def test_validate_batch_flags():
    _say("case validate")
    import torch
    import paper_2112_02752_amd as emb
    W = torch.zeros((10, 16), dtype=torch.float32, device="cuda")
    t = emb.Tables(W, [0, 4, 10])
    flag = torch.zeros(1, dtype=torch.int32, device="cuda")

    def check(offsets, idx, B):
        b = emb.Batch(torch.tensor(offsets, dtype=torch.int32, device="cuda"),
                      torch.tensor(idx, dtype=torch.int32, device="cuda"), B)
        emb.validate_batch(t, b, flag)
        torch.cuda.synchronize()
        return int(flag.item())

    assert check([0, 2, 3], [3, 0, 5], 1) == 0
    assert check([0, 2, 3], [4, 0, 5], 1) == 8          # id 4 >= rows of table 0
    assert check([0, 2, 3], [3, 0, 6], 1) == 8          # id 6 >= rows of table 1
    assert check([0, 3, 2], [3, 0, 1], 1) & 2           # decreasing offsets
    assert check([1, 2, 3], [3, 0, 1], 1) & 1           # offsets[0] != 0


# --------------------------------------------------------- full workloads

@pytest.mark.parametrize("name", ["c1", "c2", "c3", "c4", "c5"])
def test_workload_full_size_one_step(name):
    w = synth.workload(name)
    _say(f"case workload {name} rows={w.total_rows} D={w.dim} {w.dtype}")
    parity.run_workload(w, steps=1)


@pytest.mark.parametrize("rows_div,bags,concurrent", [(1, 16384, True), (1, 17000, False), (1, 23000, True),
                                                     (1, 40000, False), (50, 16384, False), (50, 23000, True)])
def test_sort_tile_modes(rows_div, bags, concurrent):
    """Batches of the 50M-row workload's shape whose sizes select each sort
    mode: co-resident passes with 2048-, 2560- and 4096-key tiles (at most
    one block per compute unit) and reduce-then-scan passes (tile counts and
    a column scan before each pass) beyond that, for 26-bit keys (three
    passes) and 20-bit keys (rows / 50: two passes)."""
    import dataclasses
    w = dataclasses.replace(synth.scaled(synth.workload("c3"), rows_div=rows_div), bags_per_table=bags,
                            name=f"c3/r{rows_div}-b{bags}")
    _say(f"case sort tile modes rows/{rows_div} bags={bags} concurrent={concurrent}")
    parity.run_workload(w, steps=1, concurrent=concurrent)


@pytest.mark.parametrize("rows_div", [1, 2, 4, 8, 16, 32])
def test_sort_key_widths_21_to_26_bits(rows_div):
    """Every key width from 26 down to 21 bits (rows of the 50M-row table
    divided by 1..32: three radix passes of 7 to 9 bits), 1024 bags."""
    w = synth.scaled(synth.workload("c3"), rows_div=rows_div, bags_div=16)
    _say(f"case sort key bits={w.key_bits} bags={w.bags_per_table}")
    assert 21 <= w.key_bits <= 26
    parity.run_workload(w, steps=1)


@pytest.mark.parametrize("name,bags", [("c3", 1), ("c3", 137), ("c3", 3000), ("c2", 2), ("c2", 500)])
def test_sort_small_batches(name, bags):
    """One tile, a ragged second tile, and several tiles, two steps on one
    workspace; one table (the ids are the keys) and eight (keys built from
    the bags)."""
    import dataclasses
    w = dataclasses.replace(synth.workload(name), bags_per_table=bags, name=f"{name}-b{bags}")
    _say(f"case sort small {name} bags={bags}")
    parity.run_workload(w, steps=2)


def test_sort_three_passes_coresident():
    """28-bit keys (the 200M-row table) in a batch small enough for
    co-resident 10-bit passes: three passes with digit-range prefix blocks."""
    w = synth.scaled(synth.workload("c5"), bags_div=8)
    _say(f"case three co-resident passes bags={w.bags_per_table}")
    parity.run_workload(w, steps=1)


# ------------------------------------------------ element-wise Adagrad variant

def _bf16_bits(Wf):
    u = Wf.view(np.uint32).astype(np.uint64)
    return ((u + 0x7FFF + ((u >> 16) & 1)) >> 16).astype(np.uint16)


@pytest.mark.parametrize("pool,dtype,D,fused", [("sum", "fp32", 64, True), ("mean", "fp32", 16, True),
                                                ("sum", "bf16", 128, True), ("sum", "fp32", 256, False)])
def test_elementwise_adagrad_small(pool, dtype, D, fused):
    """Element-wise Adagrad (state [R][D]).  The accumulators start at 1: from
    zero, the first step moves an element by lr * g / (|g| + eps), whose sign
    is that of a gradient sum that may cancel to rounding noise."""
    _say(f"case elementwise adagrad pool={pool} dtype={dtype} D={D} fused={fused}")
    rng = np.random.default_rng(40 + D)
    rows = [3000, 700]
    B = 300
    off, idx = _rand_batch(rng, rows, B, 40, empty_frac=0.05, zipf=1.3)
    Wf = rng.uniform(-0.5, 0.5, size=(sum(rows), D)).astype(np.float32)
    W = _bf16_bits(Wf) if dtype == "bf16" else Wf
    G = rng.standard_normal(size=(len(off) - 1, D)).astype(np.float32)
    state0 = rng.uniform(0.5, 1.5, size=(sum(rows), D)).astype(np.float32)
    parity.run_case(_row_offset(rows), W, off, idx, G, B, pool, "adagrad_ew", 0.01, 1e-8, state0=state0, fused=fused)


def test_elementwise_adagrad_dyadic_from_zero():
    """From zero accumulators on dyadic inputs: every gradient sum is exact, so
    no sign is in doubt."""
    _say("case elementwise adagrad dyadic from zero")
    rng = np.random.default_rng(44)
    rows = [2000, 900]
    B, D = 400, 32
    off, idx = _rand_batch(rng, rows, B, 8, empty_frac=0.1, zipf=1.5)
    W = (rng.integers(-512, 512, size=(sum(rows), D)) / 1024.0).astype(np.float32)
    G = (rng.integers(-64, 64, size=(len(off) - 1, D)) / 64.0).astype(np.float32)
    parity.run_case(_row_offset(rows), W, off, idx, G, B, "sum", "adagrad_ew", 0.01, 1e-8)


@pytest.mark.parametrize("name,steps", [("c2", 1), ("c3", 2)])
def test_elementwise_adagrad_full_size(name, steps):
    """The 8-table and the 50M-row workloads with element-wise Adagrad state
    ([R][D] fp32, starting at 1)."""
    import dataclasses
    w = dataclasses.replace(synth.workload(name), opt="adagrad_ew", name=f"{name}-ew")
    _say(f"case elementwise adagrad full size {name} x{steps}")
    parity.run_workload(w, steps=steps, h0=1.0)


# ------------------------------------------------- bf16 stochastic rounding

@pytest.mark.parametrize("opt,fused", [("adagrad", True), ("sgd", False), ("adagrad_ew", True)])
def test_stochastic_rounding_small(opt, fused):
    """bf16 tables with stochastic rounding: rows within the bf16 tolerance of
    the oracle and, element by element, the same stored value almost
    everywhere (both draw the same bits for every element)."""
    _say(f"case stochastic rounding opt={opt} fused={fused}")
    rng = np.random.default_rng(70)
    rows = [3000, 2000]
    B, D = 200, 64
    off, idx = _rand_batch(rng, rows, B, 60, zipf=1.2)
    W = _bf16_bits(rng.uniform(-0.5, 0.5, size=(sum(rows), D)).astype(np.float32))
    G = rng.standard_normal((len(off) - 1, D)).astype(np.float32)
    state0 = np.ones((sum(rows), D), np.float32) if opt == "adagrad_ew" else None
    parity.run_case(_row_offset(rows), W, off, idx, G, B, "sum", opt, 0.05, 1e-8, state0=state0, fused=fused,
                    rounding="stochastic", seed=0x1234)


def test_stochastic_rounding_full_size():
    """The 26-table bf16 workload, two steps with fresh seeds."""
    w = synth.workload("c4")
    _say("case stochastic rounding c4 x2")
    parity.run_workload(w, steps=2, rounding="stochastic", seed=77)


# ------------------------------------------------------------- int64 ids

@pytest.mark.parametrize("pool,opt", [("sum", "adagrad"), ("mean", "sgd")])
def test_int64_indices_small(pool, opt):
    _say(f"case int64 ids pool={pool} opt={opt}")
    rng = np.random.default_rng(60)
    rows = [1000, 37, 5000]
    B, D = 300, 64
    off, idx = _rand_batch(rng, rows, B, 40, empty_frac=0.05, zipf=1.3)
    W = rng.uniform(-0.5, 0.5, size=(sum(rows), D)).astype(np.float32)
    G = rng.standard_normal(size=(len(off) - 1, D)).astype(np.float32)
    parity.run_case(_row_offset(rows), W, off, idx, G, B, pool, opt, 0.01, 1e-8, idx64=True)


@pytest.mark.parametrize("name", ["c3", "c2", "c5"])
def test_int64_indices_full_size(name):
    """int64 ids (PyTorch's index type) at full size: one table with the
    co-resident sort, several tables, one table with the look-back sort."""
    w = synth.workload(name)
    _say(f"case int64 ids full size {name}")
    parity.run_workload(w, steps=1, idx64=True)


def test_int64_validate_flags_ids_beyond_32_bits():
    _say("case int64 validate")
    import torch
    import paper_2112_02752_amd as emb
    W = torch.zeros((10, 16), dtype=torch.float32, device="cuda")
    t = emb.Tables(W, [0, 10])
    flag = torch.zeros(1, dtype=torch.int32, device="cuda")
    off = torch.tensor([0, 2], dtype=torch.int32, device="cuda")
    for ids, want in (([3, 9], 0), ([3, (1 << 32) + 3], 8), ([-1, 2], 8)):
        b = emb.Batch(off, torch.tensor(ids, dtype=torch.int64, device="cuda"), 1)
        emb.validate_batch(t, b, flag)
        torch.cuda.synchronize()
        assert int(flag.item()) == want, (ids, int(flag.item()))


def test_c5_three_consecutive_steps():
    w = synth.workload("c5")
    _say("case c5 x3 steps")
    parity.run_workload(w, steps=3)


def test_c5_hundred_steps_sampled_rows():
    """All 100 steps of the 200M-row workload on the device, then a sample of
    rows (the first batch's 1000 hottest ids, 4000 more of its ids, the last
    row) against the oracle replaying every step's update of just those rows,
    and rows that no step touched against their initial values.  With sum
    pooling a row's gradient sums the upstream rows of its own id's positions
    only, so each batch is cut down to the positions of the sampled ids (bags
    kept, shortened) before the oracle's dedup, reduce and SGD step."""
    import oracle
    import paper_2112_02752_amd as emb
    torch = parity.torch_mod()
    w = synth.workload("c5")
    assert w.steps == 100 and w.pool == "sum" and w.num_tables == 1
    _say(f"case c5 x{w.steps} steps, sampled rows")
    dl = parity.device_layer_from_workload(w)
    b0 = synth.make_batch(w, 0, with_grad=False)
    ids, cnt = np.unique(b0.indices, return_counts=True)
    rng = np.random.default_rng(100)
    hot = ids[np.argsort(-cnt, kind="stable")[:1000]]
    sample = np.unique(np.concatenate([hot, rng.choice(ids, 4000, replace=False),
                                       [w.total_rows - 1]])).astype(np.uint32)
    untouched = np.setdiff1d(np.unique(rng.integers(0, w.total_rows, 2000)), sample)
    store = oracle.RowStore(synth.weight_rows(w, sample), keys=sample)
    B, M = w.bags_per_table, w.num_bags
    layer = emb.Layer(dl.tables, w.pool, w.opt, w.lr, w.eps, dl.state,
                      max_indices=M * max(t.lmax for t in w.tables), max_bags=M)
    out = torch.empty((M, w.dim), dtype=torch.float32, device=dl.W.device)
    for s in range(w.steps):
        b = synth.make_batch(w, s)
        off = torch.from_numpy(b.offsets).to(dl.W.device)
        idx = torch.from_numpy(b.indices).to(dl.W.device)
        G = torch.from_numpy(b.grad).to(dl.W.device)
        layer.step(emb.Batch(off, idx, B), out, G)
        keep = np.isin(b.indices, sample)
        bag = np.repeat(np.arange(M), np.diff(b.offsets))
        off_f = np.concatenate([[0], np.cumsum(np.bincount(bag[keep], minlength=M))]).astype(np.int32)
        idx_f = np.ascontiguousarray(b.indices[keep])
        dd = oracle.unique_ids(1, w.row_offset, B, off_f, idx_f)
        _, acc = oracle.grad_reduce(1, B, off_f, b.grad, w.pool, dd)
        oracle.sparse_update(store, dd.unique_keys, acc, w.opt, w.lr, w.eps)
        untouched = untouched[~np.isin(untouched, b.indices)]
        if s % 20 == 19:
            _say(f"  step {s + 1} done")
    torch.cuda.synchronize()
    layer.check()
    parity.check_rows(dl, store, sample, w.opt)
    assert untouched.size > 0
    np.testing.assert_array_equal(dl.rows(untouched.astype(np.uint32)), synth.weight_rows(w, untouched))


def test_graph_replay_matches_eager():
    """The serial step captured once in a HIP graph (torch.cuda.graph) and
    replayed on four batches of one size, each copied into the captured input
    buffers, with eager steps of a twin layer and host synchronisations
    between the replays: every replay's pooled output, table and Adagrad
    state equal the eager twin's bit for bit (the step launches kernels
    only, with no memset nodes)."""
    import paper_2112_02752_amd as emb
    torch = parity.torch_mod()
    _say("case graph replay vs eager")
    rows, B, D, N = 200_000, 2048, 64, 2048 * 30
    rng = np.random.default_rng(11)

    def batch():
        cuts = np.sort(rng.integers(0, N + 1, size=B - 1))
        off = np.concatenate([[0], cuts, [N]]).astype(np.int32)
        idx = ((rng.zipf(1.2, size=N) - 1) % rows).astype(np.int32)
        return off, idx, rng.standard_normal((B, D)).astype(np.float32)

    dev = "cuda"
    W0 = torch.from_numpy(rng.uniform(-0.01, 0.01, size=(rows, D)).astype(np.float32)).to(dev)
    Wa, Wb = W0.clone(), W0.clone()
    ha, hb = torch.zeros(rows, device=dev), torch.zeros(rows, device=dev)
    la = emb.Layer(emb.Tables(Wa, [0, rows]), "sum", "adagrad", 0.01, 1e-8, ha, max_indices=N, max_bags=B)
    lb = emb.Layer(emb.Tables(Wb, [0, rows]), "sum", "adagrad", 0.01, 1e-8, hb, max_indices=N, max_bags=B)
    off_s = torch.empty(B + 1, dtype=torch.int32, device=dev)
    idx_s = torch.empty(N, dtype=torch.int32, device=dev)
    G_s = torch.empty((B, D), device=dev)
    out_s = torch.empty((B, D), device=dev)
    out_a = torch.empty((B, D), device=dev)

    def step_both(b, replay=None):
        off_s.copy_(torch.from_numpy(b[0]))
        idx_s.copy_(torch.from_numpy(b[1]))
        G_s.copy_(torch.from_numpy(b[2]))
        if replay is None:
            lb.step(emb.Batch(off_s, idx_s, B), out_s, G_s)
        else:
            replay.replay()
        torch.cuda.synchronize()
        off_a, idx_a, G_a = (torch.from_numpy(x).to(dev) for x in b)
        la.step(emb.Batch(off_a, idx_a, B), out_a, G_a)
        torch.cuda.synchronize()
        assert torch.equal(out_s, out_a)
        assert torch.equal(Wb, Wa) and torch.equal(hb, ha)

    step_both(batch())  # eager warm-up on both layers
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        lb.step(emb.Batch(off_s, idx_s, B), out_s, G_s)
    for _ in range(4):
        step_both(batch(), replay=g)
    assert not torch.equal(Wb, W0)


def test_c2_unfused_path():
    w = synth.workload("c2")
    _say("case c2 unfused")
    parity.run_workload(w, steps=1, fused=False)


@pytest.mark.parametrize("name,steps", [("c3", 3), ("c2", 1), ("c4", 1)])
def test_concurrent_schedule_full_size(name, steps):
    """Layer.step with the forward on a side stream alongside the dedup
    matches the oracle at full size."""
    w = synth.workload(name)
    _say(f"case concurrent schedule {name} x{steps} steps")
    parity.run_workload(w, steps=steps, concurrent=True)


def test_concurrent_schedule_equals_serial():
    """The concurrent schedule changes nothing: tables, state and pooled
    outputs equal those of serial steps bit for bit."""
    _say("case concurrent vs serial")
    import torch
    import paper_2112_02752_amd as emb
    w = synth.scaled(synth.workload("c3"), rows_div=500, bags_div=4, name="c3-small")
    batches = [synth.make_batch(w, s) for s in range(6)]
    nmax = max(len(b.indices) for b in batches)
    dev_b = [(emb.Batch(torch.from_numpy(b.offsets).cuda(), torch.from_numpy(b.indices).cuda(), w.bags_per_table),
              torch.from_numpy(b.grad).cuda()) for b in batches]
    results = []
    for conc in (False, True):
        dl = parity.device_layer_from_workload(w)
        layer = emb.Layer(dl.tables, w.pool, w.opt, w.lr, w.eps, dl.state, max_indices=nmax, max_bags=w.num_bags,
                          concurrent=conc)
        outs = []
        for b, g in dev_b:
            out = torch.empty((w.num_bags, w.dim), dtype=torch.float32, device="cuda")
            layer.step(b, out, g)
            outs.append(out)
        torch.cuda.synchronize()
        results.append((dl.W.cpu().numpy(), dl.state.cpu().numpy(), [o.cpu().numpy() for o in outs]))
    (w0, s0, o0), (w1, s1, o1) = results
    np.testing.assert_array_equal(w0, w1)
    np.testing.assert_array_equal(s0, s1)
    for a, b in zip(o0, o1):
        np.testing.assert_array_equal(a, b)


def test_auto_schedule_full_size():
    """The 200M-row workload (3.3M lookups per batch) under the automatic
    schedule, which overlaps the forward with the dedup for it."""
    w = synth.workload("c5")
    _say("case auto schedule c5")
    parity.run_workload(w, steps=2, concurrent="auto")


@pytest.mark.parametrize("name,concurrent", [("c3", False), ("c2", True)])
def test_stale_schedule_matches_oracle_replay(name, concurrent):
    """The asynchronous schedule with staleness one (the forward of batch
    k+1 before the update of batch k) against the oracle replaying exactly
    that order: pooled outputs of every batch and the final rows."""
    _say(f"case stale schedule {name} concurrent={concurrent}")
    import oracle
    import torch
    import paper_2112_02752_amd as emb
    w = synth.scaled(synth.workload(name), rows_div=50, bags_div=4, name=f"{name}-small")
    K = 4
    batches = [synth.make_batch(w, s) for s in range(K + 1)]
    nmax = max(len(b.indices) for b in batches)
    dev_b = [(emb.Batch(torch.from_numpy(b.offsets).cuda(), torch.from_numpy(b.indices).cuda(), w.bags_per_table),
              torch.from_numpy(b.grad).cuda()) for b in batches]
    dl = parity.device_layer_from_workload(w)
    layer = emb.Layer(dl.tables, w.pool, w.opt, w.lr, w.eps, dl.state, max_indices=nmax, max_bags=w.num_bags,
                      concurrent=concurrent)
    outs = [torch.empty((w.num_bags, w.dim), dtype=torch.float32, device="cuda") for _ in range(K + 1)]
    layer.forward(dev_b[0][0], outs[0])
    for k in range(K):
        layer.step_stale(dev_b[k + 1][0], outs[k + 1], dev_b[k][0], dev_b[k][1])
    layer.backward(dev_b[K][0], dev_b[K][1])
    torch.cuda.synchronize()
    # the oracle replays the same order on the rows the batches touch
    keys = [parity.global_keys(w.row_offset, w.bags_per_table, b.offsets, b.indices) for b in batches]
    touched = np.unique(np.concatenate(keys))
    store = oracle.RowStore(synth.weight_rows(w, touched), keys=touched.astype(np.uint32),
                            state=np.zeros(len(touched), np.float32) if w.opt == "adagrad" else None)
    T, ro, B = w.num_tables, w.row_offset, w.bags_per_table

    def fwd(b):
        return oracle.pool_fwd(T, ro, B, b.offsets, b.indices, store, w.pool)

    def bwd(b):
        dd = oracle.unique_ids(T, ro, B, b.offsets, b.indices)
        _, acc = oracle.grad_reduce(T, B, b.offsets, b.grad, w.pool, dd)
        oracle.sparse_update(store, dd.unique_keys, acc, w.opt, w.lr, w.eps)

    ref = [fwd(batches[0])]
    for k in range(K):
        ref.append(fwd(batches[k + 1]))
        bwd(batches[k])
    bwd(batches[K])
    for k in range(K + 1):
        r = parity.rel_rownorm(outs[k].cpu().numpy(), ref[k])
        assert r <= parity.TOL_FP32, f"pooled output of batch {k}: rel err {r}"
    parity.check_rows(dl, store, touched, w.opt)


@pytest.mark.parametrize("group,sides,nsteps,gd,depth", [
    (1, 1, 5, False, 2), (2, 1, 7, False, 2), (4, 1, 10, False, 2), (2, 2, 7, False, 2), (6, 3, 13, False, 2),
    (1, 1, 5, True, 2), (2, 1, 7, True, 2), (6, 1, 13, True, 2), (16, 1, 20, True, 2),
    (1, 1, 9, True, 3), (2, 2, 11, False, 3), (2, 1, 15, True, 5)])
def test_pipelined_schedule_equals_serial(group, sides, nsteps, gd, depth):
    """The dedups of the next group of batches on a side stream while the main
    stream runs the forward and update of the current group change nothing:
    tables, state and pooled outputs equal those of serial steps bit for bit
    (step counts that leave a partial last group included; gd: each group's
    dedups as one emb_unique_ids_batched call; depth: buffer set parities)."""
    _say(f"case pipelined vs serial group={group} side streams={sides} steps={nsteps} group dedup={gd} "
         f"depth={depth}")
    import torch
    import paper_2112_02752_amd as emb
    w = synth.scaled(synth.workload("c3"), rows_div=500, bags_div=8, name="c3-small")
    batches = [synth.make_batch(w, s) for s in range(nsteps)]
    nmax = max(len(b.indices) for b in batches)
    dev_b = [(emb.Batch(torch.from_numpy(b.offsets).cuda(), torch.from_numpy(b.indices).cuda(), w.bags_per_table),
              torch.from_numpy(b.grad).cuda()) for b in batches]
    results = []
    for mode in ("serial", "pipelined"):
        dl = parity.device_layer_from_workload(w)
        outs = [torch.empty((w.num_bags, w.dim), dtype=torch.float32, device="cuda") for _ in dev_b]
        if mode == "serial":
            layer = emb.Layer(dl.tables, w.pool, w.opt, w.lr, w.eps, dl.state, max_indices=nmax, max_bags=w.num_bags)
            for (b, g), out in zip(dev_b, outs):
                layer.step(b, out, g)
        else:
            pipe = emb.Pipeline(dl.tables, w.pool, w.opt, w.lr, w.eps, dl.state, max_indices=nmax,
                                max_bags=w.num_bags, group=group, side_streams=sides, group_dedup=gd, depth=depth)
            # two runs: the second starts after everything the first enqueued
            half = nsteps // 2
            pipe.run([(b, o, g) for (b, g), o in zip(dev_b[:half], outs[:half])])
            pipe.run([(b, o, g) for (b, g), o in zip(dev_b[half:], outs[half:])])
        torch.cuda.synchronize()
        if mode == "pipelined":
            pipe.check()
        results.append((dl.W.cpu().numpy(), dl.state.cpu().numpy(), [o.cpu().numpy() for o in outs]))
    (w0, s0, o0), (w1, s1, o1) = results
    np.testing.assert_array_equal(w0, w1)
    np.testing.assert_array_equal(s0, s1)
    for a, b in zip(o0, o1):
        np.testing.assert_array_equal(a, b)


@pytest.mark.parametrize("group,sides,gd,chunks,depth,look", [
    (2, 1, True, (3, 4, 2), 2, 1), (4, 1, True, (5, 8, 4), 2, 1), (1, 1, False, (2, 3, 1), 2, 1),
    (8, 1, True, (5, 20, 8), 2, 1),
    (2, 2, False, (4, 3, 2), 2, 1), (6, 3, False, (7, 6, 6), 2, 1), (4, 1, True, (4, "discard", 5), 2, 1),
    # look-ahead of several groups, with as many more buffer set parities
    (2, 1, True, (3, 5, 4), 3, 2), (4, 1, True, (6, 9, 8), 3, 2), (1, 1, False, (2, 3, 2), 3, 2),
    (2, 2, False, (5, 7, 6), 4, 3), (2, 1, True, (3, 4, 2), 3, 1), (2, 1, True, (4, "discard", 5), 3, 2)])
def test_pipelined_chained_calls_equal_serial(group, sides, gd, chunks, depth, look):
    """Chained calls: each call but the last also dedups the next call's
    first `look` groups of batches, and the next call starts with those
    dedups done (a training loop's look-ahead; `depth` buffer set parities).
    Tables, state and pooled outputs equal those of serial steps bit for
    bit; a call that starts with other batches than the ones deduplicated
    ahead is refused; after discard() the next call dedups its own first
    groups."""
    _say(f"case pipelined chained group={group} side streams={sides} group dedup={gd} chunks={chunks} "
         f"depth={depth} look-ahead groups={look}")
    import torch
    import paper_2112_02752_amd as emb
    sizes = [c for c in chunks if c != "discard"]
    nsteps = sum(sizes)
    w = synth.scaled(synth.workload("c3"), rows_div=500, bags_div=8, name="c3-small")
    batches = [synth.make_batch(w, s) for s in range(nsteps)]
    nmax = max(len(b.indices) for b in batches)
    dev_b = [(emb.Batch(torch.from_numpy(b.offsets).cuda(), torch.from_numpy(b.indices).cuda(), w.bags_per_table),
              torch.from_numpy(b.grad).cuda()) for b in batches]
    results = []
    for mode in ("serial", "chained"):
        dl = parity.device_layer_from_workload(w)
        outs = [torch.empty((w.num_bags, w.dim), dtype=torch.float32, device="cuda") for _ in dev_b]
        if mode == "serial":
            layer = emb.Layer(dl.tables, w.pool, w.opt, w.lr, w.eps, dl.state, max_indices=nmax, max_bags=w.num_bags)
            for (b, g), out in zip(dev_b, outs):
                layer.step(b, out, g)
        else:
            pipe = emb.Pipeline(dl.tables, w.pool, w.opt, w.lr, w.eps, dl.state, max_indices=nmax,
                                max_bags=w.num_bags, group=group, side_streams=sides, group_dedup=gd, depth=depth)
            k = 0
            for i, c in enumerate(chunks):
                if c == "discard":
                    pipe.discard()
                    continue
                nxt = chunks[i + 1] if i + 1 < len(chunks) else None
                ahead = None
                if isinstance(nxt, int):
                    ahead = [b for b, _ in dev_b[k + c:k + c + look * group]]
                elif nxt == "discard":
                    # dedups ahead of batches that the next call will not start with
                    ahead = [b for b, _ in dev_b[k + c + 1:k + c + 1 + look * group]]
                steps = [(b, o, g) for (b, g), o in zip(dev_b[k:k + c], outs[k:k + c])]
                if k > 0 and pipe._primed is not None:
                    with pytest.raises(ValueError):
                        # batch 0 is never among the batches deduplicated ahead
                        pipe.run([(dev_b[0][0], outs[0], dev_b[0][1])])
                pipe.run(steps, ahead=ahead)
                k += c
        torch.cuda.synchronize()
        if mode == "chained":
            pipe.check()
        results.append((dl.W.cpu().numpy(), dl.state.cpu().numpy(), [o.cpu().numpy() for o in outs]))
    (w0, s0, o0), (w1, s1, o1) = results
    np.testing.assert_array_equal(w0, w1)
    np.testing.assert_array_equal(s0, s1)
    for a, b in zip(o0, o1):
        np.testing.assert_array_equal(a, b)


def test_pipelined_chained_bf16_tables_stochastic_rounding():
    """Chained pipelined calls on the 26-table bf16 workload (scaled down)
    with stochastic rounding: each step draws its bits from seed + its step
    index across the calls, as serial steps do, so tables, state and pooled
    outputs equal those of serial steps bit for bit."""
    _say("case pipelined chained c4-small bf16 stochastic rounding")
    import torch
    import paper_2112_02752_amd as emb
    w = synth.scaled(synth.workload("c4"), rows_div=100, bags_div=64, name="c4-small")
    chunks, group = (5, 4, 3), 2
    batches = [synth.make_batch(w, s) for s in range(sum(chunks))]
    nmax = max(len(b.indices) for b in batches)
    dev_b = [(emb.Batch(torch.from_numpy(b.offsets).cuda(), torch.from_numpy(b.indices).cuda(), w.bags_per_table),
              torch.from_numpy(b.grad).cuda()) for b in batches]
    results = []
    for mode in ("serial", "chained"):
        dl = parity.device_layer_from_workload(w)
        outs = [torch.empty((w.num_bags, w.dim), dtype=torch.float32, device="cuda") for _ in dev_b]
        if mode == "serial":
            layer = emb.Layer(dl.tables, w.pool, w.opt, w.lr, w.eps, dl.state, max_indices=nmax, max_bags=w.num_bags,
                              rounding="stochastic", seed=91)
            for (b, g), out in zip(dev_b, outs):
                layer.step(b, out, g)
        else:
            pipe = emb.Pipeline(dl.tables, w.pool, w.opt, w.lr, w.eps, dl.state, max_indices=nmax,
                                max_bags=w.num_bags, group=group, rounding="stochastic", seed=91)
            k = 0
            for i, c in enumerate(chunks):
                ahead = [b for b, _ in dev_b[k + c:k + c + group]] if i + 1 < len(chunks) else None
                pipe.run([(b, o, g) for (b, g), o in zip(dev_b[k:k + c], outs[k:k + c])], ahead=ahead)
                k += c
        torch.cuda.synchronize()
        if mode == "chained":
            pipe.check()
        results.append((dl.W.view(torch.int16).cpu().numpy(), dl.state.cpu().numpy(), [o.cpu().numpy() for o in outs]))
    (w0, s0, o0), (w1, s1, o1) = results
    np.testing.assert_array_equal(w0, w1)
    np.testing.assert_array_equal(s0, s1)
    for a, b in zip(o0, o1):
        np.testing.assert_array_equal(a, b)


@pytest.mark.parametrize("name,nsteps,group,sides,gd", [("c3", 6, 4, 1, False), ("c3", 13, 6, 3, False),
                                                        ("c2", 3, 2, 1, False), ("c2", 5, 4, 2, False),
                                                        ("c3", 13, 6, 1, True), ("c2", 5, 4, 1, True),
                                                        ("c3", 17, 8, 1, True)])
def test_pipelined_schedule_full_size(name, nsteps, group, sides, gd):
    """Full-size pipelined steps against the oracle replaying the same steps on
    the rows they touch: every pooled output, the final rows and state, rows
    no step touched unchanged."""
    _say(f"case pipelined full size {name} steps={nsteps} group={group} side streams={sides} group dedup={gd}")
    import oracle
    import torch
    import paper_2112_02752_amd as emb
    w = synth.workload(name)
    batches = [synth.make_batch(w, s) for s in range(nsteps)]
    nmax = max(len(b.indices) for b in batches)
    dev_b = [(emb.Batch(torch.from_numpy(b.offsets).cuda(), torch.from_numpy(b.indices).cuda(), w.bags_per_table),
              torch.from_numpy(b.grad).cuda()) for b in batches]
    dl = parity.device_layer_from_workload(w)
    pipe = emb.Pipeline(dl.tables, w.pool, w.opt, w.lr, w.eps, dl.state, max_indices=nmax, max_bags=w.num_bags,
                        group=group, side_streams=sides, group_dedup=gd)
    outs = [torch.empty((w.num_bags, w.dim), dtype=torch.float32, device="cuda") for _ in dev_b]
    pipe.run([(b, o, g) for (b, g), o in zip(dev_b, outs)])
    torch.cuda.synchronize()
    pipe.check()
    keys = [parity.global_keys(w.row_offset, w.bags_per_table, b.offsets, b.indices) for b in batches]
    touched = np.unique(np.concatenate(keys))
    store = oracle.RowStore(synth.weight_rows(w, touched), keys=touched.astype(np.uint32),
                            state=np.zeros(len(touched), np.float32) if w.opt == "adagrad" else None)
    for k, b in enumerate(batches):
        o_out, _, _ = oracle.step(w.num_tables, w.row_offset, w.bags_per_table, b.offsets, b.indices, b.grad, store,
                                  w.pool, w.opt, w.lr, w.eps)
        r = parity.rel_rownorm(outs[k].cpu().numpy(), o_out)
        assert r <= parity.TOL_FP32, f"pooled output of step {k}: rel err {r}"
    parity.check_rows(dl, store, touched, w.opt)
    parity.check_untouched(dl, w, touched)


def _dedup_concurrent_vs_oracle(row_offset, B, off, idx, M):
    import oracle
    import torch
    import paper_2112_02752_amd as emb
    N = len(idx)
    dev = "cuda"
    tables = emb.Tables(torch.empty((1, 4), dtype=torch.float32, device=dev), [int(x) for x in row_offset])
    b = emb.Batch(torch.from_numpy(np.ascontiguousarray(off, np.int32)).to(dev),
                  torch.from_numpy(np.ascontiguousarray(idx, np.int32)).to(dev), B)
    bufs = emb.DedupBuffers(dev, N, M, 4)
    emb.unique_ids(tables, b, bufs.unique_keys, bufs.counts, bufs.seg_offsets, bufs.sort_perm, bufs.num_unique,
                   bufs.ws, concurrent=True)
    torch.cuda.synchronize()
    assert emb.read_status(bufs.ws)[0] == 0
    ref = oracle.unique_ids(len(row_offset) - 1, np.asarray(row_offset, np.int64), B,
                            np.ascontiguousarray(off, np.int32), np.ascontiguousarray(idx, np.int32))
    U = int(bufs.num_unique.cpu().item())
    assert U == ref.num_unique
    np.testing.assert_array_equal(bufs.unique_keys[:U].cpu().numpy().view(np.uint32), ref.unique_keys)
    np.testing.assert_array_equal(bufs.counts[:U].cpu().numpy(), ref.counts)
    np.testing.assert_array_equal(bufs.seg_offsets[:U + 1].cpu().numpy(), ref.seg_offsets)
    np.testing.assert_array_equal(bufs.sort_perm[:N].cpu().numpy(), ref.perm)


@pytest.mark.parametrize("name", ["c1", "c2", "c3", "c5"])
def test_unique_ids_concurrent_full_size(name):
    """emb_unique_ids_concurrent (no workgroup waits for another) gives the
    oracle's dedup bit for bit at full size."""
    w = synth.workload(name)
    b = synth.make_batch(w, 2, with_grad=False)
    _say(f"case unique_ids_concurrent {name} N={len(b.indices)}")
    _dedup_concurrent_vs_oracle(w.row_offset, w.bags_per_table, b.offsets, b.indices, w.num_bags)


@pytest.mark.parametrize("case", ["empty", "one", "same", "tables"])
def test_unique_ids_concurrent_edge_cases(case):
    rng = np.random.default_rng(5)
    if case == "empty":
        rows, B = [100], 8
        off, idx = np.zeros(B + 1, np.int32), np.zeros(0, np.int32)
    elif case == "one":
        rows, B = [1000], 1
        off, idx = np.array([0, 1], np.int32), np.array([999], np.int32)
    elif case == "same":
        rows, B = [1 << 20], 2000
        lens = rng.integers(1, 60, size=B)
        off = np.concatenate([[0], np.cumsum(lens)]).astype(np.int32)
        idx = np.full(int(off[-1]), 123457, np.int32)
    else:
        rows, B = [37, 100_000, 1, 5_000_000], 3000
        off, idx = _rand_batch(rng, rows, B, 40, empty_frac=0.1, zipf=1.3)
    _say(f"case unique_ids_concurrent edge {case}")
    _dedup_concurrent_vs_oracle(_row_offset(rows), B, off, idx, len(rows) * B)


def test_workspace_shared_by_both_dedups_and_all_sizes():
    """One workspace serves both dedups and batches of very different sizes,
    in any order: co-resident passes after wait-free ones (whose plain tile
    counts must never sit where the co-resident passes poll call-tagged
    words) and small batches after large ones (whose arrays must never sit
    where a smaller batch's tagged words go).  Every dedup, and the unfused
    gradient reduce that follows it on the same workspace, matches the
    oracle, and no call reports an error."""
    import oracle
    import torch
    import paper_2112_02752_amd as emb
    dev = "cuda"
    D = 64
    rng = np.random.default_rng(11)
    small_rows, small_B = [1000, 50_000], 300
    cases = []
    for name, seed, concurrent in [("c3", 0, True), ("c3", 1, False), ("c5", 0, False), ("small", 0, False),
                                   ("c3", 2, False), ("c3", 3, True), ("c3", 6, False), ("c2", 0, False),
                                   ("small", 1, True), ("c3", 4, False), ("c2", 1, True), ("c3", 5, False)]:
        if name == "small":
            off, idx = _rand_batch(rng, small_rows, small_B, 30, empty_frac=0.05, zipf=1.2)
            G = rng.standard_normal((len(off) - 1, D)).astype(np.float32)
            cases.append((name, concurrent, _row_offset(small_rows), small_B, off, idx, G, "sum"))
        else:
            w = synth.workload(name)
            assert w.dim == D
            b = synth.make_batch(w, seed)
            cases.append((name, concurrent, w.row_offset, w.bags_per_table, b.offsets, b.indices, b.grad, w.pool))
    N = max(len(c[5]) for c in cases)
    M = max(len(c[4]) - 1 for c in cases)
    bufs = emb.DedupBuffers(dev, N, M, D)
    Wd = torch.empty((1, D), dtype=torch.float32, device=dev)  # never read: no update here
    gr = torch.zeros((N, D), dtype=torch.float32, device=dev)
    for k, (name, concurrent, ro, B, off, idx, G, pool) in enumerate(cases):
        n = len(idx)
        _say(f"case shared workspace call {k}: {name} N={n} concurrent={concurrent}")
        tables = emb.Tables(Wd, [int(x) for x in ro])
        b = emb.Batch(torch.from_numpy(np.ascontiguousarray(off, np.int32)).to(dev),
                      torch.from_numpy(np.ascontiguousarray(idx, np.int32)).to(dev), B)
        Gd = torch.from_numpy(G).to(dev)
        emb.unique_ids(tables, b, bufs.unique_keys, bufs.counts, bufs.seg_offsets, bufs.sort_perm, bufs.num_unique,
                       bufs.ws, concurrent=concurrent)
        emb.grad_reduce(tables, b, pool, Gd, bufs.sort_perm, bufs.seg_offsets, bufs.unique_keys, bufs.num_unique,
                        bufs.ws, grad_rows=gr)
        torch.cuda.synchronize()
        assert emb.read_status(bufs.ws)[0] == 0, f"call {k} ({name}) reported an error"
        ref = oracle.unique_ids(len(ro) - 1, np.asarray(ro, np.int64), B, np.ascontiguousarray(off, np.int32),
                                np.ascontiguousarray(idx, np.int32))
        U = int(bufs.num_unique.cpu().item())
        assert U == ref.num_unique, f"call {k} ({name})"
        np.testing.assert_array_equal(bufs.unique_keys[:U].cpu().numpy().view(np.uint32), ref.unique_keys)
        np.testing.assert_array_equal(bufs.counts[:U].cpu().numpy(), ref.counts)
        np.testing.assert_array_equal(bufs.seg_offsets[:U + 1].cpu().numpy(), ref.seg_offsets)
        np.testing.assert_array_equal(bufs.sort_perm[:n].cpu().numpy(), ref.perm)
        o_gr, _ = oracle.grad_reduce(len(ro) - 1, B, np.ascontiguousarray(off, np.int32), G, pool, ref)
        r = parity.rel_rownorm(gr[:U].cpu().numpy(), o_gr)
        assert r <= parity.TOL_FP32, f"call {k} ({name}): gradient rows rel err {r}"


def _batched_case(case):
    """(row_offset, dim, [(offsets, indices, bags_per_table)]) of a group."""
    rng = np.random.default_rng(17)
    if case in ("c3x6", "c3x1", "c3x2_int64"):
        w = synth.workload("c3")
        k = {"c3x6": 6, "c3x1": 1, "c3x2_int64": 2}[case]
        bs = [synth.make_batch(w, s, with_grad=False) for s in range(k)]
        dt = np.int64 if case.endswith("int64") else np.int32
        return w.row_offset, w.dim, [(b.offsets, b.indices.astype(dt), w.bags_per_table) for b in bs]
    if case == "c2_mixed":
        w = synth.workload("c2")
        bs = [synth.make_batch(w, s, with_grad=False) for s in range(3)]
        out = [(b.offsets, b.indices, w.bags_per_table) for b in bs]
        B = 4
        out.insert(1, (np.zeros(w.num_tables * B + 1, np.int32), np.zeros(0, np.int32), B))  # every bag empty
        one = np.zeros(w.num_tables * B + 1, np.int32)
        one[B * 3 + 2:] = 1  # one id, in bag 13 (the second bag of table 3)
        out.append((one, np.array([w.row_offset[4] - w.row_offset[3] - 1], np.int32), B))
        return w.row_offset, w.dim, out
    if case == "k16":
        rows = [1 << 20]
        out = []
        for i in range(16):
            off, idx = _rand_batch(rng, rows, 200 + 37 * i, 40, empty_frac=0.05, zipf=1.2)
            out.append((off, idx, 200 + 37 * i))
        return _row_offset(rows), 16, out
    raise ValueError(case)


@pytest.mark.parametrize("case", ["c3x6", "c3x1", "c3x2_int64", "c2_mixed", "k16"])
def test_unique_ids_batched_matches_single(case):
    """emb_unique_ids_batched leaves in every batch's buffers, bit for bit,
    what that batch's own emb_unique_ids leaves: the outputs, and (through
    the unfused gradient reduce that reads them) the bag ids, chunk map and
    call record in its workspace; twice in a row on the same workspaces, the
    batches' order reversed the second time.  The first batch of the first
    call is also checked against the oracle."""
    import oracle
    import torch
    import paper_2112_02752_amd as emb
    _say(f"case unique_ids_batched {case}")
    ro, D, group = _batched_case(case)
    dev = "cuda"
    tables = emb.Tables(torch.empty((1, D), dtype=torch.float32, device=dev), [int(x) for x in ro])
    T = len(ro) - 1
    bt = [emb.Batch(torch.from_numpy(np.ascontiguousarray(o, np.int32)).to(dev), torch.from_numpy(i).to(dev), B)
          for o, i, B in group]
    Ns = [len(i) for _, i, _ in group]
    Ms = [len(o) - 1 for o, _, _ in group]
    rng = np.random.default_rng(3)
    grads = [torch.from_numpy(rng.standard_normal((m, D)).astype(np.float32)).to(dev) for m in Ms]
    nmax, mmax = max(max(Ns), 1), max(Ms)
    sets_b = [emb.DedupBuffers(dev, nmax, mmax, D) for _ in group]
    sets_s = [emb.DedupBuffers(dev, nmax, mmax, D) for _ in group]
    gws = torch.empty(emb.workspace_size(max(sum(Ns), 1), sum(Ms), D), dtype=torch.uint8, device=dev)
    emb.workspace_init(gws)
    gr_b = torch.zeros((nmax, D), dtype=torch.float32, device=dev)
    gr_s = torch.zeros((nmax, D), dtype=torch.float32, device=dev)
    pool = "sum"
    for rnd, order in enumerate((list(range(len(group))), list(reversed(range(len(group)))))):
        emb.unique_ids_batched(tables, [bt[i] for i in order], [sets_b[i] for i in order], gws)
        for i in order:
            emb.unique_ids(tables, bt[i], sets_s[i].unique_keys, sets_s[i].counts, sets_s[i].seg_offsets,
                           sets_s[i].sort_perm, sets_s[i].num_unique, sets_s[i].ws)
        torch.cuda.synchronize()
        for i in order:
            n = Ns[i]
            a, b = sets_b[i], sets_s[i]
            assert emb.read_status(a.ws)[0] == 0, (rnd, i)
            U = int(b.num_unique.cpu().item())
            assert int(a.num_unique.cpu().item()) == U, (rnd, i)
            np.testing.assert_array_equal(a.unique_keys[:U].cpu().numpy(), b.unique_keys[:U].cpu().numpy())
            np.testing.assert_array_equal(a.counts[:U].cpu().numpy(), b.counts[:U].cpu().numpy())
            np.testing.assert_array_equal(a.seg_offsets[:U + 1].cpu().numpy(), b.seg_offsets[:U + 1].cpu().numpy())
            np.testing.assert_array_equal(a.sort_perm[:n].cpu().numpy(), b.sort_perm[:n].cpu().numpy())
            if n == 0:
                continue
            for sset, gr in ((a, gr_b), (b, gr_s)):
                emb.grad_reduce(tables, bt[i], pool, grads[i], sset.sort_perm, sset.seg_offsets, sset.unique_keys,
                                sset.num_unique, sset.ws, grad_rows=gr)
            torch.cuda.synchronize()
            np.testing.assert_array_equal(gr_b[:U].cpu().numpy(), gr_s[:U].cpu().numpy())
            if rnd == 0 and i == 0:
                o, idx, B = group[0]
                ref = oracle.unique_ids(T, np.asarray(ro, np.int64), B, np.ascontiguousarray(o, np.int32),
                                        np.ascontiguousarray(idx, np.int32))
                assert U == ref.num_unique
                np.testing.assert_array_equal(a.unique_keys[:U].cpu().numpy().view(np.uint32), ref.unique_keys)
                np.testing.assert_array_equal(a.sort_perm[:n].cpu().numpy(), ref.perm)


# ------------------------------------------------------------------ routing

def _route_gpu(row_offset, B, off, idx, shard, W_dev=None, idx64=False):
    import torch
    import paper_2112_02752_amd as emb
    N, M = len(idx), len(off) - 1
    Wr = len(shard) - 1
    dev = "cuda"
    if W_dev is None:
        W_dev = torch.empty((int(row_offset[-1]), 4), dtype=torch.float32, device=dev)  # never read
    tables = emb.Tables(W_dev, [int(x) for x in row_offset])
    b = emb.Batch(torch.from_numpy(np.ascontiguousarray(off, np.int32)).to(dev),
                  torch.from_numpy(np.ascontiguousarray(idx, np.int64 if idx64 else np.int32)).to(dev), B)
    i32 = dict(dtype=torch.int32, device=dev)
    cnt = torch.full((Wr,), -1, **i32)
    ids, pos, bag = (torch.full((max(N, 1),), -1, **i32) for _ in range(3))
    ws = torch.empty(emb.route_workspace_size(N, M, Wr), dtype=torch.uint8, device=dev)
    emb.route_ids(tables, b, shard, cnt, ids, pos, bag, ws)
    torch.cuda.synchronize()
    return cnt.cpu().numpy(), ids[:N].cpu().numpy(), pos[:N].cpu().numpy(), bag[:N].cpu().numpy()


def _check_route(row_offset, B, off, idx, shard, idx64=False):
    import oracle
    T = len(row_offset) - 1
    ref = oracle.route_ids(T, np.asarray(row_offset, np.int64), B, np.ascontiguousarray(off, np.int32),
                           np.ascontiguousarray(idx, np.int32), np.asarray(shard, np.int64))
    cnt, ids, pos, bag = _route_gpu(row_offset, B, off, idx, shard, idx64=idx64)
    np.testing.assert_array_equal(cnt, ref.send_counts)
    np.testing.assert_array_equal(pos, ref.send_pos)
    np.testing.assert_array_equal(ids, ref.send_ids)
    np.testing.assert_array_equal(bag, ref.send_bag)


@pytest.mark.parametrize("Wr,seed", [(1, 0), (3, 1), (8, 2), (64, 3), (256, 4)])
def test_route_small(Wr, seed):
    """Random bounds (some ranges empty) over three tables, empty bags."""
    _say(f"case route W={Wr}")
    rng = np.random.default_rng(100 + seed)
    rows = [5000, 800, 12000]
    B = 700
    off, idx = _rand_batch(rng, rows, B, 40, empty_frac=0.1, zipf=1.2)
    R = sum(rows)
    cuts = np.sort(rng.integers(0, R + 1, size=Wr - 1))
    shard = [0] + [int(x) for x in cuts] + [R]
    _check_route(_row_offset(rows), B, off, idx, shard)


def test_route_int64_indices():
    _say("case route int64 ids")
    rng = np.random.default_rng(9)
    rows = [5000, 800, 12000]
    B = 700
    off, idx = _rand_batch(rng, rows, B, 40, empty_frac=0.1, zipf=1.2)
    R = sum(rows)
    _check_route(_row_offset(rows), B, off, idx, [0, 3000, 9000, 15000, R], idx64=True)


def test_route_tablewise_and_empty_batch():
    _say("case route table-wise / empty batch")
    rng = np.random.default_rng(7)
    rows = [300, 5, 9000, 40]
    B = 500
    off, idx = _rand_batch(rng, rows, B, 20, empty_frac=0.3)
    ro = _row_offset(rows)
    _check_route(ro, B, off, idx, [int(x) for x in ro])
    off0 = np.zeros(len(rows) * B + 1, np.int32)
    cnt, _, _, _ = _route_gpu(ro, B, off0, np.zeros(0, np.int32), [0, 1000, int(ro[-1])])
    np.testing.assert_array_equal(cnt, [0, 0])


@pytest.mark.parametrize("name,Wr", [("c3", 8), ("c5", 8), ("c4", 0)])
def test_route_full_size(name, Wr):
    """Full-size batches: equal row ranges over Wr ranks, or (Wr = 0) one rank
    per table."""
    w = synth.workload(name)
    _say(f"case route full size {name} W={Wr or w.num_tables}")
    b = synth.make_batch(w, 0)
    R = w.total_rows
    shard = [int(x) for x in w.row_offset] if Wr == 0 else [R * r // Wr for r in range(Wr + 1)]
    _check_route(w.row_offset, w.bags_per_table, b.offsets, b.indices, shard)


@pytest.mark.parametrize("pool", ["sum", "mean"])
def test_route_fragments_reassemble_forward_on_gpu(pool):
    """The sharded forward on one GPU: each rank pools its fragments from its
    own slice of the table with emb_pool_fwd (sum), the fragments' rows are
    added by bag (and scaled by 1 / bag length for mean pooling); the result
    equals the unsharded forward within the fp32 tolerance."""
    _say(f"case route reassemble pool={pool}")
    import torch
    import paper_2112_02752_amd as emb
    w = synth.scaled(synth.workload("c3"), rows_div=100, bags_div=4, name="c3-small")
    b = synth.make_batch(w, 0)
    dl = parity.device_layer_from_workload(w)
    R = w.total_rows
    shard = [R * r // 8 for r in range(9)]
    cnt, ids, pos, bag = _route_gpu(w.row_offset, w.bags_per_table, b.offsets, b.indices, shard, W_dev=dl.W)
    M = w.num_bags
    full = torch.empty((M, w.dim), dtype=torch.float32, device="cuda")
    emb.pool_fwd(dl.tables, emb.Batch(torch.from_numpy(b.offsets).cuda(), torch.from_numpy(b.indices).cuda(),
                                      w.bags_per_table), pool, full)
    acc = np.zeros((M, w.dim), np.float64)
    k0 = 0
    for r in range(8):
        k1 = k0 + int(cnt[r])
        fb = bag[k0:k1]
        heads = np.concatenate([[True], fb[1:] != fb[:-1]]) if k1 > k0 else np.zeros(0, bool)
        foff = np.concatenate([np.nonzero(heads)[0], [k1 - k0]]).astype(np.int32)
        nf = len(foff) - 1
        if nf > 0:
            local = emb.Tables(dl.W[shard[r]:shard[r + 1]], [0, shard[r + 1] - shard[r]])
            part = torch.empty((nf, w.dim), dtype=torch.float32, device="cuda")
            emb.pool_fwd(local, emb.Batch(torch.from_numpy(foff).cuda(),
                                          torch.from_numpy(np.ascontiguousarray(ids[k0:k1])).cuda(), nf),
                         "sum", part)
            np.add.at(acc, fb[foff[:-1]], part.cpu().numpy())
        k0 = k1
    if pool == "mean":
        L = np.diff(b.offsets)
        acc[L > 0] /= L[L > 0, None]
    r = parity.rel_rownorm(acc, full.cpu().numpy())
    assert r <= parity.TOL_FP32, f"reassembled forward rel err {r}"
