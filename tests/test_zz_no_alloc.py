"""emb_route_ids_noalloc (the routing call for callers that cannot allocate:
its per-block counts live in the library's per-device scratch array) against
emb_route_ids on the same inputs, bit for bit, on two calls in a row, the
second with a smaller batch, and its host-side rejection of a batch whose
counts do not fit the array."""
import sys

import numpy as np
import pytest

import synth

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


def _route_both(w, step, Wr):
    import torch
    import paper_2112_02752_amd as emb
    b = synth.make_batch(w, step, with_grad=False)
    N, M = len(b.indices), w.num_bags
    dev = "cuda"
    # the routing never reads the table; a one-row stand-in carries its layout
    tables = emb.Tables(torch.empty((1, 4), dtype=torch.float32, device=dev), [int(x) for x in w.row_offset])
    db = emb.Batch(torch.from_numpy(b.offsets).to(dev), torch.from_numpy(b.indices).to(dev), w.bags_per_table)
    shard = [w.total_rows * r // Wr for r in range(Wr + 1)]
    assert emb.route_workspace_size(N, M, Wr) <= emb.ROUTE_SCRATCH_BYTES
    i32 = dict(dtype=torch.int32, device=dev)
    outs = []
    for noalloc in (False, True):
        cnt = torch.full((Wr,), -1, **i32)
        ids, pos, bag = (torch.full((N,), -1, **i32) for _ in range(3))
        if noalloc:
            emb.route_ids_noalloc(tables, db, shard, cnt, ids, pos, bag)
        else:
            ws = torch.empty(emb.route_workspace_size(N, M, Wr), dtype=torch.uint8, device=dev)
            emb.route_ids(tables, db, shard, cnt, ids, pos, bag, ws)
        torch.cuda.synchronize()
        outs.append([t.cpu().numpy() for t in (cnt, ids, pos, bag)])
    for a, b2 in zip(*outs):
        np.testing.assert_array_equal(a, b2)
    assert int(outs[0][0].sum()) == N
    return N


def test_noalloc_route_matches_route_ids_twice():
    """A 50M-row batch of 491k ids over 8 ranks, then a smaller one (4096 bags,
    about 123k ids, over 3 ranks) on the same scratch array."""
    w = synth.workload("c3")
    _say("case noalloc route: c3 batch, 8 ranks")
    n1 = _route_both(w, 0, 8)
    w2 = synth.scaled(w, bags_div=4, name="c3-b4096")
    _say("case noalloc route: smaller batch, 3 ranks")
    n2 = _route_both(w2, 1, 3)
    assert n2 < n1


def test_noalloc_route_rejects_batches_beyond_the_array():
    """A batch whose per-block counts exceed the 4 MiB array is rejected on the
    host with EMB_EUNSUPPORTED; nothing is enqueued."""
    import ctypes
    import torch
    import paper_2112_02752_amd as emb
    w = synth.workload("c5")   # 3.3M ids in 65536 bags: 13108 blocks of counts per rank
    b = synth.make_batch(w, 0, with_grad=False)
    N, M = len(b.indices), w.num_bags
    Wr = 256
    assert emb.route_workspace_size(N, M, Wr) > emb.ROUTE_SCRATCH_BYTES
    dev = "cuda"
    # the routing never reads the table; a one-row stand-in carries its layout
    tables = emb.Tables(torch.empty((1, 4), dtype=torch.float32, device=dev), [int(x) for x in w.row_offset])
    db = emb.Batch(torch.from_numpy(b.offsets).to(dev), torch.from_numpy(b.indices).to(dev), w.bags_per_table)
    shard = (ctypes.c_int64 * (Wr + 1))(*[w.total_rows * r // Wr for r in range(Wr + 1)])
    i32 = dict(dtype=torch.int32, device=dev)
    cnt = torch.full((Wr,), -7, **i32)
    ids = torch.full((N,), -7, **i32)
    st = emb.lib().emb_route_ids_noalloc(ctypes.byref(tables.c()), ctypes.byref(db.c()), Wr, shard, cnt.data_ptr(),
                                          ids.data_ptr(), ids.data_ptr(), ids.data_ptr(), None)
    assert st == emb.EMB_EUNSUPPORTED
    torch.cuda.synchronize()
    assert int(cnt.min().item()) == -7 and int(cnt.max().item()) == -7
