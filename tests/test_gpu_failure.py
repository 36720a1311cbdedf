"""The per-call failure path of the dedup on the GPU.

A dedup call whose bounded waits give up must write no table or state row,
be reported to the caller (Layer.check raises StepFailed), and leave the next
call on the workspace unaffected.  The error bits of the coming call are set
from the host before it runs, through the workspace header's documented
layout (uint32 generation at offset 0, uint64 error word (generation << 32) |
bits at emb_workspace_error_offset()), so every bounded wait of that call
gives up at its first check of them and every kernel still exits normally:
no wait is made to run out for real.  Every write of such a call stays inside
the caller's buffers (scatters are guarded by the batch size, the unique scan
returns before indexing with anything the sort wrote)."""
import dataclasses
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


def _preset_failure(ws):
    """Set bit 0 (a wait ran out) among the error bits of the next dedup call
    on workspace ``ws``."""
    import torch
    import paper_2112_02752_amd as emb
    gen = int(ws[0:4].cpu().numpy().view(np.uint32)[0])
    g = 1 if gen == 0xFFFFFFFF else gen + 1
    word = np.array([(g << 32) | 1], dtype=np.uint64).view(np.uint8)
    eo = emb.workspace_error_offset()
    ws[eo:eo + 8].copy_(torch.from_numpy(word.copy()).to(ws.device))


def _batch(w, s):
    import torch
    import paper_2112_02752_amd as emb
    b = synth.make_batch(w, s)
    return b, emb.Batch(torch.from_numpy(b.offsets).cuda(), torch.from_numpy(b.indices).cuda(), w.bags_per_table), \
        torch.from_numpy(b.grad).cuda()


@pytest.mark.parametrize("name,bags_mult", [("c3", 1), ("c3", 8)])
def test_failed_dedup_writes_nothing_and_is_reported(name, bags_mult):
    """Full 50M-row table: a step whose dedup fails leaves the table and the
    Adagrad state bit-identical and reports num_unique = 0 and the failure;
    the next step is correct and clean; emb_workspace_init clears the record.
    bags_mult 8 gives batches of about 3.9M lookups, whose sort runs the
    reduce-then-scan passes (no waits) and whose unique scan runs its
    reduce-then-scan route too."""
    import torch
    import oracle
    import paper_2112_02752_amd as emb
    w = synth.workload(name)
    if bags_mult > 1:
        w = dataclasses.replace(w, name=f"{name}-bags-x{bags_mult}", bags_per_table=w.bags_per_table * bags_mult)
    _say(f"case failed dedup {w.name}: rows={w.total_rows} bags={w.num_bags}")
    dl = parity.device_layer_from_workload(w)
    (b0, db0, g0), (b1, db1, g1) = _batch(w, 0), _batch(w, 1)
    nmax = max(len(b0.indices), len(b1.indices))
    layer = emb.Layer(dl.tables, w.pool, w.opt, w.lr, w.eps, dl.state, max_indices=nmax, max_bags=w.num_bags)
    W0, S0 = dl.W.clone(), dl.state.clone()
    out = torch.empty((w.num_bags, w.dim), dtype=torch.float32, device="cuda")
    _preset_failure(layer.ws)
    layer.step(db0, out, g0)
    torch.cuda.synchronize()
    _say("  failed step returned")
    assert int(layer.num_unique.cpu().item()) == 0
    assert torch.equal(dl.W, W0), "a failed step wrote table rows"
    assert torch.equal(dl.state, S0), "a failed step wrote optimizer state"
    bits, site, block, timeouts = layer.status()
    assert bits & 1, (bits, site, block, timeouts)
    # co-resident sort passes: a wait that kept finding a word not yet
    # published gave up at its check of the error bits and was recorded
    # (whether any wait retries that long depends on timing: the published
    # words may all be there in time)
    assert (site != 0) == (timeouts > 0), (bits, site, block, timeouts)
    _say(f"  recorded waits that gave up: {timeouts} (first site {site:#x})")
    with pytest.raises(emb.StepFailed):
        layer.check()
    # the next call starts afresh: correct against the oracle, status clean
    g = parity.gpu_step(dl, b1.offsets, b1.indices, b1.grad, w.bags_per_table, w.pool, w.opt, w.lr, w.eps,
                        layer=layer)
    keys = parity.global_keys(w.row_offset, w.bags_per_table, b1.offsets, b1.indices)
    touched = np.unique(keys)
    store = oracle.RowStore(synth.weight_rows(w, touched), keys=touched.astype(np.uint32),
                            state=np.zeros(len(touched), np.float32))
    o_out, o_dd, o_gr = oracle.step(w.num_tables, w.row_offset, w.bags_per_table, b1.offsets, b1.indices, b1.grad,
                                    store, w.pool, w.opt, w.lr, w.eps)
    parity.check_against_oracle(g, o_out, o_dd, o_gr)
    parity.check_rows(dl, store, o_dd.unique_keys, w.opt)
    layer.check()
    assert layer.status()[0] == 0
    # the record of the timed-out waits stays until the workspace is initialised again
    assert layer.status()[3] == timeouts
    emb.workspace_init(layer.ws)
    assert layer.status() == (0, 0, 0, 0)
    _say("  ok")


def test_failed_dedup_unfused_path():
    """Unfused: the reduce after a failed dedup forms no gradient rows for the
    update and emb_sparse_update then changes nothing."""
    import torch
    import paper_2112_02752_amd as emb
    w = synth.scaled(synth.workload("c3"), rows_div=100, bags_div=4, name="c3-small")
    _say(f"case failed dedup unfused {w.name}")
    dl = parity.device_layer_from_workload(w)
    b, db, g = _batch(w, 0)
    N = len(b.indices)
    layer = emb.Layer(dl.tables, w.pool, w.opt, w.lr, w.eps, dl.state, max_indices=N, max_bags=w.num_bags)
    W0, S0 = dl.W.clone(), dl.state.clone()
    grad_rows = torch.full((N, w.dim), 7.0, dtype=torch.float32, device="cuda")
    _preset_failure(layer.ws)
    emb.unique_ids(dl.tables, db, layer.unique_keys, layer.counts, layer.seg_offsets, layer.sort_perm,
                   layer.num_unique, layer.ws)
    emb.grad_reduce(dl.tables, db, w.pool, g, layer.sort_perm, layer.seg_offsets, layer.unique_keys,
                    layer.num_unique, layer.ws, grad_rows=grad_rows)
    emb.sparse_update(dl.tables, w.opt, w.lr, w.eps, dl.state, layer.unique_keys, layer.num_unique, N, grad_rows)
    torch.cuda.synchronize()
    assert int(layer.num_unique.cpu().item()) == 0
    assert torch.equal(dl.W, W0)
    assert torch.equal(dl.state, S0)
    assert layer.status()[0] & 1
    with pytest.raises(emb.StepFailed):
        layer.check()
    _say("  ok")


@pytest.mark.parametrize("group_dedup", [True, False])
def test_failed_dedup_in_pipeline_is_reported(group_dedup):
    """The pipelined schedule: a failure preset in one buffer set's workspace
    makes that step write nothing and Pipeline.check raise; the other steps
    of the run equal serial steps of the same batches minus the failed one
    (with each group's dedups as one batched call, and one call per batch)."""
    import torch
    import paper_2112_02752_amd as emb
    w = synth.scaled(synth.workload("c3"), rows_div=500, bags_div=8, name="c3-small")
    _say(f"case failed dedup in pipeline {w.name} group dedup={group_dedup}")
    bs = [_batch(w, s) for s in range(4)]
    nmax = max(len(b.indices) for b, _, _ in bs)
    dl_p = parity.device_layer_from_workload(w)
    pipe = emb.Pipeline(dl_p.tables, w.pool, w.opt, w.lr, w.eps, dl_p.state, max_indices=nmax,
                        max_bags=w.num_bags, group=2, side_streams=1, group_dedup=group_dedup)
    # set index of step 1 in the first group is 1
    _preset_failure(pipe.sets[1].ws)
    outs = [torch.empty((w.num_bags, w.dim), dtype=torch.float32, device="cuda") for _ in bs]
    pipe.run([(db, o, g) for (_, db, g), o in zip(bs, outs)])
    torch.cuda.synchronize()
    with pytest.raises(emb.StepFailed):
        pipe.check()
    dl_s = parity.device_layer_from_workload(w)
    layer = emb.Layer(dl_s.tables, w.pool, w.opt, w.lr, w.eps, dl_s.state, max_indices=nmax, max_bags=w.num_bags)
    for k, (_, db, g) in enumerate(bs):
        o = torch.empty((w.num_bags, w.dim), dtype=torch.float32, device="cuda")
        if k == 1:
            layer.forward(db, o)  # the failed step still pooled its batch, but updated nothing
        else:
            layer.step(db, o, g)
        torch.cuda.synchronize()
        assert torch.equal(o, outs[k]), f"pooled output of step {k}"
    assert torch.equal(dl_s.W, dl_p.W)
    assert torch.equal(dl_s.state, dl_p.state)
    _say("  ok")


def test_failed_group_dedup_reaches_every_batch():
    """A failure preset in a group dedup's own workspace (the error bits of its
    next call) becomes every batch's: each batch's fused gradient reduce
    writes nothing and each set reports the failure; the next group call on
    the same workspaces is clean and every batch's step then equals a serial
    step of it."""
    import torch
    import paper_2112_02752_amd as emb
    w = synth.scaled(synth.workload("c3"), rows_div=500, bags_div=8, name="c3-small")
    _say(f"case failed group dedup {w.name}")
    bs = [_batch(w, s) for s in range(3)]
    nmax = max(len(b.indices) for b, _, _ in bs)
    dl = parity.device_layer_from_workload(w)
    sets = [emb.DedupBuffers("cuda", nmax, w.num_bags, w.dim) for _ in bs]
    gws = torch.empty(emb.workspace_size(3 * nmax, 3 * w.num_bags, w.dim), dtype=torch.uint8, device="cuda")
    emb.workspace_init(gws)

    def steps():
        emb.unique_ids_batched(dl.tables, [db for _, db, _ in bs], sets, gws)
        for (_, db, g), d in zip(bs, sets):
            emb.grad_reduce(dl.tables, db, w.pool, g, d.sort_perm, d.seg_offsets, d.unique_keys, d.num_unique, d.ws,
                            opt=w.opt, lr=w.lr, eps=w.eps, state=dl.state)
        torch.cuda.synchronize()

    W0, S0 = dl.W.clone(), dl.state.clone()
    _preset_failure(gws)
    steps()
    assert torch.equal(dl.W, W0)
    assert torch.equal(dl.state, S0)
    for d in sets:
        assert emb.read_status(d.ws)[0] & 1
        assert int(d.num_unique.cpu().item()) == 0
    steps()
    for d in sets:
        assert emb.read_status(d.ws)[0] == 0
    dl_s = parity.device_layer_from_workload(w)
    layer = emb.Layer(dl_s.tables, w.pool, w.opt, w.lr, w.eps, dl_s.state, max_indices=nmax, max_bags=w.num_bags)
    for _, db, g in bs:
        layer.backward(db, g)
    torch.cuda.synchronize()
    assert torch.equal(dl_s.W, dl.W)
    assert torch.equal(dl_s.state, dl.state)
    _say("  ok")
