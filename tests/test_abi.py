"""The C ABI library without a GPU: it loads, exports every entry point the
header declares, sizes workspaces, and rejects bad arguments synchronously
(host checks run before anything touches the GPU)."""
import ctypes
import os
import re

import pytest

import paper_2112_02752_amd as emb

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "emb.h")


def declared_functions():
    src = open(HEADER).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(emb_[a-z_]+)\s*\(", src)))


def test_header_declares_the_boundary():
    names = declared_functions()
    for fn in ("emb_pool_fwd", "emb_unique_ids", "emb_grad_reduce", "emb_sparse_update"):
        assert fn in names
    assert set(names) == set(emb.EXPORTED)


def test_library_exports_every_declared_symbol():
    L = emb.lib()
    for fn in declared_functions():
        assert hasattr(L, fn), fn
        assert getattr(L, fn) is not None


def test_status_strings():
    for st in range(5):
        assert emb.lib().emb_status_string(st).decode()
    assert emb.lib().emb_status_string(99).decode() == "unknown status"


def test_workspace_size_monotone_and_invalid():
    a = emb.workspace_size(1000, 100, 64)
    b = emb.workspace_size(100_000, 100, 64)
    c = emb.workspace_size(100_000, 100, 128)
    assert 0 < a < b < c
    assert a % 256 == 0
    assert emb.workspace_size(-1, 1, 64) == 0
    assert emb.workspace_size(1 << 30, 1, 64) == 0
    assert emb.workspace_size(10, 1, 0) == 0
    assert emb.workspace_size(0, 0, 16) > 0


def _tables(row_offset=(0, 100), dim=16, dtype=0, weights=0x1000):
    ro = (ctypes.c_int64 * len(row_offset))(*row_offset)
    t = emb.CTables(len(row_offset) - 1, ro, dim, dtype, weights)
    t._keep = ro
    return t


def _batch(B=4, offsets=0x2000, indices=0x3000, n=10):
    return emb.CBatch(B, offsets, indices, n)


def call_fwd(t, b, pool=0, out=0x4000):
    return emb.lib().emb_pool_fwd(ctypes.byref(t), ctypes.byref(b), pool, out, None)


def test_fwd_argument_errors():
    assert call_fwd(_tables(weights=None), _batch()) == emb.EMB_EINVAL
    assert call_fwd(_tables(dim=3), _batch()) == emb.EMB_EUNSUPPORTED        # 12-byte rows
    assert call_fwd(_tables(dim=4, dtype=1), _batch()) == emb.EMB_EUNSUPPORTED  # 8-byte bf16 rows
    assert call_fwd(_tables(dtype=7), _batch()) == emb.EMB_EINVAL
    assert call_fwd(_tables(row_offset=(0, 1 << 32)), _batch()) == emb.EMB_EUNSUPPORTED
    assert call_fwd(_tables(row_offset=(1, 10)), _batch()) == emb.EMB_EINVAL
    assert call_fwd(_tables(row_offset=(0, 10, 5)), _batch()) == emb.EMB_EINVAL
    assert call_fwd(_tables(weights=0x1008), _batch()) == emb.EMB_EINVAL      # not 16-byte aligned
    assert call_fwd(_tables(), _batch(offsets=None)) == emb.EMB_EINVAL
    assert call_fwd(_tables(), _batch(B=-1)) == emb.EMB_EINVAL
    assert call_fwd(_tables(), _batch(n=1 << 30)) == emb.EMB_EUNSUPPORTED
    assert call_fwd(_tables(), _batch(indices=None)) == emb.EMB_EINVAL
    assert call_fwd(_tables(), _batch(), pool=2) == emb.EMB_EINVAL
    bad_width = _batch()
    bad_width.index_bytes = 2
    assert call_fwd(_tables(), bad_width) == emb.EMB_EINVAL
    assert call_fwd(_tables(), _batch(), out=None) == emb.EMB_EINVAL
    t = _tables()
    t.num_tables = 0
    assert call_fwd(t, _batch()) == emb.EMB_EINVAL
    many = _tables(row_offset=tuple(range(300)))
    assert call_fwd(many, _batch()) == emb.EMB_EUNSUPPORTED
    # an empty batch is valid and enqueues nothing
    assert call_fwd(_tables(), _batch(B=0, n=0, indices=None), out=None) == emb.EMB_OK


def test_unique_ids_workspace_errors():
    L = emb.lib()
    t, b = _tables(), _batch(n=1000)
    need = emb.workspace_size(1000, 4, 16)

    def call(ws=0x100000, nbytes=need, **kw):
        args = dict(uk=0x5000, cnt=0x6000, seg=0x7000, perm=0x8000, nu=0x9000)
        args.update(kw)
        return L.emb_unique_ids(ctypes.byref(t), ctypes.byref(b), args["uk"], args["cnt"], args["seg"],
                                args["perm"], args["nu"], ws, nbytes, None)

    assert call(nbytes=need - 1) == emb.EMB_EWORKSPACE
    assert call(ws=0x100010) == emb.EMB_EWORKSPACE  # not 256-byte aligned
    assert call(ws=None) == emb.EMB_EINVAL
    assert call(seg=None) == emb.EMB_EINVAL
    assert call(perm=None) == emb.EMB_EINVAL


def test_grad_reduce_argument_errors():
    L = emb.lib()
    t, b = _tables(), _batch(n=1000)
    need = emb.workspace_size(1000, 4, 16)
    bad_opt = emb.CUpdate(5, 0.1, 0.0, None)
    adagrad_no_state = emb.CUpdate(1, 0.1, 1e-8, None)

    def call(grad_rows=0xa000, fuse=None, pool=0, nbytes=need):
        f = ctypes.byref(fuse) if fuse is not None else None
        return L.emb_grad_reduce(ctypes.byref(t), ctypes.byref(b), pool, 0xb000, 0xc000, 0xd000, 0xe000, 0xf000,
                                 grad_rows, f, 0x100000, nbytes, None)

    assert call(grad_rows=None) == emb.EMB_EINVAL
    assert call(fuse=bad_opt) == emb.EMB_EINVAL
    assert call(fuse=adagrad_no_state) == emb.EMB_EINVAL
    assert call(pool=3) == emb.EMB_EINVAL
    assert call(nbytes=16) == emb.EMB_EWORKSPACE


def test_route_argument_errors():
    L = emb.lib()
    t, b = _tables(row_offset=(0, 100)), _batch(n=1000)
    need = emb.route_workspace_size(1000, 4, 4)
    assert need > 0
    assert emb.route_workspace_size(1000, 4, 0) == 0
    assert emb.route_workspace_size(1000, 4, 257) == 0

    def call(bounds=(0, 10, 50, 60, 100), nbytes=None, counts=0x5000, ids=0x6000):
        W = len(bounds) - 1
        ss = (ctypes.c_int64 * len(bounds))(*bounds)
        return L.emb_route_ids(ctypes.byref(t), ctypes.byref(b), W, ss, counts, ids, 0x7000, 0x8000, 0x100000,
                               need if nbytes is None else nbytes, None)

    assert call(bounds=(1, 50, 100)) == emb.EMB_EINVAL       # first bound not 0
    assert call(bounds=(0, 50, 99)) == emb.EMB_EINVAL        # last bound not R
    assert call(bounds=(0, 60, 50, 100)) == emb.EMB_EINVAL   # decreasing
    assert call(bounds=(0,)) == emb.EMB_EINVAL               # no rank
    assert call(counts=None) == emb.EMB_EINVAL
    assert call(ids=None) == emb.EMB_EINVAL
    assert call(nbytes=need - 1) == emb.EMB_EWORKSPACE


def test_sparse_update_argument_errors():
    L = emb.lib()
    t = _tables()
    ok = emb.CUpdate(0, 0.1, 0.0, None)
    assert L.emb_sparse_update(ctypes.byref(t), ctypes.byref(ok), None, 0x1, 10, 0x2, None) == emb.EMB_EINVAL
    assert L.emb_sparse_update(ctypes.byref(t), ctypes.byref(ok), 0x1, 0x1, -1, 0x2, None) == emb.EMB_EINVAL
    assert L.emb_sparse_update(ctypes.byref(t), ctypes.byref(ok), None, None, 0, None, None) == emb.EMB_OK
    big = _tables(dim=2048)
    assert L.emb_sparse_update(ctypes.byref(big), ctypes.byref(ok), 0x1, 0x1, 5, 0x2, None) == \
        emb.EMB_EUNSUPPORTED


def test_error_word_offset():
    # uint32 generation at 0, uint32 in-flight generation at 4, uint64 error word at 8
    assert emb.workspace_error_offset() == 8


def test_workspace_status_argument_checks():
    L = emb.lib()
    assert L.emb_workspace_status(None, 256, 0x100, None) == emb.EMB_EINVAL
    assert L.emb_workspace_status(0x1000, 256, None, None) == emb.EMB_EINVAL
    assert L.emb_workspace_status(0x1010, 256, 0x100, None) == emb.EMB_EWORKSPACE   # misaligned
    assert L.emb_workspace_status(0x1000, 255, 0x100, None) == emb.EMB_EWORKSPACE   # smaller than the header


def test_step_failed_message_names_the_wait():
    e = emb.StepFailed(1, 0x120, 17, 3)
    msg = str(e)
    assert "sort pass 2" in msg and "digit offsets" in msg and "workgroup 17" in msg and "3 waits" in msg
    assert "unique scan" in str(emb.StepFailed(1, 0x200, 5, 1))
    assert "inconsistent" in str(emb.StepFailed(2, 0, 0, 0))
    assert "combine" in str(emb.StepFailed(4, 0x300, 2, 1))


def test_binding_fails_loudly_without_library(monkeypatch, tmp_path):
    monkeypatch.setattr(emb, "LIB_PATH", str(tmp_path / "missing.so"))
    monkeypatch.setattr(emb, "_lib", None)
    with pytest.raises(RuntimeError, match="missing"):
        emb.lib()


def test_pipeline_steps_argument_checks():
    """Host checks of emb_pipeline_steps return before anything is enqueued."""
    L = emb.lib()
    t = _tables()
    upd = emb.CUpdate(0, 0.1, 0.0, None, 0, 0)
    b = (emb.CBatch * 1)(emb.CBatch(1, 0x1000, 0x2000, 10, 4))
    ptrs = (ctypes.c_void_p * 1)(0x3000)
    sets = (emb.CDedupSet * 2)()
    sides = (ctypes.c_void_p * 2)(0x10, 0x20)
    events = (ctypes.c_void_p * 7)(*([0x40] * 7))
    no_events = (ctypes.c_void_p * 7)(*([0x40] * 6 + [0]))
    def f(*a, group_ws=None, group_ws_bytes=0, group_base=0, primed=0, ahead=0, depth=2):
        return L.emb_pipeline_steps(*a, group_ws, group_ws_bytes, group_base, primed, ahead, depth)

    tb, ub = ctypes.byref(t), ctypes.byref(upd)
    assert f(tb, 0, ub, 0, b, ptrs, ptrs, 1, sets, None, 1, sides, events) == emb.EMB_OK   # nothing to do
    assert f(None, 0, ub, 1, b, ptrs, ptrs, 1, sets, None, 1, sides, events) == emb.EMB_EINVAL
    assert f(tb, 0, None, 1, b, ptrs, ptrs, 1, sets, None, 1, sides, events) == emb.EMB_EINVAL
    assert f(tb, 0, ub, -1, b, ptrs, ptrs, 1, sets, None, 1, sides, events) == emb.EMB_EINVAL
    assert f(tb, 0, ub, 1, b, ptrs, ptrs, 0, sets, None, 1, sides, events) == emb.EMB_EINVAL      # group 0
    assert f(tb, 0, ub, 1, b, ptrs, ptrs, 1, sets, None, 2, sides, events) == emb.EMB_EINVAL      # sides > group
    assert f(tb, 0, ub, 1, b, ptrs, ptrs, 2, sets, None, 0, sides, events) == emb.EMB_EINVAL      # no side stream
    many = (ctypes.c_void_p * 17)(*range(0x10, 0x10 + 17))
    ev17 = (ctypes.c_void_p * 37)(*([0x40] * 37))
    assert f(tb, 0, ub, 1, b, ptrs, ptrs, 17, sets, None, 17, many, ev17) == emb.EMB_EUNSUPPORTED  # > 16 sides
    assert f(tb, 0, ub, 1, None, ptrs, ptrs, 1, sets, None, 1, sides, events) == emb.EMB_EINVAL
    assert f(tb, 0, ub, 1, b, ptrs, ptrs, 1, None, None, 1, sides, events) == emb.EMB_EINVAL
    assert f(tb, 0, ub, 1, b, ptrs, ptrs, 2, sets, None, 2, sides, no_events) == emb.EMB_EINVAL   # a null event
    same = (ctypes.c_void_p * 2)(0x10, 0x77)
    assert f(tb, 0, ub, 1, b, ptrs, ptrs, 2, sets, 0x77, 2, same, events) == emb.EMB_EINVAL       # side == main

    # every step is checked before anything is enqueued: four steps in two
    # groups of two, the last one bad in turn (a valid list would go on to
    # enqueue, so it is not called here)
    n = 4
    wsb = L.emb_workspace_size(10, 1, t.dim)
    good = emb.CDedupSet(0x5000, 0x5100, 0x5200, 0x5300, 0x5400, 0x100000, wsb)
    sets4 = (emb.CDedupSet * 4)(*([good] * 4))
    b4 = (emb.CBatch * n)(*([emb.CBatch(1, 0x1000, 0x2000, 10, 4)] * n))
    outs4 = (ctypes.c_void_p * n)(*([0x3000] * n))
    grads4 = (ctypes.c_void_p * n)(*([0x3000] * n))
    no_grad = (ctypes.c_void_p * n)(*([0x3000] * (n - 1) + [0]))
    no_out = (ctypes.c_void_p * n)(*([0x3000] * (n - 1) + [0]))
    assert f(tb, 0, ub, n, b4, outs4, no_grad, 2, sets4, None, 1, sides, events) == emb.EMB_EINVAL
    assert f(tb, 0, ub, n, b4, no_out, grads4, 2, sets4, None, 1, sides, events) == emb.EMB_EINVAL
    assert f(tb, 7, ub, n, b4, outs4, grads4, 2, sets4, None, 1, sides, events) == emb.EMB_EINVAL    # pool
    small = (emb.CDedupSet * 4)(*([good] * 3 + [emb.CDedupSet(0x5000, 0x5100, 0x5200, 0x5300, 0x5400, 0x100000,
                                                              wsb - 256)]))
    assert f(tb, 0, ub, n, b4, outs4, grads4, 2, small, None, 1, sides, events) == emb.EMB_EWORKSPACE
    bad_b = (emb.CBatch * n)(*([emb.CBatch(1, 0x1000, 0x2000, 10, 4)] * (n - 1) + [emb.CBatch(1, 0x1000, 0, 10, 4)]))
    assert f(tb, 0, ub, n, bad_b, outs4, grads4, 2, sets4, None, 1, sides, events) == emb.EMB_EINVAL
    bad_upd = emb.CUpdate(9, 0.1, 0.0, None, 0, 0)
    assert f(tb, 0, ctypes.byref(bad_upd), n, b4, outs4, grads4, 2, sets4, None, 1, sides, events) == emb.EMB_EINVAL
    # one batched dedup per group: one side stream only, and a group workspace
    # large enough for every group (checked before anything is enqueued)
    gws = L.emb_workspace_size(20, 2, t.dim)
    assert f(tb, 0, ub, n, b4, outs4, grads4, 2, sets4, None, 2, sides, events,
             group_ws=0x200000, group_ws_bytes=gws) == emb.EMB_EINVAL                                    # 2 sides
    assert f(tb, 0, ub, n, b4, outs4, grads4, 2, sets4, None, 1, sides, events,
             group_ws=0x200000, group_ws_bytes=gws - 256) == emb.EMB_EWORKSPACE                           # too small
    many_sets = (emb.CDedupSet * 34)(*([good] * 34))
    b17 = (emb.CBatch * 17)(*([emb.CBatch(1, 0x1000, 0x2000, 10, 4)] * 17))
    o17 = (ctypes.c_void_p * 17)(*([0x3000] * 17))
    assert f(tb, 0, ub, 17, b17, o17, o17, 17, many_sets, None, 1, sides, events,
             group_ws=0x200000, group_ws_bytes=1 << 30) == emb.EMB_EUNSUPPORTED                           # > 16
    # chained calls: flags 0 or 1, a group base >= 0, a look-ahead only after
    # steps, and the look-ahead batches' dedups checked before anything is
    # enqueued (two steps in one group of two, then a look-ahead group of two
    # in the sets of the other parity, its last batch or set bad in turn)
    assert f(tb, 0, ub, 1, b, ptrs, ptrs, 1, sets, None, 1, sides, events, group_base=-1) == emb.EMB_EINVAL
    assert f(tb, 0, ub, 1, b, ptrs, ptrs, 1, sets, None, 1, sides, events, primed=2) == emb.EMB_EINVAL
    assert f(tb, 0, ub, 1, b, ptrs, ptrs, 1, sets, None, 1, sides, events, ahead=2) == emb.EMB_EINVAL
    assert f(tb, 0, ub, 0, b, ptrs, ptrs, 1, sets, None, 1, sides, events, ahead=1) == emb.EMB_EINVAL
    assert f(tb, 0, ub, 0, b, ptrs, ptrs, 1, sets, None, 1, sides, events, primed=1) == emb.EMB_OK
    # buffer set parities: 2..8; primed and ahead below the depth; primed
    # groups whole groups of the call's steps
    assert f(tb, 0, ub, 1, b, ptrs, ptrs, 1, sets, None, 1, sides, events, depth=1) == emb.EMB_EINVAL
    assert f(tb, 0, ub, 1, b, ptrs, ptrs, 1, sets, None, 1, sides, events, depth=9) == emb.EMB_EUNSUPPORTED
    assert f(tb, 0, ub, 1, b, ptrs, ptrs, 1, sets, None, 1, sides, events, depth=3, ahead=3) == emb.EMB_EINVAL
    assert f(tb, 0, ub, 1, b, ptrs, ptrs, 1, sets, None, 1, sides, events, depth=3, primed=2) == emb.EMB_EINVAL
    assert f(tb, 0, ub, 1, b, ptrs, ptrs, 1, sets, None, 1, sides, events, primed=-1) == emb.EMB_EINVAL
    ev_d3 = (ctypes.c_void_p * 7)(*([0x40] * 6 + [0]))   # 1 + 3 + 3 events for depth 3 and one side stream
    assert f(tb, 0, ub, 1, b, ptrs, ptrs, 1, sets, None, 1, sides, ev_d3, depth=3) == emb.EMB_EINVAL
    assert f(tb, 0, ub, 2, bad_b, outs4, grads4, 2, sets4, None, 1, sides, events, ahead=1) == emb.EMB_EINVAL
    assert f(tb, 0, ub, 2, b4, outs4, grads4, 2, small, None, 1, sides, events, ahead=1) == emb.EMB_EWORKSPACE
    # with group base 1 the steps take the last two sets and the look-ahead
    # group the first two: the small first set is a look-ahead batch's
    small0 = (emb.CDedupSet * 4)(*([emb.CDedupSet(0x5000, 0x5100, 0x5200, 0x5300, 0x5400, 0x100000, wsb - 256)]
                                   + [good] * 3))
    assert f(tb, 0, ub, 2, b4, outs4, grads4, 2, small0, None, 1, sides, events, ahead=1,
             group_base=1) == emb.EMB_EWORKSPACE
    assert f(tb, 0, ub, 2, b4, outs4, grads4, 2, sets4, None, 1, sides, events, ahead=1,
             group_ws=0x200000, group_ws_bytes=L.emb_workspace_size(20, 2, t.dim) - 256) == emb.EMB_EWORKSPACE


def test_unique_ids_batched_argument_checks():
    """Host checks of emb_unique_ids_batched return before anything is enqueued."""
    L = emb.lib()
    t = _tables()
    n = 3
    b = (emb.CBatch * n)(*([emb.CBatch(1, 0x1000, 0x2000, 10, 4)] * n))
    need = L.emb_workspace_size(10, 1, t.dim)
    gneed = L.emb_workspace_size(30, 3, t.dim)
    sets = (emb.CDedupSet * n)(*[emb.CDedupSet(0x5000, 0x5100, 0x5200, 0x5300, 0x5400, 0x100000 * (i + 1), need)
                                 for i in range(n)])
    f = L.emb_unique_ids_batched
    tb = ctypes.byref(t)
    assert f(tb, 0, b, sets, 0x800000, gneed, None) == emb.EMB_EINVAL          # no batch
    assert f(tb, n, None, sets, 0x800000, gneed, None) == emb.EMB_EINVAL
    assert f(tb, n, b, None, 0x800000, gneed, None) == emb.EMB_EINVAL
    assert f(tb, n, b, sets, 0x800000, gneed - 256, None) == emb.EMB_EWORKSPACE  # group workspace too small
    assert f(tb, n, b, sets, 0x800010, gneed, None) == emb.EMB_EWORKSPACE      # misaligned
    assert f(tb, n, b, sets, 0x100000, gneed, None) == emb.EMB_EINVAL          # a set's workspace is the group's
    same = (emb.CDedupSet * n)(*[emb.CDedupSet(0x5000, 0x5100, 0x5200, 0x5300, 0x5400, 0x100000, need)] * n)
    assert f(tb, n, b, same, 0x800000, gneed, None) == emb.EMB_EINVAL          # two sets share a workspace
    small = (emb.CDedupSet * n)(*[emb.CDedupSet(0x5000, 0x5100, 0x5200, 0x5300, 0x5400, 0x100000 * (i + 1), need - 256)
                                  for i in range(n)])
    assert f(tb, n, b, small, 0x800000, gneed, None) == emb.EMB_EWORKSPACE
    no_perm = (emb.CDedupSet * n)(*[emb.CDedupSet(0x5000, 0x5100, 0x5200, None, 0x5400, 0x100000 * (i + 1), need)
                                    for i in range(n)])
    assert f(tb, n, b, no_perm, 0x800000, gneed, None) == emb.EMB_EINVAL
    b17 = (emb.CBatch * 17)(*([emb.CBatch(1, 0x1000, 0x2000, 10, 4)] * 17))
    s17 = (emb.CDedupSet * 17)(*[emb.CDedupSet(0x5000, 0x5100, 0x5200, 0x5300, 0x5400, 0x100000 * (i + 1), need)
                                 for i in range(17)])
    assert f(tb, 17, b17, s17, 0x800000, 1 << 30, None) == emb.EMB_EUNSUPPORTED  # more than 16 batches
    # 2^31 + 1 rows need 32 key bits: no room for a batch index
    wide = _tables(row_offset=(0, (1 << 31) + 1))
    assert f(ctypes.byref(wide), 2, b, sets, 0x800000, gneed, None) == emb.EMB_EUNSUPPORTED


def test_pipeline_group_by_batch_size():
    """Groups of 8 batches, 4 once 8 batches would exceed 2^25 ids."""
    assert emb.pipeline_group(0) == 8
    assert emb.pipeline_group(491_724) == 8          # the 50M-row workload
    assert emb.pipeline_group(1 << 22) == 8          # exactly 2^25 ids in 8 batches
    assert emb.pipeline_group((1 << 22) + 1) == 4
    assert emb.pipeline_group(5_484_949) == 4        # the 26-table workload


def test_batch_descriptor_follows_its_tensors():
    """The cached C descriptor of a Batch (and its bytes, which pipelined
    calls join into one array) follows field assignments, an in-place
    shrink of the index tensor and a change of index width."""
    import torch
    b = emb.Batch(torch.zeros(17, dtype=torch.int32), torch.arange(100, dtype=torch.int32), 16)
    assert bytes(b.c()) == b._c_bytes()
    d = emb.CBatch.from_buffer_copy(b._c_bytes())
    assert (d.num_indices, d.bags_per_table, d.index_bytes) == (100, 16, 4)
    b.indices = torch.arange(50, dtype=torch.int32)
    assert emb.CBatch.from_buffer_copy(b._c_bytes()).num_indices == 50
    b.indices.resize_(40)
    assert emb.CBatch.from_buffer_copy(b._c_bytes()).num_indices == 40
    b.bags_per_table = 8
    assert emb.CBatch.from_buffer_copy(b._c_bytes()).bags_per_table == 8
    b.indices = torch.arange(30, dtype=torch.int64)
    d = emb.CBatch.from_buffer_copy(b._c_bytes())
    assert (d.num_indices, d.index_bytes, d.indices) == (30, 8, b.indices.data_ptr())
    b.offsets = torch.zeros(9, dtype=torch.int32)
    assert emb.CBatch.from_buffer_copy(b._c_bytes()).offsets == b.offsets.data_ptr()
    # an empty batch carries no index pointer
    e = emb.Batch(torch.zeros(17, dtype=torch.int32), torch.zeros(0, dtype=torch.int32), 16)
    assert emb.CBatch.from_buffer_copy(e._c_bytes()).indices is None
