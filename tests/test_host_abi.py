"""CPU tests of the C-ABI library: it loads, exports every declared symbol,
and its host-only logic (the sample plan, argument checks, workspace
queries) agrees with the oracle.  No device work is launched."""
import ctypes
import math

import numpy as np
import pytest

from oracle import sampler
from paper_2401_04829_amd import _lib as L


def test_library_exports_every_declared_function():
    lib = L.load()
    names = L.header_functions()
    assert len(names) >= 12
    for name in names:
        assert hasattr(lib, name), name
    assert set(L._SIGNATURES) == set(names)
    assert lib.gnnshap_version() >= 100
    for st in range(6):
        assert lib.gnnshap_status_str(st)


@pytest.mark.parametrize("M,p", [(2, 2), (3, 4), (5, 30), (8, 254), (12, 4094), (13, 8190), (17, 2000),
                                 (20, 10000), (33, 5000), (57, 2000), (60, 2000), (64, 3000), (65, 777 * 2),
                                 (400, 10000), (1000, 3334 * 2), (4000, 25000), (12345, 50000), (30000, 100000)])
def test_plan_matches_oracle_bit_for_bit(M, p):
    plan, classes = L.gnnshap_plan_samples(M, p, 1, 2)
    ref = sampler.plan(M, p)
    assert plan.num_rows == ref["k"]
    assert plan.words_per_row == math.ceil(M / 64)
    assert plan.random_begin == ref["random_begin"]
    assert plan.num_classes == len(ref["classes"])
    assert plan.full_fraction == ref["full_fraction"]          # exact fp64 equality
    assert plan.random_weight == ref["random_weight"]
    for got, want in zip(classes, ref["classes"]):
        assert got.size == want["c"]
        assert bool(got.full) == want["full"]
        assert got.row_begin == want["row_begin"]
        assert got.row_count == want["row_count"]
        assert got.weight == want["weight"]


def test_plan_errors_and_size_query():
    lib = L.load()
    plan = L.gnnshap_sample_plan(num_players=1, num_samples=10)
    assert lib.gnnshap_plan_samples(ctypes.byref(plan), None, 0) == L.EINVAL
    plan = L.gnnshap_sample_plan(num_players=10, num_samples=11)
    assert lib.gnnshap_plan_samples(ctypes.byref(plan), None, 0) == L.EINVAL
    plan = L.gnnshap_sample_plan(num_players=10, num_samples=0)
    assert lib.gnnshap_plan_samples(ctypes.byref(plan), None, 0) == L.EINVAL
    assert lib.gnnshap_plan_samples(None, None, 0) == L.EINVAL
    plan = L.gnnshap_sample_plan(num_players=400, num_samples=10000)
    assert lib.gnnshap_plan_samples(ctypes.byref(plan), None, 0) == L.ECAPACITY
    assert plan.num_classes > 0 and plan.num_rows == 10000
    assert "class table" in lib.gnnshap_last_error().decode()


def test_workspace_queries_and_argument_checks():
    lib = L.load()
    n = ctypes.c_size_t()
    assert lib.gnnshap_extract_workspace(2708, ctypes.byref(n)) == L.OK and n.value >= 5 * 4 * 2708
    assert lib.gnnshap_extract_workspace(0, ctypes.byref(n)) == L.EINVAL
    plan, classes = L.gnnshap_plan_samples(400, 10000, 1, 2)
    assert L.gnnshap_sample_workspace(plan) >= plan.num_classes * 32
    need = L.gnnshap_solve_workspace(plan)
    assert need >= 400 * 400 * 4
    bad = L.gnnshap_sample_plan(num_players=400, num_samples=10000)    # not planned
    assert lib.gnnshap_sample_workspace(ctypes.byref(bad), ctypes.byref(n)) == L.EINVAL
    assert lib.gnnshap_solve_workspace(ctypes.byref(bad), ctypes.byref(n)) == L.EINVAL
    # eval: a consistent 2-hop subgraph description and a 2-layer model
    sg = L.gnnshap_subgraph(num_hops=2, num_nodes=10, num_edges=12, num_dst=4)
    for i, v in enumerate([0, 1, 4, 10, 10, 10, 10, 10, 10, 10]):
        sg.hop_ptr[i] = v
    dims = (ctypes.c_int32 * 3)(8, 16, 3)
    W = (ctypes.c_void_p * 2)(1, 1)
    model = L.gnnshap_gcn(num_layers=2, dims=dims, W=W, b=None)
    assert L.gnnshap_eval_workspace(sg, model, 100) > 0
    assert lib.gnnshap_eval_workspace(ctypes.byref(sg), ctypes.byref(model), 0, ctypes.byref(n)) == L.EINVAL
    sg.hop_ptr[2] = 5                                                   # inconsistent with num_dst
    assert lib.gnnshap_eval_workspace(ctypes.byref(sg), ctypes.byref(model), 100, ctypes.byref(n)) == L.EINVAL
    sg.hop_ptr[2] = 4
    # invalid arguments are rejected before any device work
    assert lib.gnnshap_eval_coalitions(ctypes.byref(sg), ctypes.byref(model), None, 0, None, 10, 1, None, None,
                                       None, None, 0, None) == L.EINVAL
    assert lib.gnnshap_sample_coalitions(ctypes.byref(plan), classes, None, None, None, 0, None) == L.EINVAL
    assert lib.gnnshap_solve_wls(ctypes.byref(plan), classes, None, None, None, None, None, None, 0,
                                 None) == L.EINVAL
    g = L.gnnshap_graph(num_nodes=10, num_edges=0, indptr=1, indices=1)
    sub = L.gnnshap_subgraph(num_hops=2)
    assert lib.gnnshap_extract_subgraph(ctypes.byref(g), 10, ctypes.byref(sub), 1, 10 ** 6, None) == L.EINVAL
    sub.num_hops = 9
    assert lib.gnnshap_extract_subgraph(ctypes.byref(g), 0, ctypes.byref(sub), 1, 10 ** 6, None) == L.EINVAL
    sub.num_hops = 2
    assert lib.gnnshap_extract_subgraph(ctypes.byref(g), 0, ctypes.byref(sub), 1, 16, None) == L.ECAPACITY


def test_batch_entry_points_reject_bad_arguments():
    lib = L.load()
    n = ctypes.c_size_t()
    assert lib.gnnshap_extract_batch_workspace(100, 0, ctypes.byref(n)) == L.EINVAL
    assert lib.gnnshap_extract_batch_workspace(0, 4, ctypes.byref(n)) == L.EINVAL
    assert lib.gnnshap_extract_batch_workspace(100, 4, ctypes.byref(n)) == L.OK and n.value > 0
    assert lib.gnnshap_extract_batch(None, None, 1, None, None, 0, None) == L.EINVAL
    assert lib.gnnshap_extract_batch_launch(None, None, 1, None, None, 0, None) == L.EINVAL
    sgs = (L.gnnshap_subgraph * 2)()
    assert lib.gnnshap_extract_batch_finish(sgs, 2) == L.EINVAL       # nothing launched by this thread
    assert lib.gnnshap_extract_batch_finish(None, 2) == L.EINVAL
    assert lib.gnnshap_explain_batch_workspace(None, None, 1, None, ctypes.byref(n)) == L.EINVAL
    assert lib.gnnshap_explain_batch(None, None, None, 0, None, None, -1, None, None, None, None, None, None, None,
                                     None, 0, None) == L.EINVAL


def test_plan_batch_equals_single_plans():
    Ms = [7, 60, 60, 2, 400, 7, 33, 1000]
    sgs = (L.gnnshap_subgraph * len(Ms))()
    for sg, M in zip(sgs, Ms):
        sg.num_edges = M
    ids = (ctypes.c_int64 * len(Ms))(*[100 + i for i in range(len(Ms))])
    plans = (L.gnnshap_sample_plan * len(Ms))()
    st, ncls, totals = L.gnnshap_plan_batch(sgs, ids, 2000, 77, plans, None)
    assert st == L.ECAPACITY and ncls > 0
    short = (L.gnnshap_class * (ncls - 1))()
    assert L.gnnshap_plan_batch(sgs, ids, 2000, 77, plans, short)[0] == L.ECAPACITY
    classes = (L.gnnshap_class * ncls)()
    st, ncls2, totals = L.gnnshap_plan_batch(sgs, ids, 2000, 77, plans, classes)
    assert st == L.OK and ncls2 == ncls
    o, words, rows = 0, 0, 0
    for t, M in enumerate(Ms):
        plan, cl = L.gnnshap_plan_samples(M, 2000, 77, 100 + t)
        got = plans[t]
        for f, _ in L.gnnshap_sample_plan._fields_:
            assert getattr(got, f) == getattr(plan, f), (t, f)
        for i in range(plan.num_classes):
            a, b = classes[o + i], cl[i]
            assert (a.size, a.full, a.row_begin, a.row_count, a.weight) == \
                   (b.size, b.full, b.row_begin, b.row_count, b.weight)
        o += plan.num_classes
        words += plan.num_rows * plan.words_per_row
        rows += plan.num_rows
    assert o == ncls and totals == (words, rows, sum(Ms))
    sgs[3].num_edges = 1
    st = L.load().gnnshap_plan_batch(sgs, ids, len(Ms), 2000, 77, plans, classes, ncls, ctypes.byref(ctypes.c_int64()),
                                     None)
    assert st == L.EINVAL and "target 3" in L.load().gnnshap_last_error().decode()


def test_subgraph_batch_init_strides():
    sgs = (L.gnnshap_subgraph * 3)()
    L.gnnshap_subgraph_batch_init(sgs, 2, 10, 20, 1 << 20, 2 << 20, 3 << 20, 4 << 20, 5 << 20)
    for t, sg in enumerate(sgs):
        assert (sg.num_hops, sg.cap_nodes, sg.cap_edges, sg.num_edges) == (2, 10, 20, 0)
        assert sg.node_gid == (1 << 20) + 4 * 10 * t
        assert sg.dst_ptr == (2 << 20) + 4 * 11 * t
        assert sg.edge_src == (3 << 20) + 4 * 20 * t
        assert sg.edge_dst == (4 << 20) + 4 * 20 * t
        assert sg.edge_gid == (5 << 20) + 8 * 20 * t
    with pytest.raises(RuntimeError):
        L.gnnshap_subgraph_batch_init(sgs, 2, 10, 20, None, 2 << 20, 3 << 20, 4 << 20, 5 << 20)


def test_iterative_threshold_selects_path_and_workspace():
    """Above the plan's iterative threshold (0 = the default 5000 players,
    Sec. 3.5) the solve reports path 3 and needs no M x M matrix in its
    workspace; gnnshap_plan_samples keeps the threshold the caller set."""
    plan, _ = L.gnnshap_plan_samples(6000, 50000, 1, 2)
    assert plan.iterative_threshold == 0
    assert L.gnnshap_solve_info(plan) == 3
    small, _ = L.gnnshap_plan_samples(4000, 25000, 1, 2)
    assert L.gnnshap_solve_info(small) == 0
    direct = L.gnnshap_solve_workspace(small)
    small.iterative_threshold = 3999
    assert L.gnnshap_solve_info(small) == 3
    assert L.gnnshap_solve_workspace(small) < min(direct, 4000 * 4000 * 4) // 2
    again, _ = L.gnnshap_plan_samples(4000, 25000, 1, 2, iterative_threshold=3999)
    assert again.iterative_threshold == 3999 and L.gnnshap_solve_info(again) == 3
    mid, _ = L.gnnshap_plan_samples(300, 4000, 1, 2)
    assert L.gnnshap_solve_info(mid) == 2
    mid.iterative_threshold = 299
    assert L.gnnshap_solve_info(mid) == 3
    mid.iterative_threshold = -5
    assert L.gnnshap_solve_info(mid) == 2


def test_fidelity_entry_points_reject_bad_arguments():
    """Argument checks of the fidelity calls (eq. 7-8) happen before any launch."""
    lib = L.load()
    fake = ctypes.c_void_p(256)
    assert lib.gnnshap_fidelity_masks(None, 10, 0.3, 10, fake, None) == L.EINVAL
    assert lib.gnnshap_fidelity_masks(fake, 0, 0.3, 10, fake, None) == L.EINVAL
    assert lib.gnnshap_fidelity_masks(fake, 10, 1.5, 10, fake, None) == L.EINVAL
    assert lib.gnnshap_fidelity_masks(fake, 10, float("nan"), 10, fake, None) == L.EINVAL
    assert lib.gnnshap_fidelity_masks(fake, 10, 0.3, -1, fake, None) == L.EINVAL
    assert lib.gnnshap_fidelity_average(fake, 0, 3, fake, None) == L.EINVAL
    assert lib.gnnshap_fidelity_average(fake, 4, 1, fake, None) == L.EINVAL
    assert lib.gnnshap_fidelity_average(None, 4, 3, fake, None) == L.EINVAL
    sg = L.gnnshap_subgraph(num_hops=2)
    n = ctypes.c_size_t()
    assert lib.gnnshap_fidelity_workspace(ctypes.byref(sg), None, ctypes.byref(n)) == L.EINVAL


def test_gat_entry_points_reject_bad_arguments():
    """The GAT calls (App. E) check the subgraph depth and the model shape
    before any launch."""
    lib = L.load()
    fake = 256
    m = L.gnnshap_gat(heads=8, head_dim=16, num_classes=7, XW1=fake, att_src1=fake, att_dst1=fake, b1=fake, W2=fake,
                      att_src2=fake, att_dst2=fake, b2=fake, negative_slope=0.2)
    sg = L.gnnshap_subgraph(num_hops=2, num_nodes=10, num_edges=12, num_dst=4)
    n = ctypes.c_size_t()
    assert lib.gnnshap_gat_eval_workspace(ctypes.byref(sg), ctypes.byref(m), 100, ctypes.byref(n)) == L.OK
    assert n.value > 0
    sg3 = L.gnnshap_subgraph(num_hops=3, num_nodes=10, num_edges=12, num_dst=4)
    assert lib.gnnshap_gat_eval_workspace(ctypes.byref(sg3), ctypes.byref(m), 100, ctypes.byref(n)) == L.EINVAL
    for bad in (dict(heads=0), dict(head_dim=33, heads=8), dict(num_classes=0), dict(negative_slope=1.0),
                dict(XW1=None)):
        mb = L.gnnshap_gat(heads=8, head_dim=16, num_classes=7, XW1=fake, att_src1=fake, att_dst1=fake, b1=fake,
                           W2=fake, att_src2=fake, att_dst2=fake, b2=fake, negative_slope=0.2)
        for k, v in bad.items():
            setattr(mb, k, v)
        assert lib.gnnshap_gat_eval_workspace(ctypes.byref(sg), ctypes.byref(mb), 100, ctypes.byref(n)) == L.EINVAL, bad
    assert lib.gnnshap_gat_eval_workspace(ctypes.byref(sg), ctypes.byref(m), 0, ctypes.byref(n)) == L.EINVAL
