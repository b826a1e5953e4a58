"""ctypes binding of libgnnshap.so: the C ABI of include/gnnshap.h, one Python
function per entry point, with the same names.  Argument marshalling only;
every step runs in the library.  There is no fallback: if the library is not
built, loading it raises."""
import ctypes
import os
import re

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libgnnshap.so")
HEADER = os.path.join(os.path.dirname(_HERE), "include", "gnnshap.h")

OK, EINVAL, ECAPACITY, EHIP, ESINGULAR, EUNSUPPORTED = range(6)
MAX_HOPS = 8
MAX_LAYERS = 8

c_i32, c_i64, c_u64, c_dbl, c_vp = ctypes.c_int32, ctypes.c_int64, ctypes.c_uint64, ctypes.c_double, ctypes.c_void_p


class gnnshap_graph(ctypes.Structure):
    _fields_ = [("num_nodes", c_i64), ("num_edges", c_i64), ("indptr", c_vp), ("indices", c_vp)]


class gnnshap_subgraph(ctypes.Structure):
    _fields_ = [("num_hops", c_i32), ("reserved", c_i32), ("cap_nodes", c_i64), ("cap_edges", c_i64),
                ("node_gid", c_vp), ("dst_ptr", c_vp), ("edge_src", c_vp), ("edge_dst", c_vp),
                ("edge_gid", c_vp), ("num_nodes", c_i64), ("num_edges", c_i64), ("num_dst", c_i64),
                ("hop_ptr", c_i64 * (MAX_HOPS + 2))]


class gnnshap_class(ctypes.Structure):
    _fields_ = [("size", c_i32), ("full", c_i32), ("row_begin", c_i64), ("row_count", c_i64),
                ("weight", c_dbl)]


class gnnshap_sample_plan(ctypes.Structure):
    _fields_ = [("num_players", c_i64), ("num_samples", c_i64), ("seed", c_u64), ("stream_id", c_u64),
                ("num_rows", c_i64), ("words_per_row", c_i64), ("num_classes", c_i64),
                ("random_begin", c_i64), ("full_fraction", c_dbl), ("random_weight", c_dbl),
                ("iterative_threshold", c_i64)]


class gnnshap_gcn(ctypes.Structure):
    _fields_ = [("num_layers", c_i32), ("reserved", c_i32), ("dims", ctypes.POINTER(c_i32)),
                ("W", ctypes.POINTER(c_vp)), ("b", ctypes.POINTER(c_vp)), ("XW1", c_vp)]


class gnnshap_gat(ctypes.Structure):
    _fields_ = [("heads", c_i32), ("head_dim", c_i32), ("num_classes", c_i32), ("reserved", c_i32),
                ("XW1", c_vp), ("att_src1", c_vp), ("att_dst1", c_vp), ("b1", c_vp), ("W2", c_vp),
                ("att_src2", c_vp), ("att_dst2", c_vp), ("b2", c_vp), ("negative_slope", c_dbl)]


_P = ctypes.POINTER
_SIGNATURES = {
    "gnnshap_status_str": (ctypes.c_char_p, [ctypes.c_int]),
    "gnnshap_last_error": (ctypes.c_char_p, []),
    "gnnshap_version": (ctypes.c_int, []),
    "gnnshap_extract_workspace": (ctypes.c_int, [c_i64, _P(ctypes.c_size_t)]),
    "gnnshap_extract_subgraph": (ctypes.c_int, [_P(gnnshap_graph), c_i64, _P(gnnshap_subgraph), c_vp,
                                                ctypes.c_size_t, c_vp]),
    "gnnshap_plan_samples": (ctypes.c_int, [_P(gnnshap_sample_plan), _P(gnnshap_class), c_i64]),
    "gnnshap_sample_workspace": (ctypes.c_int, [_P(gnnshap_sample_plan), _P(ctypes.c_size_t)]),
    "gnnshap_sample_coalitions": (ctypes.c_int, [_P(gnnshap_sample_plan), _P(gnnshap_class), c_vp, c_vp,
                                                 c_vp, ctypes.c_size_t, c_vp]),
    "gnnshap_sample_coalitions_noalloc": (ctypes.c_int, [_P(gnnshap_sample_plan), _P(gnnshap_class), c_vp, c_vp,
                                                         c_vp]),
    "gnnshap_eval_workspace": (ctypes.c_int, [_P(gnnshap_subgraph), _P(gnnshap_gcn), c_i64,
                                              _P(ctypes.c_size_t)]),
    "gnnshap_eval_coalitions": (ctypes.c_int, [_P(gnnshap_subgraph), _P(gnnshap_gcn), c_vp, c_i32, c_vp,
                                               c_i64, c_i64, c_vp, c_vp, c_vp, c_vp, ctypes.c_size_t, c_vp]),
    "gnnshap_eval_sampled_coalitions": (ctypes.c_int, [_P(gnnshap_subgraph), _P(gnnshap_gcn), c_vp, c_i32, c_vp,
                                                       c_i64, c_i64, c_vp, c_vp, c_vp, c_vp, ctypes.c_size_t,
                                                       c_vp]),
    "gnnshap_transform_features": (ctypes.c_int, [c_vp, c_i64, c_i32, c_vp, c_i32, c_vp, c_vp]),
    "gnnshap_solve_workspace": (ctypes.c_int, [_P(gnnshap_sample_plan), _P(ctypes.c_size_t)]),
    "gnnshap_solve_wls": (ctypes.c_int, [_P(gnnshap_sample_plan), _P(gnnshap_class), c_vp, c_vp, c_vp, c_vp,
                                         c_vp, c_vp, ctypes.c_size_t, c_vp]),
    "gnnshap_extract_batch_workspace": (ctypes.c_int, [c_i64, c_i64, _P(ctypes.c_size_t)]),
    "gnnshap_extract_batch": (ctypes.c_int, [_P(gnnshap_graph), _P(c_i64), c_i64, _P(gnnshap_subgraph), c_vp,
                                             ctypes.c_size_t, c_vp]),
    "gnnshap_extract_batch_launch": (ctypes.c_int, [_P(gnnshap_graph), _P(c_i64), c_i64, _P(gnnshap_subgraph),
                                                    c_vp, ctypes.c_size_t, c_vp]),
    "gnnshap_extract_batch_finish": (ctypes.c_int, [_P(gnnshap_subgraph), c_i64]),
    "gnnshap_subgraph_batch_init": (ctypes.c_int, [_P(gnnshap_subgraph), c_i64, c_i32, c_i64, c_i64, c_vp, c_vp,
                                                    c_vp, c_vp, c_vp]),
    "gnnshap_plan_batch": (ctypes.c_int, [_P(gnnshap_subgraph), _P(c_i64), c_i64, c_i64, ctypes.c_uint64,
                                          _P(gnnshap_sample_plan), _P(gnnshap_class), c_i64, _P(c_i64),
                                          _P(c_i64)]),
    "gnnshap_explain_batch_workspace": (ctypes.c_int, [_P(gnnshap_subgraph), _P(gnnshap_sample_plan), c_i64,
                                                       _P(gnnshap_gcn), _P(ctypes.c_size_t)]),
    "gnnshap_explain_batch": (ctypes.c_int, [_P(gnnshap_subgraph), _P(gnnshap_sample_plan), _P(gnnshap_class),
                                             c_i64, _P(gnnshap_gcn), c_vp, c_i32, c_vp, c_vp, c_vp, c_vp, c_vp,
                                             c_vp, c_vp, c_vp, ctypes.c_size_t, c_vp]),
    "gnnshap_gat_explain_batch_workspace": (ctypes.c_int, [_P(gnnshap_subgraph), _P(gnnshap_sample_plan), c_i64,
                                                           _P(gnnshap_gat), _P(ctypes.c_size_t)]),
    "gnnshap_gat_explain_batch": (ctypes.c_int, [_P(gnnshap_subgraph), _P(gnnshap_sample_plan), _P(gnnshap_class),
                                                 c_i64, _P(gnnshap_gat), c_i32, c_vp, c_vp, c_vp, c_vp, c_vp,
                                                 c_vp, c_vp, c_vp, ctypes.c_size_t, c_vp]),
    "gnnshap_solve_info": (ctypes.c_int, [_P(gnnshap_sample_plan), _P(c_i32)]),
    "gnnshap_fidelity_workspace": (ctypes.c_int, [_P(gnnshap_subgraph), _P(gnnshap_gcn), _P(ctypes.c_size_t)]),
    "gnnshap_fidelity": (ctypes.c_int, [_P(gnnshap_subgraph), _P(gnnshap_gcn), c_vp, c_i32, c_vp, c_dbl, c_i64,
                                        c_vp, c_vp, ctypes.c_size_t, c_vp]),
    "gnnshap_fidelity_average": (ctypes.c_int, [c_vp, c_i64, c_i64, c_vp, c_vp]),
    "gnnshap_fidelity_masks": (ctypes.c_int, [c_vp, c_i64, c_dbl, c_i64, c_vp, c_vp]),
    "gnnshap_gat_eval_workspace": (ctypes.c_int, [_P(gnnshap_subgraph), _P(gnnshap_gat), c_i64,
                                                  _P(ctypes.c_size_t)]),
    "gnnshap_gat_eval_coalitions": (ctypes.c_int, [_P(gnnshap_subgraph), _P(gnnshap_gat), c_i32, c_vp, c_i64, c_i64,
                                                   c_vp, c_vp, c_vp, c_vp, ctypes.c_size_t, c_vp]),
    "gnnshap_timing_begin": (ctypes.c_int, [ctypes.c_char_p]),
    "gnnshap_timing_end": (ctypes.c_int, [_P(ctypes.c_double), _P(c_i64)]),
    "gnnshap_timing_solves": (ctypes.c_int, [_P(c_i64), c_i64, _P(c_i64)]),
}

_lib = None


def load():
    """Loads libgnnshap.so (built by `python -m paper_2401_04829_amd.build`)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is not built; run `python -m paper_2401_04829_amd.build`")
        lib = ctypes.CDLL(LIB_PATH)
        for name, (res, args) in _SIGNATURES.items():
            fn = getattr(lib, name)
            fn.restype = res
            fn.argtypes = args
        _lib = lib
    return _lib


def header_functions():
    """Names of the functions declared in include/gnnshap.h."""
    with open(HEADER) as f:
        text = f.read()
    return sorted(set(re.findall(r"\b(gnnshap_[a-z_]+)\s*\(", text)))


class GnnShapError(RuntimeError):
    def __init__(self, status, what):
        lib = load()
        msg = lib.gnnshap_last_error().decode()
        super().__init__(f"{what}: {lib.gnnshap_status_str(status).decode()} ({msg})")
        self.status = status


def check(status, what):
    if status != OK:
        raise GnnShapError(status, what)
    return status


# -- one wrapper per entry point (same names as the C ABI) ---------------------------------

def gnnshap_extract_workspace(num_nodes):
    n = ctypes.c_size_t()
    check(load().gnnshap_extract_workspace(num_nodes, ctypes.byref(n)), "extract_workspace")
    return n.value


def gnnshap_extract_subgraph(graph, target, sg, ws_ptr, ws_bytes, stream):
    """Returns the status (OK or ECAPACITY); raises on other failures."""
    st = load().gnnshap_extract_subgraph(ctypes.byref(graph), target, ctypes.byref(sg), ws_ptr, ws_bytes, stream)
    if st not in (OK, ECAPACITY):
        check(st, "extract_subgraph")
    return st


def gnnshap_plan_samples(num_players, num_samples, seed, stream_id, iterative_threshold=0):
    plan = gnnshap_sample_plan(num_players=num_players, num_samples=num_samples, seed=seed, stream_id=stream_id,
                               iterative_threshold=iterative_threshold)
    st = load().gnnshap_plan_samples(ctypes.byref(plan), None, 0)
    if st != ECAPACITY:
        check(st, "plan_samples")
    classes = (gnnshap_class * plan.num_classes)()
    check(load().gnnshap_plan_samples(ctypes.byref(plan), classes, plan.num_classes), "plan_samples")
    return plan, classes


def gnnshap_sample_workspace(plan):
    n = ctypes.c_size_t()
    check(load().gnnshap_sample_workspace(ctypes.byref(plan), ctypes.byref(n)), "sample_workspace")
    return n.value


def gnnshap_sample_coalitions(plan, classes, masks_ptr, weights_ptr, ws_ptr, ws_bytes, stream):
    check(load().gnnshap_sample_coalitions(ctypes.byref(plan), classes, masks_ptr, weights_ptr, ws_ptr, ws_bytes,
                                           stream), "sample_coalitions")


def gnnshap_sample_coalitions_noalloc(plan, classes, masks_ptr, weights_ptr, stream):
    check(load().gnnshap_sample_coalitions_noalloc(ctypes.byref(plan), classes, masks_ptr, weights_ptr, stream),
          "sample_coalitions_noalloc")


def gnnshap_eval_workspace(sg, model, k):
    n = ctypes.c_size_t()
    check(load().gnnshap_eval_workspace(ctypes.byref(sg), ctypes.byref(model), k, ctypes.byref(n)), "eval_workspace")
    return n.value


def gnnshap_eval_coalitions(sg, model, X_ptr, target_class, masks_ptr, k, wpr, y_ptr, fef_ptr, cls_ptr, ws_ptr,
                            ws_bytes, stream):
    check(load().gnnshap_eval_coalitions(ctypes.byref(sg), ctypes.byref(model), X_ptr, target_class, masks_ptr, k,
                                         wpr, y_ptr, fef_ptr, cls_ptr, ws_ptr, ws_bytes, stream), "eval_coalitions")


def gnnshap_eval_sampled_coalitions(sg, model, X_ptr, target_class, masks_ptr, k, wpr, y_ptr, fef_ptr, cls_ptr,
                                    ws_ptr, ws_bytes, stream):
    check(load().gnnshap_eval_sampled_coalitions(ctypes.byref(sg), ctypes.byref(model), X_ptr, target_class,
                                                 masks_ptr, k, wpr, y_ptr, fef_ptr, cls_ptr, ws_ptr, ws_bytes,
                                                 stream), "eval_sampled_coalitions")


def gnnshap_transform_features(X_ptr, n, d, W_ptr, h, Z_ptr, stream):
    check(load().gnnshap_transform_features(X_ptr, n, d, W_ptr, h, Z_ptr, stream), "transform_features")


def gnnshap_solve_workspace(plan):
    n = ctypes.c_size_t()
    check(load().gnnshap_solve_workspace(ctypes.byref(plan), ctypes.byref(n)), "solve_workspace")
    return n.value


def gnnshap_timing_begin(kernel_name):
    check(load().gnnshap_timing_begin(kernel_name.encode()), "timing_begin")


def gnnshap_timing_end():
    """Returns (total milliseconds, number of timed launches)."""
    ms, n = ctypes.c_double(), c_i64()
    check(load().gnnshap_timing_end(ctypes.byref(ms), ctypes.byref(n)), "timing_end")
    return ms.value, n.value


def gnnshap_timing_solves():
    """The iterative solves since gnnshap_timing_begin: a list of
    (players, words per row, random rows, iterations, sparse rows, their players)."""
    n = c_i64()
    lib = load()
    st = lib.gnnshap_timing_solves(None, 0, ctypes.byref(n))
    if st not in (OK, ECAPACITY):
        check(st, "timing_solves")
    buf = (c_i64 * max(6 * n.value, 1))()
    check(lib.gnnshap_timing_solves(buf, n.value, ctypes.byref(n)), "timing_solves")
    return [tuple(buf[6 * i:6 * i + 6]) for i in range(n.value)]


def gnnshap_solve_wls(plan, classes, masks_ptr, y_ptr, fef_ptr, phi_ptr, info_ptr, ws_ptr, ws_bytes, stream):
    check(load().gnnshap_solve_wls(ctypes.byref(plan), classes, masks_ptr, y_ptr, fef_ptr, phi_ptr, info_ptr,
                                   ws_ptr, ws_bytes, stream), "solve_wls")


def gnnshap_extract_batch_workspace(num_nodes, n):
    b = ctypes.c_size_t()
    check(load().gnnshap_extract_batch_workspace(num_nodes, n, ctypes.byref(b)), "extract_batch_workspace")
    return b.value


def gnnshap_extract_batch(graph, targets, sgs, ws_ptr, ws_bytes, stream):
    """targets: ctypes int64 array; sgs: ctypes array of gnnshap_subgraph.  Returns OK or ECAPACITY."""
    st = load().gnnshap_extract_batch(ctypes.byref(graph), targets, len(sgs), sgs, ws_ptr, ws_bytes, stream)
    if st not in (OK, ECAPACITY):
        check(st, "extract_batch")
    return st


def gnnshap_extract_batch_launch(graph, targets, sgs, ws_ptr, ws_bytes, stream):
    """First half of gnnshap_extract_batch: queues the extraction; sizes come
    with gnnshap_extract_batch_finish."""
    check(load().gnnshap_extract_batch_launch(ctypes.byref(graph), targets, len(sgs), sgs, ws_ptr, ws_bytes, stream),
          "extract_batch_launch")


def gnnshap_extract_batch_finish(sgs):
    """Second half: waits for the sizes of the launched extraction.  Returns OK or ECAPACITY."""
    st = load().gnnshap_extract_batch_finish(sgs, len(sgs))
    if st not in (OK, ECAPACITY):
        check(st, "extract_batch_finish")
    return st


def gnnshap_subgraph_batch_init(sgs, num_hops, cap_nodes, cap_edges, node_gid, dst_ptr, edge_src, edge_dst,
                                edge_gid):
    check(load().gnnshap_subgraph_batch_init(sgs, len(sgs), num_hops, cap_nodes, cap_edges, node_gid, dst_ptr,
                                             edge_src, edge_dst, edge_gid), "subgraph_batch_init")


def gnnshap_plan_batch(sgs, stream_ids, num_samples, seed, plans, classes):
    """Plans of a batch into `plans` and `classes` (ctypes arrays).  Returns
    (status, num_classes, totals): OK, or ECAPACITY when `classes` is too
    short (plans and the counts are filled either way)."""
    ncls = c_i64()
    tot = (c_i64 * 3)()
    cap = len(classes) if classes is not None else 0
    st = load().gnnshap_plan_batch(sgs, stream_ids, len(sgs), num_samples, seed, plans, classes, cap,
                                   ctypes.byref(ncls), tot)
    if st not in (OK, ECAPACITY):
        check(st, "plan_batch")
    return st, ncls.value, tuple(tot)


def gnnshap_explain_batch_workspace(sgs, plans, model):
    b = ctypes.c_size_t()
    check(load().gnnshap_explain_batch_workspace(sgs, plans, len(sgs), ctypes.byref(model), ctypes.byref(b)),
          "explain_batch_workspace")
    return b.value


def gnnshap_explain_batch(sgs, plans, classes, model, X_ptr, target_class, masks_ptr, weights_ptr, y_ptr, fef_ptr,
                          cls_ptr, phi_ptr, info_ptr, ws_ptr, ws_bytes, stream):
    """Returns OK, or ECAPACITY when the workspace is too small (nothing was
    queued then); raises on any other status."""
    st = load().gnnshap_explain_batch(sgs, plans, classes, len(sgs), ctypes.byref(model), X_ptr, target_class,
                                      masks_ptr, weights_ptr, y_ptr, fef_ptr, cls_ptr, phi_ptr, info_ptr, ws_ptr,
                                      ws_bytes, stream)
    if st not in (OK, ECAPACITY):
        check(st, "explain_batch")
    return st


def gnnshap_gat_explain_batch_workspace(sgs, plans, model):
    b = ctypes.c_size_t()
    check(load().gnnshap_gat_explain_batch_workspace(sgs, plans, len(sgs), ctypes.byref(model), ctypes.byref(b)),
          "gat_explain_batch_workspace")
    return b.value


def gnnshap_gat_explain_batch(sgs, plans, classes, model, target_class, masks_ptr, weights_ptr, y_ptr, fef_ptr,
                              cls_ptr, phi_ptr, info_ptr, ws_ptr, ws_bytes, stream):
    """As gnnshap_explain_batch, for the GAT: OK, or ECAPACITY when the
    workspace is too small (nothing was queued then); raises otherwise."""
    st = load().gnnshap_gat_explain_batch(sgs, plans, classes, len(sgs), ctypes.byref(model), target_class,
                                          masks_ptr, weights_ptr, y_ptr, fef_ptr, cls_ptr, phi_ptr, info_ptr, ws_ptr,
                                          ws_bytes, stream)
    if st not in (OK, ECAPACITY):
        check(st, "gat_explain_batch")
    return st


def gnnshap_solve_info(plan):
    """Solver path of the plan's system: 1 one workgroup, 2 the panel path, 0 multi-block, 3 iterative."""
    v = c_i32()
    check(load().gnnshap_solve_info(ctypes.byref(plan), ctypes.byref(v)), "solve_info")
    return v.value


def gnnshap_fidelity_workspace(sg, model):
    n = ctypes.c_size_t()
    check(load().gnnshap_fidelity_workspace(ctypes.byref(sg), ctypes.byref(model), ctypes.byref(n)),
          "fidelity_workspace")
    return n.value


def gnnshap_fidelity(sg, model, X_ptr, target_class, phi_ptr, sparsity, top_k, out_ptr, ws_ptr, ws_bytes, stream):
    check(load().gnnshap_fidelity(ctypes.byref(sg), ctypes.byref(model), X_ptr, int(target_class), phi_ptr,
                                  float(sparsity), int(top_k), out_ptr, ws_ptr, ws_bytes, stream), "fidelity")


def gnnshap_gat_eval_workspace(sg, model, k):
    n = ctypes.c_size_t()
    check(load().gnnshap_gat_eval_workspace(ctypes.byref(sg), ctypes.byref(model), int(k), ctypes.byref(n)),
          "gat_eval_workspace")
    return n.value


def gnnshap_gat_eval_coalitions(sg, model, target_class, masks_ptr, k, wpr, y_ptr, fef_ptr, cls_ptr, ws_ptr,
                                ws_bytes, stream):
    check(load().gnnshap_gat_eval_coalitions(ctypes.byref(sg), ctypes.byref(model), int(target_class), masks_ptr,
                                             int(k), int(wpr), y_ptr, fef_ptr, cls_ptr, ws_ptr, ws_bytes, stream),
          "gat_eval_coalitions")


def gnnshap_fidelity_masks(phi_ptr, M, sparsity, top_k, masks_ptr, stream):
    check(load().gnnshap_fidelity_masks(phi_ptr, int(M), float(sparsity), int(top_k), masks_ptr, stream),
          "fidelity_masks")


def gnnshap_fidelity_average(terms_ptr, n, stride, avg_ptr, stream):
    check(load().gnnshap_fidelity_average(terms_ptr, int(n), int(stride), avg_ptr, stream), "fidelity_average")
