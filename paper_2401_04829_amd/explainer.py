"""Torch-facing driver of the C-ABI calls for one graph and one GCN.

Torch provides device memory and streams; every computation runs in
libgnnshap.so.  Buffers are caller-owned torch tensors.
"""
import ctypes
from dataclasses import dataclass

import torch

from . import _lib as L


def _vp(t):
    return ctypes.c_void_p(t.data_ptr() if t is not None else 0)


class _Buffer:
    """Grow-only device byte buffer used as a library workspace."""

    def __init__(self, device):
        self.device = device
        self.t = None

    def get(self, nbytes):
        nbytes = max(int(nbytes), 256)
        if self.t is None or self.t.numel() < nbytes:
            self.t = None
            self.t = torch.empty(nbytes, dtype=torch.uint8, device=self.device)
        return self.t


@dataclass
class Subgraph:
    sg: L.gnnshap_subgraph      # sizes (host struct; pointers into the arrays below)
    node_gid: torch.Tensor      # int32 [n']
    dst_ptr: torch.Tensor       # int32 [num_dst + 1]
    edge_src: torch.Tensor      # int32 [M]
    edge_dst: torch.Tensor      # int32 [M]
    edge_gid: torch.Tensor      # int64 [M]

    @property
    def num_edges(self):
        return self.sg.num_edges

    @property
    def hop_ptr(self):
        return [self.sg.hop_ptr[i] for i in range(self.sg.num_hops + 2)]


@dataclass
class Explanation:
    target: int
    sub: Subgraph
    plan: L.gnnshap_sample_plan
    classes: object             # ctypes array of gnnshap_class
    masks: torch.Tensor         # int64 [k, wpr] (uint64 bit patterns)
    weights: torch.Tensor       # float32 [k]
    y: torch.Tensor             # float32 [k]
    f_empty_full: torch.Tensor  # float32 [2]
    cls: torch.Tensor           # int32 [1]
    phi: torch.Tensor           # float32 [M]
    info: torch.Tensor          # int32 [1]


class Explainer:
    def __init__(self, indptr, indices, X, weights, biases, hops, device="cuda"):
        L.load()
        self.device = torch.device(device)
        dev = self.device
        self.indptr = torch.as_tensor(indptr, dtype=torch.int64).to(dev).contiguous()
        self.indices = torch.as_tensor(indices, dtype=torch.int32).to(dev).contiguous()
        self.X = torch.as_tensor(X, dtype=torch.float32).to(dev).contiguous()
        self.W = [torch.as_tensor(w, dtype=torch.float32).to(dev).contiguous() for w in weights]
        self.b = [None if b is None else torch.as_tensor(b, dtype=torch.float32).to(dev).contiguous() for b in biases]
        self.hops = int(hops)
        self.dims = [int(self.X.shape[1])] + [int(w.shape[1]) for w in self.W]
        n = self.indptr.numel() - 1
        self.graph = L.gnnshap_graph(num_nodes=n, num_edges=self.indices.numel(),
                                     indptr=self.indptr.data_ptr(), indices=self.indices.data_ptr())
        nl = len(self.W)
        self._dims = (ctypes.c_int32 * (nl + 1))(*self.dims)
        self._Wp = (ctypes.c_void_p * nl)(*[w.data_ptr() for w in self.W])
        self._bp = (ctypes.c_void_p * nl)(*[0 if b is None else b.data_ptr() for b in self.b])
        self.model = L.gnnshap_gcn(num_layers=nl, dims=self._dims, W=self._Wp, b=self._bp, XW1=None)
        self.XW1 = None
        self.extract_ws = torch.zeros(L.gnnshap_extract_workspace(n), dtype=torch.uint8, device=dev)
        self._cap = [1024, 8192]                 # node and edge capacity of new subgraph buffers
        self._sub = None
        self.ws_sample = _Buffer(dev)
        self.ws_eval = _Buffer(dev)
        self.ws_solve = _Buffer(dev)
        self.ws_batch = _Buffer(dev)
        self.ws_fid = _Buffer(dev)
        self._pipe = None
        self._bx = None                          # batched extraction: (n, zero-filled workspace)
        self._plans = {}                         # (M, p) -> (plan, classes): the plan does not depend on seed
        self._ncls_hint = 1024                   # class-table length explain_batch allocates
        self._xstream = None                     # stream of the batched extraction
        self._tg_cache = None                    # (target tuple, ctypes int64 array) of the last batch
        self.iterative_threshold = 0             # players above which systems are solved iteratively (0: 5000)

    def prepare(self):
        """gnnshap_transform_features: X W_1 for every node, shared by all targets."""
        n = self.X.shape[0]
        if self.XW1 is None:
            self.XW1 = torch.empty((n, self.dims[1]), dtype=torch.float32, device=self.device)
        L.gnnshap_transform_features(_vp(self.X), n, self.dims[0], _vp(self.W[0]), self.dims[1], _vp(self.XW1),
                                     self.stream())
        self.model.XW1 = self.XW1.data_ptr()

    def stream(self):
        return ctypes.c_void_p(torch.cuda.current_stream(self.device).cuda_stream)

    def _new_sub_buffers(self):
        dev = self.device
        cn, ce = self._cap
        return dict(node_gid=torch.empty(cn, dtype=torch.int32, device=dev),
                    dst_ptr=torch.empty(cn + 1, dtype=torch.int32, device=dev),
                    edge_src=torch.empty(ce, dtype=torch.int32, device=dev),
                    edge_dst=torch.empty(ce, dtype=torch.int32, device=dev),
                    edge_gid=torch.empty(ce, dtype=torch.int64, device=dev))

    def _extract(self, target, bufs):
        """gnnshap_extract_subgraph into `bufs` (grown and retried on ECAPACITY);
        blocks the host until the sizes are known."""
        while True:
            b = bufs
            sg = L.gnnshap_subgraph(num_hops=self.hops, cap_nodes=b["node_gid"].numel(),
                                    cap_edges=b["edge_src"].numel(), node_gid=b["node_gid"].data_ptr(),
                                    dst_ptr=b["dst_ptr"].data_ptr(), edge_src=b["edge_src"].data_ptr(),
                                    edge_dst=b["edge_dst"].data_ptr(), edge_gid=b["edge_gid"].data_ptr())
            st = L.gnnshap_extract_subgraph(self.graph, int(target), sg, _vp(self.extract_ws),
                                            self.extract_ws.numel(), self.stream())
            if st == L.OK:
                break
            self._cap = [max(int(sg.num_nodes * 1.25) + 16, self._cap[0]),
                         max(int(sg.num_edges * 1.25) + 64, self._cap[1])]
            bufs.clear()
            bufs.update(self._new_sub_buffers())
        n, m, nd = sg.num_nodes, sg.num_edges, sg.num_dst
        return Subgraph(sg=sg, node_gid=b["node_gid"][:n], dst_ptr=b["dst_ptr"][:nd + 1],
                        edge_src=b["edge_src"][:m], edge_dst=b["edge_dst"][:m], edge_gid=b["edge_gid"][:m])

    def extract(self, target):
        """The computational graph of one target (arrays valid until the next extract())."""
        if self._sub is None:
            self._sub = self._new_sub_buffers()
        return self._extract(target, self._sub)

    def explain(self, target, num_samples, seed, target_class=-1, stream_id=None):
        """Alg. 1 for one target: extract, plan, sample, evaluate, solve."""
        if self.XW1 is None:
            self.prepare()
        sub = self.extract(target)
        M = sub.sg.num_edges
        if M < 2:
            raise ValueError(f"target {target} has {M} players; at least 2 are needed")
        plan, classes = L.gnnshap_plan_samples(M, int(num_samples), int(seed),
                                               int(target if stream_id is None else stream_id),
                                               self.iterative_threshold)
        return self.run(sub, plan, classes, target_class, target)

    def explain_many(self, targets, num_samples, seed, target_class=-1, n_streams=3):
        """Alg. 1 for many targets.  Extraction (the only call that waits for
        the device) runs on its own stream into fresh buffers, so it never
        waits for compute; each target's sampling, evaluation and solve are
        enqueued on one of `n_streams` compute streams, so independent targets
        overlap on the GPU.  The compute streams are joined to the current
        stream before returning; results are complete once it synchronises."""
        if self.XW1 is None:
            self.prepare()
        main = torch.cuda.current_stream(self.device)
        if self._pipe is None or len(self._pipe[1]) != n_streams:
            self._pipe = (torch.cuda.Stream(self.device), [torch.cuda.Stream(self.device) for _ in range(n_streams)],
                          [(_Buffer(self.device), _Buffer(self.device), _Buffer(self.device))
                           for _ in range(n_streams)])
        ext, lanes, wss = self._pipe
        ext.wait_stream(main)
        for st in lanes:
            st.wait_stream(main)
        out = []
        for t, v in enumerate(targets):
            lane, ws = lanes[t % n_streams], wss[t % n_streams]
            with torch.cuda.stream(ext):
                bufs = self._new_sub_buffers()
                sub = self._extract(v, bufs)
            for tensor in bufs.values():
                tensor.record_stream(lane)
            M = sub.sg.num_edges
            if M < 2:
                raise ValueError(f"target {v} has {M} players; at least 2 are needed")
            plan, classes = L.gnnshap_plan_samples(M, int(num_samples), int(seed), int(v), self.iterative_threshold)
            with torch.cuda.stream(lane):
                out.append(self.run(sub, plan, classes, target_class, v, workspaces=ws))
        for st in lanes:
            main.wait_stream(st)
        return out

    def run(self, sub, plan, classes, target_class=-1, target=-1, workspaces=None):
        """Sample, evaluate and solve on the current stream."""
        dev, s = self.device, self.stream()
        ws_sample, ws_eval, ws_solve = workspaces or (self.ws_sample, self.ws_eval, self.ws_solve)
        k, wpr, M = plan.num_rows, plan.words_per_row, plan.num_players
        masks = torch.empty((k, wpr), dtype=torch.int64, device=dev)
        weights = torch.empty(k, dtype=torch.float32, device=dev)
        ws = ws_sample.get(L.gnnshap_sample_workspace(plan))
        L.gnnshap_sample_coalitions(plan, classes, _vp(masks), _vp(weights), _vp(ws), ws.numel(), s)
        y = torch.empty(k, dtype=torch.float32, device=dev)
        fef = torch.empty(2, dtype=torch.float32, device=dev)
        cls = torch.empty(1, dtype=torch.int32, device=dev)
        self._evaluate(sub, target_class, masks, k, wpr, y, fef, cls, ws_eval, s)
        phi = torch.empty(M, dtype=torch.float32, device=dev)
        info = torch.empty(1, dtype=torch.int32, device=dev)
        ws = ws_solve.get(L.gnnshap_solve_workspace(plan))
        L.gnnshap_solve_wls(plan, classes, _vp(masks), _vp(y), _vp(fef), _vp(phi), _vp(info), _vp(ws), ws.numel(), s)
        return Explanation(target=target, sub=sub, plan=plan, classes=classes, masks=masks, weights=weights, y=y,
                           f_empty_full=fef, cls=cls, phi=phi, info=info)

    def _evaluate(self, sub, target_class, masks, k, wpr, y, fef, cls, ws_eval, s):
        """gnnshap_eval_sampled_coalitions (the masks come from the sampler) on
        the current stream."""
        ws = ws_eval.get(L.gnnshap_eval_workspace(sub.sg, self.model, k))
        L.gnnshap_eval_sampled_coalitions(sub.sg, self.model, _vp(self.X), int(target_class), _vp(masks), k, wpr,
                                          _vp(y), _vp(fef), _vp(cls), _vp(ws), ws.numel(), s)

    # -- many targets per launch sequence ------------------------------------------------------

    def _plan(self, M, num_samples, seed, stream_id):
        key = (int(M), int(num_samples))
        hit = self._plans.get(key)
        if hit is None:
            hit = L.gnnshap_plan_samples(int(M), int(num_samples), 0, 0)
            self._plans[key] = hit
        plan, classes = hit
        out = L.gnnshap_sample_plan()
        ctypes.pointer(out)[0] = plan
        out.seed = int(seed)
        out.stream_id = int(stream_id)
        return out, classes

    def extract_batch(self, targets):
        """gnnshap_extract_batch: the computational graphs of all targets with one
        host synchronisation; capacities grow and the batch is redone on
        ECAPACITY.  Extraction runs on a stream of its own, so that waiting for
        the sizes does not wait for work queued earlier on the current stream;
        it is complete when the call returns.  Returns (BatchSubgraphs, ctypes
        array of gnnshap_subgraph)."""
        return self.extract_batch_finish(self.extract_batch_start(targets))

    def extract_batch_start(self, targets):
        """First half of extract_batch (gnnshap_extract_batch_launch): queues the
        extraction on the extraction stream and returns a pending batch for
        extract_batch_finish.  One batch may be pending at a time."""
        dev = self.device
        n = len(targets)
        if self._bx is None or self._bx[0] < n:
            nbytes = L.gnnshap_extract_batch_workspace(self.indptr.numel() - 1, n)
            self._bx = (n, torch.zeros(nbytes, dtype=torch.uint8, device=dev))
            torch.cuda.current_stream(dev).synchronize()
        ws = self._bx[1]
        key = tuple(int(v) for v in targets)
        if self._tg_cache is None or self._tg_cache[0] != key:
            self._tg_cache = (key, (ctypes.c_int64 * n)(*key))
        tg = self._tg_cache[1]
        main = torch.cuda.current_stream(dev)
        if self._xstream is None:
            self._xstream = torch.cuda.Stream(device=dev)
        xs = self._xstream
        cn, ce = self._cap
        with torch.cuda.stream(xs):
            bufs = BatchSubgraphs(n, cn, ce, dev)
        sgs = (L.gnnshap_subgraph * n)()
        L.gnnshap_subgraph_batch_init(sgs, self.hops, cn, ce, _vp(bufs.node_gid), _vp(bufs.dst_ptr),
                                      _vp(bufs.edge_src), _vp(bufs.edge_dst), _vp(bufs.edge_gid))
        L.gnnshap_extract_batch_launch(self.graph, tg, sgs, _vp(ws), ws.numel(), ctypes.c_void_p(xs.cuda_stream))
        # the buffers are used on the current stream once the sizes are back
        # (the extraction is then complete, so that stream needs no wait)
        bufs.buffer.record_stream(main)
        bufs.sgs = sgs
        bufs.targets = tg
        bufs.target_ids = key
        return bufs

    def extract_batch_finish(self, bufs):
        """Second half (gnnshap_extract_batch_finish): waits for the sizes; on
        ECAPACITY the capacities grow and the batch is extracted again.
        Returns (BatchSubgraphs, ctypes array of gnnshap_subgraph)."""
        sgs = bufs.sgs
        while L.gnnshap_extract_batch_finish(sgs) != L.OK:
            cn, ce = self._cap
            self._cap = [max(max(int(sg.num_nodes * 1.25) + 16 for sg in sgs), cn),
                         max(max(int(sg.num_edges * 1.25) + 64 for sg in sgs), ce)]
            bufs = self.extract_batch_start(bufs.target_ids)
            sgs = bufs.sgs
        return bufs, sgs

    def fidelity(self, explanations, sparsity=0.3, top_k=10, target_class=-1):
        """Fidelity- and Fidelity+ (eq. 7-8) of explanations whose subgraph
        arrays are still valid (explain()'s until the next extract(), a
        BatchExplanations' until the next batch): per target
        gnnshap_fidelity with the explanation's phi (G_S drops the
        floor(sparsity M) least important players by |phi|, G_C minus S the
        top_k most important; Sec. 4.6 uses 0.3 and 10), then
        gnnshap_fidelity_average.  Returns (terms, avg): float32 [n, 3] rows
        (Fidelity- term, Fidelity+ term, f(G_C)) and [2] (eq. 7, eq. 8), on
        the device, valid once the current stream has run."""
        items = list(explanations)
        n = len(items)
        terms = torch.empty((n, 3), dtype=torch.float32, device=self.device)
        avg = torch.empty(2, dtype=torch.float32, device=self.device)
        s = self.stream()
        for t, e in enumerate(items):
            nbytes = L.gnnshap_fidelity_workspace(e.sub.sg, self.model)
            ws = self.ws_fid.get(nbytes)
            L.gnnshap_fidelity(e.sub.sg, self.model, _vp(self.X), target_class, _vp(e.phi), sparsity, top_k,
                               _vp(terms[t]), _vp(ws), ws.numel(), s)
        L.gnnshap_fidelity_average(_vp(terms), n, 3, _vp(avg), s)
        return terms, avg

    def explain_batch(self, targets, num_samples, seed, target_class=-1):
        """Alg. 1 for every target, one launch per step for the whole batch
        (gnnshap_extract_batch, then gnnshap_explain_batch); each target's
        Philox stream is its node id.  Results equal explain()'s bit for bit.
        Returns a BatchExplanations (packed tensors, valid once the current
        stream has run; indexing gives per-target Explanation views)."""
        if self.XW1 is None:
            self.prepare()
        subs, sgs = self.extract_batch(targets)
        return self._explain_extracted(subs, sgs, num_samples, seed, target_class)

    def explain_batches(self, batches, num_samples, seed, target_class=-1, prepare_each=False):
        """explain_batch over a sequence of target batches, pipelined: the next
        batch's extraction is queued before the current batch's explanation,
        so that its sizes are ready when they are needed.  prepare_each: X W_1
        again before every batch.  Yields one BatchExplanations per batch, in
        order; each equals explain_batch's for the same batch."""
        it = iter(batches)
        first = next(it, None)
        if first is None:
            return
        pend = self.extract_batch_start(first)
        try:
            while pend is not None:
                if prepare_each or self.XW1 is None:
                    self.prepare()
                subs, sgs = self.extract_batch_finish(pend)
                pend = None
                nxt = next(it, None)
                pend = self.extract_batch_start(nxt) if nxt is not None else None
                yield self._explain_extracted(subs, sgs, num_samples, seed, target_class)
        finally:
            if pend is not None:          # stopped early: collect the queued extraction
                L.gnnshap_extract_batch_finish(pend.sgs)

    def _explain_extracted(self, subs, sgs, num_samples, seed, target_class):
        """Plans and gnnshap_explain_batch for extracted subgraphs."""
        dev = self.device
        n = len(sgs)
        targets = subs.target_ids
        plans = (L.gnnshap_sample_plan * n)()
        cl = (L.gnnshap_class * self._ncls_hint)()
        st, ncls, totals = L.gnnshap_plan_batch(sgs, subs.targets, int(num_samples), int(seed), plans, cl)
        if st == L.ECAPACITY:
            self._ncls_hint = ncls + ncls // 4
            cl = (L.gnnshap_class * self._ncls_hint)()
            st, ncls, totals = L.gnnshap_plan_batch(sgs, subs.targets, int(num_samples), int(seed), plans, cl)
        for t in range(n):
            plans[t].iterative_threshold = self.iterative_threshold
        out = BatchExplanations(targets, subs, plans, cl, ncls, totals, dev)
        # the workspace is sized on demand: the call checks it before queueing anything
        ptrs = out.pointers()
        ws = self.ws_batch.t
        st = L.ECAPACITY
        if ws is not None:
            st = self._batch_call(sgs, plans, cl, target_class, ptrs, ws)
        if st == L.ECAPACITY:
            ws = self.ws_batch.get(self._batch_workspace(sgs, plans))
            L.check(self._batch_call(sgs, plans, cl, target_class, ptrs, ws), "explain_batch")
        return out

    def _batch_workspace(self, sgs, plans):
        return L.gnnshap_explain_batch_workspace(sgs, plans, self.model)

    def _batch_call(self, sgs, plans, cl, target_class, ptrs, ws):
        """gnnshap_explain_batch on the current stream (OK or ECAPACITY)."""
        return L.gnnshap_explain_batch(sgs, plans, cl, self.model, _vp(self.X), int(target_class), *ptrs,
                                       _vp(ws), ws.numel(), self.stream())


class BatchSubgraphs:
    """Packed subgraph buffers of a batch, views of one device allocation:
    target t owns row t of each array."""

    def __init__(self, n, cap_nodes, cap_edges, dev):
        shapes = (("node_gid", torch.int32, 4, (n, cap_nodes)), ("dst_ptr", torch.int32, 4, (n, cap_nodes + 1)),
                  ("edge_src", torch.int32, 4, (n, cap_edges)), ("edge_dst", torch.int32, 4, (n, cap_edges)),
                  ("edge_gid", torch.int64, 8, (n, cap_edges)))
        offs, off = [], 0
        for _, _, es, shp in shapes:
            offs.append(off)
            off = (off + shp[0] * shp[1] * es + 255) // 256 * 256
        self.buffer = torch.empty(max(off, 256), dtype=torch.uint8, device=dev)
        for (name, dt, es, shp), o in zip(shapes, offs):
            setattr(self, name, self.buffer[o:o + shp[0] * shp[1] * es].view(dt).view(shp))
        self.sgs = None

    def __getitem__(self, t):
        sg = self.sgs[t]
        m, nn, nd = sg.num_edges, sg.num_nodes, sg.num_dst
        return Subgraph(sg=sg, node_gid=self.node_gid[t, :nn], dst_ptr=self.dst_ptr[t, :nd + 1],
                        edge_src=self.edge_src[t, :m], edge_dst=self.edge_dst[t, :m], edge_gid=self.edge_gid[t, :m])


class BatchExplanations:
    """Outputs of gnnshap_explain_batch, packed in target order in one device
    allocation; entry t is materialised as an Explanation (tensor views) on
    access.  `classes` holds the concatenated class tables (the first
    num_classes records)."""

    _FIELDS = (("masks", torch.int64, 8), ("weights", torch.float32, 4), ("y", torch.float32, 4),
               ("fef", torch.float32, 4), ("cls", torch.int32, 4), ("phi", torch.float32, 4),
               ("info", torch.int32, 4))

    def __init__(self, targets, subs, plans, classes, num_classes, totals, dev):
        n = len(targets)
        self.targets, self.subs, self.plans, self.classes, self.num_classes = targets, subs, plans, classes, num_classes
        words, rows, players = totals
        self.total_rows = rows
        counts = (words, rows, rows, 2 * n, n, players, n)
        self._span, off = {}, 0
        for (name, _, size), c in zip(self._FIELDS, counts):
            self._span[name] = (off, c)
            off += (c * size + 255) // 256 * 256
        self.buf = torch.empty(max(off, 256), dtype=torch.uint8, device=dev)
        self._offs = None

    def pointers(self):
        """Device addresses of the seven outputs, in gnnshap_explain_batch's order."""
        base = self.buf.data_ptr()
        return tuple(ctypes.c_void_p(base + self._span[name][0]) for name, _, _ in self._FIELDS)

    def _view(self, name):
        off, c = self._span[name]
        dt, size = next((d, z) for f, d, z in self._FIELDS if f == name)
        return self.buf[off:off + c * size].view(dt)

    masks = property(lambda self: self._view("masks"))
    weights = property(lambda self: self._view("weights"))
    y = property(lambda self: self._view("y"))
    fef = property(lambda self: self._view("fef"))
    cls = property(lambda self: self._view("cls"))
    phi = property(lambda self: self._view("phi"))
    info = property(lambda self: self._view("info"))

    def _offsets(self):
        if self._offs is None:
            mo, ro, po, co = [0], [0], [0], [0]
            for p in self.plans:
                mo.append(mo[-1] + p.num_rows * p.words_per_row)
                ro.append(ro[-1] + p.num_rows)
                po.append(po[-1] + p.num_players)
                co.append(co[-1] + p.num_classes)
            self._offs = (mo, ro, po, co)
        return self._offs

    def __len__(self):
        return len(self.targets)

    def __getitem__(self, t):
        if t < 0:
            t += len(self)
        mo, ro, po, co = (o[t] for o in self._offsets())
        p = self.plans[t]
        k, w, M = p.num_rows, p.words_per_row, p.num_players
        tab = (L.gnnshap_class * p.num_classes)(*self.classes[co:co + p.num_classes])
        masks, weights, y, fef, cls, phi, info = (self._view(f) for f, _, _ in self._FIELDS)
        return Explanation(target=self.targets[t], sub=self.subs[t], plan=p, classes=tab,
                           masks=masks[mo:mo + k * w].view(k, w), weights=weights[ro:ro + k],
                           y=y[ro:ro + k], f_empty_full=fef[2 * t:2 * t + 2], cls=cls[t:t + 1],
                           phi=phi[po:po + M], info=info[t:t + 1])

    def __iter__(self):
        return (self[t] for t in range(len(self)))


class GatExplainer(Explainer):
    """Alg. 1 for a two-layer GAT (App. E): the same extraction (2 hops),
    plan, sampler and least squares as Explainer, with the coalition values
    of gnnshap_gat_eval_coalitions.  `params` as workloads.glorot_gat makes
    them (W1, att_src1, att_dst1, b1, W2, att_src2, att_dst2, b2).  Batches
    go through gnnshap_gat_explain_batch (explain_batch, explain_batches)."""

    def __init__(self, indptr, indices, X, params, device="cuda", negative_slope=0.2):
        heads, head_dim = (int(v) for v in params["att_src1"].shape)
        classes = int(params["W2"].shape[1])
        super().__init__(indptr, indices, X, [params["W1"], params["W2"]], [params["b1"], params["b2"]], 2, device)
        self.gat_params = {k: torch.as_tensor(v, dtype=torch.float32).to(self.device).contiguous()
                           for k, v in params.items()}
        p = self.gat_params
        self.gat = L.gnnshap_gat(heads=heads, head_dim=head_dim, num_classes=classes, XW1=None,
                                 att_src1=p["att_src1"].data_ptr(), att_dst1=p["att_dst1"].data_ptr(),
                                 b1=p["b1"].data_ptr(), W2=p["W2"].data_ptr(), att_src2=p["att_src2"].data_ptr(),
                                 att_dst2=p["att_dst2"].data_ptr(), b2=p["b2"].data_ptr(),
                                 negative_slope=float(negative_slope))

    def prepare(self):
        super().prepare()
        self.gat.XW1 = self.XW1.data_ptr()

    def _evaluate(self, sub, target_class, masks, k, wpr, y, fef, cls, ws_eval, s):
        """gnnshap_gat_eval_coalitions on the current stream."""
        ws = ws_eval.get(L.gnnshap_gat_eval_workspace(sub.sg, self.gat, k))
        L.gnnshap_gat_eval_coalitions(sub.sg, self.gat, int(target_class), _vp(masks), k, wpr, _vp(y), _vp(fef),
                                      _vp(cls), _vp(ws), ws.numel(), s)

    def _batch_workspace(self, sgs, plans):
        return L.gnnshap_gat_explain_batch_workspace(sgs, plans, self.gat)

    def _batch_call(self, sgs, plans, cl, target_class, ptrs, ws):
        """gnnshap_gat_explain_batch on the current stream (OK or ECAPACITY)."""
        if not self.gat.XW1:
            raise RuntimeError("GatExplainer.prepare() must run before explaining (X W_1 of every node)")
        return L.gnnshap_gat_explain_batch(sgs, plans, cl, self.gat, int(target_class), *ptrs, _vp(ws), ws.numel(),
                                           self.stream())

    def fidelity(self, *args, **kwargs):
        raise NotImplementedError("gnnshap_fidelity evaluates GCNs")
