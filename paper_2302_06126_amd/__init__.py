"""MI355X (gfx950) hot path of TAG's strategy search: heterogeneous-GNN
forward pass over batches of candidate deployment graphs plus the per-op
decision head, behind the C ABI in include/tag.h.

This module only marshals arguments: torch provides device memory and the
current HIP stream, and every step of the computation runs in libtag.so.
The same names as the C ABI are exported (``tag_graph_plan``,
``tag_graph_build``, ``tag_gnn_forward``, ...), plus small convenience
classes that own the device buffers those calls need.
"""
from __future__ import annotations

import ctypes as C
from typing import Dict, Optional, Sequence

import numpy as np

from . import _abi
from ._abi import (TAG_BF16, TAG_F32, TagError, check, tag_decision, tag_features, tag_graph_desc,
                   tag_graph_info, tag_model_dims, tag_slices, tag_weights)

__all__ = ["Graph", "Model", "tag_graph_plan", "tag_graph_build", "tag_graph_get_info", "tag_graph_export",
           "tag_graph_destroy", "tag_gnn_workspace", "tag_gnn_forward", "tag_gnn_decide_workspace",
           "tag_gnn_decide", "tag_last_error", "tag_version", "tag_profile_begin", "tag_profile_end",
           "forward", "decide", "TagError",
           "TAG_F32", "TAG_BF16"]


def _torch():
    import torch
    return torch


def _ptr(t) -> Optional[int]:
    return None if t is None else int(t.data_ptr())


def _stream(stream=None) -> int:
    torch = _torch()
    s = stream if stream is not None else torch.cuda.current_stream()
    return int(s.cuda_stream)


class _OnStream:
    """Orders a one-shot call on `stream` against torch's current stream: the
    given stream first waits for the current one (which allocated and filled
    the temporaries), and on exit the current stream waits for the given one,
    so results read and temporaries freed on the current stream come after
    the library's kernels."""

    def __init__(self, stream):
        self.stream = stream

    def __enter__(self):
        torch = _torch()
        self.cur = torch.cuda.current_stream()
        if self.stream is not None and self.stream != self.cur:
            self.stream.wait_stream(self.cur)
        return self

    def __exit__(self, *exc):
        if self.stream is not None and self.stream != self.cur:
            self.cur.wait_stream(self.stream)
        return False


# ------------------------------------------------------------ C-ABI names --

def tag_last_error() -> str:
    return _abi.load().tag_last_error().decode(errors="replace")


def tag_version() -> str:
    return _abi.load().tag_version().decode()


def tag_profile_begin(stage: int, capacity: int) -> int:
    return _abi.load().tag_profile_begin(stage, capacity)


def tag_profile_end():
    ms, n = C.c_double(0.0), C.c_int32(0)
    st = _abi.load().tag_profile_end(C.byref(ms), C.byref(n))
    return st, ms.value, n.value


def tag_graph_plan(desc: tag_graph_desc):
    cb, tb = C.c_size_t(0), C.c_size_t(0)
    st = _abi.load().tag_graph_plan(C.byref(desc), C.byref(cb), C.byref(tb))
    return st, cb.value, tb.value


def tag_graph_build(desc: tag_graph_desc, csr_buf, csr_bytes: int, tmp_buf, tmp_bytes: int, stream: int):
    out = C.c_void_p(None)
    st = _abi.load().tag_graph_build(C.byref(desc), csr_buf, csr_bytes, tmp_buf, tmp_bytes, stream, C.byref(out))
    return st, out.value


def tag_graph_get_info(handle: int):
    info = tag_graph_info()
    st = _abi.load().tag_graph_get_info(handle, C.byref(info))
    return st, info


def tag_graph_export(handle: int, bucket: int, rowptr, col, eid) -> int:
    return _abi.load().tag_graph_export(handle, bucket, rowptr, col, eid)


def tag_graph_destroy(handle: int) -> None:
    _abi.load().tag_graph_destroy(handle)


def tag_gnn_workspace(handle: int, dims: tag_model_dims, n_replicas: int):
    b = C.c_size_t(0)
    st = _abi.load().tag_gnn_workspace(handle, C.byref(dims), n_replicas, C.byref(b))
    return st, b.value


def tag_gnn_forward(handle, dims, weights, feats, workspace, ws_bytes, E_op, E_dev, stream) -> int:
    return _abi.load().tag_gnn_forward(handle, C.byref(dims), C.byref(weights), C.byref(feats), workspace,
                                       ws_bytes, E_op, E_dev, stream)


def tag_gnn_decide_workspace(handle, dims, n_replicas, n_slices, n_query):
    b = C.c_size_t(0)
    st = _abi.load().tag_gnn_decide_workspace(handle, C.byref(dims), n_replicas, n_slices, n_query, C.byref(b))
    return st, b.value


def tag_gnn_decide(handle, dims, weights, n_replicas, E_op, E_dev, slices, n_query, q_rep, q_graph, q_op,
                   argmax, best, prior, decision, workspace, ws_bytes, stream) -> int:
    return _abi.load().tag_gnn_decide(handle, C.byref(dims), C.byref(weights), n_replicas, E_op, E_dev,
                                      C.byref(slices), n_query, q_rep, q_graph, q_op, argmax, best, prior,
                                      decision, workspace, ws_bytes, stream)


# --------------------------------------------------------- convenience ----

class Graph:
    """A built joint graph on the GPU: a batch of G topologies.

    `topologies` is a sequence of objects with n_op, n_dev, oo_src, oo_dst,
    dd_a, dd_b, od_op, od_dev (local ids, numpy int32)."""

    def __init__(self, topologies: Sequence, device: str = "cuda", stream=None):
        torch = _torch()
        self.device = torch.device(device)
        G = len(topologies)
        cat = lambda name: np.concatenate([np.asarray(getattr(t, name), np.int32) for t in topologies]) \
            if G else np.zeros(0, np.int32)
        offs = lambda a, b: np.concatenate([[0], np.cumsum([len(getattr(t, a)) for t in topologies])]).astype(np.int64)
        self._n_op = np.array([t.n_op for t in topologies], np.int32)
        self._n_dev = np.array([t.n_dev for t in topologies], np.int32)
        self._oo_off, self._dd_off, self._od_off = offs("oo_src", 0), offs("dd_a", 0), offs("od_op", 0)
        dev = lambda a: torch.from_numpy(np.ascontiguousarray(a)).to(self.device) if len(a) else None
        self._edges = {k: dev(cat(k)) for k in ("oo_src", "oo_dst", "dd_a", "dd_b", "od_op", "od_dev")}
        d = tag_graph_desc()
        d.n_graphs = G
        d.n_op = self._n_op.ctypes.data_as(C.POINTER(C.c_int32))
        d.n_dev = self._n_dev.ctypes.data_as(C.POINTER(C.c_int32))
        d.oo_off = self._oo_off.ctypes.data_as(C.POINTER(C.c_int64))
        d.dd_off = self._dd_off.ctypes.data_as(C.POINTER(C.c_int64))
        d.od_off = self._od_off.ctypes.data_as(C.POINTER(C.c_int64))
        for k, v in self._edges.items():
            setattr(d, k, _ptr(v))
        self.desc = d
        st, cb, tb = tag_graph_plan(d)
        check(st, "tag_graph_plan")
        self.csr = torch.empty(cb, dtype=torch.uint8, device=self.device)
        tmp = torch.empty(tb, dtype=torch.uint8, device=self.device)
        with _OnStream(stream):
            st, h = tag_graph_build(d, _ptr(self.csr), cb, _ptr(tmp), tb, _stream(stream))
        check(st, "tag_graph_build")
        del tmp
        self.handle = h
        st, self.info = tag_graph_get_info(h)
        check(st, "tag_graph_get_info")
        self.op_off = np.concatenate([[0], np.cumsum(self._n_op)]).astype(np.int64)
        self.dev_off = np.concatenate([[0], np.cumsum(self._n_dev)]).astype(np.int64)

    @property
    def n_op(self) -> int:
        return int(self.info.n_op)

    @property
    def n_dev(self) -> int:
        return int(self.info.n_dev)

    def export(self, bucket: int):
        rows, nnz = int(self.info.rows[bucket]), int(self.info.nnz[bucket])
        rp = np.zeros(rows + 1, np.int32)
        col = np.zeros(max(nnz, 1), np.int32)
        eid = np.zeros(max(nnz, 1), np.int32)
        st = tag_graph_export(self.handle, bucket, rp.ctypes.data, col.ctypes.data, eid.ctypes.data)
        check(st, "tag_graph_export")
        return rp, col[:nnz], eid[:nnz]

    def close(self) -> None:
        if getattr(self, "handle", None):
            tag_graph_destroy(self.handle)
            self.handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


class Model:
    """Model dimensions plus device copies of the parameters (fp32)."""

    def __init__(self, weights: Dict[str, np.ndarray], *, f: int, heads: int, layers: int, f_op: int,
                 f_dev: int = 8, dec_hidden: Optional[int] = None, dtype: str = "f32",
                 gamma_same: float = 1.0, gamma_cross: float = 0.1, leaky_slope: float = 0.2,
                 device: str = "cuda", sigma: str = "relu", relations: int = 3, edge_act: str = "affine",
                 heads_mode: str = "concat"):
        torch = _torch()
        if dec_hidden is None:
            dec_hidden = int(weights["dec_w1"].shape[0])
        if sigma not in ("relu", "elu"):
            raise ValueError("sigma must be 'relu' or 'elu'")
        if relations not in (3, 5) or edge_act not in ("affine", "relu") or heads_mode not in ("concat", "avg"):
            raise ValueError("relations must be 3 or 5, edge_act 'affine' or 'relu', heads_mode 'concat' or 'avg'")
        self.dims = tag_model_dims(f, heads, layers, f_op, f_dev, dec_hidden,
                                   TAG_BF16 if dtype == "bf16" else TAG_F32,
                                   gamma_same, gamma_cross, leaky_slope, 1 if sigma == "elu" else 0,
                                   relations, 1 if edge_act == "relu" else 0, 1 if heads_mode == "avg" else 0)
        self.t = {k: torch.from_numpy(np.ascontiguousarray(v, np.float32).reshape(-1).copy()).to(device)
                  for k, v in weights.items()}
        # non-empty placeholders keep every pointer valid
        for k in ("dec_w1", "dec_b1"):
            if self.t[k].numel() == 0:
                self.t[k] = torch.zeros(1, dtype=torch.float32, device=device)
        w = tag_weights()
        g = lambda k: _ptr(self.t[k])
        w.enc_op_w, w.enc_op_b, w.enc_dev_w, w.enc_dev_b = g("enc_op_w"), g("enc_op_b"), g("enc_dev_w"), g("enc_dev_b")
        for r in range(3):
            w.enc_edge_w[r] = g(f"enc_edge_w{r}")
            w.enc_edge_b[r] = g(f"enc_edge_b{r}")
        w.layer_w, w.layer_b, w.att_src, w.att_dst = g("layer_w"), g("layer_b"), g("att_src"), g("att_dst")
        w.dec_w1, w.dec_b1, w.dec_w2, w.dec_b2 = g("dec_w1"), g("dec_b1"), g("dec_w2"), g("dec_b2")
        self.weights = w


def make_features(x_op, x_dev, x_oo, x_dd, x_od) -> tag_features:
    """Features for R replicas from device tensors: x_op [R,N,F_op],
    x_dev [R,M,F_dev], x_oo [E_oo] or [R,E_oo], x_dd [E_dd,2] or [R,E_dd,2],
    x_od [E_od] or [R,E_od] (uint8).  A tensor without the replica axis is
    shared by all replicas (stride 0)."""
    R = int(x_op.shape[0])
    f = tag_features()
    f.n_replicas = R
    f.x_op, f.x_dev = _ptr(x_op), _ptr(x_dev)
    f.x_oo, f.x_dd, f.x_od = _ptr(x_oo), _ptr(x_dd), _ptr(x_od)
    f.stride_oo = int(x_oo.shape[1]) if x_oo is not None and x_oo.dim() == 2 else 0
    f.stride_dd = int(x_dd.shape[1] * 2) if x_dd is not None and x_dd.dim() == 3 else 0
    f.stride_od = int(x_od.shape[1]) if x_od is not None and x_od.dim() == 2 else 0
    return f


class Forward:
    """Reusable forward call: owns the workspace and the output tensors."""

    def __init__(self, graph: Graph, model: Model, n_replicas: int):
        torch = _torch()
        self.graph, self.model, self.R = graph, model, n_replicas
        st, b = tag_gnn_workspace(graph.handle, model.dims, n_replicas)
        check(st, "tag_gnn_workspace")
        self.ws_bytes = b
        self.ws = torch.empty(b, dtype=torch.uint8, device=graph.device)
        F = model.dims.f
        self.E_op = torch.empty((n_replicas, graph.n_op, F), dtype=torch.float32, device=graph.device)
        self.E_dev = torch.empty((n_replicas, graph.n_dev, F), dtype=torch.float32, device=graph.device)

    def __call__(self, feats: tag_features, stream=None):
        st = tag_gnn_forward(self.graph.handle, self.model.dims, self.model.weights, feats, _ptr(self.ws),
                             self.ws_bytes, _ptr(self.E_op), _ptr(self.E_dev), _stream(stream))
        check(st, "tag_gnn_forward")
        return self.E_op, self.E_dev


def forward(graph: Graph, model: Model, x_op, x_dev, x_oo, x_dd, x_od, stream=None):
    fw = Forward(graph, model, int(x_op.shape[0]))
    keep = (x_op, x_dev, x_oo, x_dd, x_od)
    with _OnStream(stream):
        E_op, E_dev = fw(make_features(*keep), stream)
    return E_op, E_dev


class Decide:
    """Reusable decide call for fixed (R, slice table, queries)."""

    def __init__(self, graph: Graph, model: Model, n_replicas: int, masks, options, q_rep, q_graph, q_op,
                 want_prior: bool = True):
        torch = _torch()
        dev = graph.device
        self.graph, self.model, self.R = graph, model, n_replicas
        self.masks = torch.from_numpy(np.ascontiguousarray(masks, np.uint64).view(np.int64)).to(dev)
        self.options = torch.from_numpy(np.ascontiguousarray(options, np.uint8)).to(dev)
        self.q = [torch.from_numpy(np.ascontiguousarray(a, np.int32)).to(dev) for a in (q_rep, q_graph, q_op)]
        self.S, self.Q = len(masks), len(q_op)
        self.slices = tag_slices(self.S, _ptr(self.masks), _ptr(self.options))
        st, b = tag_gnn_decide_workspace(graph.handle, model.dims, n_replicas, self.S, self.Q)
        check(st, "tag_gnn_decide_workspace")
        self.ws_bytes = b
        self.ws = torch.empty(max(b, 1), dtype=torch.uint8, device=dev)
        Q = max(self.Q, 1)
        self.argmax = torch.empty(Q, dtype=torch.int32, device=dev)
        self.best = torch.empty(Q, dtype=torch.float32, device=dev)
        self.prior = torch.empty((Q, self.S), dtype=torch.float32, device=dev) if want_prior else None
        self.decision = torch.empty((Q, C.sizeof(tag_decision)), dtype=torch.uint8, device=dev)

    def __call__(self, E_op, E_dev, stream=None):
        st = tag_gnn_decide(self.graph.handle, self.model.dims, self.model.weights, self.R, _ptr(E_op), _ptr(E_dev),
                            self.slices, self.Q, _ptr(self.q[0]), _ptr(self.q[1]), _ptr(self.q[2]),
                            _ptr(self.argmax), _ptr(self.best), _ptr(self.prior), _ptr(self.decision),
                            _ptr(self.ws), self.ws_bytes, _stream(stream))
        check(st, "tag_gnn_decide")

    def results(self) -> dict:
        """Copy the last call's outputs to host numpy arrays."""
        Q = self.Q
        raw = self.decision[:Q].cpu().numpy()
        rec = np.frombuffer(raw.tobytes(), dtype=np.dtype([("mask", "<u8"), ("option", "<i4"), ("replicas", "<i4"),
                                                          ("sync", "<i4"), ("sfb", "<i4")]))
        out = dict(argmax=self.argmax[:Q].cpu().numpy(), best=self.best[:Q].cpu().numpy(),
                   mask=rec["mask"], option=rec["option"], replicas=rec["replicas"], sync=rec["sync"],
                   sfb=rec["sfb"])
        if self.prior is not None:
            out["prior"] = self.prior[:Q].cpu().numpy()
        return out


def decide(graph: Graph, model: Model, E_op, E_dev, masks, options, q_rep, q_graph, q_op, want_prior=True,
           stream=None) -> dict:
    d = Decide(graph, model, int(E_op.shape[0]), masks, options, q_rep, q_graph, q_op, want_prior)
    with _OnStream(stream):
        d(E_op, E_dev, stream)
    return d.results()


def decide_full(graph: Graph, model: Model, E_op, E_dev, q_rep, q_graph, q_op, want_prior: bool = True,
                stream=None) -> dict:
    """Full-enumeration decision head (tag_gnn_decide_full): every non-empty
    device mask with each option, slice a = 4 (mask - 1) + option."""
    torch = _torch()
    dev = graph.device
    lib = _abi.load()
    q = [torch.from_numpy(np.ascontiguousarray(a, np.int32)).to(dev) for a in (q_rep, q_graph, q_op)]
    Q = len(q_op)
    R = int(E_op.shape[0])
    b = C.c_size_t(0)
    check(lib.tag_gnn_decide_full_workspace(graph.handle, C.byref(model.dims), R, Q, C.byref(b)),
          "tag_gnn_decide_full_workspace")
    ws = torch.empty(max(b.value, 1), dtype=torch.uint8, device=dev)
    S_full = 4 * ((1 << int(graph.info.max_dev)) - 1)
    argmax = torch.empty(max(Q, 1), dtype=torch.int32, device=dev)
    best = torch.empty(max(Q, 1), dtype=torch.float32, device=dev)
    prior = torch.empty((max(Q, 1), S_full), dtype=torch.float32, device=dev) if want_prior else None
    decision = torch.empty((max(Q, 1), C.sizeof(tag_decision)), dtype=torch.uint8, device=dev)
    with _OnStream(stream):
        check(lib.tag_gnn_decide_full(graph.handle, C.byref(model.dims), C.byref(model.weights), R, _ptr(E_op),
                                      _ptr(E_dev), Q, _ptr(q[0]), _ptr(q[1]), _ptr(q[2]), _ptr(argmax),
                                      _ptr(best), _ptr(prior), _ptr(decision), _ptr(ws), b.value,
                                      _stream(stream)),
              "tag_gnn_decide_full")
    raw = decision[:Q].cpu().numpy()
    rec = np.frombuffer(raw.tobytes(), dtype=np.dtype([("mask", "<u8"), ("option", "<i4"), ("replicas", "<i4"),
                                                      ("sync", "<i4"), ("sfb", "<i4")]))
    out = dict(argmax=argmax[:Q].cpu().numpy(), best=best[:Q].cpu().numpy(), mask=rec["mask"],
               option=rec["option"], replicas=rec["replicas"], sync=rec["sync"], sfb=rec["sfb"])
    if want_prior:
        out["prior"] = prior[:Q].cpu().numpy()
    return out
