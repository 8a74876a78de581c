"""Binding of include/tag_search.h: the batched strategy-search service.

Argument marshalling only: the search tree, the reward model and the state
packing run in libtag.so's host code, the feature expansion, the GNN forward
pass and the decision head in its HIP kernels.  torch provides device memory,
pinned host staging and the stream.
"""
from __future__ import annotations

import ctypes as C
from typing import Dict, List, Optional, Tuple

import numpy as np

from . import _abi
from ._abi import check, tag_search_problem_desc

__all__ = ["SearchProblem", "Mcts", "SearchService"]


def _i32(a) -> np.ndarray:
    return np.ascontiguousarray(np.asarray(a, dtype=np.int32))


def _f64(a) -> np.ndarray:
    return np.ascontiguousarray(np.asarray(a, dtype=np.float64))


class SearchProblem:
    """Host handle of a search problem.  `sp` carries the topology (ops,
    devices, links, op-device pairs and their attributes), the op grouping,
    per-op parameter bytes and the slice table (``synth.SearchProblem``
    layout).  `model` picks the reward and runtime-feedback model: the
    analytic iteration-time model or the simulator."""

    def __init__(self, sp, f_op: int = 42, model: str = "analytic"):
        t = sp.topo
        self.keep = keep = {
            "group_of": _i32(sp.group_of), "op_type": _i32(t.op_type), "op_flops": _f64(t.op_flops),
            "op_bytes": _f64(t.op_bytes), "op_params": _f64(sp.op_params), "dev_tflops": _f64(t.dev_tflops),
            "dev_mem_gb": _f64(t.dev_mem), "dev_intra_gbs": _f64(t.dev_intra_bw), "dd_a": _i32(t.dd_a),
            "dd_b": _i32(t.dd_b), "dd_gbs": _f64(t.dd_bw), "oo_src": _i32(t.oo_src), "oo_dst": _i32(t.oo_dst),
            "od_op": _i32(t.od_op), "od_dev": _i32(t.od_dev),
            "slice_mask": np.ascontiguousarray(np.asarray(sp.masks, np.uint64)),
            "slice_option": np.ascontiguousarray(np.asarray(sp.options, np.uint8))}
        d = tag_search_problem_desc()
        d.n_op, d.n_dev, d.n_groups, d.n_slices, d.f_op = t.n_op, t.n_dev, sp.n_groups, len(sp.masks), f_op
        for k, v in keep.items():
            setattr(d, k, v.ctypes.data)
        d.e_dd, d.e_oo, d.e_od = t.e_dd, t.e_oo, t.e_od
        h = C.c_void_p(None)
        check(_abi.load().tag_search_problem_create(C.byref(d), C.byref(h)), "tag_search_problem_create")
        self.h = h.value
        self.n_op, self.n_dev, self.n_groups, self.n_slices, self.f_op = t.n_op, t.n_dev, sp.n_groups, len(sp.masks), f_op
        self.e_od, self.e_dd = t.e_od, t.e_dd
        if model not in ("analytic", "simulator"):
            raise ValueError("model must be 'analytic' or 'simulator'")
        if model == "simulator":
            check(_abi.load().tag_search_set_model(self.h, 1), "tag_search_set_model")
        self.model = model

    def order(self) -> Tuple[np.ndarray, np.ndarray]:
        order = np.zeros(self.n_groups, np.int32)
        rep = np.zeros(self.n_groups, np.int32)
        check(_abi.load().tag_search_order(self.h, order.ctypes.data, rep.ctypes.data), "tag_search_order")
        return order, rep

    def evaluate(self, path) -> Tuple[float, float, bool]:
        p = _i32(path)
        r, T, oom = C.c_double(0), C.c_double(0), C.c_int32(0)
        check(_abi.load().tag_search_evaluate(self.h, p.ctypes.data if p.size else None, int(p.size),
                                              C.byref(r), C.byref(T), C.byref(oom)), "tag_search_evaluate")
        return r.value, T.value, bool(oom.value)

    def simulate(self, path) -> dict:
        """Runtime feedback of the strategy ``path`` (tag_simulate)."""
        p = _i32(path)
        out = _abi.tag_sim_out()
        arrs = {"group_makespan": np.zeros(self.n_groups), "group_idle": np.zeros(self.n_groups),
                "dev_peak": np.zeros(self.n_dev), "dev_idle": np.zeros(self.n_dev),
                "link_idle": np.zeros(max(self.e_dd, 1))}
        for k, v in arrs.items():
            setattr(out, k, v.ctypes.data)
        check(_abi.load().tag_simulate(self.h, p.ctypes.data if p.size else None, int(p.size), C.byref(out)),
              "tag_simulate")
        arrs["link_idle"] = arrs["link_idle"][:self.e_dd]
        return dict(T=out.iter_time, valid=bool(out.valid), oom=bool(out.oom), n_tasks=int(out.n_tasks), **arrs)

    def simulate_batch(self, depth, path, n_threads: int = 1) -> Tuple[np.ndarray, np.ndarray]:
        """Iteration times and OOM flags of B strategies (tag_simulate_batch)."""
        d = _i32(depth)
        p = _i32(path).reshape(len(d), -1)
        B = int(d.size)
        T = np.zeros(B)
        oom = np.zeros(B, np.int32)
        check(_abi.load().tag_simulate_batch(self.h, B, d.ctypes.data, p.ctypes.data, p.shape[1], n_threads,
                                             T.ctypes.data, oom.ctypes.data), "tag_simulate_batch")
        return T, oom.astype(bool)

    def device_bytes(self) -> Tuple[int, int]:
        a, b = C.c_size_t(0), C.c_size_t(0)
        check(_abi.load().tag_search_device_bytes(self.h, C.byref(a), C.byref(b)), "tag_search_device_bytes")
        return a.value, b.value

    def pack(self, depth: np.ndarray, path: np.ndarray, states: int):
        """Rewards and query ops of B leaves; writes the records to `states`
        (host address of B * state_bytes bytes)."""
        B = int(depth.shape[0])
        rewards = np.zeros(B, np.float64)
        qop = np.zeros(B, np.int32)
        check(_abi.load().tag_search_pack(self.h, B, depth.ctypes.data, path.ctypes.data, path.shape[1], states,
                                          rewards.ctypes.data, qop.ctypes.data), "tag_search_pack")
        return rewards, qop

    def close(self) -> None:
        if getattr(self, "h", None):
            _abi.load().tag_search_problem_destroy(self.h)
            self.h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


class Mcts:
    """Host handle of a search tree."""

    def __init__(self, n_levels: int, n_actions: int, c_puct: float = 1.5, vl_value: float = 0.0):
        h = C.c_void_p(None)
        check(_abi.load().tag_mcts_create(n_levels, n_actions, float(c_puct), float(vl_value), C.byref(h)),
              "tag_mcts_create")
        self.h = h.value
        self.L, self.S = n_levels, n_actions

    def select(self, B: int):
        leaf = np.zeros(B, np.int32)
        depth = np.zeros(B, np.int32)
        path = np.zeros((B, self.L), np.int32)
        check(_abi.load().tag_mcts_select(self.h, B, leaf.ctypes.data, depth.ctypes.data, path.ctypes.data),
              "tag_mcts_select")
        return leaf, depth, path

    def update(self, leaf, depth, path, priors: Optional[np.ndarray], rewards) -> None:
        pr = None if priors is None else np.ascontiguousarray(priors, np.float32)
        rw = _f64(rewards)
        check(_abi.load().tag_mcts_update(self.h, int(leaf.shape[0]), leaf.ctypes.data, depth.ctypes.data,
                                          path.ctypes.data, None if pr is None else pr.ctypes.data,
                                          rw.ctypes.data), "tag_mcts_update")

    def root_stats(self) -> Tuple[np.ndarray, np.ndarray]:
        n = np.zeros(self.S, np.int32)
        q = np.zeros(self.S, np.float64)
        check(_abi.load().tag_mcts_root_stats(self.h, n.ctypes.data, q.ctypes.data), "tag_mcts_root_stats")
        return n, q

    def best_path(self) -> np.ndarray:
        p = np.zeros(self.L, np.int32)
        d = C.c_int32(0)
        check(_abi.load().tag_mcts_best_path(self.h, p.ctypes.data, C.byref(d)), "tag_mcts_best_path")
        return p[:d.value].copy()

    def size(self) -> Tuple[int, int]:
        v, e = C.c_int64(0), C.c_int64(0)
        check(_abi.load().tag_mcts_size(self.h, C.byref(v), C.byref(e)), "tag_mcts_size")
        return v.value, e.value

    def close(self) -> None:
        if getattr(self, "h", None):
            _abi.load().tag_mcts_destroy(self.h)
            self.h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


class SearchService:
    """Device buffers for evaluating B leaves per round: packed states,
    expanded features, the GNN workspace, embeddings and priors.  A round is
    select -> pack (host) -> features, forward, decide (GPU) -> update."""

    def __init__(self, problem: SearchProblem, sp, model, B: int, device: str = "cuda"):
        import torch
        from . import Graph, make_features, tag_gnn_decide_workspace, tag_gnn_workspace, tag_slices
        self.torch, self.problem, self.model, self.B = torch, problem, model, B
        dev = torch.device(device)
        self.dev = dev
        t = sp.topo
        self.graph = Graph([t], device=device)
        sb, rb = problem.device_bytes()
        self.state_bytes = rb
        self.static = torch.empty(sb, dtype=torch.uint8, device=dev)
        check(_abi.load().tag_search_upload(problem.h, self.static.data_ptr(), sb,
                                            int(torch.cuda.current_stream().cuda_stream)), "tag_search_upload")
        self.states_h = torch.empty(B * rb, dtype=torch.uint8, pin_memory=True)
        self.states_d = torch.empty(B * rb, dtype=torch.uint8, device=dev)
        self.x_op = torch.empty((B, t.n_op, problem.f_op), dtype=torch.float32, device=dev)
        self.x_dev = torch.empty((B, t.n_dev, 8), dtype=torch.float32, device=dev)
        self.x_od = torch.empty((B, max(t.e_od, 1)), dtype=torch.uint8, device=dev)
        # tensor sizes and link bandwidths do not depend on the strategy: shared rows
        x_oo = (np.log10(t.op_bytes[t.oo_src]) - 6.0).astype(np.float32)
        x_dd = np.stack([np.log10(t.dd_bw) - 1.0, np.zeros(t.e_dd)], axis=1).astype(np.float32) \
            if t.e_dd else np.zeros((0, 2), np.float32)
        self.x_oo = torch.from_numpy(np.ascontiguousarray(x_oo)).to(dev)
        self.x_dd = torch.from_numpy(np.ascontiguousarray(x_dd)).to(dev)
        # under the simulator model every leaf has its own link rows (idle shares)
        self.own_dd = problem.model == "simulator" and t.e_dd > 0
        if self.own_dd:
            self.x_dd_leaf = torch.empty((B, t.e_dd, 2), dtype=torch.float32, device=dev)
        self.feats = make_features(self.x_op, self.x_dev, self.x_oo, self.x_dd_leaf if self.own_dd else self.x_dd,
                                   self.x_od)
        st, self.fwd_ws_bytes = tag_gnn_workspace(self.graph.handle, model.dims, B)
        check(st, "tag_gnn_workspace")
        self.fwd_ws = torch.empty(self.fwd_ws_bytes, dtype=torch.uint8, device=dev)
        f = int(model.dims.f)
        self.E_op = torch.empty((B, t.n_op, f), dtype=torch.float32, device=dev)
        self.E_dev = torch.empty((B, t.n_dev, f), dtype=torch.float32, device=dev)
        S = problem.n_slices
        self.masks = torch.from_numpy(np.ascontiguousarray(np.asarray(sp.masks, np.uint64).view(np.int64))).to(dev)
        self.opts = torch.from_numpy(np.ascontiguousarray(np.asarray(sp.options, np.uint8))).to(dev)
        self.slices = tag_slices(S, self.masks.data_ptr(), self.opts.data_ptr())
        self.q_rep = torch.arange(B, dtype=torch.int32, device=dev)
        self.q_graph = torch.zeros(B, dtype=torch.int32, device=dev)
        self.q_op_h = torch.zeros(B, dtype=torch.int32, pin_memory=True)
        self.q_op = torch.zeros(B, dtype=torch.int32, device=dev)
        st, self.dec_ws_bytes = tag_gnn_decide_workspace(self.graph.handle, model.dims, B, S, B)
        check(st, "tag_gnn_decide_workspace")
        self.dec_ws = torch.empty(max(self.dec_ws_bytes, 1), dtype=torch.uint8, device=dev)
        self.argmax = torch.empty(B, dtype=torch.int32, device=dev)
        self.best = torch.empty(B, dtype=torch.float32, device=dev)
        self.prior = torch.empty((B, S), dtype=torch.float32, device=dev)
        self.prior_h = torch.empty((B, S), dtype=torch.float32, pin_memory=True)

    def evaluate(self, depth: np.ndarray, path: np.ndarray, stream=None):
        """Rewards (host) and priors (host float32 [B, S]) of B leaves."""
        from . import tag_gnn_decide, tag_gnn_forward
        torch = self.torch
        B = int(depth.shape[0])
        assert B == self.B, "the service is sized for a fixed batch"
        st = torch.cuda.current_stream() if stream is None else stream
        sh = int(st.cuda_stream)
        rewards, qop = self.problem.pack(depth, path, self.states_h.data_ptr())
        self.q_op_h.numpy()[:] = qop
        with torch.cuda.stream(st):
            self.states_d.copy_(self.states_h, non_blocking=True)
            self.q_op.copy_(self.q_op_h, non_blocking=True)
        lib = _abi.load()
        check(lib.tag_search_features(self.problem.h, B, self.static.data_ptr(), self.states_d.data_ptr(),
                                      self.x_op.data_ptr(), self.x_dev.data_ptr(), self.x_od.data_ptr(), sh),
              "tag_search_features")
        if self.own_dd:
            check(lib.tag_search_link_features(self.problem.h, B, self.static.data_ptr(), self.states_d.data_ptr(),
                                               self.x_dd_leaf.data_ptr(), sh), "tag_search_link_features")
        check(tag_gnn_forward(self.graph.handle, self.model.dims, self.model.weights, self.feats,
                              self.fwd_ws.data_ptr(), self.fwd_ws_bytes, self.E_op.data_ptr(),
                              self.E_dev.data_ptr(), sh), "tag_gnn_forward")
        check(tag_gnn_decide(self.graph.handle, self.model.dims, self.model.weights, B, self.E_op.data_ptr(),
                             self.E_dev.data_ptr(), self.slices, B, self.q_rep.data_ptr(), self.q_graph.data_ptr(),
                             self.q_op.data_ptr(), self.argmax.data_ptr(), self.best.data_ptr(),
                             self.prior.data_ptr(), None, self.dec_ws.data_ptr(), self.dec_ws_bytes, sh),
              "tag_gnn_decide")
        with torch.cuda.stream(st):
            self.prior_h.copy_(self.prior, non_blocking=True)
        st.synchronize()
        return rewards, self.prior_h.numpy()

    def round(self, tree: Mcts, stream=None) -> np.ndarray:
        """One search round on `tree`; returns the leaves' rewards."""
        leaf, depth, path = tree.select(self.B)
        rewards, priors = self.evaluate(depth, path, stream)
        tree.update(leaf, depth, path, priors, rewards)
        return rewards

    def run(self, tree: Mcts, rounds: int, pipelined: bool = True, record: bool = False, stream=None):
        """`rounds` rounds in native code (tag_search_run).  With `record`,
        returns the rounds' depths, paths, rewards and priors (host arrays in
        selection order)."""
        import ctypes as C
        from ._abi import tag_search_run_args
        torch = self.torch
        if not hasattr(self, "run_ws"):
            db, hb = C.c_size_t(0), C.c_size_t(0)
            check(_abi.load().tag_search_run_workspace(self.problem.h, self.graph.handle, C.byref(self.model.dims),
                                                       self.B, C.byref(db), C.byref(hb)), "tag_search_run_workspace")
            self.run_ws = torch.empty(db.value, dtype=torch.uint8, device=self.dev)
            self.run_host = torch.empty(hb.value, dtype=torch.uint8, pin_memory=True)
        B, L, S = self.B, tree.L, tree.S
        rec = None
        if record:
            rec = {"depth": np.zeros(rounds * B, np.int32), "path": np.zeros(rounds * B * L, np.int32),
                   "reward": np.zeros(rounds * B, np.float64), "prior": np.zeros(rounds * B * S, np.float32)}
        a = tag_search_run_args()
        a.problem, a.tree, a.graph = self.problem.h, tree.h, self.graph.handle
        a.dims = C.addressof(self.model.dims)
        a.weights = C.addressof(self.model.weights)
        a.x_oo, a.x_dd = self.x_oo.data_ptr(), self.x_dd.data_ptr()
        a.slices = C.addressof(self.slices)
        a.batch, a.rounds, a.pipelined = B, rounds, 1 if pipelined else 0
        a.workspace, a.ws_bytes = self.run_ws.data_ptr(), self.run_ws.numel()
        a.host_buf, a.host_bytes = self.run_host.data_ptr(), self.run_host.numel()
        if rec is not None:
            a.depth_out, a.path_out = rec["depth"].ctypes.data, rec["path"].ctypes.data
            a.reward_out, a.prior_out = rec["reward"].ctypes.data, rec["prior"].ctypes.data
        st = torch.cuda.current_stream() if stream is None else stream
        check(_abi.load().tag_search_run(C.byref(a), int(st.cuda_stream)), "tag_search_run")
        if rec is None:
            return None
        return {"depth": rec["depth"].reshape(rounds, B), "path": rec["path"].reshape(rounds, B, L),
                "reward": rec["reward"].reshape(rounds, B), "prior": rec["prior"].reshape(rounds, B, S)}

    def close(self) -> None:
        self.graph.close()
