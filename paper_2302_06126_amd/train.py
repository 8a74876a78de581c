"""Binding of the GNN training step (include/tag_train.h): one call runs the
forward pass, the cross entropy between the decoder's priors and target
distributions over the slice table (Section 4.2.2), every parameter's
gradient and, when lr > 0, the SGD update of the model's device parameters.

Argument marshalling only; the step runs in libtag.so's HIP kernels.
"""
from __future__ import annotations

from typing import Dict

import numpy as np

from . import Graph, Model, _ptr, _stream, _torch
from . import _abi
from ._abi import check, tag_grads, tag_slices, tag_train_batch

PARAM_NAMES = ("enc_op_w", "enc_op_b", "enc_dev_w", "enc_dev_b", "enc_edge_w0", "enc_edge_b0",
               "enc_edge_w1", "enc_edge_b1", "enc_edge_w2", "enc_edge_b2", "layer_w", "layer_b",
               "att_src", "att_dst", "dec_w1", "dec_b1", "dec_w2", "dec_b2")


class Trainer:
    """Reusable training step for fixed (R, slice table, queries).

    Owns the workspace, the gradient tensors (flat fp32, one per parameter
    of ``model``) and the loss.  ``step`` updates ``model``'s parameters in
    place when lr > 0."""

    def __init__(self, graph: Graph, model: Model, n_replicas: int, masks, options, q_rep, q_graph, q_op):
        torch = _torch()
        dev = graph.device
        self.graph, self.model, self.R = graph, model, int(n_replicas)
        self.masks = torch.from_numpy(np.ascontiguousarray(masks, np.uint64).view(np.int64)).to(dev)
        self.options = torch.from_numpy(np.ascontiguousarray(options, np.uint8)).to(dev)
        self.q = [torch.from_numpy(np.ascontiguousarray(a, np.int32)).to(dev) for a in (q_rep, q_graph, q_op)]
        self.S, self.Q = len(masks), len(q_op)
        self.slices = tag_slices(self.S, _ptr(self.masks), _ptr(self.options))
        b = _abi.C.c_size_t()
        check(_abi.load().tag_train_workspace(graph.handle, _abi.C.byref(model.dims), self.R, self.S, self.Q,
                                              _abi.C.byref(b)), "tag_train_workspace")
        self.ws_bytes = b.value
        self.ws = torch.empty(max(self.ws_bytes, 1), dtype=torch.uint8, device=dev)
        self.grads: Dict[str, "torch.Tensor"] = {k: torch.zeros_like(model.t[k]) for k in PARAM_NAMES}
        g = tag_grads()
        p = lambda k: _ptr(self.grads[k])
        g.enc_op_w, g.enc_op_b, g.enc_dev_w, g.enc_dev_b = p("enc_op_w"), p("enc_op_b"), p("enc_dev_w"), p("enc_dev_b")
        for r in range(3):
            g.enc_edge_w[r] = p(f"enc_edge_w{r}")
            g.enc_edge_b[r] = p(f"enc_edge_b{r}")
        g.layer_w, g.layer_b, g.att_src, g.att_dst = p("layer_w"), p("layer_b"), p("att_src"), p("att_dst")
        g.dec_w1, g.dec_b1, g.dec_w2, g.dec_b2 = p("dec_w1"), p("dec_b1"), p("dec_w2"), p("dec_b2")
        self.grad_struct = g
        self.loss = torch.zeros(1, dtype=torch.float32, device=dev)
        self.target = torch.zeros((max(self.Q, 1), self.S), dtype=torch.float32, device=dev)

    def set_targets(self, target) -> None:
        """Target distributions [Q, S] (host array or device tensor)."""
        torch = _torch()
        t = target if isinstance(target, torch.Tensor) else torch.from_numpy(np.ascontiguousarray(target, np.float32))
        self.target.copy_(t.reshape(self.Q, self.S))

    def step(self, feats, lr: float = 0.0, stream=None):
        """One step on the features ``feats`` (a tag_features); returns the
        loss tensor (device, [1]).  Gradients are in ``self.grads``."""
        batch = tag_train_batch(self.Q, _ptr(self.q[0]), _ptr(self.q[1]), _ptr(self.q[2]), _ptr(self.target))
        st = _abi.load().tag_train_step(self.graph.handle, _abi.C.byref(self.model.dims),
                                        _abi.C.byref(self.model.weights), _abi.C.byref(feats),
                                        _abi.C.byref(self.slices), _abi.C.byref(batch),
                                        _abi.C.byref(self.grad_struct), float(lr), _ptr(self.loss), _ptr(self.ws),
                                        self.ws_bytes, _stream(stream))
        check(st, "tag_train_step")
        return self.loss
