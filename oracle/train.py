"""Reference training step: the cross-entropy between the decoder's priors and
the search's visit distribution, and its gradient with respect to every
parameter (Section 4.2.2: the GNN is trained to minimise the cross entropy
between its prior G(s, a) and the MCTS selection probability pi(s, a)).

TEST INFRASTRUCTURE ONLY (like the rest of ``oracle/``).  Plain PyTorch CPU
ops in float64 restate the forward pass of Section 4.2.1 (encoders, the
heterogeneous GAT layers, the decoder) under the readings of the C oracle,
and autograd differentiates it.  The forward is pinned to the C oracle and
the gradient to central differences of the C oracle's loss (tests).

Loss over Q queries (replica r_q, op i_q, target distribution pi_q over
the S slices):  L = -(1/Q) sum_q sum_a pi_qa log softmax_a(score_qa).
"""
from __future__ import annotations

from typing import Dict, List, Sequence

import numpy as np
import torch

PARAMS = ("enc_op_w", "enc_op_b", "enc_dev_w", "enc_dev_b", "enc_edge_w0", "enc_edge_b0",
          "enc_edge_w1", "enc_edge_b1", "enc_edge_w2", "enc_edge_b2", "layer_w", "layer_b",
          "att_src", "att_dst", "dec_w1", "dec_b1", "dec_w2", "dec_b2")


def _t(a, grad=False):
    x = torch.tensor(np.asarray(a, dtype=np.float64))
    return x.requires_grad_(grad)


def _buckets(topo):
    """(destination, source, edge id) of the four buckets; neighbour sets are
    undirected inside a link type, so op-op and device-device links feed
    both of their ends."""
    oo_s, oo_d = torch.as_tensor(topo.oo_src, dtype=torch.long), torch.as_tensor(topo.oo_dst, dtype=torch.long)
    dd_a, dd_b = torch.as_tensor(topo.dd_a, dtype=torch.long), torch.as_tensor(topo.dd_b, dtype=torch.long)
    od_o, od_d = torch.as_tensor(topo.od_op, dtype=torch.long), torch.as_tensor(topo.od_dev, dtype=torch.long)
    e_oo, e_dd, e_od = oo_s.numel(), dd_a.numel(), od_o.numel()
    b0 = (torch.cat([oo_d, oo_s]), torch.cat([oo_s, oo_d]), torch.cat([torch.arange(e_oo)] * 2))
    b1 = (od_o, od_d, torch.arange(e_od))
    b2 = (od_d, od_o, torch.arange(e_od))
    b3 = (torch.cat([dd_a, dd_b]), torch.cat([dd_b, dd_a]), torch.cat([torch.arange(e_dd)] * 2))
    return b0, b1, b2, b3


def _aggregate(bucket, n_dst, ysrc, ydst, te, a, ad, heads, slope, sigma="relu"):
    """sum over the destination's entries of softmax_e(logit_e) m_e, per head:
    m_e = sigma(W^h h_src + W^e e + b) (ReLU, or ELU as a variant),
    logit_e = LeakyReLU(a . m_e + a~ . W^h h_dst)."""
    dst, src, eid = bucket
    f = ysrc.shape[1]
    d = f // heads
    E = dst.numel()
    if E == 0:
        return torch.zeros((n_dst, f), dtype=torch.float64)
    pre = ysrc[src] + te[eid]
    m = torch.nn.functional.elu(pre) if sigma == "elu" else torch.relu(pre)
    s = (m * a).view(E, heads, d).sum(-1) + (ydst * ad).view(-1, heads, d).sum(-1)[dst]
    s = torch.where(s > 0, s, slope * s)
    mx = torch.full((n_dst, heads), -np.inf, dtype=torch.float64)
    mx = mx.scatter_reduce(0, dst[:, None].expand(E, heads), s.detach(), "amax", include_self=True)
    ex = torch.exp(s - mx[dst])
    z = torch.zeros((n_dst, heads), dtype=torch.float64).index_add(0, dst, ex)
    al = ex / z[dst]
    out = torch.zeros((n_dst, heads, d), dtype=torch.float64).index_add(0, dst, al[:, :, None] * m.view(E, heads, d))
    return out.view(n_dst, f)


def forward(topo, x_op, x_dev, x_oo, x_dd, x_od, P: Dict[str, torch.Tensor], *, f, heads, layers,
            gamma_same=1.0, gamma_cross=0.1, slope=0.2, sigma="relu"):
    """E_op [N, f], E_dev [M, f] as float64 tensors."""
    xo, xd = _t(x_op), _t(x_dev)
    h_op = torch.relu(xo @ P["enc_op_w"].T + P["enc_op_b"])
    h_dev = torch.relu(xd @ P["enc_dev_w"].T + P["enc_dev_b"])
    enc_oo = _t(x_oo).reshape(-1, 1) @ P["enc_edge_w0"].T + P["enc_edge_b0"]
    enc_od = _t(np.asarray(x_od, np.float64)).reshape(-1, 1) @ P["enc_edge_w1"].T + P["enc_edge_b1"]
    enc_dd = _t(x_dd).reshape(-1, 2) @ P["enc_edge_w2"].T + P["enc_edge_b2"]
    b0, b1, b2, b3 = _buckets(topo)
    N, M = topo.n_op, topo.n_dev
    for l in range(layers):
        W = [P["layer_w"][l, r] for r in range(3)]
        Wh = [w[:, :f] for w in W]
        We = [w[:, f:] for w in W]
        b = [P["layer_b"][l, r] for r in range(3)]
        a = [P["att_src"][l, r] for r in range(3)]
        ad = [P["att_dst"][l, r] for r in range(3)]
        te_oo = enc_oo @ We[0].T + b[0]
        te_od = enc_od @ We[1].T + b[1]
        te_dd = enc_dd @ We[2].T + b[2]
        y_oo = h_op @ Wh[0].T
        y_od_op = h_op @ Wh[1].T
        y_od_dev = h_dev @ Wh[1].T
        y_dd = h_dev @ Wh[2].T
        n_op = gamma_same * _aggregate(b0, N, y_oo, y_oo, te_oo, a[0], ad[0], heads, slope, sigma) \
            + gamma_cross * _aggregate(b1, N, y_od_dev, y_od_op, te_od, a[1], ad[1], heads, slope, sigma)
        n_dev = gamma_cross * _aggregate(b2, M, y_od_op, y_od_dev, te_od, a[1], ad[1], heads, slope, sigma) \
            + gamma_same * _aggregate(b3, M, y_dd, y_dd, te_dd, a[2], ad[2], heads, slope, sigma)
        h_op, h_dev = n_op, n_dev
    return h_op, h_dev


def scores(E_op, E_dev, masks, options, query_op, P, *, f):
    """Decoder scores [Q, S]: w2 . ReLU(W1 [sum_{j in mask} E_dev[j]; E_op[i]; onehot(option)] + b1) + b2."""
    M = E_dev.shape[0]
    S = len(masks)
    Mk = np.zeros((S, M))
    for a, m in enumerate(masks):
        for j in range(min(M, 64)):
            if (int(m) >> j) & 1:
                Mk[a, j] = 1.0
    devsum = _t(Mk) @ E_dev                                     # [S, f]
    oh = _t(np.eye(4)[np.asarray(options, np.int64)])            # [S, 4]
    q = torch.as_tensor(np.asarray(query_op, np.int64))
    Q = q.numel()
    x = torch.cat([devsum[None].expand(Q, S, f), E_op[q][:, None].expand(Q, S, f),
                   oh[None].expand(Q, S, 4)], dim=2)
    h = torch.relu(x @ P["dec_w1"].T + P["dec_b1"])
    return h @ P["dec_w2"] + P["dec_b2"][0]


def loss_and_grads(items: Sequence[dict], w: Dict[str, np.ndarray], *, f, heads, layers, masks, options,
                   gamma_same=1.0, gamma_cross=0.1, slope=0.2, sigma="relu"):
    """`items`: one dict per replica with its topology, features, query ops
    and targets [Q_r, S].  Returns (loss, {name: gradient as float64 numpy
    in the parameter's own shape}); the loss is the mean over all queries."""
    P = {}
    for k in PARAMS:
        P[k] = _t(w[k], grad=True)
    total, Qn = 0.0, 0
    terms: List[torch.Tensor] = []
    for it in items:
        E_op, E_dev = forward(it["topo"], it["x_op"], it["x_dev"], it["x_oo"], it["x_dd"], it["x_od"], P,
                              f=f, heads=heads, layers=layers, gamma_same=gamma_same,
                              gamma_cross=gamma_cross, slope=slope, sigma=sigma)
        sc = scores(E_op, E_dev, masks, options, it["query_op"], P, f=f)
        lp = torch.log_softmax(sc, dim=1)
        terms.append(-(_t(it["target"]) * lp).sum())
        Qn += len(it["query_op"])
    loss = torch.stack(terms).sum() / Qn
    loss.backward()
    return float(loss.detach()), {k: P[k].grad.numpy().copy() for k in PARAMS}
