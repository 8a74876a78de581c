"""GPU parity of the ELU variant of the message non-linearity (sigma of the
layer equation, which the paper leaves open; ReLU is the default reading):
the forward pass on every aggregation path (MFMA tiles with heads of 16-64
channels, the per-row path for narrower heads, and the device-message
preparation pass for heads wider than 64 channels) against the oracle with
sigma = ELU at the fp32 tolerance (row-relative 1e-4), the saturated case
whose output is minus the sum of gamma over a node's link types, the
training step against the reference training step with ELU, and the
rejection of ELU with bf16 transforms."""
import numpy as np
import pytest

import oracle
import paper_2302_06126_amd as P
import synth
from tests._gpu import FP32_TOL, Case, dev_tensor, say
from tests._helpers import row_rel_err

pytestmark = pytest.mark.gpu


def _elu_forward(c, w=None):
    w = w if w is not None else c.w
    g = P.Graph([c.topo])
    m = P.Model(w, f=c.f, heads=c.heads, layers=c.layers, f_op=c.f_op, dec_hidden=c.dec_hidden, sigma="elu")
    E_op, E_dev = P.forward(g, m, dev_tensor(c.x_op), dev_tensor(c.x_dev), dev_tensor(c.x_oo), dev_tensor(c.x_dd),
                            dev_tensor(c.x_od))
    return E_op.cpu().numpy(), E_dev.cpu().numpy()


@pytest.mark.parametrize("f,heads,layers", [(64, 4, 2), (128, 4, 3), (128, 16, 2), (256, 2, 2), (256, 64, 1)])
def test_elu_forward_matches_oracle(f, heads, layers):
    say(f"[elu] forward f={f} K={heads} L={layers}")
    topo = synth.random_topology(400 + heads, 150, 7, 300, od_per_op=4, dd_density=0.8)
    c = Case(topo, 3, f, heads, layers, seed=heads + layers)
    E_op, E_dev = _elu_forward(c)
    worst = 0.0
    for r in range(c.R):
        R_op, R_dev = oracle.forward(c.topo, c.x_op[r], c.x_dev[r], c.x_oo[r], c.x_dd[r], c.x_od[r], c.w, f=f,
                                     heads=heads, layers=layers, sigma="elu")
        got = np.vstack([E_op[r], E_dev[r]])
        assert np.all(np.isfinite(got))
        err = row_rel_err(got, np.vstack([R_op, R_dev]))
        worst = max(worst, err)
        assert err <= FP32_TOL, (r, err)
    # ELU differs from ReLU on these inputs (negative messages are present)
    R_relu, _ = oracle.forward(c.topo, c.x_op[0], c.x_dev[0], c.x_oo[0], c.x_dd[0], c.x_od[0], c.w, f=f,
                               heads=heads, layers=layers)
    assert row_rel_err(E_op[0], R_relu) > 1e-3
    say(f"  worst row-relative error {worst:.2e}")


def test_elu_forward_many_devices_wide_rows():
    # 40 devices at f = 256: the op<-device contraction on sparse split
    # products over the ELU message table, two 32-device steps (the second ragged)
    say("[elu] forward f=256, 40 devices")
    topo = synth.random_topology(440, 120, 40, 250, od_per_op=None, dd_density=0.3)
    c = Case(topo, 2, 256, 4, 2, seed=40)
    E_op, E_dev = _elu_forward(c)
    for r in range(c.R):
        R_op, R_dev = oracle.forward(c.topo, c.x_op[r], c.x_dev[r], c.x_oo[r], c.x_dd[r], c.x_od[r], c.w, f=256,
                                     heads=4, layers=2, sigma="elu")
        got = np.vstack([E_op[r], E_dev[r]])
        assert np.all(np.isfinite(got))
        err = row_rel_err(got, np.vstack([R_op, R_dev]))
        assert err <= FP32_TOL, (r, err)


def test_elu_saturated_messages_give_minus_gamma_sums():
    say("[elu] saturated messages")
    topo = synth.random_topology(410, 90, 5, 150, od_per_op=3, dd_density=0.6)
    c = Case(topo, 2, 128, 4, 1, seed=3)
    w = {k: v.copy() for k, v in c.w.items()}
    w["layer_b"][:] = -100.0
    E_op, E_dev = _elu_forward(c, w)
    has_oo = np.zeros(topo.n_op, bool)
    has_oo[topo.oo_src] = True
    has_oo[topo.oo_dst] = True
    has_od_op = np.zeros(topo.n_op, bool)
    has_od_op[topo.od_op] = True
    has_od_dev = np.zeros(topo.n_dev, bool)
    has_od_dev[topo.od_dev] = True
    has_dd = np.zeros(topo.n_dev, bool)
    has_dd[topo.dd_a] = True
    has_dd[topo.dd_b] = True
    want_op = -(1.0 * has_oo + 0.1 * has_od_op)
    want_dev = -(0.1 * has_od_dev + 1.0 * has_dd)
    for r in range(2):
        np.testing.assert_allclose(E_op[r], np.repeat(want_op[:, None], 128, 1), rtol=0, atol=1e-6)
        np.testing.assert_allclose(E_dev[r], np.repeat(want_dev[:, None], 128, 1), rtol=0, atol=1e-6)


def test_elu_training_step_matches_reference():
    import torch
    from tests.test_gpu_train import TrainCase, _compare
    from oracle import train as OT
    import paper_2302_06126_amd.train as PT
    say("[elu] training step")
    topo = synth.make_topology("tiny")
    c = TrainCase([topo], 2, 64, 4, 2, 60, 2, seed=11)
    graph = P.Graph([topo])
    model = P.Model(c.w, f=64, heads=4, layers=2, f_op=c.f_op, dec_hidden=64, sigma="elu")
    tr = PT.Trainer(graph, model, c.R, c.masks, c.opts, c.q_rep, c.q_graph, c.q_op)
    tr.set_targets(c.target)
    d = lambda a: torch.from_numpy(np.ascontiguousarray(a)).cuda()
    keep = [d(c.x_op), d(c.x_dev), d(c.x_oo), d(c.x_dd), d(c.x_od)]
    loss = float(tr.step(P.make_features(*keep)).cpu()[0])
    ref_loss, ref_g = OT.loss_and_grads(c.items, c.w, f=64, heads=4, layers=2, masks=c.masks, options=c.opts,
                                        sigma="elu")
    worst = _compare(tr, loss, ref_loss, ref_g, c.w)
    say(f"  loss {loss:.6f} ref {ref_loss:.6f}; worst relative gradient error {max(worst.values()):.2e}")


def test_elu_needs_fp32():
    from paper_2302_06126_amd import _abi
    import ctypes as C
    say("[elu] bf16 rejected")
    topo = synth.random_topology(420, 20, 3, 30)
    g = P.Graph([topo])
    m = P.Model(synth.make_weights(128, 4, 1, 42, 128), f=128, heads=4, layers=1, f_op=42, dtype="bf16",
                sigma="elu")
    b = C.c_size_t()
    assert _abi.load().tag_gnn_workspace(g.handle, C.byref(m.dims), 1, C.byref(b)) == _abi.TAG_ESHAPE
