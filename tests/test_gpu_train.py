"""GPU parity of the training step (Section 4.2.2): loss and every
parameter's gradient from tag_train_step against the reference training
step (oracle/train.py, float64 autograd over the reference forward pass,
itself pinned to the C oracle and to central differences), plus the SGD
update, bitwise repeatability and the argument checks.

Tolerance (fp32 kernels against float64): the loss within 2e-5 relative;
each gradient array within 1e-3 of its largest magnitude, plus 2e-6.  The
gradients are sums of up to ~1e5 fp32 products with cancellation between
terms, so their absolute error scales with the array's magnitude, not with
each element's; the floor covers arrays whose exact value is zero (the
decoder's output bias: its gradient is sum_q (sum_a p_qa T_q - T_q) / Q = 0
when the target rows sum to T_q), where only the rounding of the S Q summed
terms (each at most 1/Q) remains."""
import numpy as np
import pytest

import paper_2302_06126_amd as P
import synth
from oracle import train as OT

pytestmark = pytest.mark.gpu

GRAD_TOL = 1e-3
GRAD_FLOOR = 2e-6
LOSS_TOL = 2e-5


def _say(msg):
    print(msg, flush=True)


@pytest.fixture(scope="module")
def torch():
    import torch
    assert torch.cuda.is_available()
    return torch


class TrainCase:
    """R candidates of each of the topologies (candidate (r, g) uses
    topology g), Q_per queries per candidate, random targets."""

    def __init__(self, topos, R, f, heads, layers, S, Q_per, seed, f_op=40, invalid=0, dup=False):
        self.topos, self.R, self.f, self.heads, self.layers = topos, R, f, heads, layers
        self.f_op = f_op
        self.w = synth.make_weights(f, heads, layers, f_op, f, bias_scale=0.3, seed_extra=seed)
        rng = synth.rng_for(91, seed)
        m_min = min(t.n_dev for t in topos)
        self.masks = np.array([int(rng.integers(1, 1 << min(m_min, 62))) | (1 << int(rng.integers(0, 64)))
                               for _ in range(S)], np.uint64)
        self.opts = rng.integers(0, 4, size=S).astype(np.uint8)
        self.items, q_rep, q_graph, q_op, tg = [], [], [], [], []
        per_r = []
        for r in range(R):
            feats = []
            for g, t in enumerate(topos):
                x = dict(topo=t, x_op=rng.uniform(-1, 1, (t.n_op, f_op)).astype(np.float32),
                         x_dev=rng.uniform(-1, 1, (t.n_dev, 8)).astype(np.float32),
                         x_oo=rng.uniform(-1, 1, t.e_oo).astype(np.float32),
                         x_dd=rng.uniform(-1, 1, (t.e_dd, 2)).astype(np.float32),
                         x_od=rng.integers(0, 2, t.e_od).astype(np.uint8),
                         query_op=rng.integers(0, t.n_op, size=Q_per).astype(np.int32))
                if dup:                   # two queries of one candidate read the same op row
                    x["query_op"][-1] = x["query_op"][0]
                tt = rng.random((Q_per, S)) ** 3
                x["target"] = tt / tt.sum(1, keepdims=True)
                feats.append(x)
                self.items.append(x)
                for i in range(Q_per):
                    q_rep.append(r); q_graph.append(g); q_op.append(int(x["query_op"][i])); tg.append(x["target"][i])
            per_r.append(feats)
        for i in range(invalid):          # out-of-range queries: no loss, no gradient
            q_rep.append(R + i); q_graph.append(0); q_op.append(0); tg.append(np.full(S, 1.0 / S))
        self.q_rep, self.q_graph, self.q_op = (np.array(a, np.int32) for a in (q_rep, q_graph, q_op))
        self.target = np.array(tg, np.float32)
        self.n_valid = len(self.items) * Q_per
        cat = lambda key: np.stack([np.concatenate([x[key] for x in feats]) for feats in per_r])
        self.x_op, self.x_dev, self.x_oo, self.x_dd, self.x_od = (cat(k) for k in ("x_op", "x_dev", "x_oo", "x_dd",
                                                                                    "x_od"))

    def reference(self):
        loss, g = OT.loss_and_grads(self.items, self.w, f=self.f, heads=self.heads, layers=self.layers,
                                    masks=self.masks, options=self.opts)
        scale = self.n_valid / len(self.q_op)      # the library averages over every query
        return loss * scale, {k: v * scale for k, v in g.items()}

    def trainer(self, torch, weights=None):
        graph = P.Graph(self.topos)
        model = P.Model(weights or self.w, f=self.f, heads=self.heads, layers=self.layers, f_op=self.f_op,
                        dec_hidden=self.f)
        import paper_2302_06126_amd.train as PT
        tr = PT.Trainer(graph, model, self.R, self.masks, self.opts, self.q_rep, self.q_graph, self.q_op)
        tr.set_targets(self.target)
        d = lambda a: torch.from_numpy(np.ascontiguousarray(a)).cuda()
        self._keep = [d(self.x_op), d(self.x_dev), d(self.x_oo), d(self.x_dd), d(self.x_od)]
        feats = P.make_features(*self._keep)
        return graph, model, tr, feats


def _compare(tr, loss_gpu, ref_loss, ref_g, w):
    assert abs(loss_gpu - ref_loss) <= LOSS_TOL * abs(ref_loss), (loss_gpu, ref_loss)
    worst = {}
    for k in OT.PARAMS:
        got = tr.grads[k].cpu().numpy().astype(np.float64)
        ref = ref_g[k].reshape(-1)
        assert np.all(np.isfinite(got)), k
        scale = np.abs(ref).max()
        err = np.abs(got - ref).max()
        worst[k] = err / max(scale, GRAD_FLOOR / GRAD_TOL)   # relative, below the floor's scale absolute
        assert err <= GRAD_TOL * scale + GRAD_FLOOR, f"{k}: max error {err:.3e} vs max |grad| {scale:.3e}"
    return worst


@pytest.mark.parametrize("name,R,S,Q_per,invalid", [("tiny", 3, 60, 2, 1), ("cnn", 2, 256, 2, 0)])
def test_train_step_matches_reference_workload_topology(torch, name, R, S, Q_per, invalid):
    wl = synth.WORKLOADS[name]
    topo = synth.make_topology(name)
    _say(f"[train] {name} R={R} S={S} f={wl.f} K={wl.heads} L={wl.layers}")
    c = TrainCase([topo], R, wl.f, wl.heads, wl.layers, S, Q_per, seed=3 + R, f_op=wl.f_op, invalid=invalid)
    graph, model, tr, feats = c.trainer(torch)
    loss = float(tr.step(feats).cpu()[0])
    ref_loss, ref_g = c.reference()
    worst = _compare(tr, loss, ref_loss, ref_g, c.w)
    _say(f"[train] {name}: loss {loss:.6f} ref {ref_loss:.6f}; relative gradient errors "
         + " ".join(f"{k}={v:.1e}" for k, v in worst.items()))


@pytest.mark.parametrize("f,heads", [(256, 8), (128, 16)])
def test_train_step_long_device_rows(torch, f, heads):
    """cnn topology (device rows of 1200 op links): at f = 256 its 16 device
    rows do not fit in LDS, so the generic passes run and the device<-op
    softmax takes the entry-per-lane path for long rows; at f = 128 with 16
    heads the op-device tile path runs with 8-channel heads."""
    topo = synth.make_topology("cnn")
    _say(f"[train] cnn long device rows f={f} K={heads}")
    c = TrainCase([topo], 1, f, heads, 1, 64, 2, seed=f + heads)
    graph, model, tr, feats = c.trainer(torch)
    loss = float(tr.step(feats).cpu()[0])
    ref_loss, ref_g = c.reference()
    worst = _compare(tr, loss, ref_loss, ref_g, c.w)
    _say(f"[train] cnn f={f} K={heads}: worst relative gradient error {max(worst.values()):.2e}")


@pytest.mark.parametrize("f,heads,layers", [(64, 1, 2), (64, 2, 1), (128, 8, 2), (256, 64, 1)])
def test_train_step_matches_reference_union_of_topologies(torch, f, heads, layers):
    """Two topologies in one graph, long device rows (chunked passes), sparse
    placements, every head width."""
    topos = [synth.random_topology(21, 300, 5, 500, od_per_op=3, dd_density=0.7),
             synth.random_topology(22, 40, 9, 70)]
    _say(f"[train] union f={f} K={heads} L={layers}")
    c = TrainCase(topos, 2, f, heads, layers, 24, 3, seed=f + heads, dup=True)
    graph, model, tr, feats = c.trainer(torch)
    loss = float(tr.step(feats).cpu()[0])
    ref_loss, ref_g = c.reference()
    worst = _compare(tr, loss, ref_loss, ref_g, c.w)
    _say(f"[train] union: worst relative gradient error {max(worst.values()):.2e}")


def test_train_step_repeatable_and_sgd_update(torch):
    topo = synth.make_topology("tiny")
    _say("[train] repeatability and update")
    c = TrainCase([topo], 2, 64, 4, 2, 60, 3, seed=7)
    graph, model, tr, feats = c.trainer(torch)
    l1 = tr.step(feats).clone()
    g1 = {k: v.clone() for k, v in tr.grads.items()}
    l2 = tr.step(feats).clone()
    assert torch.equal(l1, l2)
    for k in OT.PARAMS:
        assert torch.equal(g1[k], tr.grads[k]), k
    before = {k: model.t[k].clone() for k in OT.PARAMS}
    lr = 0.05
    tr.step(feats, lr=lr)
    torch.cuda.synchronize()
    for k in OT.PARAMS:
        assert torch.equal(tr.grads[k], g1[k]), k          # gradients of the parameters before the update
        w0 = before[k].cpu().numpy().astype(np.float64)
        want = (w0 - np.float64(np.float32(lr)) * g1[k].cpu().numpy().astype(np.float64)).astype(np.float32)
        got = model.t[k].cpu().numpy()
        assert np.array_equal(got, want) or np.abs(got - want).max() <= np.spacing(np.abs(want)).max(), k
    # a few steps toward fixed targets lower the loss
    losses = [float(tr.step(feats, lr=0.2).cpu()[0]) for _ in range(6)]
    assert losses[-1] < losses[0], losses


def test_train_argument_checks(torch):
    import ctypes as C
    from paper_2302_06126_amd import _abi
    topo = synth.make_topology("tiny")
    _say("[train] argument checks")
    graph = P.Graph([topo])
    lib = _abi.load()
    b = C.c_size_t()
    base = dict(f=64, heads=4, layers=2, f_op=40, f_dev=8, dec_hidden=64, dtype=_abi.TAG_F32,
                gamma_same=1.0, gamma_cross=0.1, leaky_slope=0.2)
    def dims(**kw):
        d = dict(base, **kw)
        return _abi.tag_model_dims(*[d[k] for k in ("f", "heads", "layers", "f_op", "f_dev", "dec_hidden", "dtype",
                                                     "gamma_same", "gamma_cross", "leaky_slope")])
    assert lib.tag_train_workspace(graph.handle, C.byref(dims()), 2, 60, 4, C.byref(b)) == _abi.TAG_OK
    assert b.value > 0
    assert lib.tag_train_workspace(graph.handle, C.byref(dims(dtype=_abi.TAG_BF16)), 2, 60, 4,
                                   C.byref(b)) == _abi.TAG_ESHAPE
    assert lib.tag_train_workspace(graph.handle, C.byref(dims(dec_hidden=0)), 2, 60, 4, C.byref(b)) == _abi.TAG_ESHAPE
    assert lib.tag_train_workspace(graph.handle, C.byref(dims()), 2, 4097, 4, C.byref(b)) == _abi.TAG_ESHAPE
    assert lib.tag_train_workspace(graph.handle, C.byref(dims()), 2, 60, 0, C.byref(b)) == _abi.TAG_EINVAL
    # a workspace one byte short is refused before anything runs
    c = TrainCase([topo], 2, 64, 4, 2, 60, 2, seed=8)
    _, model, tr, feats = c.trainer(torch)
    tr.ws_bytes -= 1
    with pytest.raises(_abi.TagError) as e:
        tr.step(feats)
    assert e.value.status == _abi.TAG_ENOSPACE
