"""Pins of the reference training step (oracle/train.py): its forward pass
equals the C oracle's, its loss equals the cross entropy of the C oracle's
priors, its gradient matches central differences of that loss, and a target
equal to the current priors has zero gradient.  CPU only."""
import numpy as np
import pytest

import oracle
import synth
from oracle import train as OT


def _case(seed, n=14, m=3, e=20, f=32, heads=4, layers=2, R=2, S=12, Q=3):
    topo = synth.random_topology(seed, n, m, e)
    w = synth.make_weights(f, heads, layers, 40, f, bias_scale=0.3, seed_extra=seed)
    rng = synth.rng_for(71, seed)
    masks = np.array([int(rng.integers(1, 1 << m)) for _ in range(S)], np.uint64)
    opts = rng.integers(0, 4, size=S).astype(np.uint8)
    items = []
    for r in range(R):
        t = rng.random((Q, S)) + 0.05
        items.append(dict(topo=topo, x_op=rng.uniform(-1, 1, (n, 40)).astype(np.float32),
                          x_dev=rng.uniform(-1, 1, (m, 8)).astype(np.float32),
                          x_oo=rng.uniform(-1, 1, topo.e_oo).astype(np.float32),
                          x_dd=rng.uniform(-1, 1, (topo.e_dd, 2)).astype(np.float32),
                          x_od=rng.integers(0, 2, topo.e_od).astype(np.uint8),
                          query_op=rng.integers(0, n, size=Q).astype(np.int32),
                          target=t / t.sum(1, keepdims=True)))
    return topo, w, masks, opts, items, dict(f=f, heads=heads, layers=layers)


def _c_loss(w, masks, opts, items, dims, sigma="relu"):
    """Cross entropy of the C oracle's priors (float64)."""
    tot, Qn = 0.0, 0
    for it in items:
        E_op, E_dev = oracle.forward(it["topo"], it["x_op"], it["x_dev"], it["x_oo"], it["x_dd"], it["x_od"], w,
                                     f=dims["f"], heads=dims["heads"], layers=dims["layers"], sigma=sigma)
        od = oracle.decide(E_op, E_dev, masks, opts, it["query_op"], w, f=dims["f"], dec_hidden=dims["f"],
                           n_dev=it["topo"].n_dev, want_prior=True)
        tot -= float((it["target"] * np.log(od["prior"])).sum())
        Qn += len(it["query_op"])
    return tot / Qn


@pytest.mark.parametrize("sigma", ["relu", "elu"])
def test_forward_matches_c_oracle(sigma):
    for seed in (1, 2):
        topo, w, masks, opts, items, dims = _case(seed)
        P = {k: OT._t(w[k]) for k in OT.PARAMS}
        it = items[0]
        E_op, E_dev = OT.forward(topo, it["x_op"], it["x_dev"], it["x_oo"], it["x_dd"], it["x_od"], P, **dims,
                                 sigma=sigma)
        R_op, R_dev = oracle.forward(topo, it["x_op"], it["x_dev"], it["x_oo"], it["x_dd"], it["x_od"], w, **dims,
                                     sigma=sigma)
        np.testing.assert_allclose(E_op.detach().numpy(), R_op, rtol=1e-11, atol=1e-13)
        np.testing.assert_allclose(E_dev.detach().numpy(), R_dev, rtol=1e-11, atol=1e-13)


def test_loss_matches_c_oracle_cross_entropy():
    topo, w, masks, opts, items, dims = _case(3)
    loss, _ = OT.loss_and_grads(items, w, masks=masks, options=opts, **dims)
    assert loss == pytest.approx(_c_loss(w, masks, opts, items, dims), rel=1e-11)


@pytest.mark.parametrize("sigma", ["relu", "elu"])
def test_gradient_matches_central_differences(sigma):
    """Every parameter array: a few entries, differentiated numerically
    through the C oracle (perturbations representable in float32)."""
    topo, w, masks, opts, items, dims = _case(4, f=16, heads=2, layers=2, S=8)
    _, g = OT.loss_and_grads(items, w, masks=masks, options=opts, **dims, sigma=sigma)
    rng = synth.rng_for(72)
    for k in OT.PARAMS:
        flat = w[k].reshape(-1)
        picks = rng.choice(flat.size, size=min(3, flat.size), replace=False)
        for i in picks:
            x0 = float(flat[i])
            h = 1e-4 * max(1.0, abs(x0))
            wp = {kk: vv.copy() for kk, vv in w.items()}
            wm = {kk: vv.copy() for kk, vv in w.items()}
            wp[k].reshape(-1)[i] = np.float32(x0 + h)
            wm[k].reshape(-1)[i] = np.float32(x0 - h)
            hp = float(wp[k].reshape(-1)[i]) - x0
            hm = x0 - float(wm[k].reshape(-1)[i])
            lp, lm = _c_loss(wp, masks, opts, items, dims, sigma), _c_loss(wm, masks, opts, items, dims, sigma)
            fd = (lp - lm) / (hp + hm)
            an = float(g[k].reshape(-1)[i])
            if abs(fd - an) <= 1e-4 * max(abs(an), abs(fd)) + 2e-8:
                continue
            # a ReLU / LeakyReLU kink inside [x - h, x + h]: the one-sided
            # differences then disagree and the derivative lies between them
            l0 = _c_loss(w, masks, opts, items, dims, sigma)
            up, dn = (lp - l0) / hp, (l0 - lm) / hm
            lo, hi = min(up, dn), max(up, dn)
            tol = 1e-4 * max(abs(up), abs(dn)) + 2e-8
            assert lo - tol <= an <= hi + tol, (k, int(i), fd, an, up, dn)


def test_targets_equal_to_priors_give_zero_gradient():
    topo, w, masks, opts, items, dims = _case(5)
    for it in items:
        E_op, E_dev = oracle.forward(it["topo"], it["x_op"], it["x_dev"], it["x_oo"], it["x_dd"], it["x_od"], w,
                                     **dims)
        it["target"] = oracle.decide(E_op, E_dev, masks, opts, it["query_op"], w, f=dims["f"],
                                     dec_hidden=dims["f"], n_dev=it["topo"].n_dev)["prior"]
    _, g = OT.loss_and_grads(items, w, masks=masks, options=opts, **dims)
    for k in OT.PARAMS:
        assert np.abs(g[k]).max() <= 1e-12, k


def _biased(seed, bias):
    """A case whose message pre-activations all share the sign of `bias`
    (the folded bias c' = W^e c + b dominates every W^h h + U x)."""
    topo, w, masks, opts, items, dims = _case(seed, layers=1)
    w = {k: v.copy() for k, v in w.items()}
    w["layer_b"][:] = bias
    return topo, w, items, dims


def test_elu_equals_relu_when_every_message_is_positive():
    topo, w, items, dims = _biased(6, 100.0)
    it = items[0]
    a = oracle.forward(topo, it["x_op"], it["x_dev"], it["x_oo"], it["x_dd"], it["x_od"], w, **dims, sigma="relu")
    b = oracle.forward(topo, it["x_op"], it["x_dev"], it["x_oo"], it["x_dd"], it["x_od"], w, **dims, sigma="elu")
    assert np.array_equal(a[0], b[0]) and np.array_equal(a[1], b[1])


def test_elu_saturates_to_minus_gamma_sum_for_negative_messages():
    """Every message is ELU(z) with z about -100, i.e. -1 to double precision,
    so each head's softmax average is -1 and a node's output is minus the sum
    of gamma over the link types it has neighbours in (ReLU gives zeros)."""
    topo, w, items, dims = _biased(7, -100.0)
    it = items[0]
    E_op, E_dev = oracle.forward(topo, it["x_op"], it["x_dev"], it["x_oo"], it["x_dd"], it["x_od"], w, **dims,
                                 sigma="elu")
    R_op, R_dev = oracle.forward(topo, it["x_op"], it["x_dev"], it["x_oo"], it["x_dd"], it["x_od"], w, **dims)
    assert not np.any(R_op) and not np.any(R_dev)
    n, m = topo.n_op, topo.n_dev
    has_oo = np.zeros(n, bool)
    has_oo[np.asarray(topo.oo_src)] = True
    has_oo[np.asarray(topo.oo_dst)] = True
    has_od_op = np.zeros(n, bool)
    has_od_op[np.asarray(topo.od_op)] = True
    has_od_dev = np.zeros(m, bool)
    has_od_dev[np.asarray(topo.od_dev)] = True
    has_dd = np.zeros(m, bool)
    has_dd[np.asarray(topo.dd_a)] = True
    has_dd[np.asarray(topo.dd_b)] = True
    want_op = -(1.0 * has_oo + 0.1 * has_od_op)
    want_dev = -(0.1 * has_od_dev + 1.0 * has_dd)
    np.testing.assert_allclose(E_op, np.repeat(want_op[:, None], dims["f"], 1), rtol=0, atol=1e-12)
    np.testing.assert_allclose(E_dev, np.repeat(want_dev[:, None], dims["f"], 1), rtol=0, atol=1e-12)
