"""GPU parity of the readings of Section 4.2.1 that the paper leaves open
(five directed relations, ReLU edge encoders, averaged full-width heads)
against the oracle: max row-relative error <= 1e-4 (fp32), on ragged random
graphs, a chain (both directions at every inner op) and a workload
topology, with per-replica and shared edge features; plus the argument
checks of the variant path."""
import ctypes as C

import numpy as np
import pytest

import oracle
import synth
from tests._helpers import mk_topo

pytestmark = pytest.mark.gpu

P = pytest.importorskip("paper_2302_06126_amd")


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    P._abi.load()
    torch.cuda.set_device(0)
    yield
    torch.cuda.synchronize()


from tests._gpu import FP32_TOL, dev_tensor, say  # noqa: E402
from tests._helpers import row_rel_err  # noqa: E402


def _features(topo, R, seed, shared_oo):
    rng = np.random.default_rng((2302, 66, seed))
    x_op = rng.uniform(-1, 1, (R, topo.n_op, 42)).astype(np.float32)
    x_dev = rng.uniform(-1, 1, (R, topo.n_dev, 8)).astype(np.float32)
    x_oo = rng.uniform(-1, 1, topo.e_oo if shared_oo else (R, topo.e_oo)).astype(np.float32)
    x_dd = rng.uniform(-1, 1, (R, topo.e_dd, 2)).astype(np.float32)
    x_od = rng.integers(0, 2, (R, topo.e_od)).astype(np.uint8)
    return x_op, x_dev, x_oo, x_dd, x_od


def _run(topo, R, f, heads, layers, relations, edge_act, heads_mode, seed=0, shared_oo=False):
    w = synth.make_weights(f, heads, layers, 42, f, bias_scale=0.3, seed_extra=seed, relations=relations,
                           heads_mode=heads_mode)
    x_op, x_dev, x_oo, x_dd, x_od = _features(topo, R, seed, shared_oo)
    g = P.Graph([topo])
    m = P.Model(w, f=f, heads=heads, layers=layers, f_op=42, relations=relations, edge_act=edge_act,
                heads_mode=heads_mode)
    E_op, E_dev = P.forward(g, m, dev_tensor(x_op), dev_tensor(x_dev), dev_tensor(x_oo), dev_tensor(x_dd),
                            dev_tensor(x_od))
    worst = 0.0
    for r in range(R):
        xo = x_oo if shared_oo else x_oo[r]
        R_op, R_dev = oracle.forward(topo, x_op[r], x_dev[r], xo, x_dd[r], x_od[r], w, f=f, heads=heads,
                                     layers=layers, relations=relations, edge_act=edge_act, heads_mode=heads_mode)
        got = np.vstack([E_op[r].cpu().numpy(), E_dev[r].cpu().numpy()])
        assert np.all(np.isfinite(got))
        err = row_rel_err(got, np.vstack([R_op, R_dev]))
        worst = max(worst, err)
        assert err <= FP32_TOL, f"candidate {r}: row-relative error {err:.3e}"
    g.close()
    return worst


VARIANTS = [(5, "affine", "concat"), (3, "relu", "concat"), (3, "affine", "avg"), (5, "relu", "avg")]


@pytest.mark.parametrize("relations,edge_act,heads_mode", VARIANTS)
@pytest.mark.parametrize("f,heads,layers", [(64, 4, 2), (128, 2, 2), (256, 8, 1)])
def test_variant_forward_random_graphs(relations, edge_act, heads_mode, f, heads, layers):
    topo = synth.random_topology(400 + f + heads, 130, 7, 260, od_per_op=None, dd_density=0.7)
    say(f"variant R={relations} edge={edge_act} heads={heads_mode} f={f} K={heads} L={layers}")
    err = _run(topo, 3, f, heads, layers, relations, edge_act, heads_mode, seed=f + heads)
    say(f"  worst row-rel err {err:.2e}")


@pytest.mark.parametrize("relations,edge_act,heads_mode", VARIANTS)
def test_variant_chain_and_shared_edge_features(relations, edge_act, heads_mode):
    # a chain: every inner op has one link in each direction; x_oo shared by the replicas
    n = 90
    topo = mk_topo(n, 3, oo=[(i, i + 1) for i in range(n - 1)], dd=[(0, 1), (1, 2), (0, 2)],
                   od=[(u, j) for u in range(n) for j in range(3) if (u + j) % 2 == 0])
    err = _run(topo, 2, 128, 4, 3, relations, edge_act, heads_mode, seed=3, shared_oo=True)
    say(f"chain R={relations} edge={edge_act} heads={heads_mode}: {err:.2e}")


def test_variant_workload_topology():
    topo = synth.make_topology("cnn")
    err = _run(topo, 2, 128, 4, 3, 5, "relu", "concat", seed=7, shared_oo=True)
    say(f"cnn topology, 5 relations + ReLU edges: {err:.2e}")


def test_variant_argument_checks():
    topo = synth.random_topology(5, 20, 3, 30)
    g = P.Graph([topo])
    w = synth.make_weights(64, 4, 1, 42, 64, relations=5)
    lib = P._abi.load()

    def status(**kw):
        d = P._abi.tag_model_dims(64, kw.get("heads", 4), 1, 42, 8, 64, kw.get("dtype", P.TAG_F32), 1.0, 0.1, 0.2,
                                  kw.get("sigma", 0), kw.get("relations", 5), kw.get("edge_act", 0),
                                  kw.get("head_mode", 0))
        b = C.c_size_t(0)
        return lib.tag_gnn_workspace(g.handle, C.byref(d), 2, C.byref(b))

    assert status() == P._abi.TAG_OK
    assert status(dtype=P.TAG_BF16) == P._abi.TAG_ESHAPE
    assert status(sigma=1) == P._abi.TAG_ESHAPE
    assert status(relations=4) == P._abi.TAG_EINVAL
    assert status(relations=3, edge_act=2) == P._abi.TAG_EINVAL
    assert status(relations=3, head_mode=1, heads=16) == P._abi.TAG_ESHAPE
    assert status(relations=3, head_mode=1, heads=8) == P._abi.TAG_OK
    # the training step takes the default readings only
    d = P._abi.tag_model_dims(64, 4, 1, 42, 8, 64, P.TAG_F32, 1.0, 0.1, 0.2, 0, 5, 0, 0)
    b = C.c_size_t(0)
    st = lib.tag_train_workspace(g.handle, C.byref(d), 2, 16, 4, C.byref(b))
    assert st == P._abi.TAG_ESHAPE
    del w
    g.close()
