"""Small helpers shared by the tests (no method arithmetic here)."""
import numpy as np

import synth


def mk_topo(n_op, n_dev, oo=(), dd=(), od=None):
    """A Topology from explicit edge lists; od=None means every (op, device) pair."""
    oo = np.asarray(list(oo), np.int32).reshape(-1, 2)
    dd = np.asarray(list(dd), np.int32).reshape(-1, 2)
    if od is None:
        od = np.array([(u, j) for u in range(n_op) for j in range(n_dev)], np.int32).reshape(-1, 2)
    else:
        od = np.asarray(list(od), np.int32).reshape(-1, 2)
    z = np.zeros
    return synth.Topology(
        n_op=n_op, n_dev=n_dev, oo_src=oo[:, 0].copy(), oo_dst=oo[:, 1].copy(),
        dd_a=dd[:, 0].copy(), dd_b=dd[:, 1].copy(), od_op=od[:, 0].copy(), od_dev=od[:, 1].copy(),
        op_type=z(n_op, int), op_flops=np.ones(n_op), op_bytes=np.ones(n_op),
        dev_tflops=np.ones(n_dev), dev_mem=np.ones(n_dev), dev_intra_bw=np.ones(n_dev),
        dd_bw=np.ones(dd.shape[0]))


def zero_weights(f, layers, f_op, dec_hidden=0):
    w = synth.make_weights(f, 1, layers, f_op, dec_hidden)
    return {k: np.zeros_like(v) for k, v in w.items()}


def random_features(topo, f_op, seed, nonneg=False):
    rng = np.random.default_rng((2302, 55, seed))
    lo = 0.0 if nonneg else -1.0
    x_op = rng.uniform(lo, 1.0, size=(topo.n_op, f_op)).astype(np.float32)
    x_dev = rng.uniform(lo, 1.0, size=(topo.n_dev, 8)).astype(np.float32)
    x_oo = rng.uniform(lo, 1.0, size=topo.e_oo).astype(np.float32)
    x_dd = rng.uniform(lo, 1.0, size=(topo.e_dd, 2)).astype(np.float32)
    x_od = rng.integers(0, 2, size=topo.e_od).astype(np.uint8)
    return x_op, x_dev, x_oo, x_dd, x_od


def row_rel_err(got, ref):
    """max over rows of ||got - ref||_inf / max(||ref||_inf, floor), with the
    floor at 1e-6 of the largest row norm: rows that are all zero (or nearly
    so) in the reference are compared on that absolute scale, every other row
    on its own norm."""
    got = np.asarray(got, np.float64).reshape(ref.shape[0], -1)
    ref = np.asarray(ref, np.float64).reshape(ref.shape[0], -1)
    if ref.size == 0:
        return 0.0
    nrm = np.abs(ref).max(axis=1)
    floor = max(1e-6 * float(nrm.max()), 1e-30)
    return float((np.abs(got - ref).max(axis=1) / np.maximum(nrm, floor)).max())
