"""GPU parity of the full-enumeration decision head (tag_gnn_decide_full)
against the C oracle's decide on the explicit table of every non-empty
device mask with each option (slice a = 4 (mask - 1) + option), on the same
embeddings: argmax exact outside a 1e-5 score band (otherwise the pick is
within the band), decoded decisions exact, best score 1e-5, priors within
1e-4 relative (fp32 against fp64: the enumeration updates the device sum by
one row per mask, at most 2^16 / (waves) steps from a fresh sum).  Also a
union of topologies with different device counts (zero-padded prior rows),
invalid queries and the argument limits."""
import numpy as np
import pytest

import oracle
import paper_2302_06126_amd as P
import synth
from tests._gpu import decide_gap_ok, dev_tensor, say

pytestmark = pytest.mark.gpu


def _full_table(m):
    masks = np.array([k for k in range(1, 1 << m) for _ in range(4)], np.uint64)
    opts = np.array([o for _ in range(1, 1 << m) for o in range(4)], np.uint8)
    return masks, opts


def _check(res, q, od, S_q):
    if decide_gap_ok(od["prior"][0], od["best"][0], 1e-5):
        assert res["argmax"][q] == od["argmax"][0]
        for k in ("mask", "option", "replicas", "sync", "sfb"):
            assert res[k][q] == od[k][0], k
    else:
        a = res["argmax"][q]
        s_pick = od["best"][0] + np.log(od["prior"][0][a] / od["prior"][0][od["argmax"][0]])
        assert s_pick >= od["best"][0] - 1e-5 * max(1.0, abs(od["best"][0]))
    np.testing.assert_allclose(res["best"][q], od["best"][0], rtol=1e-5, atol=1e-5)
    np.testing.assert_allclose(res["prior"][q][:S_q], od["prior"][0], rtol=1e-4, atol=1e-7)
    assert not np.any(res["prior"][q][S_q:])
    assert abs(res["prior"][q].sum() - 1.0) < 1e-4


@pytest.mark.parametrize("m_dev,f,H,Q", [(4, 64, 64, 20), (5, 64, 0, 20), (10, 128, 128, 12), (16, 128, 128, 2),
                                         (13, 256, 512, 4), (1, 64, 32, 5)])
def test_full_enumeration_matches_oracle(m_dev, f, H, Q):
    say(f"[decide_full] M={m_dev} f={f} H={H} Q={Q}")
    rng = np.random.default_rng((2302, 89, m_dev, H))
    n, R = 30, 2
    topo = synth.random_topology(200 + m_dev, n, m_dev, 40)
    E_op = rng.uniform(0, 1, (R, n, f)).astype(np.float32)
    E_dev = rng.uniform(0, 1, (R, m_dev, f)).astype(np.float32)
    w = synth.make_weights(f, 4, 1, 42, H, bias_scale=0.5, seed_extra=m_dev)
    g = P.Graph([topo])
    m = P.Model(w, f=f, heads=4, layers=1, f_op=42, dec_hidden=H)
    qr = rng.integers(0, R, Q).astype(np.int32)
    qo = rng.integers(0, n, Q).astype(np.int32)
    res = P.decide_full(g, m, dev_tensor(E_op), dev_tensor(E_dev), qr, np.zeros(Q, np.int32), qo)
    masks, opts = _full_table(m_dev)
    for q in range(Q):
        od = oracle.decide(E_op[qr[q]].astype(np.float64), E_dev[qr[q]].astype(np.float64), masks, opts,
                           qo[q:q + 1], w, f=f, dec_hidden=H, n_dev=m_dev)
        _check(res, q, od, len(masks))
    if m_dev <= 10:   # the table-driven head on the explicit table agrees too
        tab = P.decide(g, m, dev_tensor(E_op), dev_tensor(E_dev), masks, opts, qr, np.zeros(Q, np.int32), qo)
        np.testing.assert_allclose(res["prior"], tab["prior"], rtol=1e-4, atol=1e-7)


def test_full_enumeration_union_and_invalid_queries():
    say("[decide_full] union of topologies, invalid queries")
    rng = np.random.default_rng((2302, 90))
    topos = [synth.random_topology(301, 20, 3, 30), synth.random_topology(302, 25, 6, 40)]
    f, H, R = 64, 32, 2
    g = P.Graph(topos)
    n_op, n_dev = sum(t.n_op for t in topos), sum(t.n_dev for t in topos)
    E_op = rng.uniform(0, 1, (R, n_op, f)).astype(np.float32)
    E_dev = rng.uniform(0, 1, (R, n_dev, f)).astype(np.float32)
    w = synth.make_weights(f, 4, 1, 42, H, bias_scale=0.5, seed_extra=7)
    m = P.Model(w, f=f, heads=4, layers=1, f_op=42, dec_hidden=H)
    qr = np.array([0, 1, 1, 0, 5, 0], np.int32)
    qg = np.array([0, 1, 0, 1, 0, 2], np.int32)
    qo = np.array([3, 7, 19, 24, 0, 0], np.int32)
    res = P.decide_full(g, m, dev_tensor(E_op), dev_tensor(E_dev), qr, qg, qo)
    op_off = [0, topos[0].n_op]
    dev_off = [0, topos[0].n_dev]
    for q in range(4):
        t = topos[qg[q]]
        masks, opts = _full_table(t.n_dev)
        eo = E_op[qr[q], op_off[qg[q]]:op_off[qg[q]] + t.n_op].astype(np.float64)
        ed = E_dev[qr[q], dev_off[qg[q]]:dev_off[qg[q]] + t.n_dev].astype(np.float64)
        od = oracle.decide(eo, ed, masks, opts, qo[q:q + 1], w, f=f, dec_hidden=H, n_dev=t.n_dev)
        _check(res, q, od, len(masks))
    assert list(res["argmax"][4:]) == [-1, -1]
    assert np.all(np.isnan(res["best"][4:]))
    assert not np.any(res["prior"][4:])


def test_full_enumeration_limits():
    from paper_2302_06126_amd import _abi
    import ctypes as C
    say("[decide_full] limits")
    lib = _abi.load()
    b = C.c_size_t()
    big = P.Graph([synth.random_topology(303, 10, 17, 10)])
    m = P.Model(synth.make_weights(64, 4, 1, 42, 64), f=64, heads=4, layers=1, f_op=42)
    assert lib.tag_gnn_decide_full_workspace(big.handle, C.byref(m.dims), 1, 1, C.byref(b)) == _abi.TAG_ESHAPE
    small = P.Graph([synth.random_topology(304, 10, 4, 10)])
    m2 = P.Model(synth.make_weights(64, 4, 1, 42, 600), f=64, heads=4, layers=1, f_op=42)
    assert lib.tag_gnn_decide_full_workspace(small.handle, C.byref(m2.dims), 1, 1, C.byref(b)) == _abi.TAG_ESHAPE
    assert lib.tag_gnn_decide_full_workspace(small.handle, C.byref(m.dims), 1, 1, C.byref(b)) == _abi.TAG_OK
