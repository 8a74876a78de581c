"""Pins for the CPU oracle: each test checks it against something other than
itself -- brute force, a closed form of a special case, an invariant of the
method, hand-worked numbers, or a library routine -- so that a dropped term, a
wrong sign or index, or a transposed operand fails at least one of them.

Paper passages: Section 4.2.1 (joint graph with two node types and three link
types; per-link-type affine map of the concatenation of neighbour embedding
and edge feature, non-linearity, gamma-weighted multi-head attention
aggregation; decoder over strategy slices) and Section 4.2 (strategy encoding
P, O with four replication options).
"""
import itertools
import math

import numpy as np
import pytest

import synth
from tests._helpers import mk_topo, random_features, zero_weights

pytestmark = pytest.mark.filterwarnings("ignore::RuntimeWarning")


# ---------------------------------------------------------------- CSR ------

def _expected_buckets(topo):
    """Brute force: expand every link into its destination entries and sort."""
    b0 = [(int(c), int(p), i) for i, (p, c) in enumerate(zip(topo.oo_src, topo.oo_dst))]
    b0 += [(int(p), int(c), i) for i, (p, c) in enumerate(zip(topo.oo_src, topo.oo_dst))]
    b1 = [(int(u), int(j), i) for i, (u, j) in enumerate(zip(topo.od_op, topo.od_dev))]
    b2 = [(int(j), int(u), i) for i, (u, j) in enumerate(zip(topo.od_op, topo.od_dev))]
    b3 = [(int(a), int(b), i) for i, (a, b) in enumerate(zip(topo.dd_a, topo.dd_b))]
    b3 += [(int(b), int(a), i) for i, (a, b) in enumerate(zip(topo.dd_a, topo.dd_b))]
    out = []
    for ent, nrows in ((b0, topo.n_op), (b1, topo.n_op), (b2, topo.n_dev), (b3, topo.n_dev)):
        ent = sorted(ent)
        rp = np.zeros(nrows + 1, np.int64)
        for r, _, _ in ent:
            rp[r + 1] += 1
        out.append((np.cumsum(rp), [e[1] for e in ent], [e[2] for e in ent]))
    return out


def _csr(orc, topo):
    return orc.csr(topo.n_op, topo.n_dev, topo.oo_src, topo.oo_dst,
                   topo.dd_a, topo.dd_b, topo.od_op, topo.od_dev)


@pytest.mark.parametrize("seed,n,m,e,per", [(0, 30, 4, 60, None), (1, 57, 7, 200, 3),
                                           (2, 5, 1, 4, None), (3, 40, 9, 0, 2)])
def test_csr_brute_force(orc, seed, n, m, e, per):
    topo = synth.random_topology(seed, n, m, e, od_per_op=per, dd_density=0.6)
    st, buckets = _csr(orc, topo)
    assert st == 0
    for (rp, col, eid), (erp, ecol, eeid) in zip(buckets, _expected_buckets(topo)):
        assert np.array_equal(rp, erp)
        assert list(col) == ecol and list(eid) == eeid
        assert np.all(np.diff(rp) >= 0)


def test_csr_input_order_invariance(orc):
    topo = synth.random_topology(11, 40, 6, 90, od_per_op=4)
    st, ref = _csr(orc, topo)
    rng = np.random.default_rng(5)
    p_oo, p_dd, p_od = (rng.permutation(k) for k in (topo.e_oo, topo.e_dd, topo.e_od))
    st2, got = orc.csr(topo.n_op, topo.n_dev, topo.oo_src[p_oo], topo.oo_dst[p_oo],
                       topo.dd_b[p_dd], topo.dd_a[p_dd], topo.od_op[p_od], topo.od_dev[p_od])
    assert st == st2 == 0
    inv = [np.argsort(p) for p in (p_oo, p_od, p_od, p_dd)]
    for (rp, col, eid), (rp2, col2, eid2), iv in zip(ref, got, inv):
        assert np.array_equal(rp, rp2) and np.array_equal(col, col2)
        # the same entries, with edge ids renamed by the input permutation
        assert np.array_equal(iv[eid], eid2)


@pytest.mark.parametrize("case,status", [
    ("oo_range", -2), ("od_range", -2), ("dd_range", -2), ("self_oo", -3), ("self_dd", -3),
    ("dup_oo", -3), ("both_dirs", -3), ("dup_od", -3), ("dup_dd_swapped", -3),
    ("range_beats_dup", -2)])
def test_csr_rejects(orc, case, status):
    oo = [(0, 1), (1, 2)]
    dd = [(0, 1)]
    od = [(0, 0), (1, 1)]
    n, m = 3, 2
    if case == "oo_range": oo.append((2, 3))
    if case == "od_range": od.append((0, 2))
    if case == "dd_range": dd.append((-1, 0))
    if case == "self_oo": oo.append((2, 2))
    if case == "self_dd": dd.append((1, 1))
    if case == "dup_oo": oo.append((0, 1))
    if case == "both_dirs": oo.append((1, 0))
    if case == "dup_od": od.append((1, 1))
    if case == "dup_dd_swapped": dd.append((1, 0))
    if case == "range_beats_dup": oo += [(0, 1), (5, 0)]
    t = mk_topo(n, m, oo, dd, od)
    st, _ = _csr(orc, t)
    assert st == status


# ------------------------------------------------------- layer maths -------

def _identity_encoders(w, f):
    w["enc_op_w"][:] = np.eye(f, w["enc_op_w"].shape[1])
    w["enc_dev_w"][:] = np.eye(f, 8)


def _adjacency(topo):
    """Per link type, the (N+M)x(N+M) 0/1 neighbour matrix built from the raw links."""
    n, m = topo.n_op, topo.n_dev
    A = [np.zeros((n + m, n + m)) for _ in range(3)]
    for p, c in zip(topo.oo_src, topo.oo_dst):
        A[0][c, p] = A[0][p, c] = 1
    for u, j in zip(topo.od_op, topo.od_dev):
        A[1][u, n + j] = A[1][n + j, u] = 1
    for a, b in zip(topo.dd_a, topo.dd_b):
        A[2][n + a, n + b] = A[2][n + b, n + a] = 1
    return A


def _rownorm(A):
    s = A.sum(axis=1, keepdims=True)
    return np.divide(A, s, out=np.zeros_like(A), where=s > 0)


@pytest.mark.parametrize("seed,layers", [(0, 1), (1, 2), (2, 4)])
def test_uniform_attention_is_mean_aggregation(orc, seed, layers):
    """a = adst = 0, W^h = I, W^e = 0, b = 0, non-negative features: every
    layer is gamma-weighted mean aggregation, so H^L = P^L H^0 with
    P = sum_t gamma_t D_t^-1 A_t."""
    f = 8
    topo = synth.random_topology(20 + seed, 14, 4, 25, od_per_op=2, dd_density=0.7)
    w = zero_weights(f, layers, f)
    _identity_encoders(w, f)
    w["layer_w"][:, :, :, :f] = np.eye(f)
    x_op, x_dev, x_oo, x_dd, x_od = random_features(topo, f, seed, nonneg=True)
    E_op, E_dev = orc.forward(topo, x_op, x_dev, x_oo, x_dd, x_od, w, f=f, heads=2, layers=layers)
    A = _adjacency(topo)
    P = _rownorm(A[0]) + 0.1 * _rownorm(A[1]) + _rownorm(A[2])
    H = np.linalg.matrix_power(P, layers) @ np.vstack([x_op, x_dev]).astype(np.float64)
    np.testing.assert_allclose(np.vstack([E_op, E_dev]), H, rtol=0, atol=1e-12)


def test_relation_transforms_are_applied_per_link_type(orc):
    """W^h_t = a distinct permutation matrix per link type: one layer gives
    H' = sum_t gamma_t P_t H Pi_t^T (catches a transposed or swapped W^h)."""
    f = 8
    topo = synth.random_topology(31, 12, 3, 20, dd_density=1.0)
    w = zero_weights(f, 1, f)
    _identity_encoders(w, f)
    perms = [np.roll(np.eye(f), s, axis=0)[:, np.random.default_rng(s).permutation(f)] for s in (1, 2, 3)]
    for r in range(3):
        w["layer_w"][0, r, :, :f] = perms[r]
    x_op, x_dev, x_oo, x_dd, x_od = random_features(topo, f, 7, nonneg=True)
    E_op, E_dev = orc.forward(topo, x_op, x_dev, x_oo, x_dd, x_od, w, f=f, heads=4, layers=1)
    A = _adjacency(topo)
    H = np.vstack([x_op, x_dev]).astype(np.float64)
    want = sum(g * _rownorm(A[r]) @ H @ perms[r].T for r, g in zip(range(3), (1.0, 0.1, 1.0)))
    np.testing.assert_allclose(np.vstack([E_op, E_dev]), want, rtol=0, atol=1e-12)


def test_edge_features_closed_form(orc):
    """H^0 = 0 and uniform attention: one layer averages ReLU(W^e e_uv + b)
    over each link type.  With one-hot edge encoders and permutation W^e,
    each raw edge feature lands in a known channel."""
    f = 8
    topo = synth.random_topology(41, 16, 4, 30, od_per_op=3, dd_density=0.8)
    w = zero_weights(f, 1, f)
    rng = np.random.default_rng(3)
    w["layer_w"][0, :, :, :f] = rng.normal(size=(3, f, f))   # irrelevant: h = 0
    w["enc_edge_w0"][0, 0] = 1.0          # oo: raw value -> channel 0
    w["enc_edge_w1"][1, 0] = 1.0          # od: bit -> channel 1
    w["enc_edge_w2"][2, 0] = 1.0          # dd: (x0, x1) -> channels 2, 3
    w["enc_edge_w2"][3, 1] = 1.0
    pi = {0: {0: 5}, 1: {1: 2}, 2: {2: 6, 3: 7}}
    for r, mp in pi.items():
        for k, c in mp.items():
            w["layer_w"][0, r, c, f + k] = 1.0
    x_op, x_dev, x_oo, x_dd, x_od = random_features(topo, f, 9, nonneg=True)
    E_op, E_dev = orc.forward(topo, x_op, x_dev, x_oo, x_dd, x_od, w, f=f, heads=2, layers=1)
    n, m = topo.n_op, topo.n_dev
    want_op = np.zeros((n, f))
    want_dev = np.zeros((m, f))
    for u in range(n):
        vals = [float(x_oo[i]) for i in range(topo.e_oo) if topo.oo_src[i] == u or topo.oo_dst[i] == u]
        if vals:
            want_op[u, 5] = np.mean(vals)
        bits = [float(x_od[i]) for i in range(topo.e_od) if topo.od_op[i] == u]
        if bits:
            want_op[u, 2] = 0.1 * np.mean(bits)
    for j in range(m):
        bits = [float(x_od[i]) for i in range(topo.e_od) if topo.od_dev[i] == j]
        if bits:
            want_dev[j, 2] = 0.1 * np.mean(bits)
        rows = [x_dd[i].astype(np.float64) for i in range(topo.e_dd) if topo.dd_a[i] == j or topo.dd_b[i] == j]
        if rows:
            want_dev[j, 6], want_dev[j, 7] = np.mean(rows, axis=0)
    np.testing.assert_allclose(E_op, want_op, rtol=0, atol=1e-12)
    np.testing.assert_allclose(E_dev, want_dev, rtol=0, atol=1e-12)


@pytest.mark.parametrize("scale,slope", [(1.0, 0.2), (2.0, 0.2), (1.0, 0.01)])
def test_attention_hand_worked(orc, scale, slope):
    """Ops 0 -> 2 and 1 -> 2, f = 4, two heads of 2 channels, W^h = scale*I.
    Scores, worked by hand (m_v = scale*h_v, destination term scale*adst.h_2):
      head 0: scale*(1 + 0.5) = 1.5s  and  LeakyReLU(scale*(-1 + 0.5))
      head 1: scale*(1 - 1)   = 0     and  scale*(1.5 - 1) = 0.5s
    op 2 gets the softmax mix; ops 0 and 1 have op 2 as single neighbour."""
    f = 4
    topo = mk_topo(3, 1, oo=[(0, 2), (1, 2)], od=[])
    w = zero_weights(f, 1, f)
    w["enc_op_w"][:] = np.eye(f)
    w["layer_w"][0, 0, :, :f] = scale * np.eye(f)
    w["att_src"][0, 0] = [1.0, -1.0, 0.5, 0.5]
    w["att_dst"][0, 0] = [0.25, 0.25, -1.0, 0.0]
    x_op = np.array([[1, 0, 2, 0], [0, 1, 0, 3], [1, 1, 1, 1]], np.float32)
    x_dev = np.zeros((1, 8), np.float32)
    E_op, E_dev = orc.forward(topo, x_op, x_dev, np.zeros(2, np.float32), np.zeros((0, 2), np.float32),
                              np.zeros(0, np.uint8), w, f=f, heads=2, layers=1, leaky_slope=slope)
    lk = lambda t: t if t > 0 else slope * t
    s00, s01 = lk(scale * 1.5), lk(scale * -0.5)
    s10, s11 = lk(0.0), lk(scale * 0.5)
    a0 = math.exp(s00) / (math.exp(s00) + math.exp(s01))
    b0 = math.exp(s10) / (math.exp(s10) + math.exp(s11))
    want2 = scale * np.array([a0 * 1, (1 - a0) * 1, b0 * 2, (1 - b0) * 3])
    np.testing.assert_allclose(E_op[2], want2, rtol=0, atol=1e-14)
    np.testing.assert_allclose(E_op[0], scale * np.ones(4), atol=1e-14)
    np.testing.assert_allclose(E_op[1], scale * np.ones(4), atol=1e-14)
    assert np.all(E_dev == 0.0)


def test_attention_weights_sum_to_one(orc):
    topo = synth.random_topology(51, 25, 5, 60, od_per_op=3)
    wl = 16
    w = synth.make_weights(wl, 4, 2, 42, 0)
    x_op, x_dev, x_oo, x_dd, x_od = random_features(topo, 42, 1)
    _, _, alpha = orc.forward(topo, x_op, x_dev, x_oo, x_dd, x_od, w, f=wl, heads=4, layers=2,
                              want_alpha=True)
    st, buckets = orc.csr(topo.n_op, topo.n_dev, topo.oo_src, topo.oo_dst, topo.dd_a, topo.dd_b,
                          topo.od_op, topo.od_dev)
    off = 0
    for rp, col, _ in buckets:
        for r in range(len(rp) - 1):
            seg = alpha[off + rp[r]: off + rp[r + 1]]
            if len(seg):
                np.testing.assert_allclose(seg.sum(axis=0), 1.0, atol=1e-12)
                assert np.all(seg >= 0)
                if len(seg) == 1:
                    assert np.all(seg == 1.0)
        off += len(col)
    assert off == alpha.shape[0]


def test_identical_messages_ignore_attention(orc):
    """W^h = 0, W^e = 0: every message of a link type is ReLU(b_t), so the
    output is sum_t gamma_t ReLU(b_t) over the link types present, whatever
    the attention vectors are."""
    f = 8
    topo = synth.random_topology(61, 10, 3, 12, od_per_op=2, dd_density=0.5)
    w = synth.make_weights(f, 2, 1, 42, 0)
    w["layer_w"][:] = 0.0
    b = np.array([[0.3, -0.2, 0.5, 0.1, -0.7, 0.2, 0.9, 0.0],
                  [0.1, 0.2, -0.3, 0.4, 0.5, -0.6, 0.7, 0.8],
                  [-0.1, 0.6, 0.2, 0.3, 0.0, 0.4, -0.5, 0.25]], np.float32)
    w["layer_b"][0] = b
    x = random_features(topo, 42, 2)
    E_op, E_dev = orc.forward(topo, *x, w, f=f, heads=2, layers=1)
    A = _adjacency(topo)
    n = topo.n_op
    rb = np.maximum(b.astype(np.float64), 0)
    has = [A[r].sum(axis=1) > 0 for r in range(3)]
    want = (has[0][:, None] * rb[0] + 0.1 * has[1][:, None] * rb[1] + has[2][:, None] * rb[2])
    np.testing.assert_allclose(np.vstack([E_op, E_dev]), want, rtol=0, atol=1e-15)


def _dense_forward(topo, x_op, x_dev, x_oo, x_dd, x_od, w, f, heads, layers, slope=0.2, relations=3,
                   edge_act="affine", heads_mode="concat"):
    """Independent dense formulation: masked (dst x src x f) message tensors,
    -inf-masked softmax over the source axis, einsum aggregation.  Variants:
    5 directed relations (op<-op along / against the tensor as separate
    relations with their own parameters and softmax, op<-device and
    device<-op separate), ReLU after the edge encoders, K full-width heads
    averaged."""
    n, m = topo.n_op, topo.n_dev
    avg = heads_mode == "avg"
    d = f if avg else f // heads
    relu = lambda t: np.maximum(t, 0)
    W = w["layer_w"].astype(np.float64)
    h_op = relu(x_op.astype(np.float64) @ w["enc_op_w"].T.astype(np.float64) + w["enc_op_b"])
    h_dev = relu(x_dev.astype(np.float64) @ w["enc_dev_w"].T.astype(np.float64) + w["enc_dev_b"])
    # edge-feature tensors [dst, src, f] per bucket (NaN where no link)
    def etensor(nd, ns, pairs, feats, r):
        A = w[f"enc_edge_w{r}"].astype(np.float64)
        c = w[f"enc_edge_b{r}"].astype(np.float64)
        T = np.full((nd, ns, f), np.nan)
        for (dst, src), x in zip(pairs, feats):
            e = A @ np.atleast_1d(np.asarray(x, np.float64)) + c
            T[dst, src] = relu(e) if edge_act == "relu" else e
        return T
    fwd = list(zip(topo.oo_dst, topo.oo_src))     # consumer <- producer
    bwd = list(zip(topo.oo_src, topo.oo_dst))     # producer <- consumer
    if relations == 3:
        E0 = [etensor(n, n, fwd + bwd, list(x_oo) + list(x_oo), 0)]
    else:
        E0 = [etensor(n, n, fwd, list(x_oo), 0), etensor(n, n, bwd, list(x_oo), 0)]
    E1 = etensor(n, m, list(zip(topo.od_op, topo.od_dev)), list(x_od.astype(np.float64)), 1)
    E2 = etensor(m, n, list(zip(topo.od_dev, topo.od_op)), list(x_od.astype(np.float64)), 1)
    dd_pairs = list(zip(topo.dd_a, topo.dd_b)) + list(zip(topo.dd_b, topo.dd_a))
    E3 = etensor(m, m, dd_pairs, list(x_dd) + list(x_dd), 2)

    def bucket(hs, hd, E, l, r):
        Wh, We = W[l, r, :, :f], W[l, r, :, f:]
        b = w["layer_b"][l, r].astype(np.float64)
        mask = ~np.isnan(E[..., 0])
        Ys, Yd = hs @ Wh.T, hd @ Wh.T
        Z = Ys[None, :, :] + np.einsum("dsk,ck->dsc", np.nan_to_num(E), We) + b
        M = relu(Z)
        out = np.zeros((hd.shape[0], f))
        for k in range(heads):
            sl = slice(0, f) if avg else slice(k * d, (k + 1) * d)
            a = w["att_src"][l, r][k] if avg else w["att_src"][l, r]
            ad = w["att_dst"][l, r][k] if avg else w["att_dst"][l, r]
            a, ad = a.astype(np.float64), ad.astype(np.float64)
            s = np.einsum("dsc,c->ds", M[:, :, sl], a[sl]) + (Yd[:, sl] @ ad[sl])[:, None]
            s = np.where(s > 0, s, slope * s)
            s = np.where(mask, s, -np.inf)
            mx = s.max(axis=1, keepdims=True)
            mx = np.where(np.isfinite(mx), mx, 0.0)
            p = np.where(mask, np.exp(s - mx), 0.0)
            z = p.sum(axis=1, keepdims=True)
            al = np.divide(p, z, out=np.zeros_like(p), where=z > 0)
            out[:, sl] += np.einsum("ds,dsc->dc", al, M[:, :, sl]) / (heads if avg else 1)
        return out

    for l in range(layers):
        if relations == 3:
            n_op_new = bucket(h_op, h_op, E0[0], l, 0) + 0.1 * bucket(h_dev, h_op, E1, l, 1)
            n_dev_new = 0.1 * bucket(h_op, h_dev, E2, l, 1) + bucket(h_dev, h_dev, E3, l, 2)
        else:
            n_op_new = (bucket(h_op, h_op, E0[0], l, 0) + bucket(h_op, h_op, E0[1], l, 1)
                        + 0.1 * bucket(h_dev, h_op, E1, l, 2))
            n_dev_new = 0.1 * bucket(h_op, h_dev, E2, l, 3) + bucket(h_dev, h_dev, E3, l, 4)
        h_op, h_dev = n_op_new, n_dev_new
    return h_op, h_dev


@pytest.mark.parametrize("seed,n,m,e,per,f,heads,layers", [
    (0, 12, 3, 20, None, 8, 2, 2), (1, 20, 4, 35, 2, 16, 4, 3), (2, 6, 2, 5, 1, 8, 1, 1),
    (3, 24, 4, 60, 3, 32, 4, 4)])
def test_dense_recomputation(orc, seed, n, m, e, per, f, heads, layers):
    topo = synth.random_topology(70 + seed, n, m, e, od_per_op=per, dd_density=0.7)
    w = synth.make_weights(f, heads, layers, 42, 0, bias_scale=0.3, seed_extra=seed)
    x = random_features(topo, 42, 30 + seed)
    E_op, E_dev = orc.forward(topo, *x, w, f=f, heads=heads, layers=layers)
    R_op, R_dev = _dense_forward(topo, *x, w, f, heads, layers)
    np.testing.assert_allclose(E_op, R_op, rtol=0, atol=1e-12)
    np.testing.assert_allclose(E_dev, R_dev, rtol=0, atol=1e-12)


# ---------------------------------------- variants of the layer readings ---

VARIANTS = [(5, "affine", "concat"), (3, "relu", "concat"), (3, "affine", "avg"), (5, "relu", "avg")]


@pytest.mark.parametrize("relations,edge_act,heads_mode", VARIANTS)
@pytest.mark.parametrize("seed,n,m,e,per,f,heads,layers", [
    (0, 12, 3, 20, None, 8, 2, 2), (1, 20, 4, 35, 2, 16, 4, 3), (3, 24, 4, 60, 3, 32, 4, 2)])
def test_variants_dense_recomputation(orc, relations, edge_act, heads_mode, seed, n, m, e, per, f, heads, layers):
    """Each reading the paper leaves open (directed relations, ReLU edge
    encoders, averaged full-width heads) against the independent dense
    formulation."""
    topo = synth.random_topology(170 + seed, n, m, e, od_per_op=per, dd_density=0.7)
    w = synth.make_weights(f, heads, layers, 42, 0, bias_scale=0.3, seed_extra=seed, relations=relations,
                           heads_mode=heads_mode)
    x = random_features(topo, 42, 130 + seed)
    kw = dict(relations=relations, edge_act=edge_act, heads_mode=heads_mode)
    E_op, E_dev = orc.forward(topo, *x, w, f=f, heads=heads, layers=layers, **kw)
    R_op, R_dev = _dense_forward(topo, *x, w, f, heads, layers, **kw)
    np.testing.assert_allclose(E_op, R_op, rtol=0, atol=1e-12)
    np.testing.assert_allclose(E_dev, R_dev, rtol=0, atol=1e-12)
    # the variant changes the result (it is not silently the default)
    D_op, _ = orc.forward(topo, *x, synth.make_weights(f, heads, layers, 42, 0, bias_scale=0.3, seed_extra=seed),
                          f=f, heads=heads, layers=layers)
    assert np.abs(E_op - D_op).max() > 1e-6


def test_directed_relations_reduce_on_a_bipartite_dag(orc):
    """Two op layers (producers 0..4, consumers 5..11): every op row has
    links in one direction only, so with the forward and backward relations
    sharing the op-op parameters and op<-device / device<-op sharing the
    placement parameters, the directed reading equals the undirected one."""
    rng = np.random.default_rng(9)
    pairs = sorted({(int(p), int(c)) for p, c in zip(rng.integers(0, 5, 30), rng.integers(5, 12, 30))})
    topo = mk_topo(12, 3, oo=pairs, dd=[(0, 1), (1, 2)])
    f, heads, layers = 16, 4, 2
    w3 = synth.make_weights(f, heads, layers, 42, 0, bias_scale=0.3)
    w5 = dict(w3)
    for k in ("layer_w", "layer_b", "att_src", "att_dst"):
        w5[k] = np.ascontiguousarray(w3[k][:, [0, 0, 1, 1, 2]])
    x = random_features(topo, 42, 12)
    A = orc.forward(topo, *x, w3, f=f, heads=heads, layers=layers)
    B = orc.forward(topo, *x, w5, f=f, heads=heads, layers=layers, relations=5)
    for a, b in zip(A, B):
        np.testing.assert_allclose(a, b, rtol=0, atol=1e-13)
    # a chain has both directions at its inner ops: there the readings differ
    chain = mk_topo(12, 3, oo=[(i, i + 1) for i in range(11)], dd=[(0, 1), (1, 2)])
    xc = random_features(chain, 42, 13)
    C3 = orc.forward(chain, *xc, w3, f=f, heads=heads, layers=layers)[0]
    C5 = orc.forward(chain, *xc, w5, f=f, heads=heads, layers=layers, relations=5)[0]
    assert np.abs(C3 - C5).max() > 1e-6


def test_directed_relation_transforms_are_applied_per_direction(orc):
    """Uniform attention, W^e = 0, b = 0, W^h_r a distinct permutation per
    relation: one layer gives H' = sum_r gamma_r P_r H Pi_r^T with P_r the
    row-normalised adjacency of relation r (forward: consumer <- producer;
    backward: producer <- consumer); catches swapped directions or
    relations."""
    f = 8
    topo = synth.random_topology(31, 12, 3, 20, dd_density=1.0)
    w = zero_weights(f, 1, f)
    _identity_encoders(w, f)
    w["layer_w"] = np.zeros((1, 5, f, 2 * f), np.float32)
    for k in ("layer_b", "att_src", "att_dst"):
        w[k] = np.zeros((1, 5, f), np.float32)
    perms = [np.roll(np.eye(f), s, axis=0)[:, np.random.default_rng(s).permutation(f)] for s in range(1, 6)]
    for r in range(5):
        w["layer_w"][0, r, :, :f] = perms[r]
    x_op, x_dev, x_oo, x_dd, x_od = random_features(topo, f, 7, nonneg=True)
    E_op, E_dev = orc.forward(topo, x_op, x_dev, x_oo, x_dd, x_od, w, f=f, heads=4, layers=1, relations=5)
    n, m = topo.n_op, topo.n_dev
    Af, Ab = np.zeros((n, n)), np.zeros((n, n))
    for p, c in zip(topo.oo_src, topo.oo_dst):
        Af[c, p] = 1
        Ab[p, c] = 1
    Aod, Ado = np.zeros((n, m)), np.zeros((m, n))
    for u, j in zip(topo.od_op, topo.od_dev):
        Aod[u, j] = 1
        Ado[j, u] = 1
    Add = np.zeros((m, m))
    for a, b in zip(topo.dd_a, topo.dd_b):
        Add[a, b] = Add[b, a] = 1
    Ho, Hd = x_op.astype(np.float64), x_dev.astype(np.float64)
    want_op = (_rownorm(Af) @ Ho @ perms[0].T + _rownorm(Ab) @ Ho @ perms[1].T
               + 0.1 * _rownorm(Aod) @ Hd @ perms[2].T)
    want_dev = 0.1 * _rownorm(Ado) @ Ho @ perms[3].T + _rownorm(Add) @ Hd @ perms[4].T
    np.testing.assert_allclose(E_op, want_op, rtol=0, atol=1e-12)
    np.testing.assert_allclose(E_dev, want_dev, rtol=0, atol=1e-12)


def test_relu_edge_encoder_special_cases(orc):
    """ReLU after the edge encoders: with encoder biases that keep every
    pre-activation positive it is the identity (equals the affine reading);
    with encoder rows A = -1, c = 0 and non-negative raw features every edge
    vector is zero, so each message is ReLU(W^h h_v + b) alone."""
    topo = synth.random_topology(44, 16, 4, 30, od_per_op=2, dd_density=0.8)
    f, heads, layers = 16, 4, 2
    w = synth.make_weights(f, heads, layers, 42, 0, bias_scale=0.3)
    x = random_features(topo, 42, 8, nonneg=True)
    wp = dict(w)
    for r in range(3):
        wp[f"enc_edge_b{r}"] = w[f"enc_edge_b{r}"] + 50.0
    A = orc.forward(topo, *x, wp, f=f, heads=heads, layers=layers)
    B = orc.forward(topo, *x, wp, f=f, heads=heads, layers=layers, edge_act="relu")
    for a, b in zip(A, B):
        np.testing.assert_allclose(a, b, rtol=0, atol=1e-12)
    wn = dict(w)
    for r in range(3):
        wn[f"enc_edge_w{r}"] = -np.ones_like(w[f"enc_edge_w{r}"])
        wn[f"enc_edge_b{r}"] = np.zeros_like(w[f"enc_edge_b{r}"])
    wz = dict(wn)
    wz["layer_w"] = w["layer_w"].copy()
    wz["layer_w"][:, :, :, f:] = 0.0      # no edge term at all
    C = orc.forward(topo, *x, wn, f=f, heads=heads, layers=layers, edge_act="relu")
    D = orc.forward(topo, *x, wz, f=f, heads=heads, layers=layers)
    for a, b in zip(C, D):
        np.testing.assert_allclose(a, b, rtol=0, atol=1e-12)
    E = orc.forward(topo, *x, wn, f=f, heads=heads, layers=layers)   # affine: the negative edge vectors count
    assert np.abs(E[0] - C[0]).max() > 1e-6


def test_averaged_heads_special_cases(orc):
    """K full-width heads averaged: one head is one concatenated head of f
    channels; K identical heads equal one head; with zero attention vectors
    every head is uniform and the layer is the gamma-weighted mean
    aggregation of the messages."""
    topo = synth.random_topology(52, 14, 3, 26, od_per_op=2, dd_density=0.7)
    f, layers = 16, 2
    w1 = synth.make_weights(f, 1, layers, 42, 0, bias_scale=0.3)
    x = random_features(topo, 42, 5)
    A = orc.forward(topo, *x, w1, f=f, heads=1, layers=layers)
    wa = dict(w1)
    wa["att_src"] = w1["att_src"][:, :, None, :].copy()
    wa["att_dst"] = w1["att_dst"][:, :, None, :].copy()
    B = orc.forward(topo, *x, wa, f=f, heads=1, layers=layers, heads_mode="avg")
    for a, b in zip(A, B):
        np.testing.assert_allclose(a, b, rtol=0, atol=1e-14)
    wk = dict(w1)
    wk["att_src"] = np.repeat(w1["att_src"][:, :, None, :], 4, axis=2)
    wk["att_dst"] = np.repeat(w1["att_dst"][:, :, None, :], 4, axis=2)
    C = orc.forward(topo, *x, wk, f=f, heads=4, layers=layers, heads_mode="avg")
    for a, b in zip(A, C):
        np.testing.assert_allclose(a, b, rtol=0, atol=1e-13)
    # uniform attention in every head: mean aggregation of ReLU(W^h h + W^e e + b)
    f8 = 8
    wu = zero_weights(f8, 1, f8)
    _identity_encoders(wu, f8)
    wu["layer_w"][0, :, :, :f8] = np.eye(f8)
    wu["att_src"] = np.zeros((1, 3, 4, f8), np.float32)
    wu["att_dst"] = np.zeros((1, 3, 4, f8), np.float32)
    xu = random_features(topo, f8, 6, nonneg=True)
    E_op, E_dev = orc.forward(topo, *xu, wu, f=f8, heads=4, layers=1, heads_mode="avg")
    Aj = _adjacency(topo)
    Pm = _rownorm(Aj[0]) + 0.1 * _rownorm(Aj[1]) + _rownorm(Aj[2])
    H = Pm @ np.vstack([xu[0], xu[1]]).astype(np.float64)
    np.testing.assert_allclose(np.vstack([E_op, E_dev]), H, rtol=0, atol=1e-12)


def test_relabelling_equivariance(orc):
    topo = synth.random_topology(81, 30, 5, 55, od_per_op=3, dd_density=0.8)
    f, heads, layers = 16, 4, 3
    w = synth.make_weights(f, heads, layers, 42, 0, bias_scale=0.2)
    x_op, x_dev, x_oo, x_dd, x_od = random_features(topo, 42, 4)
    E_op, E_dev = orc.forward(topo, x_op, x_dev, x_oo, x_dd, x_od, w, f=f, heads=heads, layers=layers)
    rng = np.random.default_rng(9)
    po, pd = rng.permutation(topo.n_op), rng.permutation(topo.n_dev)
    t2 = mk_topo(topo.n_op, topo.n_dev,
                 oo=list(zip(po[topo.oo_src], po[topo.oo_dst])),
                 dd=list(zip(pd[topo.dd_a], pd[topo.dd_b])),
                 od=list(zip(po[topo.od_op], pd[topo.od_dev])))
    x_op2 = np.empty_like(x_op); x_op2[po] = x_op
    x_dev2 = np.empty_like(x_dev); x_dev2[pd] = x_dev
    F_op, F_dev = orc.forward(t2, x_op2, x_dev2, x_oo, x_dd, x_od, w, f=f, heads=heads, layers=layers)
    np.testing.assert_allclose(F_op[po], E_op, rtol=0, atol=1e-12)
    np.testing.assert_allclose(F_dev[pd], E_dev, rtol=0, atol=1e-12)


def test_edge_order_invariance_bitwise(orc):
    topo = synth.random_topology(91, 30, 5, 55, od_per_op=3)
    f, heads, layers = 16, 4, 2
    w = synth.make_weights(f, heads, layers, 42, 0)
    x_op, x_dev, x_oo, x_dd, x_od = random_features(topo, 42, 5)
    E_op, E_dev = orc.forward(topo, x_op, x_dev, x_oo, x_dd, x_od, w, f=f, heads=heads, layers=layers)
    rng = np.random.default_rng(1)
    a, b, c = rng.permutation(topo.e_oo), rng.permutation(topo.e_dd), rng.permutation(topo.e_od)
    t2 = mk_topo(topo.n_op, topo.n_dev, oo=list(zip(topo.oo_src[a], topo.oo_dst[a])),
                 dd=list(zip(topo.dd_b[b], topo.dd_a[b])), od=list(zip(topo.od_op[c], topo.od_dev[c])))
    F_op, F_dev = orc.forward(t2, x_op, x_dev, x_oo[a], x_dd[b], x_od[c], w, f=f, heads=heads, layers=layers)
    assert np.array_equal(E_op, F_op) and np.array_equal(E_dev, F_dev)


def test_cross_type_separation_and_sign(orc):
    """gamma_cross = 0 cuts ops off from devices: device features cannot
    reach E_op (bitwise).  All outputs are >= 0 (ReLU messages, alpha >= 0)."""
    topo = synth.random_topology(101, 20, 4, 40)
    f = 16
    w = synth.make_weights(f, 4, 3, 42, 0)
    x_op, x_dev, x_oo, x_dd, x_od = random_features(topo, 42, 6)
    E1, D1 = orc.forward(topo, x_op, x_dev, x_oo, x_dd, x_od, w, f=f, heads=4, layers=3, gamma_cross=0.0)
    E2, D2 = orc.forward(topo, x_op, x_dev * 3 + 1, x_oo, x_dd + 2, 1 - x_od, w, f=f, heads=4, layers=3,
                         gamma_cross=0.0)
    assert np.array_equal(E1, E2)
    assert not np.array_equal(D1, D2)
    E3, D3 = orc.forward(topo, x_op, x_dev, x_oo, x_dd, x_od, w, f=f, heads=4, layers=3)
    assert np.all(E3 >= 0) and np.all(D3 >= 0)
    assert not np.array_equal(E1, E3)


# ------------------------------------------------------------- bf16 --------

def test_round_bf16_matches_torch(orc):
    torch = pytest.importorskip("torch")
    rng = np.random.default_rng(0)
    vals = np.concatenate([
        rng.normal(size=4000).astype(np.float32),
        (rng.normal(size=1000) * 1e-30).astype(np.float32),
        (rng.normal(size=1000) * 1e30).astype(np.float32),
        np.array([1 + 2 ** -8, 1 + 3 * 2 ** -8, -(1 + 2 ** -8), 2 ** -130, 1.0, 0.0, -0.0,
                  1 + 2 ** -8 + 2 ** -20, 255.5, 3 * 2 ** -133], np.float32)])
    want = torch.from_numpy(vals).to(torch.bfloat16).to(torch.float64).numpy()
    got = np.array([orc.round_bf16(float(v)) for v in vals])
    assert np.array_equal(got, want)


def test_bf16_variant_rounds_transforms(orc):
    topo = synth.random_topology(111, 20, 4, 40)
    f = 32
    w = synth.make_weights(f, 4, 2, 42, 0)
    x = random_features(topo, 42, 8)
    A, B = orc.forward(topo, *x, w, f=f, heads=4, layers=2)
    C_, D = orc.forward(topo, *x, w, f=f, heads=4, layers=2, bf16=True)
    rel = np.abs(C_ - A).max() / np.abs(A).max()
    assert 1e-5 < rel < 3e-2
    # when every operand of W^h h is already a bf16 value with a short
    # significand, products and their sums are exact and the variants agree
    w2 = zero_weights(f, 1, 42)
    w2["enc_op_w"][:] = np.eye(f, 42)
    w2["layer_w"][0, :, :, :f] = np.eye(f) * 0.5
    x_op = np.round(np.abs(x[0]) * 8) / 8
    E1, _ = orc.forward(topo, x_op, *x[1:], w2, f=f, heads=4, layers=1)
    E2, _ = orc.forward(topo, x_op, *x[1:], w2, f=f, heads=4, layers=1, bf16=True)
    np.testing.assert_allclose(E1, E2, rtol=0, atol=1e-15)


def test_bf16_rounding_points_hand_worked(orc):
    """The bf16 variant rounds exactly three quantities of the relation
    transform (Section 4.2.1 layer equation, W^h acting on h_v): the input
    row h, the weights W^h and the product W^h h; the edge term W^e e + b,
    the message and the output stay unrounded.  Worked by hand with
    u = 2^-10 (bf16 keeps 8 significant bits, so its spacing on [1, 2) is 8u
    and on [2, 4) is 16u):

      h   = (1 + 5u, 5u)          -> bf16 (1 + 8u, 5u)
      W^h = [[1, 1], [1 + 5u, 1]] -> bf16 [[1, 1], [1 + 8u, 1]]
      Y_0 = (1 + 8u) + 5u = 1 + 13u                 -> bf16 1 + 16u
      Y_1 = (1 + 8u)(1 + 8u) + 5u = 1 + 21u + 64u^2 -> bf16 1 + 24u
      te  = W^e e + b = (1 + u, 1 + u)   (W^e = 0, b = 1 + u: not a bf16 value)

    Op 1 has the single op neighbour 0, so alpha = 1 and its output is the
    message m = ReLU(Y + te) = (2 + 17u, 2 + 25u).  Dropping any one rounding
    or adding one gives a different number:
      no rounding of h: Y = (1 + 8u, 1 + 16u) after rounding the sums;
      no rounding of W: Y_1 = (1 + 5u)(1 + 8u) + 5u -> 1 + 16u;
      no rounding of Y: Y = (1 + 13u, 1 + 21u + 64u^2);
      rounding te or m: 2 + 16u or 2 + 24u in place of 2 + 17u, 2 + 25u."""
    u = 2.0 ** -10
    topo = mk_topo(2, 1, oo=[(0, 1)], od=[])
    w = zero_weights(2, 1, 2)
    w["enc_op_w"][:] = np.eye(2)
    w["layer_w"][0, 0, :, :2] = [[1.0, 1.0], [1.0 + 5 * u, 1.0]]
    w["layer_b"][0, 0, :] = 1.0 + u
    x_op = np.array([[1 + 5 * u, 5 * u], [0.0, 0.0]], np.float32)
    args = (x_op, np.zeros((1, 8), np.float32), np.zeros(1, np.float32), np.zeros((0, 2), np.float32),
            np.zeros(0, np.uint8), w)
    E, _ = orc.forward(topo, *args, f=2, heads=1, layers=1, bf16=True)
    assert E[1].tolist() == [2 + 17 * u, 2 + 25 * u]
    # the fp32 variant takes the unrounded values: Y = (1 + 10u, (1 + 5u)^2 + 5u)
    F, _ = orc.forward(topo, *args, f=2, heads=1, layers=1)
    assert F[1].tolist() == [2 + 11 * u, 2 + 16 * u + 25 * u * u]


# ----------------------------------------------------------- decoder -------

def _full_table(m):
    masks, opts = [], []
    for msk in range(1, 1 << m):
        for o in range(4):
            masks.append(msk); opts.append(o)
    return np.array(masks, np.uint64), np.array(opts, np.uint8)


def _linear_best(t, w_opt, masks, opts):
    pos = [j for j in range(len(t)) if t[j] > 0]
    best_mask = sum(1 << j for j in pos) if pos else 1 << int(np.argmax(t))
    best_opt = int(np.argmax(w_opt))
    idx = [a for a in range(len(masks)) if int(masks[a]) == best_mask and int(opts[a]) == best_opt]
    assert len(idx) == 1
    return idx[0]


@pytest.mark.parametrize("seed,m", [(0, 4), (1, 5), (2, 3)])
def test_linear_decoder_closed_form(orc, seed, m):
    """Linear Dense decoder over the full slice table: the best slice places
    op i on exactly the devices with positive t_j = w_dev . E_dev[j] (or the
    single best one) with the option of largest weight."""
    f, n = 8, 6
    rng = np.random.default_rng(seed)
    E_op, E_dev = rng.normal(size=(n, f)), rng.normal(size=(m, f))
    w = zero_weights(f, 1, 8, 0)
    w["dec_w2"][:] = rng.normal(size=2 * f + 4)
    w["dec_b2"][:] = 0.3
    masks, opts = _full_table(m)
    out = orc.decide(E_op, E_dev, masks, opts, np.arange(n), w, f=f, dec_hidden=0, n_dev=m)
    t = E_dev @ w["dec_w2"][:f].astype(np.float64)
    want = _linear_best(t, w["dec_w2"][2 * f:], masks, opts)
    assert np.all(out["argmax"] == want)
    np.testing.assert_allclose(out["prior"].sum(axis=1), 1.0, atol=1e-12)


def test_mlp_decoder_reduces_to_linear(orc):
    """With every hidden pre-activation positive the ReLU is the identity and
    the MLP decoder is the linear one with weights W1^T w2."""
    f, n, m, H = 8, 5, 4, 16
    rng = np.random.default_rng(4)
    E_op, E_dev = rng.uniform(0, 1, size=(n, f)), rng.uniform(0, 1, size=(m, f))
    w = zero_weights(f, 1, 8, H)
    w["dec_w1"][:] = rng.normal(size=(H, 2 * f + 4)) * 0.1
    w["dec_b1"][:] = 50.0
    w["dec_w2"][:] = rng.normal(size=H)
    masks, opts = _full_table(m)
    out = orc.decide(E_op, E_dev, masks, opts, np.arange(n), w, f=f, dec_hidden=H, n_dev=m)
    weff = w["dec_w1"].astype(np.float64).T @ w["dec_w2"].astype(np.float64)
    want = _linear_best(E_dev @ weff[:f], weff[2 * f:], masks, opts)
    assert np.all(out["argmax"] == want)


def test_decoder_invariances_and_decoding(orc):
    f, n, m, H = 16, 7, 6, 16
    rng = np.random.default_rng(6)
    E_op, E_dev = rng.uniform(0, 1, size=(n, f)), rng.uniform(0, 1, size=(m, f))
    w = synth.make_weights(f, 4, 1, 42, H, bias_scale=0.5)
    masks, opts = synth.make_slices("cnn", m, 64)
    q = np.arange(n)
    a = orc.decide(E_op, E_dev, masks, opts, q, w, f=f, dec_hidden=H, n_dev=m)
    w2 = dict(w); w2["dec_b2"] = w["dec_b2"] + 5.0
    b = orc.decide(E_op, E_dev, masks, opts, q, w2, f=f, dec_hidden=H, n_dev=m)
    assert np.array_equal(a["argmax"], b["argmax"])
    np.testing.assert_allclose(a["prior"], b["prior"], atol=1e-12)
    np.testing.assert_allclose(b["best"] - a["best"], 5.0, atol=1e-12)
    # mask bits at or above the device count are ignored
    hi = masks | np.uint64(1 << 63) | np.uint64(1 << m)
    c = orc.decide(E_op, E_dev, hi, opts, q, w, f=f, dec_hidden=H, n_dev=m)
    assert np.array_equal(a["argmax"], c["argmax"]) and np.array_equal(a["best"], c["best"])
    assert np.array_equal(c["mask"], masks[a["argmax"]])
    # decoded decision
    for qq in range(n):
        o = int(opts[a["argmax"][qq]])
        pc = bin(int(masks[a["argmax"][qq]])).count("1")
        assert a["option"][qq] == o
        assert a["replicas"][qq] == (1 if o == 3 else pc)
        assert a["sync"][qq] == {0: 0, 1: 1, 2: 2, 3: 2}[o]
        assert a["sfb"][qq] == (o == 2)
    assert np.all(a["prior"].argmax(axis=1) == a["argmax"])
