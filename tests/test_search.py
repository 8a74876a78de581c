"""Strategy search (Section 4.2.2): pins of the reference search against hand
computations and closed forms, and parity of the library's host search
(tree, reward model, state packing) with the reference.  CPU only."""
import math

import numpy as np
import pytest

import synth
from oracle import search as OS


# ---------------------------------------------------------------- helpers --

def _tiny_problem(M=2, K=3, S=None, params=1e6, flops=1e9, mem_gb=16.0, seed=0):
    """A hand-sized problem: K groups of 2 chained ops, M devices."""
    n = 2 * K
    t = synth.Topology(
        n_op=n, n_dev=M,
        oo_src=np.arange(n - 1, dtype=np.int32), oo_dst=np.arange(1, n, dtype=np.int32),
        dd_a=np.array([a for a in range(M) for b in range(a + 1, M)], np.int32),
        dd_b=np.array([b for a in range(M) for b in range(a + 1, M)], np.int32),
        od_op=np.repeat(np.arange(n, dtype=np.int32), M), od_dev=np.tile(np.arange(M, dtype=np.int32), n),
        op_type=np.arange(n) % 32, op_flops=np.full(n, flops) * (1.0 + np.arange(n)),
        op_bytes=np.full(n, 1e6), dev_tflops=np.full(M, 10.0), dev_mem=np.full(M, mem_gb),
        dev_intra_bw=np.full(M, 100.0), dd_bw=np.full(M * (M - 1) // 2, 10.0))
    masks, opts = [], []
    for m in range(1, 1 << M):
        for o in range(4):
            masks.append(m); opts.append(o)
    sp = synth.SearchProblem(name="hand", topo=t, group_of=(np.arange(n) // 2).astype(np.int32), n_groups=K,
                             op_params=np.full(n, params), masks=np.array(masks, np.uint64),
                             options=np.array(opts, np.uint8))
    return sp


def _priors(S, key):
    r = synth.rng_for(55, *key)
    p = r.random(S).astype(np.float32) + np.float32(0.01)
    return (p / p.sum()).astype(np.float32)


# ------------------------------------------------------ reference pins ----

def test_order_is_descending_flops():
    P = OS.Problem(_tiny_problem(K=3))
    # group g holds ops 2g, 2g+1 with FLOPs (2g+1, 2g+2) * 1e9 -> totals increase with g
    assert P.order == [2, 1, 0]


def test_cost_model_single_device_closed_form():
    sp = _tiny_problem(M=1, K=2)
    P = OS.Problem(sp)
    ev = OS.evaluate(P, OS.full_strategy(P, []))
    # one device: no communication, no transfers, compute = total FLOPs / speed
    assert ev["T"] == pytest.approx(sp.topo.op_flops.sum() / 10e12, rel=1e-15)
    assert OS.reward(P, []) == 1.0


def test_cost_model_allreduce_closed_form():
    sp = _tiny_problem(M=2, K=1, params=3e6, flops=2e9)
    P = OS.Problem(sp)
    ev = OS.evaluate(P, OS.full_strategy(P, []))
    FL, PB = sp.topo.op_flops.sum(), sp.op_params.sum()
    comp = FL / (2 * 10e12)
    sync = 2.0 * (2 - 1) / 2 * PB / 10e9
    assert ev["T"] == pytest.approx(comp + sync, rel=1e-15)
    # the same group on one device: compute only, speed-up = (comp + sync) / (FL / speed)
    one = [a for a in range(P.S) if P.masks[a] == 1 and P.options[a] == OS.AR][0]
    assert OS.reward(P, [one]) == pytest.approx((comp + sync) / (FL / 10e12), rel=1e-15)


def test_cost_model_transfer_and_duplicate():
    sp = _tiny_problem(M=2, K=2, params=0.0)
    P = OS.Problem(sp)
    # order: group 1 first; put group 1 on device 0 and group 0 on device 1 (AllReduce, r = 1)
    a0 = [a for a in range(P.S) if P.masks[a] == 1 and P.options[a] == OS.AR][0]
    a1 = [a for a in range(P.S) if P.masks[a] == 2 and P.options[a] == OS.AR][0]
    ev = OS.evaluate(P, OS.full_strategy(P, [a0, a1]))
    f = sp.topo.op_flops
    # the single cross-group tensor (op 1 -> op 2) crosses the 10 GB/s link
    assert ev["T"] == pytest.approx(max((f[0] + f[1]), (f[2] + f[3])) / 10e12 + 1e6 / 10e9, rel=1e-15)
    # duplicate on both devices: full compute on each, inputs broadcast
    dup = [a for a in range(P.S) if P.masks[a] == 3 and P.options[a] == OS.DUP][0]
    ev = OS.evaluate(P, OS.full_strategy(P, [dup, dup]))
    ab = 2e6
    per = (f[0] + f[1]) / 10e12 + 0.5 * ab / 10e9 + (f[2] + f[3]) / 10e12 + 0.5 * ab / 10e9
    assert ev["T"] == pytest.approx(per, rel=1e-15)


def test_oom_and_undeployable_masks_give_minus_one():
    sp = _tiny_problem(M=2, K=2, params=5e9, mem_gb=16.0)
    P = OS.Problem(sp)
    assert OS.reward(P, []) == -1.0
    sp2 = _tiny_problem(M=2, K=2)
    sp2.masks = sp2.masks.copy()
    sp2.masks[0] = np.uint64(1 << 5)          # names no device of a 2-device topology
    P2 = OS.Problem(sp2)
    assert OS.reward(P2, [0]) == -1.0


def test_puct_hand_worked_sequence():
    """Two actions, priors (0.75, 0.25), c = 1, reward 1 for action 0 and 0.5
    for action 1.  U = Q + c G sqrt(sum N) / (1 + N), Q = 0 unvisited."""
    T = OS.Tree(n_levels=2, n_actions=2, c_puct=1.0)
    leaves = T.select(1)
    assert leaves == [(0, [])]                 # the unexpanded root
    T.update(leaves, [[0.75, 0.25]], [0.0])
    picks = []
    for _ in range(4):
        (vid, path), = T.select(1)
        picks.append(path[0])
        T.update([(vid, path)], [[0.5, 0.5]], [1.0 if path[0] == 0 else 0.5])
    # round 1: sum N = 0 -> U = (0, 0) -> first maximum: action 0
    # round 2: N = (1, 0), Q = (1, 0): U0 = 1 + .75*1/2 = 1.375, U1 = .25 -> 0
    # round 3: N = (2, 0): U0 = 1 + .75*sqrt2/3 = 1.354, U1 = .25*sqrt2 = .354 -> 0
    # round 4: N = (3, 0): U0 = 1 + .75*sqrt3/4 = 1.325, U1 = .25*sqrt3 = .433 -> 0
    assert picks == [0, 0, 0, 0]
    T2 = OS.Tree(n_levels=1, n_actions=2, c_puct=10.0)
    T2.update(T2.select(1), [[0.75, 0.25]], [0.0])
    picks = []
    for _ in range(3):
        (vid, path), = T2.select(1)
        picks.append(path[0])
        T2.update([(vid, path)], [[0, 0]], [1.0 if path[0] == 0 else 0.5])
    # c = 10: round 2: U0 = 1 + 7.5/2 = 4.75, U1 = 2.5 -> 0; round 3: U0 = 1 + 7.5 sqrt2/3 = 4.54,
    # U1 = 2.5 sqrt2 = 3.54 -> 0 ... the first pick is 0 (tie at 0), then 0, then 0
    assert picks == [0, 0, 0]
    n, q = T2.root_stats()
    assert n == [3, 0] and q == [1.0, 0.0]


def test_running_mean_and_virtual_loss():
    T = OS.Tree(n_levels=1, n_actions=1, c_puct=1.0, vl_value=-5.0)
    T.update(T.select(1), [[1.0]], [0.0])
    rs = [0.3, 1.7, -1.0, 2.25]
    sel = T.select(4)                           # one action: all four in flight together
    assert all(p == [0] for _, p in sel)
    assert T.verts[0]["VL"] == [4]
    T.update(sel, [[1.0]] * 4, rs)
    n, q = T.root_stats()
    assert n == [4] and q[0] == pytest.approx(sum(rs) / 4, abs=1e-15)
    assert T.verts[0]["VL"] == [0]


def test_virtual_loss_spreads_a_batch():
    T = OS.Tree(n_levels=1, n_actions=3, c_puct=0.5, vl_value=-1.0)
    T.update(T.select(1), [[0.4, 0.35, 0.25]], [0.0])
    sel = T.select(3)
    assert sorted(p[0] for _, p in sel) == [0, 1, 2]


def test_features_encode_the_partial_strategy():
    sp = synth.make_search_problem("tiny")
    P = OS.Problem(sp)
    path = [5, 17, 42]
    x, xd, xod, rep = OS.features(P, path, f_op=40)
    dec = set(P.order[:3])
    g = P.group_of
    assert np.array_equal(x[:, 38] == 1, np.isin(g, list(dec)))
    assert np.array_equal(x[:, 39] == 1, g == P.order[3])
    assert np.all(x[:, 34:38].sum(1) == x[:, 38])
    strat = OS.full_strategy(P, path)
    t = sp.topo
    for e in range(t.e_od):
        gg = int(g[t.od_op[e]])
        assert xod[e] == (gg in dec and (strat[gg][0] >> int(t.od_dev[e])) & 1)
    assert g[rep] == P.order[3]
    assert t.op_flops[rep] == t.op_flops[g == P.order[3]].max()


# ------------------------------------------- library vs reference (CPU) --

@pytest.fixture(scope="module")
def L():
    import paper_2302_06126_amd.search as PS
    PS._abi.load()
    return PS


@pytest.mark.parametrize("name", ["tiny", "cnn", "transformer"])
def test_library_order_and_rewards_match_reference(L, name):
    sp = synth.make_search_problem(name)
    P = OS.Problem(sp)
    prob = L.SearchProblem(sp, f_op=40 if name == "tiny" else 42)
    order, rep = prob.order()
    assert list(order) == P.order
    rng = synth.rng_for(56, len(name))
    T_base = OS.evaluate(P, OS.full_strategy(P, []))["T"]
    for d in [0, 1, 2, 5, P.K]:
        for _ in range(4):
            path = rng.integers(0, P.S, size=d).tolist()
            r, T, oom = prob.evaluate(path)
            ev = OS.evaluate(P, OS.full_strategy(P, path))
            assert T == pytest.approx(ev["T"], rel=1e-12)
            assert oom == ev["oom"]
            assert r == pytest.approx(OS.reward(P, path, T_base), rel=1e-12)
    prob.close()


@pytest.mark.parametrize("B,c,vl", [(1, 1.5, 0.0), (4, 1.5, 0.0), (16, 0.7, -1.0)])
def test_library_tree_matches_reference(L, B, c, vl):
    """Same priors and rewards into both trees: every selected path, and the
    final root statistics, are identical."""
    sp = synth.make_search_problem("tiny")
    P = OS.Problem(sp)
    ref = OS.Tree(P.K, P.S, c, vl)
    lib = L.Mcts(P.K, P.S, c, vl)
    T_base = OS.evaluate(P, OS.full_strategy(P, []))["T"]
    for rnd in range(12):
        leaves = ref.select(B)
        leaf, depth, path = lib.select(B)
        assert [len(p) for _, p in leaves] == list(depth)
        for b, (_, p) in enumerate(leaves):
            assert list(path[b, :depth[b]]) == p, (rnd, b)
        pri = np.stack([_priors(P.S, (rnd, b)) for b in range(B)])
        rw = [OS.reward(P, p, T_base) for _, p in leaves]
        ref.update(leaves, pri, rw)
        lib.update(leaf, depth, path, pri, rw)
    n, q = lib.root_stats()
    rn, rq = ref.root_stats()
    assert list(n) == rn
    assert list(q) == rq                       # bit-exact: same doubles in the same order
    assert list(lib.best_path()) == ref.best_path()
    v, e = lib.size()
    assert v == len(ref.verts) and e == sum(1 for x in ref.verts if x["expanded"])
    lib.close()


def test_library_pack_rewards_and_queries(L):
    sp = synth.make_search_problem("cnn")
    P = OS.Problem(sp)
    prob = L.SearchProblem(sp)
    _, rep = prob.order()
    rng = synth.rng_for(57)
    B = 5
    depth = np.array([0, 1, 7, P.K - 1, P.K], np.int32)
    path = rng.integers(0, P.S, size=(B, P.K)).astype(np.int32)
    _, rb = prob.device_bytes()
    buf = np.zeros(B * rb, np.uint8)
    rewards, qop = prob.pack(depth, path, buf.ctypes.data)
    T_base = OS.evaluate(P, OS.full_strategy(P, []))["T"]
    for b in range(B):
        p = path[b, :depth[b]].tolist()
        assert rewards[b] == pytest.approx(OS.reward(P, p, T_base), rel=1e-12)
        _, _, _, r = OS.features(P, p)
        assert qop[b] == (r if r >= 0 else 0)
    prob.close()


def test_library_rejects_bad_search_arguments(L):
    sp = synth.make_search_problem("tiny")
    prob = L.SearchProblem(sp, f_op=40)
    with pytest.raises(L._abi.TagError):
        prob.evaluate([10 ** 6])
    with pytest.raises(L._abi.TagError):
        L.SearchProblem(sp, f_op=41)
    t = L.Mcts(3, 4)
    leaf, depth, path = t.select(1)
    t.update(leaf, depth, path, np.full((1, 4), 0.25, np.float32), [1.0])
    leaf, depth, path = t.select(1)
    bad = path.copy()
    bad[0, 0] = (bad[0, 0] + 1) % 4            # a path the tree never handed out
    with pytest.raises(L._abi.TagError):
        t.update(leaf, depth, bad, np.full((1, 4), 0.25, np.float32), [1.0])
    with pytest.raises(L._abi.TagError):
        t.update(leaf, depth, path, np.full((1, 4), -1.0, np.float32), [1.0])
    t.update(leaf, depth, path, np.full((1, 4), 0.25, np.float32), [1.0])
    with pytest.raises(L._abi.TagError):      # no in-flight visit left on the path
        t.update(leaf, depth, path, np.full((1, 4), 0.25, np.float32), [1.0])
    t.close()
    prob.close()


def _records(prob, buf, B, K, M, E_dd=0):
    """Decode packed state records: (gfeat [B][K][2], dfeat [B][M][2], lfeat [B][E_dd])."""
    _, rb = prob.device_bytes()
    g0 = 8 + 8 * K + 4 * K + 4 * K
    l0 = g0 + 8 * K + 8 * M
    out_g, out_d, out_l = [], [], []
    for b in range(B):
        rec = buf[b * rb:(b + 1) * rb]
        out_g.append(np.frombuffer(rec[g0:g0 + 8 * K].tobytes(), np.float32).reshape(K, 2))
        out_d.append(np.frombuffer(rec[g0 + 8 * K:l0].tobytes(), np.float32).reshape(M, 2))
        out_l.append(np.frombuffer(rec[l0:l0 + 4 * E_dd].tobytes(), np.float32))
    return out_g, out_d, out_l


@pytest.mark.parametrize("name", ["tiny", "cnn"])
def test_library_simulator_model_matches_reference(L, name):
    """With the simulator as the reward and feedback model: rewards, times,
    OOM flags and the runtime feedback in the packed records equal the
    reference search's (built on the reference simulator)."""
    sp = synth.make_search_problem(name)
    P = OS.Problem(sp, model="simulator")
    prob = L.SearchProblem(sp, f_op=40 if name == "tiny" else 42, model="simulator")
    T_base = OS.feedback(P, OS.full_strategy(P, []))["T"]
    rng = synth.rng_for(59, len(name))
    B = 6
    depth = np.array([0, 1, 2, P.K // 2, P.K - 1, P.K], np.int32)
    path = rng.integers(0, P.S, size=(B, P.K)).astype(np.int32)
    for b in range(B):
        p = path[b, :depth[b]].tolist()
        r, T, oom = prob.evaluate(p)
        fb = OS.feedback(P, OS.full_strategy(P, p))
        assert T == pytest.approx(fb["T"], rel=1e-12) and oom == fb["oom"]
        assert r == pytest.approx(OS.reward(P, p, T_base), rel=1e-12)
    _, rb = prob.device_bytes()
    buf = np.zeros(B * rb, np.uint8)
    rewards, _ = prob.pack(depth, path, buf.ctypes.data)
    gf, df, lf = _records(prob, buf, B, P.K, P.M, sp.topo.e_dd)
    for b in range(B):
        p = path[b, :depth[b]].tolist()
        assert rewards[b] == pytest.approx(OS.reward(P, p, T_base), rel=1e-12)
        fb = OS.feedback(P, OS.full_strategy(P, p))
        for i in range(depth[b]):
            g = P.order[i]
            assert gf[b][g, 0] == np.float32(math.log10(max(fb["makespan"][g], 1e-12) * 1e3))
            assert gf[b][g, 1] == np.float32(fb["gidle"][g])
        assert np.array_equal(df[b][:, 0], np.array(fb["memf"], np.float32))
        assert np.array_equal(df[b][:, 1], np.array(fb["didle"], np.float32))
        assert np.array_equal(lf[b], np.array(fb["lidle"], np.float32))
        assert np.array_equal(OS.link_features(P, p)[:, 1], lf[b])
    # the two models agree on the baseline's iteration time only by construction of the workloads,
    # not in general; both give a positive, finite time
    assert 0 < T_base < math.inf
    prob.close()
