"""GPU parity of the batched search service (Section 4.2.2): the feature
kernel against the reference encoding of search states, and whole search
rounds (select -> reward + features -> forward -> decide -> update) against
the reference tree fed with the same priors, whose priors in turn match the
reference GNN."""
import numpy as np
import pytest

import oracle
import synth
from oracle import search as OS

pytestmark = pytest.mark.gpu


def _say(msg):
    print(msg, flush=True)


@pytest.fixture(scope="module")
def torch():
    import torch
    assert torch.cuda.is_available()
    return torch


@pytest.mark.parametrize("name,f_op,model", [("tiny", 40, "analytic"), ("cnn", 42, "analytic"),
                                             ("large", 42, "analytic"), ("cnn", 42, "simulator")])
def test_features_kernel_matches_reference(torch, name, f_op, model):
    import paper_2302_06126_amd.search as PS
    _say(f"[search] features {name} {model}")
    sp = synth.make_search_problem(name)
    P = OS.Problem(sp, model=model)
    prob = PS.SearchProblem(sp, f_op=f_op, model=model)
    rng = synth.rng_for(58, len(name))
    depth = np.array([0, 1, 3, P.K // 2, P.K - 1, P.K], np.int32)
    B = len(depth)
    path = rng.integers(0, P.S, size=(B, P.K)).astype(np.int32)
    sb, rb = prob.device_bytes()
    dev = torch.device("cuda")
    static = torch.empty(sb, dtype=torch.uint8, device=dev)
    PS.check(PS._abi.load().tag_search_upload(prob.h, static.data_ptr(), sb, 0), "upload")
    host = np.zeros(B * rb, np.uint8)
    prob.pack(depth, path, host.ctypes.data)
    states = torch.from_numpy(host).to(dev)
    t = sp.topo
    x_op = torch.full((B, t.n_op, f_op), np.nan, dtype=torch.float32, device=dev)
    x_dev = torch.full((B, t.n_dev, 8), np.nan, dtype=torch.float32, device=dev)
    x_od = torch.full((B, t.e_od), 7, dtype=torch.uint8, device=dev)
    PS.check(PS._abi.load().tag_search_features(prob.h, B, static.data_ptr(), states.data_ptr(), x_op.data_ptr(),
                                                x_dev.data_ptr(), x_od.data_ptr(), 0), "features")
    torch.cuda.synchronize()
    x_dd = torch.full((B, max(t.e_dd, 1), 2), np.nan, dtype=torch.float32, device=dev)
    PS.check(PS._abi.load().tag_search_link_features(prob.h, B, static.data_ptr(), states.data_ptr(),
                                                     x_dd.data_ptr(), 0), "link features")
    torch.cuda.synchronize()
    g_op, g_dev, g_od, g_dd = x_op.cpu().numpy(), x_dev.cpu().numpy(), x_od.cpu().numpy(), x_dd.cpu().numpy()
    for b in range(B):
        assert np.array_equal(g_dd[b][:t.e_dd], OS.link_features(P, path[b, :depth[b]].tolist())), b
        x, xd, xod, _ = OS.features(P, path[b, :depth[b]].tolist(), f_op=f_op)
        exact = list(range(32)) + list(range(34, 40))          # one-hots and flags
        assert np.array_equal(g_op[b][:, exact], x[:, exact]), b
        np.testing.assert_allclose(g_op[b], x, rtol=2e-6, atol=1e-6)
        np.testing.assert_allclose(g_dev[b], xd, rtol=2e-6, atol=1e-6)
        assert np.array_equal(g_od[b], xod), b
    prob.close()


@pytest.mark.parametrize("name,B,rounds,model", [("tiny", 8, 6, "analytic"), ("cnn", 16, 4, "analytic"),
                                                  ("cnn", 16, 3, "simulator")])
def test_search_rounds_match_reference_tree(torch, name, B, rounds, model):
    """The service's rounds, replayed through the reference tree with the
    priors the GPU produced and the reference rewards, select the same
    leaves and end with the same statistics; round 0's priors (the root
    expansion) match the reference GNN's."""
    import paper_2302_06126_amd as P0
    import paper_2302_06126_amd.search as PS
    _say(f"[search] rounds {name} B={B} {model}")
    wl = synth.WORKLOADS[name]
    sp = synth.make_search_problem(name)
    P = OS.Problem(sp, model=model)
    w = synth.make_weights(wl.f, wl.heads, wl.layers, wl.f_op, wl.f)
    gnn = P0.Model(w, f=wl.f, heads=wl.heads, layers=wl.layers, f_op=wl.f_op, dtype=wl.dtype)
    prob = PS.SearchProblem(sp, f_op=wl.f_op, model=model)
    svc = PS.SearchService(prob, sp, gnn, B)
    lib = PS.Mcts(P.K, P.S, 1.5, 0.0)
    ref = OS.Tree(P.K, P.S, 1.5, 0.0)
    T_base = OS.feedback(P, OS.full_strategy(P, []))["T"]
    first = None
    for rnd in range(rounds):
        leaf, depth, path = lib.select(B)
        leaves = ref.select(B)
        for b, (_, p) in enumerate(leaves):
            assert list(path[b, :depth[b]]) == p, (rnd, b)
        rewards, priors = svc.evaluate(depth, path)
        priors = priors.copy()
        for b, (_, p) in enumerate(leaves):
            assert rewards[b] == pytest.approx(OS.reward(P, p, T_base), rel=1e-12)
        if first is None:
            first = (path[0, :depth[0]].tolist(), priors[0].copy())
        lib.update(leaf, depth, path, priors, rewards)
        ref.update(leaves, priors, rewards)
    n, q = lib.root_stats()
    rn, rq = ref.root_stats()
    assert list(n) == rn and list(q) == rq
    # round 0, leaf 0 is the root: its priors against the reference GNN on the reference features
    p0, pr0 = first
    x, xd, xod, rep = OS.features(P, p0, f_op=wl.f_op)
    t = sp.topo
    x_oo = (np.log10(t.op_bytes[t.oo_src]) - 6.0).astype(np.float32)
    x_dd = OS.link_features(P, p0)   # under the analytic model the idle column is 0
    if model == "analytic":
        assert np.array_equal(x_dd, np.stack([np.log10(t.dd_bw) - 1.0, np.zeros(t.e_dd)], axis=1).astype(np.float32))
    E_op, E_dev = oracle.forward(t, x, xd, x_oo, x_dd, xod, w, f=wl.f, heads=wl.heads, layers=wl.layers)
    od = oracle.decide(E_op, E_dev, sp.masks, sp.options, np.array([rep], np.int32), w, f=wl.f,
                       dec_hidden=wl.f, n_dev=t.n_dev, want_prior=True)
    np.testing.assert_allclose(pr0, od["prior"][0], rtol=1e-3, atol=1e-6)
    svc.close()
    lib.close()
    prob.close()


@pytest.mark.parametrize("name,B,rounds,pipelined,model", [("tiny", 8, 6, True, "analytic"),
                                                            ("cnn", 16, 5, True, "analytic"),
                                                            ("cnn", 16, 4, False, "analytic"),
                                                            ("tiny", 8, 6, True, "simulator")])
def test_native_rounds_match_reference_schedule(torch, name, B, rounds, pipelined, model):
    """tag_search_run: the recorded leaves, replayed through the reference
    tree in the same select / update schedule (pipelined: round k+1 is
    selected before round k's update) with the recorded priors and the
    reference rewards, give the same paths and the same root statistics."""
    import paper_2302_06126_amd as P0
    import paper_2302_06126_amd.search as PS
    _say(f"[search] native rounds {name} B={B} pipelined={pipelined} {model}")
    wl = synth.WORKLOADS[name]
    sp = synth.make_search_problem(name)
    P = OS.Problem(sp, model=model)
    w = synth.make_weights(wl.f, wl.heads, wl.layers, wl.f_op, wl.f)
    gnn = P0.Model(w, f=wl.f, heads=wl.heads, layers=wl.layers, f_op=wl.f_op, dtype=wl.dtype)
    prob = PS.SearchProblem(sp, f_op=wl.f_op, model=model)
    svc = PS.SearchService(prob, sp, gnn, B)
    lib = PS.Mcts(P.K, P.S, 1.5, 0.0)
    rec = svc.run(lib, rounds, pipelined=pipelined, record=True)
    ref = OS.Tree(P.K, P.S, 1.5, 0.0)
    T_base = OS.feedback(P, OS.full_strategy(P, []))["T"]
    sel = {0: ref.select(B)}
    for k in range(rounds):
        if pipelined and k + 1 < rounds:
            sel[k + 1] = ref.select(B)
        for b, (_, p) in enumerate(sel[k]):
            assert rec["depth"][k, b] == len(p) and list(rec["path"][k, b, :len(p)]) == p, (k, b)
            assert rec["reward"][k, b] == pytest.approx(OS.reward(P, p, T_base), rel=1e-12)
        ref.update(sel[k], rec["prior"][k], rec["reward"][k])
        if not pipelined and k + 1 < rounds:
            sel[k + 1] = ref.select(B)
    n, q = lib.root_stats()
    rn, rq = ref.root_stats()
    assert list(n) == rn and list(q) == rq
    # the step-wise binding, strictly per round, builds the same tree as the native rounds
    if not pipelined:
        lib2 = PS.Mcts(P.K, P.S, 1.5, 0.0)
        for _ in range(rounds):
            svc.round(lib2)
        n2, q2 = lib2.root_stats()
        assert list(n2) == list(n) and list(q2) == list(q)
        lib2.close()
    svc.close()
    lib.close()
    prob.close()
