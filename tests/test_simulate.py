"""Parity of the host simulator (tag_simulate, tag_simulate_batch) with the
reference simulator (oracle/simulate.py, itself pinned in
tests/test_sim_oracle.py) on the workload search problems and on random
problems whose slice tables exercise every replication option.  Both sides
run the same event rules in double precision with the same operation
order, so the discrete results (validity, OOM, task count) must agree
exactly and the times, memories and idle shares to 1e-12 relative.  CPU
only: the simulator is host code."""
import numpy as np
import pytest

import synth
from oracle import search as OSR
from oracle import simulate as SIM

REL = 1e-12


@pytest.fixture(scope="module")
def PS():
    import paper_2302_06126_amd.search as ps
    return ps


def _compare(got, ref):
    assert got["valid"] == ref["valid"]
    if not ref["valid"]:
        assert got["oom"] and np.isinf(got["T"])
        return
    assert got["oom"] == ref["oom"]
    assert got["n_tasks"] == ref["n_tasks"]
    assert got["T"] == pytest.approx(ref["T"], rel=REL)
    for k in ("group_makespan", "group_idle", "dev_peak", "dev_idle", "link_idle"):
        r = np.asarray(ref[k], float)
        scale = max(np.abs(r).max(initial=0.0), 1e-300)
        assert np.abs(np.asarray(got[k]) - r).max(initial=0.0) <= REL * scale, k


def _random_problem(seed, n=80, m=6, e=160, K=7, S=40):
    topo = synth.random_topology(seed, n, m, e)
    rng = synth.rng_for(94, seed)
    groups = np.sort(rng.integers(0, K, size=n)).astype(np.int32)
    groups[:K] = np.arange(K)
    groups = np.sort(groups)
    masks = np.array([int(rng.integers(1, 1 << m)) for _ in range(S - 1)] + [1 << 63], np.uint64)
    opts = rng.integers(0, 4, size=S).astype(np.uint8)
    params = np.where(rng.random(n) < 0.3, 0.0, rng.lognormal(16, 1.5, size=n))
    return synth.SearchProblem(name="rand", topo=topo, group_of=groups, n_groups=K, op_params=params,
                               masks=masks, options=opts)


def _paths(sp, order, count, seed):
    rng = synth.rng_for(95, seed)
    out = [[]]
    for _ in range(count):
        d = int(rng.integers(1, sp.n_groups + 1))
        out.append([int(x) for x in rng.integers(0, len(sp.masks) - 1, size=d)])
    return out


@pytest.mark.parametrize("name,count", [("tiny", 25), ("cnn", 4)])
def test_simulator_matches_reference_on_workloads(PS, name, count):
    sp = synth.make_search_problem(name)
    order = OSR.Problem(sp).order
    P = SIM.SimProblem(sp)
    prob = PS.SearchProblem(sp)
    for path in _paths(sp, order, count, len(name)):
        ref = SIM.simulate(P, SIM.strategy_of(sp, path, order))
        _compare(prob.simulate(path), ref)
    prob.close()


@pytest.mark.parametrize("seed", [1, 2, 3, 4])
def test_simulator_matches_reference_every_option(PS, seed):
    sp = _random_problem(seed)
    order = OSR.Problem(sp).order
    P = SIM.SimProblem(sp)
    prob = PS.SearchProblem(sp, f_op=40)
    seen = set()
    for path in _paths(sp, order, 30, seed):
        strat = SIM.strategy_of(sp, path, order)
        seen.update(o for _, o in strat)
        _compare(prob.simulate(path), SIM.simulate(P, strat))
    assert seen == {0, 1, 2, 3}
    # the last slice names no device of the topology: invalid
    bad = [len(sp.masks) - 1]
    assert SIM.simulate(P, SIM.strategy_of(sp, bad, order))["valid"] is False
    _compare(prob.simulate(bad), dict(valid=False))
    prob.close()


def test_batch_matches_single_and_threads(PS):
    sp = _random_problem(7)
    prob = PS.SearchProblem(sp, f_op=40)
    paths = _paths(sp, OSR.Problem(sp).order, 40, 7)
    B, K = len(paths), sp.n_groups
    depth = np.array([len(p) for p in paths], np.int32)
    pm = np.zeros((B, K), np.int32)
    for b, p in enumerate(paths):
        pm[b, :len(p)] = p
    T1, o1 = prob.simulate_batch(depth, pm, n_threads=1)
    T4, o4 = prob.simulate_batch(depth, pm, n_threads=4)
    assert np.array_equal(T1, T4) and np.array_equal(o1, o4)
    for b, p in enumerate(paths):
        r = prob.simulate(p)
        assert T1[b] == r["T"] and bool(o1[b]) == r["oom"]
    prob.close()


def test_simulator_argument_checks(PS):
    from paper_2302_06126_amd import _abi
    sp = _random_problem(8)
    prob = PS.SearchProblem(sp, f_op=40)
    with pytest.raises(_abi.TagError) as e:
        prob.simulate([0] * (sp.n_groups + 1))
    assert e.value.status == _abi.TAG_EINVAL
    with pytest.raises(_abi.TagError) as e:
        prob.simulate([len(sp.masks)])
    assert e.value.status == _abi.TAG_ERANGE
    prob.close()
    # a cycle in the tensor graph
    t = synth.random_topology(9, 4, 2, 0)
    t.oo_src = np.array([0, 1, 2], np.int32)
    t.oo_dst = np.array([1, 2, 0], np.int32)
    cyc = synth.SearchProblem(name="cyc", topo=t, group_of=np.array([0, 0, 1, 1], np.int32), n_groups=2,
                              op_params=np.ones(4), masks=np.array([1, 2], np.uint64), options=np.zeros(2, np.uint8))
    prob = PS.SearchProblem(cyc, f_op=40)
    with pytest.raises(_abi.TagError) as e:
        prob.simulate([0, 1])
    assert e.value.status == _abi.TAG_EINVAL
    with pytest.raises(ValueError):
        SIM.simulate(SIM.SimProblem(cyc), SIM.strategy_of(cyc, [0, 1], OSR.Problem(cyc).order))
    prob.close()
