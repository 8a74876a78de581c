"""Pins of the reference simulator (oracle/simulate.py): micro problems with
closed-form iteration times, idle times and peak memories (a chain on one
device, a transfer, link contention in FIFO order, AllReduce and parameter
server sync, model-parallel gather, duplicate), the invalid strategy, and on
random problems the serial identity on one device and the critical-path /
serial bounds computed independently of the task graph.  CPU only."""
import math

import numpy as np
import pytest

import synth
from oracle import simulate as SIM

AR, PS, DUP, MP = 0, 1, 2, 3


def _micro(flops, out, params, groups, edges, tflops, mem_gb, links):
    """A search problem from explicit numbers; links: {(a, b): GB/s} for every pair."""
    n, m = len(flops), len(tflops)
    a = np.array([p[0] for p in links], np.int32)
    b = np.array([p[1] for p in links], np.int32)
    topo = synth.Topology(
        n_op=n, n_dev=m, oo_src=np.array([e[0] for e in edges], np.int32),
        oo_dst=np.array([e[1] for e in edges], np.int32), dd_a=a, dd_b=b,
        od_op=np.zeros(0, np.int32), od_dev=np.zeros(0, np.int32), op_type=np.zeros(n, np.int64),
        op_flops=np.array(flops, float), op_bytes=np.array(out, float), dev_tflops=np.array(tflops, float),
        dev_mem=np.array(mem_gb, float), dev_intra_bw=np.full(m, 100.0), dd_bw=np.array(list(links.values()), float))
    sp = synth.SearchProblem(name="micro", topo=topo, group_of=np.array(groups, np.int32), n_groups=max(groups) + 1,
                             op_params=np.array(params, float), masks=np.zeros(1, np.uint64),
                             options=np.zeros(1, np.uint8))
    return SIM.SimProblem(sp)


def test_chain_on_one_device():
    P = _micro([2e12, 4e12, 1e12], [3e9, 5e9, 2e9], [1e8, 0.0, 2e8], [0, 0, 0], [(0, 1), (1, 2)],
               [10.0], [80.0], {})
    r = SIM.simulate(P, [(1, AR)])
    assert r["T"] == pytest.approx(0.2 + 0.4 + 0.1, rel=1e-15)
    assert r["group_makespan"] == [pytest.approx(0.7, rel=1e-15)]
    res = 4.0 * 3e8
    assert r["dev_peak"][0] == pytest.approx(res + max(3e9 + 5e9, 5e9 + 2e9), rel=1e-15)
    assert r["dev_idle"][0] == pytest.approx(0.0, abs=1e-15)
    assert not r["oom"]
    r = SIM.simulate(P, [(1, AR)])
    P.mem[0] = res + 7.9e9
    assert SIM.simulate(P, [(1, AR)])["oom"]


def test_transfer_between_devices():
    # op 0 on device 0 (group 0), op 1 on device 1 (group 1), tensor 0 -> 1 over a 20 GB/s link
    P = _micro([1e12, 2e12], [4e9, 1e9], [0.0, 0.0], [0, 1], [(0, 1)], [10.0, 20.0], [80.0, 80.0],
               {(0, 1): 20.0})
    r = SIM.simulate(P, [(0b01, AR), (0b10, AR)])
    t0, x, t1 = 0.1, 4e9 / 20e9, 0.1
    T = t0 + x + t1
    assert r["T"] == pytest.approx(T, rel=1e-15)
    assert r["group_makespan"] == [pytest.approx(t0), pytest.approx(t1)]
    assert r["group_idle"] == [0.0, 0.0]
    assert r["dev_idle"][0] == pytest.approx(1 - t0 / T, rel=1e-14)
    assert r["link_idle"][0] == pytest.approx(1 - x / T, rel=1e-14)
    assert r["dev_peak"][0] == pytest.approx(4e9)            # freed when the transfer ends
    assert r["dev_peak"][1] == pytest.approx(4e9 + 1e9)      # received copy + the sink's output


def test_link_contention_is_fifo():
    # ops 0, 1 on device 0 (group 0) feed op 2 on device 1 (group 1); the
    # second transfer waits for the link
    P = _micro([1e12, 0.5e12, 1e12], [6e9, 2e9, 1e9], [0.0, 0.0, 0.0], [0, 0, 1], [(0, 2), (1, 2)],
               [10.0, 10.0], [80.0, 80.0], {(0, 1): 10.0})
    r = SIM.simulate(P, [(0b01, AR), (0b10, AR)])
    t0, t1, x0, x1, t2 = 0.1, 0.05, 0.6, 0.2, 0.1
    start_x1 = t0 + x0                       # > t0 + t1, when op 1's output is ready
    assert r["T"] == pytest.approx(start_x1 + x1 + t2, rel=1e-15)
    assert r["group_idle"][0] == pytest.approx((0.0 + (start_x1 - (t0 + t1))) / 2, rel=1e-14)
    assert r["link_idle"][0] == pytest.approx(1 - (x0 + x1) / r["T"], rel=1e-14)


def test_allreduce_and_parameter_server_sync():
    P = _micro([4e12], [1e9], [3e9], [0], [], [10.0, 10.0, 10.0], [80.0] * 3,
               {(0, 1): 30.0, (0, 2): 15.0, (1, 2): 60.0})
    r = SIM.simulate(P, [(0b011, AR)])
    assert r["T"] == pytest.approx(4e12 / (2 * 10e12) + 2 * 0.5 * 3e9 / 30e9, rel=1e-15)
    assert r["dev_peak"][0] == pytest.approx(4 * 3e9 + 0.5e9)
    assert r["dev_peak"][2] == 0.0
    r = SIM.simulate(P, [(0b111, AR)])     # ring bound by the slowest link
    assert r["T"] == pytest.approx(4e12 / (3 * 10e12) + 2 * (2 / 3) * 3e9 / 15e9, rel=1e-15)
    r = SIM.simulate(P, [(0b110, PS)])     # server = device 1, its link to 2
    assert r["T"] == pytest.approx(4e12 / (2 * 10e12) + 2 * 0.5 * 3e9 / 60e9, rel=1e-15)


def test_model_parallel_gather_and_duplicate():
    P = _micro([4e12], [2e9], [3e9], [0], [], [10.0, 10.0], [80.0] * 2, {(0, 1): 20.0})
    r = SIM.simulate(P, [(0b11, MP)])
    assert r["T"] == pytest.approx(0.2 + 0.5 * 2e9 / 20e9, rel=1e-15)
    assert r["dev_peak"][0] == pytest.approx(4 * 1.5e9 + 1e9 + 2e9)   # partition, then the gathered tensor
    r = SIM.simulate(P, [(0b11, DUP)])
    assert r["T"] == pytest.approx(0.4, rel=1e-15)                     # whole op on each, no sync
    assert r["dev_peak"][1] == pytest.approx(4 * 3e9 + 2e9)


def test_empty_device_set_is_invalid():
    P = _micro([1e12, 1e12], [1e9, 1e9], [0.0, 0.0], [0, 1], [(0, 1)], [10.0], [80.0], {})
    r = SIM.simulate(P, [(1, AR), (0, AR)])
    assert r["valid"] is False and r["oom"] and math.isinf(r["T"])


def _single_device_case(seed):
    topo = synth.random_topology(seed, 60, 5, 120)
    rng = synth.rng_for(93, seed)
    K = 6
    groups = np.sort(rng.integers(0, K, size=topo.n_op)).astype(np.int32)
    groups[:K] = np.arange(K)
    sp = synth.SearchProblem(name="r", topo=topo, group_of=groups, n_groups=K,
                             op_params=rng.lognormal(15, 1, size=topo.n_op), masks=np.zeros(1, np.uint64),
                             options=np.zeros(1, np.uint8))
    dev = rng.integers(0, topo.n_dev, size=K)
    return SIM.SimProblem(sp), [(1 << int(d), AR) for d in dev], dev


@pytest.mark.parametrize("seed", [1, 2, 3])
def test_serial_identity_and_critical_path_bounds(seed):
    P, strat, dev = _single_device_case(seed)
    # everything on device 0: the device never idles, T is the serial sum
    one = [(1, AR)] * P.K
    r = SIM.simulate(P, one)
    assert r["T"] == pytest.approx(sum(f / P.speed[0] for f in P.flops), rel=1e-12)
    # one device per group: longest path of compute + transfer times <= T <= sum of all durations
    r = SIM.simulate(P, strat)
    d = [int(dev[P.group_of[i]]) for i in range(P.N)]
    comp = [P.flops[i] / P.speed[d[i]] for i in range(P.N)]
    preds = [[] for _ in range(P.N)]
    for (p, c) in P.edges:
        preds[c].append(p)
    lp = [0.0] * P.N
    for i in range(P.N):            # random_topology edges go from lower to higher ids
        best = 0.0
        for p in preds[i]:
            x = 0.0 if d[p] == d[i] else P.out[p] / P.bw[d[p]][d[i]]
            best = max(best, lp[p] + x)
        lp[i] = best + comp[i]
    serial = sum(comp) + sum(P.out[p] / P.bw[d[p]][d[c]] for (p, c) in P.edges if d[p] != d[c])
    assert max(lp) <= r["T"] * (1 + 1e-12)
    assert r["T"] <= serial * (1 + 1e-12)
    for j in range(P.M):
        busy = sum(comp[i] for i in range(P.N) if d[i] == j)
        assert r["dev_idle"][j] == pytest.approx(1 - busy / r["T"], rel=1e-9, abs=1e-12)
    assert all(0.0 <= x <= 1.0 for x in r["link_idle"])
