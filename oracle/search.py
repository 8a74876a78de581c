"""Reference strategy search: PUCT tree search over per-group strategy slices.

TEST INFRASTRUCTURE ONLY (like the rest of ``oracle/``): the tests, the
package smoke check and the benchmark's CPU-baseline leg may use it; the
library never does.  Plain Python and numpy, double precision, written from
the paper's description of its search (Section 4.2.2, Monte-Carlo Tree
Search) and of its reward (speed-up of the simulated training iteration over
data parallelism with AllReduce; -1 when a device runs out of memory).

Pieces and the readings they take where the paper is silent:

* Order.  Op groups are considered in descending order of computation time
  (total FLOPs of the group; equal totals keep the lower group id first).
  Tree depth d means the first d groups of that order are decided.
* Actions.  An edge of the tree picks one slice (device mask, replication
  option) of the slice table for the next group.
* Reward.  ``cost_model`` below, a deterministic analytic iteration-time
  model standing in for the paper's simulator (which needs profiles of real
  TensorFlow graphs).  Undecided groups take the decided strategy of the most
  computation-expensive group (the paper's footnote); with nothing decided,
  every group takes the baseline (all devices, AllReduce).
* Selection (PUCT).  U(s, a) = Q(s, a) + c G(s, a) sqrt(sum_a' N(s, a')) /
  (1 + N(s, a)), the first maximum wins, an unvisited edge has Q = 0.
* Back-propagation.  The paper writes Q := Q + r / N; that is not the running
  average it names, so Q := Q + (r - Q) / N (running mean).
* Batching.  A round selects B leaves one after another; every edge on a
  selected path carries one in-flight visit (virtual loss) until the round's
  update, counted as a visit with reward `vl_value`:
  N_eff = N + VL, Q_eff = (N Q + VL vl_value) / N_eff.  Updates then apply
  the B leaves in selection order: expand (priors) if not yet expanded, then
  remove the in-flight visit and add the real one on every edge of the path.
  With B = 1 this is the paper's sequential search.

Feature encoding of a search state for the GNN follows the op / device /
placement-edge layouts of the generators (``synth``), with the runtime
feedback taken from the problem's model (the analytic cost model, or the
reference simulator of Section 4.3.2 in oracle/simulate.py).
"""
from __future__ import annotations

import math
from typing import Dict, List, Optional, Sequence, Tuple

import numpy as np

AR, PS, DUP, MP = 0, 1, 2, 3
MEM_FACTOR = 4.0   # weights + gradients + two optimizer moments per parameter byte


class Problem:
    """Static quantities of one search problem (double precision).
    ``model`` picks the reward and runtime-feedback model: "analytic"
    (``evaluate`` below) or "simulator" (oracle/simulate.py)."""

    def __init__(self, sp, model: str = "analytic"):
        t = sp.topo
        self.sp = sp
        if model not in ("analytic", "simulator"):
            raise ValueError(model)
        self.model = model
        self.sim = None
        if model == "simulator":
            from oracle import simulate as _sim
            self.sim = _sim.SimProblem(sp)
        self.N, self.M, self.K = t.n_op, t.n_dev, sp.n_groups
        self.S = len(sp.masks)
        g = sp.group_of.astype(np.int64)
        self.group_of = g
        self.FL = np.zeros(self.K)
        self.PB = np.zeros(self.K)
        self.AB = np.zeros(self.K)
        for u in range(self.N):       # plain sums in op order
            self.FL[g[u]] += t.op_flops[u]
            self.PB[g[u]] += sp.op_params[u]
            self.AB[g[u]] += t.op_bytes[u]
        # descending computation time, lower id first on ties
        self.order = sorted(range(self.K), key=lambda k: (-self.FL[k], k))
        self.speed = t.dev_tflops * 1e12
        self.mem = t.dev_mem * 1e9
        self.bw = np.zeros((self.M, self.M))
        for j in range(self.M):
            self.bw[j, j] = t.dev_intra_bw[j] * 1e9
        for e in range(t.e_dd):
            a, b = int(t.dd_a[e]), int(t.dd_b[e])
            self.bw[a, b] = self.bw[b, a] = t.dd_bw[e] * 1e9
        # cross-group tensor bytes, pairs in first-appearance order of the edge list
        self.xpairs: List[Tuple[int, int]] = []
        self.xbytes: List[float] = []
        idx: Dict[Tuple[int, int], int] = {}
        for e in range(t.e_oo):
            s, d = int(t.oo_src[e]), int(t.oo_dst[e])
            gs, gd = int(g[s]), int(g[d])
            if gs == gd:
                continue
            key = (gs, gd)
            if key not in idx:
                idx[key] = len(self.xpairs)
                self.xpairs.append(key)
                self.xbytes.append(0.0)
            self.xbytes[idx[key]] += t.op_bytes[s]
        self.masks = [int(m) for m in sp.masks]
        self.options = [int(o) for o in sp.options]

    def devices(self, mask: int) -> List[int]:
        return [j for j in range(self.M) if (mask >> j) & 1]


def full_strategy(P: Problem, path: Sequence[int]) -> List[Tuple[int, int]]:
    """(mask, option) of every group for a partial strategy: `path[i]` is the
    slice of the i-th group in search order."""
    d = len(path)
    if d == 0:
        base = ((1 << P.M) - 1, AR)
        return [base] * P.K
    first = (P.masks[path[0]] & ((1 << P.M) - 1), P.options[path[0]])
    strat = [first] * P.K
    for i, a in enumerate(path):
        strat[P.order[i]] = (P.masks[a] & ((1 << P.M) - 1), P.options[a])
    return strat


def _bwmin(P: Problem, devs: List[int]) -> float:
    m = math.inf
    for x in range(len(devs)):
        for y in range(x + 1, len(devs)):
            m = min(m, P.bw[devs[x], devs[y]])
    return m


def evaluate(P: Problem, strat: List[Tuple[int, int]]) -> dict:
    """Iteration time, per-device loads and memory of a full strategy."""
    load = np.zeros(P.M)
    memu = np.zeros(P.M)
    invalid = False
    comp = np.zeros(P.K)     # slowest participating device's compute time
    sync = np.zeros(P.K)
    for g in range(P.K):
        mask, o = strat[g]
        devs = P.devices(mask)
        r = len(devs)
        if r == 0:   # a mask with no device of the topology cannot be deployed
            invalid = True
            continue
        s = 0.0   # per-iteration communication of the group on each of its devices
        if r > 1 and o == AR:      # ring AllReduce of the gradients
            s = 2.0 * (r - 1) / r * P.PB[g] / _bwmin(P, devs)
        elif r > 1 and o == PS:    # push and pull through the first device
            p = devs[0]
            bps = math.inf
            for j in devs[1:]:
                bps = min(bps, P.bw[p, j])
            s = 2.0 * (r - 1) / r * P.PB[g] / bps
        elif r > 1:                # duplicate: inputs broadcast; model parallel: activations exchanged
            s = (r - 1) / r * P.AB[g] / _bwmin(P, devs)
        sync[g] = s
        cmax = 0.0
        for j in devs:
            c = P.FL[g] / P.speed[j] if o == DUP else P.FL[g] / (r * P.speed[j])
            cmax = max(cmax, c)
            load[j] += c + s
            wbytes = P.PB[g] / r if o == MP else P.PB[g]
            abytes = P.AB[g] if o == DUP else P.AB[g] / r
            memu[j] += MEM_FACTOR * wbytes + abytes
        comp[g] = cmax
    xfer = 0.0
    for (g1, g2), b in zip(P.xpairs, P.xbytes):
        m1, m2 = strat[g1][0], strat[g2][0]
        if m1 == m2 or m1 == 0 or m2 == 0:
            continue
        p1 = (m1 & -m1).bit_length() - 1
        p2 = (m2 & -m2).bit_length() - 1
        xfer += b / P.bw[p1, p2]
    T = float(load.max()) + xfer
    oom = bool(np.any(memu > P.mem)) or invalid
    return {"T": T, "load": load, "mem": memu, "comp": comp, "sync": sync, "oom": oom}


def feedback(P: Problem, strat: List[Tuple[int, int]]) -> dict:
    """Iteration time, OOM flag and runtime feedback of a full strategy
    under the problem's model: per group its makespan (s) and idle share, per
    device its memory share (capped at 1) and idle share.
      analytic:  makespan = slowest replica's compute, idle share = sync /
                 (compute + sync), memory = modelled use, idle = 1 - load / T
      simulator: simulated makespan, mean idle before the group's output
                 transfers / T, peak / capacity, simulated idle share"""
    if P.model == "analytic":
        ev = evaluate(P, strat)
        gidle = [ev["sync"][g] / (ev["comp"][g] + ev["sync"][g]) if ev["comp"][g] + ev["sync"][g] > 0 else 0.0
                 for g in range(P.K)]
        memf = [min(ev["mem"][j] / P.mem[j], 1.0) for j in range(P.M)]
        didle = [1.0 - ev["load"][j] / ev["T"] if ev["T"] > 0 else 0.0 for j in range(P.M)]
        return dict(T=ev["T"], oom=ev["oom"], makespan=list(ev["comp"]), gidle=gidle, memf=memf, didle=didle,
                    lidle=[0.0] * P.sp.topo.e_dd)
    from oracle import simulate as _sim
    r = _sim.simulate(P.sim, strat)
    if not r["valid"]:
        return dict(T=math.inf, oom=True, makespan=[0.0] * P.K, gidle=[0.0] * P.K, memf=[0.0] * P.M,
                    didle=[0.0] * P.M, lidle=[0.0] * P.sp.topo.e_dd)
    T = r["T"]
    return dict(T=T, oom=r["oom"], makespan=r["group_makespan"],
                gidle=[min(x / T, 1.0) if T > 0 else 0.0 for x in r["group_idle"]],
                memf=[min(r["dev_peak"][j] / P.mem[j], 1.0) for j in range(P.M)], didle=r["dev_idle"],
                lidle=r["link_idle"])


def reward(P: Problem, path: Sequence[int], T_base: Optional[float] = None) -> float:
    """Speed-up of the partial strategy's iteration time over the baseline
    (every group on every device with AllReduce); -1 when a device runs out
    of memory or a group's mask names no device of the topology."""
    if T_base is None:
        T_base = feedback(P, full_strategy(P, []))["T"]
    ev = feedback(P, full_strategy(P, path))
    if ev["oom"]:
        return -1.0
    return T_base / ev["T"]


def link_features(P: Problem, path: Sequence[int]) -> np.ndarray:
    """Link rows of a search state, x_dd [E_dd, 2] float32: log10(GB/s) - 1
    and the link's idle share (the simulator's; 0 under the analytic model)."""
    t = P.sp.topo
    fb = feedback(P, full_strategy(P, path))
    x = np.zeros((t.e_dd, 2), np.float32)
    for e in range(t.e_dd):
        x[e, 0] = np.float32(math.log10(t.dd_bw[e]) - 1.0)
        x[e, 1] = np.float32(fb["lidle"][e])
    return x


def features(P: Problem, path: Sequence[int], f_op: int = 42):
    """GNN inputs of a search state: x_op [N, f_op], x_dev [M, 8], x_od [E_od]
    (float32 / uint8), and the representative (most FLOPs, lowest id first)
    op of the next group, or -1 when every group is decided."""
    t = P.sp.topo
    d = len(path)
    strat = full_strategy(P, path)
    fb = feedback(P, strat)
    decided_g = np.zeros(P.K, bool)
    for i in range(d):
        decided_g[P.order[i]] = True
    nxt = P.order[d] if d < P.K else -1
    x = np.zeros((P.N, f_op), np.float32)
    for u in range(P.N):
        g = int(P.group_of[u])
        x[u, int(t.op_type[u]) % 32] = 1.0
        x[u, 32] = np.float32(math.log10(t.op_flops[u]) - 8.0)
        x[u, 33] = np.float32(math.log10(t.op_bytes[u]) - 6.0)
        if decided_g[g]:
            x[u, 34 + strat[g][1]] = 1.0
            x[u, 38] = 1.0
            if f_op >= 42:
                x[u, 40] = np.float32(math.log10(max(fb["makespan"][g], 1e-12) * 1e3))
                x[u, 41] = np.float32(fb["gidle"][g])
        if g == nxt:
            x[u, 39] = 1.0
    xd = np.zeros((P.M, 8), np.float32)
    for j in range(P.M):
        xd[j, 0] = np.float32(t.dev_tflops[j] / 10.0)
        xd[j, 1] = np.float32(t.dev_mem[j] / 32.0)
        xd[j, 2] = 1.0
        xd[j, 3] = np.float32(math.log10(t.dev_intra_bw[j]))
        xd[j, 4] = np.float32(fb["memf"][j])
        xd[j, 5] = np.float32(fb["didle"][j])
    xod = np.zeros(t.e_od, np.uint8)
    for e in range(t.e_od):
        u, j = int(t.od_op[e]), int(t.od_dev[e])
        g = int(P.group_of[u])
        if decided_g[g] and (strat[g][0] >> j) & 1:
            xod[e] = 1
    rep = -1
    if nxt >= 0:
        best = -1.0
        for u in range(P.N):
            if int(P.group_of[u]) == nxt and t.op_flops[u] > best:
                best, rep = t.op_flops[u], u
    return x, xd, xod, rep


class Tree:
    """PUCT search tree with batched selection (see the module docstring)."""

    def __init__(self, n_levels: int, n_actions: int, c_puct: float, vl_value: float = 0.0):
        self.L, self.S, self.c, self.vl = n_levels, n_actions, float(c_puct), float(vl_value)
        self.verts: List[dict] = []
        self._new_vertex(0)

    def _new_vertex(self, depth: int) -> int:
        self.verts.append({"depth": depth, "expanded": False, "G": None,
                           "N": [0] * self.S, "Q": [0.0] * self.S, "VL": [0] * self.S,
                           "child": [-1] * self.S})
        return len(self.verts) - 1

    def _pick(self, v: dict) -> int:
        total = 0
        for a in range(self.S):
            total += v["N"][a] + v["VL"][a]
        sq = math.sqrt(float(total))
        best, arg = -math.inf, 0
        for a in range(self.S):
            n, vl = v["N"][a], v["VL"][a]
            ne = n + vl
            q = (n * v["Q"][a] + vl * self.vl) / ne if ne > 0 else 0.0
            u = q + self.c * v["G"][a] * sq / (1.0 + ne)
            if u > best:
                best, arg = u, a
        return arg

    def select(self, B: int) -> List[Tuple[int, List[int]]]:
        """B leaves as (vertex id, action path), in-flight visits applied."""
        out = []
        for _ in range(B):
            vid, path = 0, []
            while self.verts[vid]["expanded"] and self.verts[vid]["depth"] < self.L:
                v = self.verts[vid]
                a = self._pick(v)
                v["VL"][a] += 1
                path.append(a)
                if v["child"][a] < 0:
                    v["child"][a] = self._new_vertex(v["depth"] + 1)
                vid = v["child"][a]
            out.append((vid, path))
        return out

    def update(self, leaves: List[Tuple[int, List[int]]], priors: Sequence[Sequence[float]],
               rewards: Sequence[float]) -> None:
        for (vid, path), pr, r in zip(leaves, priors, rewards):
            leaf = self.verts[vid]
            if leaf["depth"] < self.L and not leaf["expanded"]:
                leaf["G"] = [float(p) for p in pr]
                leaf["expanded"] = True
            u = 0
            for a in path:
                v = self.verts[u]
                v["VL"][a] -= 1
                v["N"][a] += 1
                v["Q"][a] += (float(r) - v["Q"][a]) / v["N"][a]
                u = v["child"][a]

    def root_stats(self):
        r = self.verts[0]
        return list(r["N"]), list(r["Q"])

    def best_path(self) -> List[int]:
        """Most visited action at every level (first maximum)."""
        path, vid = [], 0
        while self.verts[vid]["expanded"] and self.verts[vid]["depth"] < self.L:
            v = self.verts[vid]
            a = int(np.argmax(v["N"]))
            if v["N"][a] == 0 or v["child"][a] < 0:
                break
            path.append(a)
            vid = v["child"][a]
        return path
