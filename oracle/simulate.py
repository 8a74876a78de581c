"""Reference simulator of one training iteration under a deployment strategy.

TEST INFRASTRUCTURE ONLY (like the rest of ``oracle/``): the tests, the
package smoke check and the benchmark's CPU-baseline leg may use it; the
library never does.  Plain Python, double precision, written from the
paper's virtual runtime (Section 4.3.1, the compiler that inserts auxiliary
ops for a strategy; Section 4.3.2, the simulator: a FIFO task queue per
device, an op enters the queue when all its inputs are ready, devices run
their queues independently, and reference counting of tensors gives the
peak memory of every device).  Its outputs are the runtime feedback of the
GNN input features (Section 4.2.1): makespan of each op group, idle time
before a group's output transfers, peak memory and idle share of each
device, idle share of each device link.

Readings (the paper leaves these open):

* Strategy.  Every op takes its group's (device set D, option); r = |D|.
  Options: 0 replicate + AllReduce, 1 replicate + parameter server,
  2 duplicate (SFB: every replica does the whole op, no gradient sync),
  3 model parallel.
* Compute.  Op i runs one task on each device j of D: FLOPs / speed_j for
  duplicate or r = 1, FLOPs / (r speed_j) otherwise.
* Model-parallel gather (Concat of the partitions).  With option 3 and
  r > 1, each device of D runs a gather task after all partitions are done:
  (r - 1) / r * out_bytes / min bandwidth inside D; consumers read the
  gathered tensor.
* Gradient sync (the inserted AllReduce / AddN).  With option 0 or 1, r > 1
  and parameters > 0, each device of D runs a sync task after all replicas
  are done: AllReduce 2 (r - 1) / r params / min bandwidth inside D;
  parameter server 2 (r - 1) / r params / min bandwidth from D's first
  device to the others.
* Tensors (Split / Concat to another placement).  For a tensor p -> c and
  every device j of c: when j also holds p, the input is local; otherwise a
  transfer from the device of p with the highest bandwidth to j (first
  maximum in device order) runs on that link's FIFO queue, of
  out_bytes(p) / r_c bytes when c splits its batch (options 0, 1) and the
  whole tensor otherwise, taking bytes / bandwidth.
* Queues.  One FIFO queue per device and per device pair (link).  Tasks are
  numbered: for each op in id order its compute tasks (device order), then
  its gather tasks, then its sync tasks; then for each tensor in input order
  its transfers (consumer device order).  Task completions are processed in
  order of (finish time, task number); the tasks a completion makes ready
  enter their queues in task-number order; an idle resource starts the head
  of its queue at once.
* Memory (bytes).  Resident from the start on every device of D: 4 x
  parameters (divided by r for model parallel).  A task's output is
  allocated on its device when it finishes: a compute output holds
  out_bytes (duplicate or r = 1) or out_bytes / r; a gather output the whole
  tensor; a transfer the transferred bytes.  Then the task releases its
  inputs; a tensor is freed when its last use finishes (a tensor without
  uses right after its allocation).  Uses: a compute output is used by the
  gather task (model parallel, r > 1) or else, like a gather output, by the
  local consumer compute tasks and the transfers that leave its device; a
  transfer output by its consumer's compute task.
* Outputs.  Iteration time T = last finish.  Group makespan = last finish
  of the group's compute / gather / sync tasks - first start of its compute
  tasks.  Group idle = mean, over transfers from an op of the group to an op
  of another group, of transfer start - finish of the task it waits for
  (0 without such transfers).  Device / link idle share = 1 - busy / T.  OOM
  when a device's peak exceeds its memory.  A strategy with an empty device
  set is invalid.
"""
from __future__ import annotations

import heapq
import math
from collections import deque
from typing import Dict, List, Optional, Sequence, Tuple

AR, PS, DUP, MP = 0, 1, 2, 3
MEM_FACTOR = 4.0   # weights + gradients + two optimizer moments per parameter byte


class SimProblem:
    """Per-op and per-device quantities of a search problem (double precision)."""

    def __init__(self, sp):
        t = sp.topo
        self.N, self.M = t.n_op, t.n_dev
        self.group_of = [int(x) for x in sp.group_of]
        self.K = sp.n_groups
        self.flops = [float(x) for x in t.op_flops]
        self.out = [float(x) for x in t.op_bytes]
        self.params = [float(x) for x in sp.op_params]
        self.speed = [float(x) * 1e12 for x in t.dev_tflops]
        self.mem = [float(x) * 1e9 for x in t.dev_mem]
        M = self.M
        self.bw = [[0.0] * M for _ in range(M)]
        for j in range(M):
            self.bw[j][j] = float(t.dev_intra_bw[j]) * 1e9
        for e in range(t.e_dd):
            a, b = int(t.dd_a[e]), int(t.dd_b[e])
            self.bw[a][b] = self.bw[b][a] = float(t.dd_bw[e]) * 1e9
        self.links = [(int(t.dd_a[e]), int(t.dd_b[e])) for e in range(t.e_dd)]
        self.edges = [(int(t.oo_src[e]), int(t.oo_dst[e])) for e in range(t.e_oo)]


def _bwmin(P: SimProblem, D: List[int]) -> float:
    m = math.inf
    for x in range(len(D)):
        for y in range(x + 1, len(D)):
            m = min(m, P.bw[D[x]][D[y]])
    return m


class _Task:
    __slots__ = ("res", "dur", "deps", "kind", "op", "dev", "start", "finish", "size", "uses", "inputs", "src_task")

    def __init__(self, res, dur, kind, op, dev):
        self.res, self.dur, self.kind, self.op, self.dev = res, dur, kind, op, dev
        self.deps: List[int] = []
        self.start = self.finish = 0.0
        self.size = 0.0          # bytes of the output tensor
        self.uses = 0            # tasks that use the output
        self.inputs: List[int] = []   # tasks whose outputs this task uses
        self.src_task = -1       # transfers: the task whose output is sent


def _link(P: SimProblem, a: int, b: int) -> int:
    a, b = min(a, b), max(a, b)
    return P.M + a * P.M + b


def build_tasks(P: SimProblem, strat: Sequence[Tuple[int, int]]) -> Optional[List[_Task]]:
    """Task graph of a full strategy ((mask, option) per group), or None
    when a group's device set is empty (Section 4.3.1 readings above)."""
    devs = []
    for i in range(P.N):
        mask, _ = strat[P.group_of[i]]
        D = [j for j in range(P.M) if (mask >> j) & 1]
        if not D:
            return None
        devs.append(D)
    opt = [strat[P.group_of[i]][1] for i in range(P.N)]
    T: List[_Task] = []
    comp: Dict[Tuple[int, int], int] = {}
    ready: Dict[Tuple[int, int], int] = {}   # task giving op i's usable output on device j
    for i in range(P.N):
        D, r, o = devs[i], len(devs[i]), opt[i]
        for j in D:
            dur = P.flops[i] / P.speed[j] if (o == DUP or r == 1) else P.flops[i] / (r * P.speed[j])
            t = _Task(j, dur, "C", i, j)
            t.size = P.out[i] if (o == DUP or r == 1) else P.out[i] / r
            comp[(i, j)] = len(T)
            ready[(i, j)] = len(T)
            T.append(t)
        if o == MP and r > 1:
            dur = (r - 1) / r * P.out[i] / _bwmin(P, D)
            for j in D:
                t = _Task(j, dur, "G", i, j)
                t.deps = [comp[(i, x)] for x in D]
                t.inputs = [comp[(i, j)]]
                t.size = P.out[i]
                T[comp[(i, j)]].uses += 1
                ready[(i, j)] = len(T)
                T.append(t)
        if P.params[i] > 0 and r > 1 and o in (AR, PS):
            if o == AR:
                dur = 2.0 * (r - 1) / r * P.params[i] / _bwmin(P, D)
            else:
                bps = min(P.bw[D[0]][x] for x in D[1:])
                dur = 2.0 * (r - 1) / r * P.params[i] / bps
            for j in D:
                t = _Task(j, dur, "S", i, j)
                t.deps = [comp[(i, x)] for x in D]
                T.append(t)
    for (p, c) in P.edges:
        Dp, Dc = devs[p], devs[c]
        share = 1.0 / len(Dc) if opt[c] in (AR, PS) else 1.0
        for j in Dc:
            cons = T[comp[(c, j)]]
            if j in Dp:
                src = ready[(p, j)]
                cons.deps.append(src)
                cons.inputs.append(src)
                T[src].uses += 1
                continue
            s = Dp[0]
            for x in Dp[1:]:
                if P.bw[x][j] > P.bw[s][j]:
                    s = x
            nbytes = P.out[p] * share
            t = _Task(_link(P, s, j), nbytes / P.bw[s][j], "X", p, j)
            src = ready[(p, s)]
            t.deps = [src]
            t.inputs = [src]
            t.src_task = src
            t.size = nbytes
            t.uses = 1
            T[src].uses += 1
            xid = len(T)
            T.append(t)
            cons.deps.append(xid)
            cons.inputs.append(xid)
    return T


def simulate(P: SimProblem, strat: Sequence[Tuple[int, int]]) -> dict:
    """Event simulation of the task graph; see the module notes for the rules."""
    T = build_tasks(P, strat)
    if T is None:
        return dict(valid=False, T=math.inf, oom=True)
    n = len(T)
    dependents: List[List[int]] = [[] for _ in range(n)]
    waiting = [0] * n
    for k, t in enumerate(T):
        waiting[k] = len(t.deps)
        for d in t.deps:
            dependents[d].append(k)
    nres = P.M + P.M * P.M
    queue = [deque() for _ in range(nres)]
    running = [False] * nres
    busy = [0.0] * nres
    heap: List[Tuple[float, int]] = []

    def start_next(res: int, now: float) -> None:
        k = queue[res].popleft()
        T[k].start = now
        T[k].finish = now + T[k].dur
        busy[res] += T[k].dur
        running[res] = True
        heapq.heappush(heap, (T[k].finish, k))

    def make_ready(k: int, now: float) -> None:
        queue[T[k].res].append(k)
        if not running[T[k].res]:
            start_next(T[k].res, now)

    # memory: resident parameters, then live tensors
    cur = [0.0] * P.M
    for i in range(P.N):
        mask, o = strat[P.group_of[i]]
        D = [j for j in range(P.M) if (mask >> j) & 1]
        for j in D:
            cur[j] += MEM_FACTOR * (P.params[i] / len(D) if o == MP else P.params[i])
    peak = list(cur)
    left = [t.uses for t in T]

    for k in range(n):
        if waiting[k] == 0:
            make_ready(k, 0.0)
    done = 0
    while heap:
        now, k = heapq.heappop(heap)
        t = T[k]
        running[t.res] = False
        done += 1
        d = t.dev
        if t.kind != "S":
            cur[d] += t.size
            peak[d] = max(peak[d], cur[d])
        for q in t.inputs:
            left[q] -= 1
            if left[q] == 0:
                cur[T[q].dev] -= T[q].size
        if t.kind != "S" and left[k] == 0:
            cur[d] -= t.size
        for q in dependents[k]:
            waiting[q] -= 1
            if waiting[q] == 0:
                make_ready(q, now)
        if not running[t.res] and queue[t.res]:
            start_next(t.res, now)
    if done != n:
        raise ValueError("the tensor graph has a cycle")
    Tit = max((t.finish for t in T), default=0.0)
    gstart = [math.inf] * P.K
    gend = [0.0] * P.K
    for t in T:
        g = P.group_of[t.op]
        if t.kind == "C":
            gstart[g] = min(gstart[g], t.start)
        if t.kind in ("C", "G", "S"):
            gend[g] = max(gend[g], t.finish)
    # idle before output transfers: transfers whose consumer (the compute
    # task listing them as an input) is in another group
    cons_of = {}
    for t in T:
        if t.kind == "C":
            for q in t.inputs:
                if T[q].kind == "X":
                    cons_of[q] = t.op
    isum = [0.0] * P.K
    icnt = [0] * P.K
    for k, t in enumerate(T):
        if t.kind != "X":
            continue
        gp, gc = P.group_of[t.op], P.group_of[cons_of[k]]
        if gp != gc:
            isum[gp] += t.start - T[t.src_task].finish
            icnt[gp] += 1
    makespan = [gend[g] - gstart[g] for g in range(P.K)]
    gidle = [isum[g] / icnt[g] if icnt[g] else 0.0 for g in range(P.K)]
    didle = [1.0 - busy[j] / Tit if Tit > 0 else 0.0 for j in range(P.M)]
    lidle = [1.0 - busy[_link(P, a, b)] / Tit if Tit > 0 else 0.0 for (a, b) in P.links]
    oom = any(peak[j] > P.mem[j] for j in range(P.M))
    return dict(valid=True, T=Tit, oom=oom, group_makespan=makespan, group_idle=gidle, dev_peak=peak,
                dev_idle=didle, link_idle=lidle, n_tasks=n)


def strategy_of(sp, path: Sequence[int], order: Sequence[int]) -> List[Tuple[int, int]]:
    """Full strategy of a partial one (the search's rule: undecided groups
    follow the first decided group; nothing decided: all devices, AllReduce)."""
    M, K = sp.topo.n_dev, sp.n_groups
    full = (1 << M) - 1
    if not path:
        return [(full, AR)] * K
    first = (int(sp.masks[path[0]]) & full, int(sp.options[path[0]]))
    strat = [first] * K
    for i, a in enumerate(path):
        strat[order[i]] = (int(sp.masks[a]) & full, int(sp.options[a]))
    return strat
