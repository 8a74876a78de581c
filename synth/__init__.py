"""Seeded synthetic inputs for the heterogeneous-GNN hot path.

This module only draws numbers: topologies, per-candidate strategy features,
slice tables and weights.  It holds none of the method's arithmetic (no
encoders, no layers, no attention, no decoder), so both the GPU path and the
CPU oracle can take their inputs from it without sharing any computation.

Workload shapes follow the paper's evaluation set-up: op counts of the
benchmark models (Section 5.2, table of benchmark DNN models), at most 60 op
groups per graph (Section 4.1.1, grouping ops), and device topologies of
machines with several same-type GPUs joined by slower inter-machine links
(Section 5.2, hardware and random training topologies).  The paper's real
TensorFlow graphs, profiles and clusters are not available; these generators
stand in for them.

Feature layouts (the paper lists the features in its GNN input table,
Section 4.2.1; the exact encoding is this module's reading):

op node, width 40 (tiny) or 42 (all other workloads)
    [0:32)  op-type one-hot (tiny workload) / same for the rest
    [32]    log10(compute FLOPs) - 8            computation time proxy
    [33]    log10(output bytes) - 6             parameter/size proxy
    [34:38) replication-option one-hot (zero if undecided)
    [38]    decided flag
    [39]    to-be-produced-next flag
    [40]    log10(makespan in ms)               runtime feedback (42 only)
    [41]    idle fraction before output transfer runtime feedback (42 only)
device node, width 8
    [TFLOPs/10, memory GB/32, #GPUs in group, log10(intra-group GB/s),
     peak-memory fraction, idle fraction, 0, 0]
op-op edge, width 1     log10(tensor bytes) - 6
device-device edge, 2   log10(GB/s) - 1, link idle fraction
op-device edge, 1 byte  placement bit (0/1)
"""
from __future__ import annotations

import dataclasses
import math
from typing import Dict, List, Optional

import numpy as np

SEED_ROOT = 2302
WEIGHT_STREAM = 99

# relation order used everywhere: 0 = op-op, 1 = op-device, 2 = device-device
REL_OO, REL_OD, REL_DD = 0, 1, 2
EDGE_DIMS = (1, 1, 2)
F_DEV = 8


@dataclasses.dataclass
class Topology:
    """One joint graph: op DAG + device graph + op-device pairs (local ids)."""
    n_op: int
    n_dev: int
    oo_src: np.ndarray  # int32 [E_oo] producer op
    oo_dst: np.ndarray  # int32 [E_oo] consumer op
    dd_a: np.ndarray    # int32 [E_dd] unordered device pair
    dd_b: np.ndarray
    od_op: np.ndarray   # int32 [E_od]
    od_dev: np.ndarray
    # raw attributes the feature generator reads
    op_type: np.ndarray      # int [N]
    op_flops: np.ndarray     # float [N]
    op_bytes: np.ndarray     # float [N] output bytes of each op
    dev_tflops: np.ndarray   # float [M]
    dev_mem: np.ndarray      # float [M] GB
    dev_intra_bw: np.ndarray  # float [M] GB/s inside the device's machine
    dd_bw: np.ndarray        # float [E_dd] GB/s

    @property
    def e_oo(self) -> int:
        return int(self.oo_src.shape[0])

    @property
    def e_dd(self) -> int:
        return int(self.dd_a.shape[0])

    @property
    def e_od(self) -> int:
        return int(self.od_op.shape[0])

    def entries(self) -> int:
        """Directed message entries of one forward layer (all four buckets)."""
        return 2 * self.e_oo + 2 * self.e_od + 2 * self.e_dd


@dataclasses.dataclass
class Candidate:
    """Per-candidate strategy features for one topology."""
    x_op: np.ndarray   # float32 [N, F_op]
    x_dev: np.ndarray  # float32 [M, 8]
    x_oo: np.ndarray   # float32 [E_oo]
    x_dd: np.ndarray   # float32 [E_dd, 2]
    x_od: np.ndarray   # uint8 [E_od]
    next_ops: np.ndarray  # int32: ops of the group whose strategy is produced next


@dataclasses.dataclass
class Workload:
    name: str
    cfg_id: int
    f: int
    heads: int
    layers: int
    f_op: int
    batch: int
    dtype: str          # "f32" or "bf16"
    n_slices: int
    description: str


WORKLOADS: Dict[str, Workload] = {
    "tiny": Workload("tiny", 0, 64, 4, 2, 40, 1, "f32", 60,
                     "1 graph, 200-op random DAG (400 edges), 4 devices, 2 layers, f=64, fp32"),
    "cnn": Workload("cnn", 1, 128, 4, 3, 42, 64, "f32", 256,
                    "ResNet-shaped 1200-op chain with skips, 16 devices, 3 layers, f=128, fp32, 64 candidates"),
    "transformer": Workload("transformer", 2, 256, 4, 3, 42, 128, "f32", 256,
                            "BERT-shaped 6000-op DAG, 32 devices, 3 layers, f=256, fp32, 128 candidates"),
    "large": Workload("large", 3, 256, 4, 4, 42, 256, "bf16", 256,
                      "10000-op layered DAG, 64 devices, 16 devices/op, 4 layers, f=256, bf16, 256 candidates"),
    "sweep": Workload("sweep", 4, 128, 4, 3, 42, 1024, "f32", 256,
                      "transformer graph, 1024 candidates, 3 layers, f=128, fp32"),
}


def rng_for(*key: int) -> np.random.Generator:
    return np.random.default_rng((SEED_ROOT,) + tuple(int(k) for k in key))


# --------------------------------------------------------------------------
# device topologies
# --------------------------------------------------------------------------

def _all_pairs(m: int):
    a, b = np.triu_indices(m, k=1)
    return a.astype(np.int32), b.astype(np.int32)


def _devices(kind: str, rng: np.random.Generator):
    """Return (tflops[M], mem[M], intra_bw[M], pair_bw(a, b) -> GB/s)."""
    if kind == "tiny":
        m = 4
        tfl = rng.choice([9.0, 15.0, 19.5], size=m)
        mem = rng.choice([11.0, 16.0, 32.0], size=m)
        a, b = _all_pairs(m)
        bw = rng.uniform(8.0, 300.0, size=a.shape[0])
        intra = np.full(m, 300.0)
        return tfl, mem, intra, a, b, bw
    if kind == "cnn":
        m = 16
        machine = np.arange(m) // 4
        tfl = np.full(m, 15.0)
        mem = np.full(m, 16.0)
        a, b = _all_pairs(m)
        bw = np.where(machine[a] == machine[b], 150.0, 12.5)
        return tfl, mem, np.full(m, 150.0), a, b, bw
    if kind == "transformer":
        m = 32
        machine = np.arange(m) // 4          # 8 machines
        rack = machine // 4                  # 2 racks
        types = [(19.5, 32.0)] * 3 + [(15.0, 16.0)] * 3 + [(9.0, 11.0)] * 2
        tfl = np.array([types[mc][0] for mc in machine])
        mem = np.array([types[mc][1] for mc in machine])
        a, b = _all_pairs(m)
        bw = np.where(machine[a] == machine[b], 150.0,
                      np.where(rack[a] == rack[b], 12.5, 3.0))
        return tfl, mem, np.full(m, 150.0), a, b, bw
    if kind == "large":
        m = 64
        island = np.arange(m) // 4           # 16 islands of 4
        machine = island // 2                # 8 machines
        rack = machine // 2                  # 4 racks
        types = [(19.5, 32.0), (15.0, 16.0), (9.0, 11.0)]
        tfl = np.array([types[mc % 3][0] for mc in machine])
        mem = np.array([types[mc % 3][1] for mc in machine])
        a, b = _all_pairs(m)
        bw = np.where(island[a] == island[b], 300.0,
                      np.where(machine[a] == machine[b], 32.0,
                               np.where(rack[a] == rack[b], 12.5, 3.0)))
        return tfl, mem, np.full(m, 300.0), a, b, bw
    raise ValueError(kind)


# --------------------------------------------------------------------------
# op DAGs
# --------------------------------------------------------------------------

def _dag_tiny(rng):
    n = 200
    pairs = [(i, j) for i in range(n) for j in range(i + 1, min(n, i + 17))]
    pick = rng.choice(len(pairs), size=400, replace=False)
    pick.sort()
    src = np.array([pairs[k][0] for k in pick], np.int32)
    dst = np.array([pairs[k][1] for k in pick], np.int32)
    return n, src, dst


def _dag_cnn():
    n = 1200
    src = list(range(n - 1))
    dst = list(range(1, n))
    for i in range(0, n - 3, 3):
        src.append(i)
        dst.append(i + 3)
    return n, np.array(src, np.int32), np.array(dst, np.int32)


def _dag_transformer():
    """24 blocks of 250 ops: entry -> 4 parallel 55-op chains -> merge
    (+ residual from entry) -> 28-op FFN chain (+ residual) -> next block."""
    src, dst = [], []
    n_blocks, per = 24, 250
    for blk in range(n_blocks):
        base = blk * per
        entry = base
        merge = base + 1 + 4 * 55
        for c in range(4):
            first = base + 1 + c * 55
            src.append(entry); dst.append(first)
            for k in range(54):
                src.append(first + k); dst.append(first + k + 1)
            src.append(first + 54); dst.append(merge)
        src.append(entry); dst.append(merge)
        f0 = merge + 1
        src.append(merge); dst.append(f0)
        for k in range(27):
            src.append(f0 + k); dst.append(f0 + k + 1)
        src.append(merge); dst.append(f0 + 27)
        if blk + 1 < n_blocks:
            src.append(f0 + 27); dst.append(base + per)
    return n_blocks * per, np.array(src, np.int32), np.array(dst, np.int32)


def _dag_layered(rng, n_layers=200, width=50, mean_deg=3.0):
    src, dst = [], []
    for layer in range(n_layers - 1):
        for i in range(width):
            d = min(int(rng.poisson(mean_deg)), width)
            if d == 0:
                continue
            tg = rng.choice(width, size=d, replace=False)
            tg.sort()
            u = layer * width + i
            for t in tg:
                src.append(u); dst.append((layer + 1) * width + int(t))
    return n_layers * width, np.array(src, np.int32), np.array(dst, np.int32)


_TOPO_KIND = {"tiny": "tiny", "cnn": "cnn", "transformer": "transformer",
              "large": "large", "sweep": "transformer"}
_TOPO_CFG = {"tiny": 0, "cnn": 1, "transformer": 2, "large": 3, "sweep": 2}


def make_topology(name: str) -> Topology:
    """The shared topology of a workload (seeded by the workload's config id)."""
    kind = _TOPO_KIND[name]
    cfg = _TOPO_CFG[name]
    rng = rng_for(cfg, 1_000_000)
    if kind == "tiny":
        n, src, dst = _dag_tiny(rng)
    elif kind == "cnn":
        n, src, dst = _dag_cnn()
    elif kind == "transformer":
        n, src, dst = _dag_transformer()
    else:
        n, src, dst = _dag_layered(rng)
    tfl, mem, intra, a, b, bw = _devices(kind, rng)
    m = tfl.shape[0]
    if kind == "large":
        ops, devs = [], []
        for u in range(n):
            ch = rng.choice(m, size=16, replace=False)
            ch.sort()
            ops.append(np.full(16, u, np.int32))
            devs.append(ch.astype(np.int32))
        od_op = np.concatenate(ops)
        od_dev = np.concatenate(devs)
    else:
        od_op = np.repeat(np.arange(n, dtype=np.int32), m)
        od_dev = np.tile(np.arange(m, dtype=np.int32), n)
    return Topology(
        n_op=n, n_dev=m, oo_src=src, oo_dst=dst, dd_a=a, dd_b=b,
        od_op=od_op.astype(np.int32), od_dev=od_dev.astype(np.int32),
        op_type=rng.integers(0, 32, size=n),
        op_flops=rng.lognormal(math.log(1e8), 1.5, size=n),
        op_bytes=rng.lognormal(math.log(1e6), 1.5, size=n),
        dev_tflops=tfl.astype(np.float64), dev_mem=mem.astype(np.float64),
        dev_intra_bw=intra.astype(np.float64), dd_bw=bw.astype(np.float64))


def random_topology(seed: int, n_op: int, n_dev: int, e_oo: int,
                    od_per_op: Optional[int] = None, dd_density: float = 1.0) -> Topology:
    """A small random joint graph for tests (distinct DAG pairs, distinct
    device pairs, distinct op-device pairs; ids local)."""
    rng = rng_for(7, seed)
    cand = [(i, j) for i in range(n_op) for j in range(i + 1, n_op)]
    e_oo = min(e_oo, len(cand))
    pick = rng.choice(len(cand), size=e_oo, replace=False) if e_oo else np.zeros(0, int)
    src = np.array([cand[k][0] for k in pick], np.int32)
    dst = np.array([cand[k][1] for k in pick], np.int32)
    a, b = _all_pairs(n_dev)
    if dd_density < 1.0 and a.shape[0]:
        keep = rng.random(a.shape[0]) < dd_density
        a, b = a[keep], b[keep]
    if od_per_op is None or od_per_op >= n_dev:
        od_op = np.repeat(np.arange(n_op, dtype=np.int32), n_dev)
        od_dev = np.tile(np.arange(n_dev, dtype=np.int32), n_op)
    else:
        ops, devs = [], []
        for u in range(n_op):
            ch = np.sort(rng.choice(n_dev, size=od_per_op, replace=False))
            ops.append(np.full(od_per_op, u, np.int32)); devs.append(ch.astype(np.int32))
        od_op = np.concatenate(ops) if ops else np.zeros(0, np.int32)
        od_dev = np.concatenate(devs) if devs else np.zeros(0, np.int32)
    return Topology(
        n_op=n_op, n_dev=n_dev, oo_src=src, oo_dst=dst,
        dd_a=a.astype(np.int32), dd_b=b.astype(np.int32),
        od_op=od_op.astype(np.int32), od_dev=od_dev.astype(np.int32),
        op_type=rng.integers(0, 32, size=n_op),
        op_flops=rng.lognormal(math.log(1e8), 1.5, size=n_op),
        op_bytes=rng.lognormal(math.log(1e6), 1.5, size=n_op),
        dev_tflops=rng.choice([9.0, 15.0, 19.5], size=n_dev),
        dev_mem=rng.choice([11.0, 16.0, 32.0], size=n_dev),
        dev_intra_bw=rng.uniform(64.0, 300.0, size=n_dev),
        dd_bw=rng.uniform(3.0, 300.0, size=a.shape[0]))


# --------------------------------------------------------------------------
# candidates (strategy encodings + synthetic runtime feedback)
# --------------------------------------------------------------------------

def _groups(name: str, n: int, rng) -> List[np.ndarray]:
    """Contiguous op groups, as a list of op-id ranges."""
    if name == "tiny":
        k = 10
    elif name == "cnn":
        k = int(rng.integers(20, 61))
    else:
        k = 60
    cuts = np.sort(rng.choice(np.arange(1, n), size=k - 1, replace=False)) if name == "cnn" \
        else np.array([round(i * n / k) for i in range(1, k)])
    bounds = np.concatenate([[0], cuts, [n]]).astype(int)
    return [np.arange(bounds[i], bounds[i + 1], dtype=np.int32) for i in range(k)]


def make_candidate(name: str, topo: Topology, cand: int, f_op: int) -> Candidate:
    """Strategy features of candidate `cand` (seed (2302, cfg, cand))."""
    cfg = WORKLOADS[name].cfg_id if name in WORKLOADS else 9
    rng = rng_for(cfg, cand)
    n, m = topo.n_op, topo.n_dev
    groups = _groups(name if name in WORKLOADS else "transformer", n, rng)
    k = len(groups)
    if name == "tiny":
        n_dec, nxt = 5, 5
    else:
        n_dec = int(rng.integers(0, k))
        nxt = n_dec
    option = rng.integers(0, 4, size=k)
    masks = np.zeros((k, m), np.uint8)
    for g in range(k):
        r = int(rng.integers(1, min(8, m) + 1)) if name != "tiny" else int(rng.integers(1, m + 1))
        masks[g, rng.choice(m, size=r, replace=False)] = 1
    group_of = np.empty(n, np.int64)
    for g, ops in enumerate(groups):
        group_of[ops] = g
    decided = group_of < n_dec

    x = np.zeros((n, f_op), np.float32)
    x[np.arange(n), topo.op_type % 32] = 1.0
    x[:, 32] = np.log10(topo.op_flops) - 8.0
    x[:, 33] = np.log10(topo.op_bytes) - 6.0
    rep = np.zeros((n, 4), np.float32)
    rep[np.arange(n), option[group_of]] = 1.0
    x[:, 34:38] = rep * decided[:, None]
    x[:, 38] = decided
    x[:, 39] = (group_of == nxt)
    if f_op >= 42:
        x[:, 40] = np.log10(rng.lognormal(math.log(1.0), 1.0, size=n)) * decided
        x[:, 41] = rng.uniform(0.0, 1.0, size=n) * decided

    xd = np.zeros((m, F_DEV), np.float32)
    xd[:, 0] = topo.dev_tflops / 10.0
    xd[:, 1] = topo.dev_mem / 32.0
    xd[:, 2] = 1.0
    xd[:, 3] = np.log10(topo.dev_intra_bw)
    xd[:, 4] = rng.uniform(0.0, 1.0, size=m)
    xd[:, 5] = rng.uniform(0.0, 1.0, size=m)

    x_oo = (np.log10(topo.op_bytes[topo.oo_src]) - 6.0).astype(np.float32)
    x_dd = np.stack([np.log10(topo.dd_bw) - 1.0,
                     rng.uniform(0.0, 1.0, size=topo.e_dd)], axis=1).astype(np.float32) \
        if topo.e_dd else np.zeros((0, 2), np.float32)
    g_of_edge = group_of[topo.od_op]
    x_od = (masks[g_of_edge, topo.od_dev].astype(bool) & decided[topo.od_op]).astype(np.uint8)
    next_ops = groups[nxt] if nxt < k else np.zeros(0, np.int32)
    return Candidate(x_op=x, x_dev=xd, x_oo=x_oo, x_dd=x_dd, x_od=x_od,
                     next_ops=next_ops.astype(np.int32))


@dataclasses.dataclass
class Batch:
    """R candidates sharing one topology, stacked replica-major."""
    x_op: np.ndarray   # [R, N, F_op]
    x_dev: np.ndarray  # [R, M, 8]
    x_oo: np.ndarray   # [E_oo] (shared: tensor sizes do not depend on the strategy)
    x_dd: np.ndarray   # [R, E_dd, 2]
    x_od: np.ndarray   # [R, E_od]
    query_rep: np.ndarray  # int32 [Q]
    query_op: np.ndarray   # int32 [Q]


def make_batch(name: str, topo: Topology, n_cand: int, f_op: int,
               first: int = 0) -> Batch:
    cands = [make_candidate(name, topo, first + c, f_op) for c in range(n_cand)]
    qr = np.concatenate([np.full(c.next_ops.shape[0], i, np.int32) for i, c in enumerate(cands)])
    qo = np.concatenate([c.next_ops for c in cands]).astype(np.int32)
    return Batch(
        x_op=np.stack([c.x_op for c in cands]),
        x_dev=np.stack([c.x_dev for c in cands]),
        x_oo=cands[0].x_oo,
        x_dd=np.stack([c.x_dd for c in cands]),
        x_od=np.stack([c.x_od for c in cands]),
        query_rep=qr, query_op=qo)


# --------------------------------------------------------------------------
# slice tables (candidate strategies for one op group)
# --------------------------------------------------------------------------

def make_slices(name: str, n_dev: int, n_slices: int):
    """Masks (uint64) and options (uint8).  The tiny workload enumerates every
    non-empty device subset with each of the 4 replication options."""
    if name == "tiny":
        masks, opts = [], []
        for msk in range(1, 1 << n_dev):
            for o in range(4):
                masks.append(msk); opts.append(o)
        return np.array(masks, np.uint64), np.array(opts, np.uint8)
    rng = rng_for(WORKLOADS[name].cfg_id if name in WORKLOADS else 9, 2_000_000)
    masks = np.zeros(n_slices, np.uint64)
    for s in range(n_slices):
        r = int(rng.integers(1, min(8, n_dev) + 1))
        bits = rng.choice(n_dev, size=r, replace=False)
        v = 0
        for bt in bits:
            v |= 1 << int(bt)
        masks[s] = np.uint64(v)
    opts = rng.integers(0, 4, size=n_slices).astype(np.uint8)
    return masks, opts


# --------------------------------------------------------------------------
# weights (Glorot-uniform, seeded per (layer, relation))
# --------------------------------------------------------------------------

def _glorot(rng, rows, cols):
    lim = math.sqrt(6.0 / (rows + cols))
    return rng.uniform(-lim, lim, size=(rows, cols)).astype(np.float32)


def make_weights(f: int, heads: int, layers: int, f_op: int, dec_hidden: int,
                 bias_scale: float = 0.1, seed_extra: int = 0, relations: int = 3,
                 heads_mode: str = "concat") -> Dict[str, np.ndarray]:
    """All parameters, float32, in the library's documented layouts:
    enc_op_w [f, f_op], enc_op_b [f], enc_dev_w [f, 8], enc_dev_b [f],
    enc_edge_w{r} [f, d_r], enc_edge_b{r} [f],
    layer_w [L, R, f, 2f] (= [W^h | W^e] per relation), layer_b [L, R, f],
    att_src [L, R, f], att_dst [L, R, f] (heads_mode "avg": [L, R, K, f]),
    dec_w1 [H, 2f+4], dec_b1 [H], dec_w2 [H], dec_b2 [1] (H = dec_hidden > 0)
    or dec_w2 [2f+4], dec_b2 [1] (linear decoder, H = 0).  R = relations
    (3 undirected link types, or 5 directed relations); the first three
    relations draw the same numbers whatever R is."""
    avg = heads_mode == "avg"
    d = f if avg else f // heads
    R = relations
    w: Dict[str, np.ndarray] = {}
    r0 = rng_for(WEIGHT_STREAM, 100, seed_extra)
    w["enc_op_w"] = _glorot(r0, f, f_op)
    w["enc_op_b"] = (r0.uniform(-1, 1, f) * bias_scale).astype(np.float32)
    w["enc_dev_w"] = _glorot(r0, f, F_DEV)
    w["enc_dev_b"] = (r0.uniform(-1, 1, f) * bias_scale).astype(np.float32)
    for r, dr in enumerate(EDGE_DIMS):
        w[f"enc_edge_w{r}"] = _glorot(r0, f, dr)
        w[f"enc_edge_b{r}"] = (r0.uniform(-1, 1, f) * bias_scale).astype(np.float32)
    lw = np.zeros((layers, R, f, 2 * f), np.float32)
    lb = np.zeros((layers, R, f), np.float32)
    ashape = (layers, R, heads, f) if avg else (layers, R, f)
    asrc = np.zeros(ashape, np.float32)
    adst = np.zeros(ashape, np.float32)
    for layer in range(layers):
        for r in range(R):
            rg = rng_for(WEIGHT_STREAM, layer, r, seed_extra)
            lw[layer, r] = _glorot(rg, f, 2 * f)
            lb[layer, r] = rg.uniform(-1, 1, f) * bias_scale
            lim = math.sqrt(6.0 / (d + 1))
            asrc[layer, r] = rg.uniform(-lim, lim, ashape[2:])
            adst[layer, r] = rg.uniform(-lim, lim, ashape[2:])
    w["layer_w"], w["layer_b"], w["att_src"], w["att_dst"] = lw, lb, asrc, adst
    rd = rng_for(WEIGHT_STREAM, 200, seed_extra)
    din = 2 * f + 4
    if dec_hidden > 0:
        w["dec_w1"] = _glorot(rd, dec_hidden, din)
        w["dec_b1"] = (rd.uniform(-1, 1, dec_hidden) * bias_scale).astype(np.float32)
        w["dec_w2"] = _glorot(rd, 1, dec_hidden)[0]
    else:
        w["dec_w1"] = np.zeros((0, din), np.float32)
        w["dec_b1"] = np.zeros(0, np.float32)
        w["dec_w2"] = _glorot(rd, 1, din)[0]
    w["dec_b2"] = np.array([rd.uniform(-1, 1) * bias_scale], np.float32)
    return w


def workload_inputs(name: str, n_cand: Optional[int] = None, first: int = 0):
    """(workload, topology, batch, slices, weights) for a named workload."""
    wl = WORKLOADS[name]
    topo = make_topology(name)
    batch = make_batch(name, topo, wl.batch if n_cand is None else n_cand, wl.f_op, first)
    masks, opts = make_slices(name, topo.n_dev, wl.n_slices)
    weights = make_weights(wl.f, wl.heads, wl.layers, wl.f_op, wl.f)
    return wl, topo, batch, (masks, opts), weights


# --------------------------------------------------------------------------
# search problems (op grouping, parameter sizes, slice tables)
# --------------------------------------------------------------------------

@dataclasses.dataclass
class SearchProblem:
    """Inputs of the strategy search over one joint graph: the topology, a
    contiguous op grouping (the paper groups ops before the search; the
    grouping here is given, not computed), per-op parameter bytes, the
    training batch's activation scale and the slice table the search picks
    from for every group."""
    name: str
    topo: Topology
    group_of: np.ndarray    # int32 [N] group id of every op
    n_groups: int
    op_params: np.ndarray   # float64 [N] parameter bytes of every op
    masks: np.ndarray       # uint64 [S]
    options: np.ndarray     # uint8 [S]


def make_search_problem(name: str, n_groups: Optional[int] = None) -> SearchProblem:
    """The workload's topology cut into `n_groups` contiguous groups (10 for
    tiny, 60 otherwise) with log-normal parameter sizes (seed (2302, cfg,
    3_000_000)) and the workload's slice table."""
    wl = WORKLOADS[name]
    topo = make_topology(name)
    k = n_groups if n_groups is not None else (10 if name == "tiny" else 60)
    n = topo.n_op
    bounds = [round(i * n / k) for i in range(k + 1)]
    group_of = np.empty(n, np.int32)
    for g in range(k):
        group_of[bounds[g]:bounds[g + 1]] = g
    rng = rng_for(wl.cfg_id, 3_000_000)
    params = rng.lognormal(math.log(2e4), 2.0, size=n)
    masks, opts = make_slices(name, topo.n_dev, wl.n_slices)
    return SearchProblem(name=name, topo=topo, group_of=group_of, n_groups=k,
                         op_params=params, masks=masks, options=opts)
