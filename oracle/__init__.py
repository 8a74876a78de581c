"""Python access to the CPU reference oracle (``tag_oracle.c``).

TEST INFRASTRUCTURE ONLY.  The test suite, the package smoke check and the
benchmark's CPU-baseline leg may import this module; the GPU library and its
binding never do.  It shares no code with the GPU path: it takes numpy arrays
from the seeded generators and returns float64 results.
"""
from __future__ import annotations

import ctypes as C
import os
import subprocess
from typing import Dict, Optional, Tuple

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "tag_oracle.c")
_LIB = os.path.join(_HERE, "liboracle.so")

OK, EINVAL, ERANGE, EDUP, ESHAPE = 0, -1, -2, -3, -4


def build(force: bool = True) -> str:
    """Compile the oracle with gcc -O2 (no fast-math) into liboracle.so."""
    if force or not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
        tmp = _LIB + ".tmp"
        subprocess.check_call(["gcc", "-O2", "-std=c99", "-fPIC", "-shared", "-Wall",
                               "-o", tmp, _SRC, "-lm"])
        os.replace(tmp, _LIB)
    return _LIB


class _Dims(C.Structure):
    _fields_ = [("f", C.c_int32), ("heads", C.c_int32), ("layers", C.c_int32),
                ("f_op", C.c_int32), ("f_dev", C.c_int32), ("dec_hidden", C.c_int32),
                ("bf16", C.c_int32), ("gamma_same", C.c_double),
                ("gamma_cross", C.c_double), ("leaky_slope", C.c_double), ("sigma", C.c_int32),
                ("relations", C.c_int32), ("edge_act", C.c_int32), ("head_mode", C.c_int32)]


_FP = C.POINTER(C.c_float)


class _Weights(C.Structure):
    _fields_ = [("enc_op_w", _FP), ("enc_op_b", _FP), ("enc_dev_w", _FP), ("enc_dev_b", _FP),
                ("enc_edge_w", _FP * 3), ("enc_edge_b", _FP * 3),
                ("layer_w", _FP), ("layer_b", _FP), ("att_src", _FP), ("att_dst", _FP),
                ("dec_w1", _FP), ("dec_b1", _FP), ("dec_w2", _FP), ("dec_b2", _FP)]


_lib: Optional[C.CDLL] = None


def lib() -> C.CDLL:
    global _lib
    if _lib is None:
        alt = os.environ.get("TAG_ORACLE_LIBRARY")   # a sanitizer build of the same source
        if alt:
            _lib = C.CDLL(alt)
        else:
            if not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
                build(force=True)
            _lib = C.CDLL(_LIB)
        _lib.tago_round_bf16.restype = C.c_double
        _lib.tago_round_bf16.argtypes = [C.c_double]
    return _lib


def _p(a: np.ndarray, ct):
    return a.ctypes.data_as(C.POINTER(ct))


def _i32(a) -> np.ndarray:
    return np.ascontiguousarray(np.asarray(a, dtype=np.int32))


def _f32(a) -> np.ndarray:
    return np.ascontiguousarray(np.asarray(a, dtype=np.float32))


def round_bf16(x: float) -> float:
    return lib().tago_round_bf16(float(x))


def csr(n_op: int, n_dev: int, oo_src, oo_dst, dd_a, dd_b, od_op, od_dev
        ) -> Tuple[int, Optional[list]]:
    """Four destination buckets [(rowptr, col, eid)] for B0 op<-op, B1 op<-dev,
    B2 dev<-op, B3 dev<-dev, or (status, None) on rejection."""
    oo_src, oo_dst, dd_a, dd_b = _i32(oo_src), _i32(oo_dst), _i32(dd_a), _i32(dd_b)
    od_op, od_dev = _i32(od_op), _i32(od_dev)
    e_oo, e_dd, e_od = len(oo_src), len(dd_a), len(od_op)
    shapes = [(n_op, 2 * e_oo), (n_op, e_od), (n_dev, e_od), (n_dev, 2 * e_dd)]
    outs = [(np.zeros(max(r, 0) + 1, np.int32), np.zeros(max(n, 1), np.int32),
             np.zeros(max(n, 1), np.int32)) for r, n in shapes]
    args = []
    for rp, c, e in outs:
        args += [_p(rp, C.c_int32), _p(c, C.c_int32), _p(e, C.c_int32)]
    st = lib().tago_csr(C.c_int32(n_op), C.c_int32(n_dev),
                        C.c_int32(e_oo), _p(oo_src, C.c_int32), _p(oo_dst, C.c_int32),
                        C.c_int32(e_dd), _p(dd_a, C.c_int32), _p(dd_b, C.c_int32),
                        C.c_int32(e_od), _p(od_op, C.c_int32), _p(od_dev, C.c_int32), *args)
    if st != OK:
        return st, None
    return OK, [(rp, c[:n], e[:n]) for (rp, c, e), (_, n) in zip(outs, shapes)]


def _dims(f, heads, layers, f_op, f_dev, dec_hidden, bf16, gamma_same, gamma_cross, slope, sigma=0,
          relations=3, edge_act=0, head_mode=0):
    return _Dims(f, heads, layers, f_op, f_dev, dec_hidden, 1 if bf16 else 0,
                 gamma_same, gamma_cross, slope, sigma, relations, edge_act, head_mode)


def _weights(w: Dict[str, np.ndarray]):
    keep = {k: _f32(v) for k, v in w.items()}
    ws = _Weights()
    ws.enc_op_w, ws.enc_op_b = _p(keep["enc_op_w"], C.c_float), _p(keep["enc_op_b"], C.c_float)
    ws.enc_dev_w, ws.enc_dev_b = _p(keep["enc_dev_w"], C.c_float), _p(keep["enc_dev_b"], C.c_float)
    for r in range(3):
        ws.enc_edge_w[r] = _p(keep[f"enc_edge_w{r}"], C.c_float)
        ws.enc_edge_b[r] = _p(keep[f"enc_edge_b{r}"], C.c_float)
    ws.layer_w, ws.layer_b = _p(keep["layer_w"], C.c_float), _p(keep["layer_b"], C.c_float)
    ws.att_src, ws.att_dst = _p(keep["att_src"], C.c_float), _p(keep["att_dst"], C.c_float)
    ws.dec_w1, ws.dec_b1 = _p(keep["dec_w1"], C.c_float), _p(keep["dec_b1"], C.c_float)
    ws.dec_w2, ws.dec_b2 = _p(keep["dec_w2"], C.c_float), _p(keep["dec_b2"], C.c_float)
    return ws, keep


def forward(topo, x_op, x_dev, x_oo, x_dd, x_od, w: Dict[str, np.ndarray], *,
            f: int, heads: int, layers: int, bf16: bool = False,
            gamma_same: float = 1.0, gamma_cross: float = 0.1, leaky_slope: float = 0.2,
            want_alpha: bool = False, sigma: str = "relu", relations: int = 3,
            edge_act: str = "affine", heads_mode: str = "concat"):
    """E_op [N, f], E_dev [M, f] (float64) for one candidate graph; with
    want_alpha also the layer-0 attention weights [T, heads] in bucket order
    B0, B1, B2, B3 (each bucket in CSR order; three relations only).
    relations: 3 undirected link types or 5 directed relations (weights
    [L][5][...]); edge_act: "affine" or "relu" edge encoders; heads_mode:
    "concat" (K heads of f/K channels) or "avg" (K full-width heads averaged,
    att_src / att_dst [L][R][K][f])."""
    x_op, x_dev = _f32(x_op), _f32(x_dev)
    x_oo, x_dd = _f32(x_oo).reshape(-1), _f32(x_dd).reshape(-1)
    x_od = np.ascontiguousarray(np.asarray(x_od, dtype=np.uint8)).reshape(-1)
    n, m = topo.n_op, topo.n_dev
    if sigma not in ("relu", "elu") or relations not in (3, 5) or edge_act not in ("affine", "relu") \
            or heads_mode not in ("concat", "avg"):
        raise ValueError((sigma, relations, edge_act, heads_mode))
    if relations == 5:
        want_alpha = False
    dims = _dims(f, heads, layers, x_op.shape[1] if x_op.ndim == 2 else 0, 8,
                 0, bf16, gamma_same, gamma_cross, leaky_slope, 1 if sigma == "elu" else 0,
                 relations, 1 if edge_act == "relu" else 0, 1 if heads_mode == "avg" else 0)
    ws, keep = _weights(w)
    E_op = np.zeros((n, f), np.float64)
    E_dev = np.zeros((m, f), np.float64)
    T = 2 * topo.e_oo + 2 * topo.e_od + 2 * topo.e_dd
    alpha = np.zeros((max(T, 1), heads), np.float64) if want_alpha else None
    src, dst, a, b = _i32(topo.oo_src), _i32(topo.oo_dst), _i32(topo.dd_a), _i32(topo.dd_b)
    oop, odv = _i32(topo.od_op), _i32(topo.od_dev)
    st = lib().tago_forward(
        C.byref(dims), C.c_int32(n), C.c_int32(m),
        C.c_int32(topo.e_oo), _p(src, C.c_int32), _p(dst, C.c_int32),
        C.c_int32(topo.e_dd), _p(a, C.c_int32), _p(b, C.c_int32),
        C.c_int32(topo.e_od), _p(oop, C.c_int32), _p(odv, C.c_int32),
        _p(x_op, C.c_float), _p(x_dev, C.c_float), _p(x_oo, C.c_float),
        _p(x_dd, C.c_float), _p(x_od, C.c_uint8), C.byref(ws),
        _p(E_op, C.c_double), _p(E_dev, C.c_double),
        _p(alpha, C.c_double) if want_alpha else None)
    del keep
    if st != OK:
        raise RuntimeError(f"oracle forward failed with status {st}")
    if want_alpha:
        return E_op, E_dev, alpha[:T]
    return E_op, E_dev


def decide(E_op, E_dev, masks, options, query_op, w: Dict[str, np.ndarray], *,
           f: int, dec_hidden: int, n_dev: int, want_prior: bool = True):
    """Per query: argmax slice, best score, prior [Q, S] and the decoded
    decision (mask, replicas, option, sync, sfb)."""
    E_op = np.ascontiguousarray(E_op, np.float64)
    E_dev = np.ascontiguousarray(E_dev, np.float64)
    masks = np.ascontiguousarray(masks, np.uint64)
    options = np.ascontiguousarray(options, np.uint8)
    query_op = _i32(query_op)
    S, Q = len(masks), len(query_op)
    dims = _dims(f, 1, 0, 0, 8, dec_hidden, False, 1.0, 0.1, 0.2)
    ws, keep = _weights(w)
    am = np.zeros(max(Q, 1), np.int32)
    best = np.zeros(max(Q, 1), np.float64)
    prior = np.zeros((max(Q, 1), S), np.float64) if want_prior else None
    dm = np.zeros(max(Q, 1), np.uint64)
    dr, do, dsy, dsf = (np.zeros(max(Q, 1), np.int32) for _ in range(4))
    st = lib().tago_decide(
        C.byref(dims), C.c_int32(E_op.shape[0]), C.c_int32(n_dev),
        _p(E_op, C.c_double), _p(E_dev, C.c_double),
        C.c_int32(S), _p(masks, C.c_uint64), _p(options, C.c_uint8),
        C.c_int32(Q), _p(query_op, C.c_int32), C.byref(ws),
        _p(am, C.c_int32), _p(best, C.c_double),
        _p(prior, C.c_double) if want_prior else None,
        _p(dm, C.c_uint64), _p(dr, C.c_int32), _p(do, C.c_int32),
        _p(dsy, C.c_int32), _p(dsf, C.c_int32))
    del keep
    if st != OK:
        raise RuntimeError(f"oracle decide failed with status {st}")
    out = dict(argmax=am[:Q], best=best[:Q], mask=dm[:Q], replicas=dr[:Q],
               option=do[:Q], sync=dsy[:Q], sfb=dsf[:Q])
    if want_prior:
        out["prior"] = prior[:Q]
    return out
