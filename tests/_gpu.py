"""GPU-side helpers for the parity tests: upload seeded inputs, call the
library through its binding, and compare with the oracle candidate by
candidate.  (Imported only by tests marked gpu.)"""
from concurrent.futures import ThreadPoolExecutor

import numpy as np

import oracle
import paper_2302_06126_amd as P
import synth
from tests._helpers import row_rel_err

FP32_TOL = 1e-4
BF16_TOL = 2e-2


def dev_tensor(a, device="cuda"):
    import torch
    return torch.from_numpy(np.ascontiguousarray(a)).to(device)


def say(msg):
    print(msg, flush=True)


class Case:
    """R candidates sharing one topology (G = 1) with seeded features."""

    def __init__(self, topo, R, f, heads, layers, f_op=42, dtype="f32", dec_hidden=None, seed=0,
                 weights=None, batch=None, name=None):
        self.topo, self.R, self.f, self.heads, self.layers = topo, R, f, heads, layers
        self.f_op, self.dtype = f_op, dtype
        self.dec_hidden = f if dec_hidden is None else dec_hidden
        self.w = weights if weights is not None else synth.make_weights(
            f, heads, layers, f_op, self.dec_hidden, bias_scale=0.2, seed_extra=seed)
        if batch is None:
            batch = synth.make_batch(name or "cnn", topo, R, f_op, first=seed * 1000) if name else None
        if batch is None:
            feats = [self._rand_feats(seed * 100 + r) for r in range(R)]
            self.x_op = np.stack([x[0] for x in feats])
            self.x_dev = np.stack([x[1] for x in feats])
            self.x_oo = np.stack([x[2] for x in feats])
            self.x_dd = np.stack([x[3] for x in feats])
            self.x_od = np.stack([x[4] for x in feats])
        else:
            self.x_op, self.x_dev, self.x_dd, self.x_od = batch.x_op, batch.x_dev, batch.x_dd, batch.x_od
            self.x_oo = np.broadcast_to(batch.x_oo, (R,) + batch.x_oo.shape)
            self.shared_oo = batch.x_oo
        self.batch = batch

    def _rand_feats(self, s):
        rng = np.random.default_rng((2302, 77, s))
        t = self.topo
        return (rng.uniform(-1, 1, (t.n_op, self.f_op)).astype(np.float32),
                rng.uniform(-1, 1, (t.n_dev, 8)).astype(np.float32),
                rng.uniform(-1, 1, t.e_oo).astype(np.float32),
                rng.uniform(-1, 1, (t.e_dd, 2)).astype(np.float32),
                rng.integers(0, 2, t.e_od).astype(np.uint8))

    def model(self):
        return P.Model(self.w, f=self.f, heads=self.heads, layers=self.layers, f_op=self.f_op,
                       dec_hidden=self.dec_hidden, dtype=self.dtype)

    def gpu_forward(self, graph=None, model=None):
        import torch
        graph = graph or P.Graph([self.topo])
        model = model or self.model()
        x_oo = dev_tensor(self.shared_oo) if self.batch is not None else dev_tensor(self.x_oo)
        E_op, E_dev = P.forward(graph, model, dev_tensor(self.x_op), dev_tensor(self.x_dev), x_oo,
                                dev_tensor(self.x_dd), dev_tensor(self.x_od))
        torch.cuda.synchronize()
        return graph, model, E_op, E_dev

    def oracle_forward(self, r):
        return oracle.forward(self.topo, self.x_op[r], self.x_dev[r], self.x_oo[r], self.x_dd[r], self.x_od[r],
                              self.w, f=self.f, heads=self.heads, layers=self.layers, bf16=self.dtype == "bf16")

    def oracle_many(self, reps):
        """Oracle outputs of several candidates, computed in parallel threads
        (each call is single-threaded C that releases the interpreter lock)."""
        with ThreadPoolExecutor(max_workers=max(1, min(len(reps), 8))) as ex:
            return dict(zip(reps, ex.map(self.oracle_forward, reps)))

    def check(self, E_op, E_dev, reps, refs=None):
        tol = BF16_TOL if self.dtype == "bf16" else FP32_TOL
        refs = refs if refs is not None else self.oracle_many(list(reps))
        worst = 0.0
        for r in reps:
            R_op, R_dev = refs[r]
            got = np.vstack([E_op[r].cpu().numpy(), E_dev[r].cpu().numpy()])
            err = row_rel_err(got, np.vstack([R_op, R_dev]))
            worst = max(worst, err)
            assert np.all(np.isfinite(got))
            assert err <= tol, f"candidate {r}: row-relative error {err:.3e} > {tol}"
        return worst


def decide_gap_ok(prior_row, best, delta_rel):
    """True when the oracle's top-two score gap exceeds delta (a unique winner)."""
    return top_gap(prior_row) > delta_rel * max(1.0, abs(best))


def top_gap(prior_row):
    """The oracle's gap between its best and second-best score (from the
    priors: log p_a - log p_b = s_a - s_b)."""
    s = np.sort(np.log(np.maximum(prior_row, 1e-300)))[::-1]
    return np.inf if len(s) < 2 else float(s[0] - s[1])


def score_error_bound(w, f, H, E_op, E_dev, masks, query_op, n_dev, emb_err):
    """Per query, a bound on how far any slice's decoder score can move when
    every embedding row x moves by at most emb_err * ||x||_inf (the measured
    row-relative error of the forward pass).  The decoder input is
    [sum_j mask_j E_dev[j] ; E_op[i] ; onehot], the first layer is linear and
    ReLU is 1-Lipschitz, so
      |d score| <= sum_h |w2_h| (sum_{c<f} |W1_hc| D_a + sum_c |W1_h,f+c| ||E_op[i]||) emb_err
    with D_a = sum_{j in mask a} ||E_dev[j]||_inf (H = 0: |w2| in place of
    the sum over h); row norms are floored as in the error measure (1e-6 of
    the largest).  Two scores move by at most twice the largest bound."""
    w1 = np.abs(np.asarray(w["dec_w1"], np.float64))
    w2 = np.abs(np.asarray(w["dec_w2"], np.float64))
    if H > 0:
        alpha = float(w2 @ w1[:, :f].sum(axis=1))
        beta = float(w2 @ w1[:, f:2 * f].sum(axis=1))
    else:
        alpha, beta = float(w2[:f].sum()), float(w2[f:2 * f].sum())
    dev_n = np.abs(np.asarray(E_dev, np.float64)).max(axis=1)
    all_op = np.abs(np.asarray(E_op, np.float64)).max(axis=1)
    floor = 1e-6 * max(float(dev_n.max(initial=0.0)), float(all_op.max(initial=0.0)))
    dev_n = np.maximum(dev_n, floor)
    bits = ((np.asarray(masks, np.uint64)[:, None] >> np.arange(n_dev, dtype=np.uint64)) & np.uint64(1)).astype(bool)
    d_max = float((bits * dev_n[None, :]).sum(axis=1).max())
    op_n = np.maximum(all_op[np.asarray(query_op)], floor)
    return emb_err * (alpha * d_max + beta * op_n)
