"""GPU-side helpers for the parity tests: upload seeded inputs, call the
library through its binding, and compare with the oracle candidate by
candidate.  (Imported only by tests marked gpu.)"""
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

    def check(self, E_op, E_dev, reps):
        tol = BF16_TOL if self.dtype == "bf16" else FP32_TOL
        worst = 0.0
        for r in reps:
            R_op, R_dev = self.oracle_forward(r)
            got = np.vstack([E_op[r].cpu().numpy(), E_dev[r].cpu().numpy()])
            err = row_rel_err(got, np.vstack([R_op, R_dev]))
            worst = max(worst, err)
            assert np.all(np.isfinite(got))
            assert err <= tol, f"candidate {r}: row-relative error {err:.3e} > {tol}"
        return worst


def decide_gap_ok(prior_row, best, delta_rel):
    """True when the oracle's top-two score gap exceeds delta (a unique winner)."""
    s = np.sort(np.log(np.maximum(prior_row, 1e-300)))[::-1]
    if len(s) < 2:
        return True
    return (s[0] - s[1]) > delta_rel * max(1.0, abs(best))
