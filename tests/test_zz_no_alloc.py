"""The allocation-free decision head (tag_gnn_decide_noalloc) against the
workspace entry point (tag_gnn_decide) through the C ABI: the same kernels
on the same inputs, so every output must be identical.  Two calls in a row,
the second on a smaller problem (the static scratch keeps the first call's
contents), and the size limit rejected on the host."""
import ctypes as C

import numpy as np
import pytest

import synth

pytestmark = pytest.mark.gpu

P = pytest.importorskip("paper_2302_06126_amd")


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    P._abi.load()
    torch.cuda.set_device(0)
    yield
    torch.cuda.synchronize()


def _problem(seed, n_op, n_dev, R, f, H, S, Q):
    import torch
    rng = np.random.default_rng((2302, 91, seed))
    topo = synth.random_topology(300 + seed, n_op, n_dev, 2 * n_op)
    w = synth.make_weights(f, 4, 1, 42, H, bias_scale=0.5, seed_extra=seed)
    g = P.Graph([topo])
    m = P.Model(w, f=f, heads=4, layers=1, f_op=42, dec_hidden=H)
    dev = torch.device("cuda")
    t = lambda a: torch.from_numpy(np.ascontiguousarray(a)).to(dev)
    E_op = t(rng.uniform(0, 1, (R, n_op, f)).astype(np.float32))
    E_dev = t(rng.uniform(0, 1, (R, n_dev, f)).astype(np.float32))
    masks, opts = synth.make_slices("cnn", n_dev, S)
    q_rep = rng.integers(0, R, Q).astype(np.int32)
    q_op = rng.integers(0, n_op, Q).astype(np.int32)
    q_rep[-1] = R   # one invalid query: argmax -1, NaN score
    return dict(g=g, m=m, R=R, E_op=E_op, E_dev=E_dev, masks=t(masks.view(np.int64)), opts=t(opts), S=S, Q=Q,
                q=[t(q_rep), t(np.zeros(Q, np.int32)), t(q_op)])


def _outputs(pb):
    import torch
    Q, S = pb["Q"], pb["S"]
    return dict(argmax=torch.full((Q,), -7, dtype=torch.int32, device="cuda"),
                best=torch.full((Q,), 7.0, dtype=torch.float32, device="cuda"),
                prior=torch.full((Q, S), 7.0, dtype=torch.float32, device="cuda"),
                dec=torch.full((Q, C.sizeof(P.tag_decision)), 7, dtype=torch.uint8, device="cuda"))


def _call(pb, noalloc):
    import torch
    lib = P._abi.load()
    out = _outputs(pb)
    sl = P.tag_slices(pb["S"], pb["masks"].data_ptr(), pb["opts"].data_ptr())
    sh = int(torch.cuda.current_stream().cuda_stream)
    common = (pb["g"].handle, C.byref(pb["m"].dims), C.byref(pb["m"].weights), pb["R"], pb["E_op"].data_ptr(),
              pb["E_dev"].data_ptr(), C.byref(sl), pb["Q"], pb["q"][0].data_ptr(), pb["q"][1].data_ptr(),
              pb["q"][2].data_ptr(), out["argmax"].data_ptr(), out["best"].data_ptr(), out["prior"].data_ptr(),
              out["dec"].data_ptr())
    if noalloc:
        st = lib.tag_gnn_decide_noalloc(*common, sh)
    else:
        b = C.c_size_t(0)
        P._abi.check(lib.tag_gnn_decide_workspace(pb["g"].handle, C.byref(pb["m"].dims), pb["R"], pb["S"], pb["Q"],
                                                  C.byref(b)), "workspace")
        ws = torch.empty(b.value, dtype=torch.uint8, device="cuda")
        st = lib.tag_gnn_decide(*common, ws.data_ptr(), b.value, sh)
        torch.cuda.synchronize()
        del ws
    P._abi.check(st, "decide")
    torch.cuda.synchronize()
    return {k: v.cpu().numpy() for k, v in out.items()}


def _same(a, b):
    for k in a:
        assert np.array_equal(a[k], b[k], equal_nan=(k != "dec")) if a[k].dtype.kind == "f" else \
            np.array_equal(a[k], b[k]), k


def test_noalloc_matches_workspace_entry_point_twice():
    big = _problem(1, 300, 16, 8, 128, 128, 256, 200)
    small = _problem(2, 40, 5, 2, 64, 32, 17, 9)
    print("noalloc: big problem (R=8, N=300, M=16, f=128, H=128, S=256, Q=200)", flush=True)
    a = _call(big, noalloc=True)
    _same(a, _call(big, noalloc=False))
    assert a["argmax"][-1] == -1 and np.isnan(a["best"][-1])
    assert np.all(a["argmax"][:-1] >= 0)
    print("noalloc: second, smaller problem (R=2, N=40, M=5, f=64, H=32, S=17, Q=9)", flush=True)
    b = _call(small, noalloc=True)
    _same(b, _call(small, noalloc=False))
    assert np.all(b["argmax"][:-1] >= 0)


def test_noalloc_rejects_problems_beyond_its_scratch():
    import torch
    lib = P._abi.load()
    limit = lib.tag_gnn_decide_noalloc_max_bytes()
    assert limit == 64 << 20
    # slice terms alone: R * H * S * 4 bytes > 64 MiB
    pb = _problem(3, 20, 4, 64, 256, 1024, 300, 4)
    b = C.c_size_t(0)
    P._abi.check(lib.tag_gnn_decide_workspace(pb["g"].handle, C.byref(pb["m"].dims), pb["R"], pb["S"], pb["Q"],
                                              C.byref(b)), "workspace")
    assert b.value > limit
    out = _outputs(pb)
    sl = P.tag_slices(pb["S"], pb["masks"].data_ptr(), pb["opts"].data_ptr())
    st = lib.tag_gnn_decide_noalloc(pb["g"].handle, C.byref(pb["m"].dims), C.byref(pb["m"].weights), pb["R"],
                                    pb["E_op"].data_ptr(), pb["E_dev"].data_ptr(), C.byref(sl), pb["Q"],
                                    pb["q"][0].data_ptr(), pb["q"][1].data_ptr(), pb["q"][2].data_ptr(),
                                    out["argmax"].data_ptr(), out["best"].data_ptr(), out["prior"].data_ptr(),
                                    out["dec"].data_ptr(), int(torch.cuda.current_stream().cuda_stream))
    assert st == P._abi.TAG_ENOSPACE
    assert "static decide scratch" in P.tag_last_error()
    torch.cuda.synchronize()
    assert np.all(out["argmax"].cpu().numpy() == -7)   # nothing was enqueued
