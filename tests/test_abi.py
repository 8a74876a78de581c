"""Host-side checks of the C ABI that need no GPU: the library loads, exports
every symbol include/tag.h declares, and rejects bad arguments before
touching the device."""
import ctypes as C
import os
import re

import numpy as np
import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _declared():
    import glob
    src = "".join(open(h).read() for h in sorted(glob.glob(os.path.join(ROOT, "include", "*.h"))))
    return sorted(set(re.findall(r"^\s*(?:tag_status|void|size_t|const char \*)\s*\*?\s*(tag_\w+)\s*\(", src, re.M)))


@pytest.fixture(scope="module")
def P():
    import paper_2302_06126_amd as pkg
    pkg._abi.load()
    return pkg


def test_exports_every_declared_symbol(P):
    lib = P._abi.load()
    names = _declared()
    assert len(names) >= 13
    for n in names:
        assert hasattr(lib, n), n
    assert set(names) == set(P._abi.EXPORTS) | set(P._abi.SEARCH_EXPORTS) | set(P._abi.TRAIN_EXPORTS)
    assert "gfx950" in P.tag_version()


def _desc(P, n_op, n_dev, oo_off=(0, 0), dd_off=(0, 0), od_off=(0, 0)):
    keep = [np.asarray(n_op, np.int32), np.asarray(n_dev, np.int32), np.asarray(oo_off, np.int64),
            np.asarray(dd_off, np.int64), np.asarray(od_off, np.int64)]
    d = P.tag_graph_desc()
    d.n_graphs = len(keep[0])
    d.n_op = keep[0].ctypes.data_as(C.POINTER(C.c_int32))
    d.n_dev = keep[1].ctypes.data_as(C.POINTER(C.c_int32))
    d.oo_off = keep[2].ctypes.data_as(C.POINTER(C.c_int64))
    d.dd_off = keep[3].ctypes.data_as(C.POINTER(C.c_int64))
    d.od_off = keep[4].ctypes.data_as(C.POINTER(C.c_int64))
    return d, keep


def test_plan_sizes_and_validation(P):
    d, keep = _desc(P, [10, 3], [4, 2], oo_off=(0, 5, 7), dd_off=(0, 6, 7), od_off=(0, 40, 46))
    d.oo_src = d.oo_dst = d.dd_a = d.dd_b = d.od_op = d.od_dev = 256  # never dereferenced by plan
    st, cb, tb = P.tag_graph_plan(d)
    assert st == 0 and cb > 0 and tb > 0
    bad = [
        (dict(n_dev=[65]), -4), (dict(n_dev=[0]), -1), (dict(n_op=[0]), -1),
        (dict(oo_off=(1, 2)), -1), (dict(od_off=(0, -1)), -1),
    ]
    for kw, status in bad:
        args = dict(n_op=[5], n_dev=[2])
        args.update(kw)
        d, keep = _desc(P, **args)
        d.oo_src = d.oo_dst = d.dd_a = d.dd_b = d.od_op = d.od_dev = 256
        st, _, _ = P.tag_graph_plan(d)
        assert st == status, (kw, st, P.tag_last_error())
        assert P.tag_last_error()
    # positive counts need edge arrays
    d, keep = _desc(P, [5], [2], oo_off=(0, 3))
    st, _, _ = P.tag_graph_plan(d)
    assert st == -1


def test_build_rejects_before_launch(P):
    d, keep = _desc(P, [5], [2])
    out = C.c_void_p(None)
    lib = P._abi.load()
    assert lib.tag_graph_build(None, None, 0, None, 0, None, C.byref(out)) == -1
    assert lib.tag_graph_build(C.byref(d), None, 0, None, 0, None, C.byref(out)) == -1
    assert lib.tag_graph_build(C.byref(d), 256, 1, 256, 1, None, C.byref(out)) == -5
    assert out.value is None


def test_forward_and_decide_reject_null_arguments(P):
    lib = P._abi.load()
    dims = P.tag_model_dims(64, 4, 2, 40, 8, 64, 0, 1.0, 0.1, 0.2)
    b = C.c_size_t(0)
    assert lib.tag_gnn_workspace(None, C.byref(dims), 1, C.byref(b)) == -1
    assert lib.tag_gnn_forward(None, C.byref(dims), None, None, None, 0, None, None, None) == -1
    assert lib.tag_gnn_decide_workspace(None, C.byref(dims), 1, 1, 1, C.byref(b)) == -1
    assert lib.tag_graph_get_info(None, None) == -1
    assert lib.tag_graph_export(None, 0, None, None, None) == -1
    lib.tag_graph_destroy(None)


def test_missing_library_fails_loudly(tmp_path, monkeypatch):
    import paper_2302_06126_amd._abi as abi
    monkeypatch.setattr(abi, "_lib", None)
    monkeypatch.setattr(abi, "LIB_PATH", str(tmp_path / "libtag.so"))
    with pytest.raises(RuntimeError, match="missing"):
        abi.load()
