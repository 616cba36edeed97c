"""The scatter-add entry point that allocates nothing
(polyglot_scatter_add_noalloc), called through the C ABI, against the
context entry point it is a variant of (polyglot_scatter_add, sorted mode):
two calls in a row, the second with a smaller input, then a call with an
out-of-range index and a clean call after it."""
import ctypes

import numpy as np
import pytest

import oracle
import workloads

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


def _inputs(seed, rows, d, N, s):
    rng = np.random.default_rng(seed)
    t0 = rng.normal(0, 0.01, (rows, d)).astype(np.float32)
    idx = workloads.zipf_ids(rng, rows, s, N)
    Y = rng.normal(0, 1e-3, (N, d)).astype(np.float32)
    return t0, idx, Y


def _bound(t0, idx, Y, alpha):
    cnt = np.bincount(idx, minlength=t0.shape[0]).astype(np.float64)[:, None] + 1.0
    mag = np.abs(t0.astype(np.float64))
    np.add.at(mag, idx, np.abs(alpha * Y.astype(np.float64)))
    return cnt * 2.0 ** -24 * mag + 1e-30


def test_noalloc_scatter_add_equals_context_scatter_add():
    import paper_1404_1521_amd as pg
    lib = pg.load_library()
    rows, d = 100_000, 64
    ctx = pg.Context(1000, 16, 5, 8, max_batch=1, max_scatter=pg.NOALLOC_MAX_N, max_rows=rows)
    status = torch.full((1,), 123, dtype=torch.int32, device="cuda")
    stream = torch.cuda.current_stream()
    for call, (N, s, alpha) in enumerate([(pg.NOALLOC_MAX_N, 1.2, 0.75), (3001, 1.0, -1.5)]):
        t0, idx, Y = _inputs(100 + call, rows, d, N, s)
        ta, tb = torch.from_numpy(t0).cuda(), torch.from_numpy(t0).cuda()
        di, dY = torch.from_numpy(idx).cuda(), torch.from_numpy(Y).cuda()
        rc = lib.polyglot_scatter_add_noalloc(
            ctypes.c_void_p(ta.data_ptr()), rows, d, ctypes.c_void_p(di.data_ptr()),
            ctypes.c_void_p(dY.data_ptr()), N, ctypes.c_float(alpha),
            ctypes.c_void_p(status.data_ptr()), ctypes.c_void_p(stream.cuda_stream))
        assert rc == pg.OK
        ctx.scatter_add(tb, di, dY, alpha, pg.SCATTER_SORTED)
        torch.cuda.synchronize()
        assert int(status.cpu()[0]) == pg.OK
        assert ctx.status() == pg.OK
        ga, gb = ta.cpu().numpy(), tb.cpu().numpy()
        assert np.array_equal(ga, gb), call  # same kernels, same order: bit-identical
        ref = t0.copy()
        oracle.scatter_add(ref, idx, Y, alpha)
        err = np.abs(ga.astype(np.float64) - ref.astype(np.float64))
        assert np.all(err <= _bound(t0, idx, Y, alpha)), call
    # an out-of-range index: the table is left untouched, the status says EID
    t0, idx, Y = _inputs(7, rows, d, 500, 1.1)
    idx[250] = rows
    ta = torch.from_numpy(t0).cuda()
    di, dY = torch.from_numpy(idx).cuda(), torch.from_numpy(Y).cuda()
    pg.scatter_add_noalloc(ta, di, dY, 1.0, status)
    torch.cuda.synchronize()
    assert int(status.cpu()[0]) == pg.EID
    assert np.array_equal(ta.cpu().numpy(), t0)
    # nothing is sticky: the next valid call applies and reports OK
    idx[250] = 3
    di = torch.from_numpy(idx).cuda()
    pg.scatter_add_noalloc(ta, di, dY, 1.0, status)
    torch.cuda.synchronize()
    assert int(status.cpu()[0]) == pg.OK
    ref = t0.copy()
    oracle.scatter_add(ref, idx, Y, 1.0)
    got = ta.cpu().numpy()
    assert np.all(np.abs(got.astype(np.float64) - ref) <= _bound(t0, idx, Y, 1.0))
    # host-side limits: nothing enqueued
    for N, rws, dd, code in ((pg.NOALLOC_MAX_N + 1, rows, d, pg.EBATCH), (0, rows, d, pg.EBATCH),
                             (10, rows, 6, pg.EINVAL), (10, (1 << 26) + 1, d, pg.EINVAL)):
        rc = lib.polyglot_scatter_add_noalloc(
            ctypes.c_void_p(ta.data_ptr()), rws, dd, ctypes.c_void_p(di.data_ptr()),
            ctypes.c_void_p(dY.data_ptr()), N, ctypes.c_float(1.0), None,
            ctypes.c_void_p(stream.cuda_stream))
        assert rc == code, (N, rws, dd)
    assert lib.polyglot_scatter_add_noalloc(None, rows, d, None, None, 10, ctypes.c_float(1.0),
                                            None, None) == pg.ENULL
    torch.cuda.synchronize()
    assert np.array_equal(ta.cpu().numpy(), got)
