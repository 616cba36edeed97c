"""Pins of the CPU oracle against what the model definition fixes.

The paper prints no model outputs, so the oracle is pinned by hand-derived
closed forms (tests/golden/worked_examples.json), central finite differences
of its own loss, library routines (numpy.add.at, numpy fancy indexing,
numpy.unique, torch autograd) and invariants that hold exactly.
"""
import json
import math
import os

import numpy as np
import pytest

import oracle
import workloads

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "worked_examples.json")


def golden(name):
    with open(GOLDEN) as f:
        return json.load(f)[name]


def params_from(g, dtype=np.float64):
    return {k: np.array(g[k], dtype=dtype).reshape(-1 if k in ("b1", "w2", "b2") else
                                                    (len(g[k]), -1))
            for k in ("E", "W1", "b1", "w2", "b2")}


def ids_from(g):
    return np.array(g["windows"], np.int32), np.array(g["corrupt"], np.int32)


def rand_params(rng, V, d, win, H, std=0.5):
    return {"E": rng.normal(0, std, (V, d)), "W1": rng.normal(0, std, (H, win * d)),
            "b1": rng.normal(0, std, H), "w2": rng.normal(0, std, H),
            "b2": rng.normal(0, std, 1)}


def copy(p):
    return {k: v.copy() for k, v in p.items()}


# ---------------------------------------------------------------- closed forms

def test_w1_closed_form_loss_and_gradients():
    g = golden("W1")
    p = params_from(g)
    w, c = ids_from(g)
    ex = g["expect"]
    # closed forms re-evaluated here, and the stored numbers
    assert ex["loss"] == pytest.approx(1 - 2 * math.tanh(0.5), abs=1e-15)
    L, gr = oracle.gradients(p, w, c)
    assert L == pytest.approx(ex["loss"], abs=1e-14)
    np.testing.assert_allclose(gr["w2"], ex["dw2"], atol=1e-14)
    np.testing.assert_allclose(gr["W1"], ex["dW1"], atol=1e-14)
    np.testing.assert_allclose(gr["b1"], ex["db1"], atol=1e-14)
    np.testing.assert_allclose(gr["b2"], ex["db2"], atol=1e-14)
    np.testing.assert_allclose(gr["E"], ex["dE"], atol=1e-14)
    assert gr["E"][0, 0] == 0.0  # the two context contributions cancel exactly
    np.testing.assert_allclose(oracle.score(p, w), [ex["s"]], atol=1e-15)


def test_w1_closed_form_step():
    g = golden("W1")
    p = params_from(g)
    w, c = ids_from(g)
    L = oracle.train_step(p, w, c, g["lr"])
    ex = g["expect"]
    assert L == pytest.approx(ex["loss"], abs=1e-14)
    for k, v in ex["after_step"].items():
        np.testing.assert_allclose(p[k].reshape(np.array(v).shape), v, atol=1e-13, err_msg=k)


@pytest.mark.parametrize("name", ["W1_margin_met", "W1_margin_zero"])
def test_margin_not_positive_leaves_everything_bit_identical(name):
    g = golden(name)
    for dtype in (np.float64, np.float32):
        p = params_from(g, dtype)
        before = copy(p)
        w, c = ids_from(g)
        L = oracle.train_step(p, w, c, g["lr"])
        assert L == 0.0
        for k in p:
            assert np.array_equal(p[k], before[k]), k


def test_l2_layout_closed_form():
    g = golden("L2")
    p = params_from(g)
    w, c = ids_from(g)
    ex = g["expect"]
    assert ex["s"] == pytest.approx(0.3 + 2 * math.tanh(0.75) + math.tanh(1.1), abs=1e-15)
    np.testing.assert_allclose(oracle.score(p, w), [ex["s"]], atol=1e-14)
    # the corrupted window's score, through a window that holds the corrupt id
    wc = w.copy()
    wc[0, 1] = c[0]
    np.testing.assert_allclose(oracle.score(p, wc), [ex["s_corrupt"]], atol=1e-14)
    assert oracle.loss(p, w, c) == pytest.approx(ex["loss"], abs=1e-14)


def test_scatter_w2_duplicates_accumulate():
    g = golden("W2_scatter")
    for dtype in (np.float64, np.float32):
        t = np.array(g["table"], dtype)
        oracle.scatter_add(t, np.array(g["idx"], np.int32), np.array(g["Y"], dtype), g["alpha"])
        np.testing.assert_array_equal(t, np.array(g["expect"]["table"], dtype))


# ------------------------------------------------------- finite differences

def _fd_setup(seed, V=7, d=3, win=3, H=4, B=5, std=0.5):
    rng = np.random.default_rng(seed)
    while True:
        p = rand_params(rng, V, d, win, H, std)
        w = rng.integers(0, V, (B, win)).astype(np.int32)
        c = rng.integers(0, V, B).astype(np.int32)
        # keep every margin away from the hinge kink so the loss is smooth there
        s = oracle.score(p, w)
        wc = w.copy()
        wc[:, win // 2] = c
        st = oracle.score(p, wc)
        m = 1 - s + st
        if np.all(np.abs(m) > 1e-3) and np.any(m > 0):
            return p, w, c


@pytest.mark.parametrize("seed", [0, 1, 2, 3])
def test_gradients_match_central_differences(seed):
    p, w, c = _fd_setup(seed)
    _, g = oracle.gradients(p, w, c)
    eps = 1e-6
    for k in p:
        flat = p[k].reshape(-1)
        fd = np.empty_like(flat)
        for i in range(flat.size):
            old = flat[i]
            flat[i] = old + eps
            lp = oracle.loss(p, w, c)
            flat[i] = old - eps
            lm = oracle.loss(p, w, c)
            flat[i] = old
            fd[i] = (lp - lm) / (2 * eps)
        an = g[k].reshape(-1)
        err = np.abs(fd - an)
        assert np.all(err <= 1e-7 + 1e-6 * np.abs(an)), (k, np.max(err))


def test_gradients_fd_with_duplicates_in_window_and_corrupt():
    # ids repeated inside a window and the corrupt id equal to a context id
    rng = np.random.default_rng(11)
    p = rand_params(rng, 4, 2, 5, 3)
    w = np.array([[1, 1, 2, 1, 3], [0, 2, 2, 0, 0], [3, 3, 3, 3, 3]], np.int32)
    c = np.array([1, 0, 2], np.int32)
    _, g = oracle.gradients(p, w, c)
    eps = 1e-6
    flat = p["E"].reshape(-1)
    for i in range(flat.size):
        old = flat[i]
        flat[i] = old + eps
        lp = oracle.loss(p, w, c)
        flat[i] = old - eps
        lm = oracle.loss(p, w, c)
        flat[i] = old
        fd = (lp - lm) / (2 * eps)
        assert abs(fd - g["E"].reshape(-1)[i]) <= 1e-7 + 1e-6 * abs(fd)


def test_step_is_sgd_on_the_fd_gradient():
    p, w, c = _fd_setup(5)
    _, g = oracle.gradients(p, w, c)
    q = copy(p)
    lr = 0.37
    oracle.train_step(q, w, c, lr)
    for k in p:
        # the step's update equals lr times the gradient taken at the pre-step params
        np.testing.assert_allclose((p[k] - q[k]) / lr, g[k], atol=1e-12, err_msg=k)


def test_torch_autograd_cross_check():
    torch = pytest.importorskip("torch")
    rng = np.random.default_rng(21)
    V, d, win, H, B = 9, 4, 5, 6, 8
    p = rand_params(rng, V, d, win, H)
    w = rng.integers(0, V, (B, win)).astype(np.int32)
    c = rng.integers(0, V, B).astype(np.int32)
    L, g = oracle.gradients(p, w, c)
    tp = {k: torch.tensor(v, dtype=torch.float64, requires_grad=True) for k, v in p.items()}
    tw = torch.tensor(w, dtype=torch.long)
    tc = torch.tensor(c, dtype=torch.long)
    x = tp["E"][tw].reshape(B, -1)
    wt = tw.clone()
    wt[:, win // 2] = tc
    xt = tp["E"][wt].reshape(B, -1)

    def s(v):
        return torch.tanh(v @ tp["W1"].T + tp["b1"]) @ tp["w2"] + tp["b2"][0]

    loss = torch.relu(1 - s(x) + s(xt)).mean()
    loss.backward()
    assert L == pytest.approx(loss.item(), abs=1e-14)
    for k in p:
        np.testing.assert_allclose(g[k], tp[k].grad.numpy(), atol=1e-14, err_msg=k)


# ---------------------------------------------------------------- invariants

def _tiny_f32(seed=0, B=32):
    w = workloads.PRESETS["tiny"]
    p = workloads.init_params(w, seed=seed)
    win, cor = workloads.batch(w, 0, B)
    return w, p, win, cor


def test_untouched_rows_bit_identical_and_b2_constant():
    w, p, win, cor = _tiny_f32()
    before = copy(p)
    oracle.train_step(p, win, cor, 0.5)
    touched = np.zeros(w.V, bool)
    touched[win.reshape(-1)] = True
    touched[cor] = True
    assert np.array_equal(p["E"][~touched], before["E"][~touched])
    assert not np.array_equal(p["E"][touched], before["E"][touched])
    assert np.array_equal(p["b2"], before["b2"])


def test_all_margins_met_no_change():
    # H=1, d=1: s = 10 tanh(10 e_c), centre row +1, corrupt row -1 -> margin = 1 - 20 tanh(10) < 0
    E = np.array([[1.0], [-1.0], [0.3]])
    p = {"E": E, "W1": np.array([[0.7, 10.0, -0.2]]), "b1": np.zeros(1), "w2": np.array([10.0]),
         "b2": np.array([0.1])}
    w = np.array([[2, 0, 2], [0, 0, 1], [1, 0, 0], [2, 0, 0]], np.int32)
    c = np.array([1, 1, 1, 1], np.int32)
    before = copy(p)
    assert oracle.train_step(p, w, c, 1.0) == 0.0
    for k in p:
        assert np.array_equal(p[k], before[k])


def test_corrupt_equal_centre_gives_zero_gradient_exactly():
    rng = np.random.default_rng(3)
    p = rand_params(rng, 12, 3, 5, 4)
    w = rng.integers(0, 12, (6, 5)).astype(np.int32)
    c = w[:, 2].copy()
    L, g = oracle.gradients(p, w, c)
    assert L == 1.0
    for k in g:
        assert not np.any(g[k]), k
    for dtype in (np.float64, np.float32):
        q = {k: v.astype(dtype) for k, v in p.items()}
        before = copy(q)
        oracle.train_step(q, w, c, 0.3)
        for k in q:
            assert np.array_equal(q[k], before[k])


def test_lr_zero_is_identity():
    w, p, win, cor = _tiny_f32(1)
    before = copy(p)
    oracle.train_step(p, win, cor, 0.0)
    for k in p:
        assert np.array_equal(p[k], before[k])


def test_batch_mean_duplication_and_permutation_invariance():
    rng = np.random.default_rng(4)
    p = rand_params(rng, 10, 3, 5, 4)
    w = rng.integers(0, 10, (7, 5)).astype(np.int32)
    c = rng.integers(0, 10, 7).astype(np.int32)
    L, g = oracle.gradients(p, w, c)
    L2, g2 = oracle.gradients(p, np.concatenate([w, w]), np.concatenate([c, c]))
    perm = rng.permutation(7)
    L3, g3 = oracle.gradients(p, w[perm].copy(), c[perm].copy())
    assert L2 == pytest.approx(L, rel=1e-13) and L3 == pytest.approx(L, rel=1e-13)
    for k in g:
        np.testing.assert_allclose(g2[k], g[k], rtol=1e-12, atol=1e-15)
        np.testing.assert_allclose(g3[k], g[k], rtol=1e-12, atol=1e-15)


# ------------------------------------------------------ library routines

def test_scatter_add_equals_numpy_add_at():
    rng = np.random.default_rng(5)
    rows, d, N = 50, 7, 400
    idx = workloads.zipf_ids(rng, rows, 1.2, N)
    Y = rng.normal(0, 1, (N, d))
    t0 = rng.normal(0, 1, (rows, d))
    t = t0.copy()
    oracle.scatter_add(t, idx, Y, 0.75)
    ref = t0.copy()
    np.add.at(ref, idx, 0.75 * Y)
    assert np.array_equal(t, ref)  # same order, same float64 operations
    # float32 storage: the float64 result rounded once
    t32 = t0.astype(np.float32)
    Y32 = Y.astype(np.float32)
    oracle.scatter_add(t32, idx, Y32, 0.75)
    ref = t0.astype(np.float32).astype(np.float64)
    np.add.at(ref, idx, 0.75 * Y32.astype(np.float64))
    assert np.array_equal(t32, ref.astype(np.float32))


def test_gather_equals_fancy_indexing():
    w = workloads.PRESETS["tiny"]
    p = workloads.init_params(w)
    win, cor = workloads.batch(w, 3, 40)
    X, Xc = oracle.gather(p["E"], win, cor)
    assert np.array_equal(X, p["E"][win].reshape(40, -1))
    assert np.array_equal(Xc, p["E"][cor])


def test_touched_rows_equals_unique():
    w = workloads.PRESETS["tiny"]
    win, cor = workloads.batch(w, 7, 64)
    assert np.array_equal(oracle.touched_rows(w.V, win, cor),
                          np.unique(np.concatenate([win.reshape(-1), cor])))


def test_f32_storage_step_close_to_f64_step():
    w, p, win, cor = _tiny_f32(2)
    p64 = {k: v.astype(np.float64) for k, v in p.items()}
    L32 = oracle.train_step(p, win, cor, 0.5)
    L64 = oracle.train_step(p64, win, cor, 0.5)
    assert L32 == pytest.approx(L64, rel=1e-7)
    for k in p:
        np.testing.assert_allclose(p[k], p64[k], rtol=1e-6, atol=1e-9)


# ---------------------------------------------------------------- errors

def test_error_codes_leave_params_untouched():
    w, p, win, cor = _tiny_f32(3)
    before = copy(p)
    bad = win.copy()
    bad[3, 1] = w.V
    with pytest.raises(oracle.OracleError) as e:
        oracle.train_step(p, bad, cor, 0.1)
    assert e.value.rc == oracle.EID
    badc = cor.copy()
    badc[0] = -1
    with pytest.raises(oracle.OracleError) as e:
        oracle.train_step(p, win, badc, 0.1)
    assert e.value.rc == oracle.EID
    with pytest.raises(oracle.OracleError) as e:
        oracle.train_step(p, win, cor, float("nan"))
    assert e.value.rc == oracle.EINVAL
    with pytest.raises(oracle.OracleError) as e:
        oracle.train_step(p, win[:, :4].copy(), cor, 0.1)  # even window
    assert e.value.rc == oracle.EINVAL
    for k in p:
        assert np.array_equal(p[k], before[k])


def test_zipf_generator_head_mass():
    rng = np.random.default_rng(0)
    V, s = 1000, 1.0
    ids = workloads.zipf_ids(rng, V, s, 200_000)
    assert ids.min() >= 0 and ids.max() < V
    hv = np.sum(1.0 / np.arange(1, V + 1))
    assert np.mean(ids == 0) == pytest.approx(1 / hv, rel=0.03)
    assert np.mean(ids == 1) == pytest.approx(0.5 / hv, rel=0.05)


# ------------------------------------------- the general advanced-indexing op

def _probe_doubles(rng, n):
    """Doubles over the interesting ranges of the 16-bit formats: normal,
    subnormal, near overflow, exact halfway points, both signs."""
    x = np.concatenate([
        rng.standard_normal(n) * 10.0 ** rng.uniform(-9, 5, n),
        np.ldexp(rng.integers(1, 2048, n).astype(np.float64) + 0.5, -24),  # fp16 halfway points
        np.ldexp(rng.integers(256, 512, n).astype(np.float64) + 0.5, rng.integers(-20, 20, n) - 8),
        [0.0, -0.0, 65504.0, 65519.99, 65520.0, 2.0 ** -24, 2.0 ** -25, 3 * 2.0 ** -26, 1e300],
    ])
    return x * np.where(rng.random(x.size) < 0.5, -1.0, 1.0)


def test_f16_rounding_matches_numpy():
    """binary16 encoding is numpy's float64 -> float16 cast (round to nearest even)."""
    x = _probe_doubles(np.random.default_rng(11), 4000)
    with np.errstate(over="ignore"):
        ref = x.astype(np.float16).view(np.uint16)
    assert np.array_equal(oracle.encode(x, oracle.F16), ref)
    finite = np.isfinite(ref.view(np.float16))
    assert np.array_equal(oracle.decode(ref[finite], oracle.F16),
                          ref[finite].view(np.float16).astype(np.float64))


def test_f32_rounding_matches_numpy():
    x = _probe_doubles(np.random.default_rng(12), 4000)
    with np.errstate(over="ignore"):
        ref = x.astype(np.float32)
    assert np.array_equal(oracle.encode(x, oracle.F32).view(np.uint32), ref.view(np.uint32))


def test_bf16_rounding_is_nearest_even_by_brute_force():
    """Each bfloat16 code is the nearest representable value to x (compared
    exactly in float64 against both neighbours of the code), and on a tie the
    one with an even last mantissa bit; decoding is the upper half of a
    binary32."""
    x = _probe_doubles(np.random.default_rng(13), 3000)
    x = x[np.abs(x) < 3e38]
    h = oracle.encode(x, oracle.BF16)
    v = oracle.decode(h, oracle.BF16)
    assert np.array_equal(v, (h.astype(np.uint32) << 16).view(np.float32).astype(np.float64))
    for hk, xk, vk in zip(h, x, v):
        mag = int(hk) & 0x7FFF
        sign = int(hk) & 0x8000
        nbrs = [sign | m for m in (mag - 1, mag + 1) if 0 <= m < 0x7F80]
        dv = abs(vk - xk)
        for nb in nbrs:
            dn = abs(oracle.decode(np.array([nb], np.uint16), oracle.BF16)[0] - xk)
            assert dv <= dn
            if dv == dn:
                assert mag % 2 == 0


def test_scatter_add_ex_f32_inc_is_scatter_add():
    rng = np.random.default_rng(14)
    t0 = rng.normal(0, 0.01, (50, 7)).astype(np.float32)
    idx = workloads.zipf_ids(rng, 50, 1.2, 400)
    Y = rng.normal(0, 1e-3, (400, 7)).astype(np.float32)
    a, b = t0.copy(), t0.copy()
    oracle.scatter_add(a, idx, Y, -0.3)
    oracle.scatter_add_ex(b, idx.astype(np.int64), Y, -0.3, oracle.OP_INC)
    assert np.array_equal(a.view(np.uint32), b.view(np.uint32))


def test_scatter_add_ex_set_last_entry_wins():
    rng = np.random.default_rng(15)
    for dt in (np.float32, np.float16):
        t0 = rng.normal(0, 1, (30, 5)).astype(dt)
        idx = rng.integers(0, 30, 200).astype(np.int32)
        Y = rng.normal(0, 1, (200, 5)).astype(dt)
        got = t0.copy()
        oracle.scatter_add_ex(got, idx, Y, 0.0, oracle.OP_SET)
        ref = t0.copy()
        last = {}
        for k, r in enumerate(idx):
            last[int(r)] = k
        for r, k in last.items():
            ref[r] = Y[k]
        assert np.array_equal(got.view(np.uint16 if dt == np.float16 else np.uint32),
                              ref.view(np.uint16 if dt == np.float16 else np.uint32))


def test_scatter_add_ex_rounds_each_row_once():
    """bfloat16 has 8 significant bits: 1 + 2^-9 rounds back to 1, so adding
    2^-9 three times entry by entry would leave 1.0; the op carries the row
    exactly and rounds 1 + 3*2^-9 once, to 1 + 2^-7.  binary16 likewise with
    2^-12 steps on 1.0 (spacing 2^-10)."""
    for code, step, want in ((oracle.BF16, 2.0 ** -9, 1 + 2.0 ** -7),
                             (oracle.F16, 2.0 ** -12, 1 + 2.0 ** -10)):
        t = oracle.encode(np.array([[1.0, -2.0]]), code)
        Y = oracle.encode(np.full((3, 2), step), code)
        if code == oracle.F16:
            t, Y = t.view(np.float16), Y.view(np.float16)
        oracle.scatter_add_ex(t, np.zeros(3, np.int64), Y, 1.0, oracle.OP_INC,
                              bf16=code == oracle.BF16)
        got = oracle.decode(t.view(np.uint16) if code == oracle.F16 else t, code)
        assert got[0, 0] == want
        assert got[0, 1] == oracle.decode(oracle.encode(np.array([-2.0 + 3 * step]), code), code)[0]


def test_scatter_add_ex_rejects_bad_ids_before_writing():
    t0 = np.ones((4, 2), np.float32)
    for idx in (np.array([0, 4], np.int32), np.array([1, -1], np.int64),
                np.array([2, 1 << 33], np.int64)):
        t = t0.copy()
        with pytest.raises(oracle.OracleError):
            oracle.scatter_add_ex(t, idx, np.ones((2, 2), np.float32), 1.0)
        assert np.array_equal(t, t0)


def test_planted_task_generator():
    """The planted rule holds for the expected share of training windows and
    for every held-out window; ids stay in range; the corrupted held-out copy
    differs only in the centre."""
    t = workloads.PLANTED
    rule = t.rule()
    assert sorted(rule.tolist()) == list(range(t.V))
    c = t.win // 2
    w, cor = t.batch(np.random.default_rng(0), 20000)
    assert w.dtype == np.int32 and cor.dtype == np.int32
    assert w.min() >= 0 and w.max() < t.V and cor.min() >= 0 and cor.max() < t.V
    hold = np.mean(w[:, c] == rule[w[:, c - 1]])
    assert abs(hold - (1 - t.noise)) < 0.02 + 1.0 / t.V * 5
    hw, hwc = t.held_out(512)
    assert np.all(hw[:, c] == rule[hw[:, c - 1]])
    assert np.array_equal(np.delete(hw, c, axis=1), np.delete(hwc, c, axis=1))
