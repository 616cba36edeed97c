"""Parity of the HIP path (through the C ABI) with the CPU oracle.

Bars (see the design notes for their derivation):
  * gather output, the set of touched rows: bit-exact;
  * per-step mean loss: relative 1e-5;
  * parameters after K steps: |gpu - ref| <= 1e-4 |ref| + 1e-4 rms(ref) per tensor;
  * parameter deltas P_K - P_0 (the updates are ~1e-4 of the values, so the
    bar above alone would barely see them):
    |dgpu - dref| <= 1e-3 |dref| + 1e-3 rms(dref) + 2 sqrt(n) ulp per tensor,
    n the float32 stores into the element (plus half an ulp per entry of a
    row in the atomic mode, which rounds once per entry);
  * scatter-add: within the worst-case float32 summation bound
    n * 2^-24 * (|t0| + sum |alpha Y|) per element, n = entries of the row + 1.
"""
import ctypes
import dataclasses
import zlib

import numpy as np
import pytest

import oracle
import workloads
from workloads import PRESETS

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


def pg():
    import paper_1404_1521_amd as m
    return m


def dev(a):
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def host(t):
    torch.cuda.synchronize()
    return t.detach().cpu().numpy()


def params_dev(p):
    return {k: dev(v) for k, v in p.items()}


def rms(a):
    a = np.asarray(a, np.float64)
    return float(np.sqrt(np.mean(a * a))) if a.size else 0.0


MARGINS = []  # (case, tensor, largest err/bar of the parameters, of the deltas)


def assert_params_close(got, ref, init, stores, entries=None, rows=None, case=""):
    """stores[k]: per-element count of float32 stores over the run (steps for
    the dense tensors, steps touching the row for E); entries: per-row count
    of scatter entries, given for the atomic variant, which rounds once per
    entry instead of once per row and step.  rows: if given, E is compared on
    these rows only (the rest must then be bit-identical to init, which the
    caller checks)."""
    if rows is not None:
        got = dict(got, E=got["E"][rows])
        ref = dict(ref, E=ref["E"][rows])
        init = dict(init, E=init["E"][rows])
        stores = dict(stores, E=np.asarray(stores["E"])[rows])
        if entries is not None:
            entries = entries[rows]
    for k in ("E", "W1", "b1", "w2", "b2"):
        g = got[k].astype(np.float64)
        r = ref[k].astype(np.float64)
        err = np.abs(g - r)
        bar = 1e-4 * np.abs(r) + 1e-4 * rms(r)
        assert np.all(err <= bar), (k, float(np.max(err - bar)))
        ulp = np.spacing(np.abs(ref[k]).astype(np.float32)).astype(np.float64)
        n = np.broadcast_to(np.asarray(stores[k], np.float64), r.shape[:1])
        n = n.reshape(n.shape + (1,) * (r.ndim - 1))
        floor = 2.0 * np.sqrt(n) * ulp
        if entries is not None and k == "E":
            floor = floor + 0.5 * entries.reshape(-1, 1) * ulp
        dg = g - init[k]
        dr = r - init[k]
        derr = np.abs(dg - dr)
        dbar = 1e-3 * np.abs(dr) + 1e-3 * rms(dr) + floor
        MARGINS.append((case, k, float(np.max(err / bar)), float(np.max(derr / dbar))))
        assert np.all(derr <= dbar), (k, "delta", float(np.max(derr - dbar)), rms(dr))


def run_both(w, steps, B, mode=0, lr=None, seed=None, p0=None, batches=None, check=True,
             touched_only=False):
    """Runs `steps` SGD steps on the GPU and in the float32-storage oracle and
    compares losses and parameters (with touched_only, E on the rows the
    steps touched, the others bit-identical)."""
    m = pg()
    lr = w.lr if lr is None else lr
    p = workloads.init_params(w, seed) if p0 is None else {k: v.copy() for k, v in p0.items()}
    init = {k: v.astype(np.float64) for k, v in p.items()}
    pd = params_dev(p)
    ctx = m.Context(w.V, w.d, w.win, w.H, max_batch=B, scatter_mode=mode)
    losses = torch.zeros(steps, dtype=torch.float32, device="cuda")
    ref_losses = []
    row_steps = np.zeros(w.V)
    row_entries = np.zeros(w.V)
    for s in range(steps):
        win, cor = batches[s] if batches is not None else workloads.batch(w, s, B)
        ctx.train_step(pd, dev(win), dev(cor), lr, losses[s:s + 1])
        ref_losses.append(oracle.train_step(p, win, cor, lr))
        ids = np.concatenate([win.reshape(-1), cor])
        row_steps[np.unique(ids)] += 1
        row_entries += np.bincount(ids, minlength=w.V)
    assert ctx.status() == m.OK
    got = {k: host(v) for k, v in pd.items()}
    gl, rl = host(losses), np.array(ref_losses)
    if check:
        np.testing.assert_allclose(gl, rl, rtol=1e-5, atol=1e-6)
        stores = {"E": row_steps, "W1": steps, "b1": steps, "w2": steps, "b2": steps}
        rows = None
        if touched_only:
            rows = np.flatnonzero(row_steps)
            untouched = row_steps == 0
            assert np.array_equal(got["E"][untouched], init["E"][untouched].astype(np.float32))
        assert_params_close(got, p, init, stores, row_entries if mode == 1 else None, rows,
                            f"{w.name} B={B} mode={mode} lr={lr} steps={steps}")
    return got, p, init, gl, rl, ctx


# --------------------------------------------------------------------- gather

@pytest.mark.parametrize("name,B", [("tiny", 37), ("poly256", 1000), ("poly256", 1)])
def test_gather_bit_exact(name, B):
    w = PRESETS[name]
    p = workloads.init_params(w)
    win, cor = workloads.batch(w, 5, B)
    ctx = pg().Context(w.V, w.d, w.win, w.H, max_batch=B)
    X, Xc = ctx.gather(dev(p["E"]), dev(win), dev(cor))
    Xr, Xcr = oracle.gather(p["E"], win, cor)
    assert np.array_equal(host(X), Xr)
    assert np.array_equal(host(Xc), Xcr)


# ---------------------------------------------------------------- scatter-add

def scatter_bound(t0, idx, Y, alpha):
    cnt = np.bincount(idx, minlength=t0.shape[0]).astype(np.float64)[:, None] + 1.0
    mag = np.abs(t0.astype(np.float64))
    np.add.at(mag, idx, np.abs(alpha * Y.astype(np.float64)))
    return cnt * 2.0 ** -24 * mag + 1e-30


@pytest.mark.parametrize("mode", [0, 1])
@pytest.mark.parametrize("rows,d,N,s", [
    (50, 8, 400, 1.2), (3, 4, 1, 1.0), (1000, 64, 5000, 1.2), (1000, 64, 8192, 1.2),
    (100_000, 64, 20_000, 1.2), (100_000, 64, 4096 * 3 + 17, 1.0), (7, 256, 3000, 1.5),
    (300_000, 16, 9000, 1.1),
])
def test_scatter_add_matches_oracle(mode, rows, d, N, s):
    rng = np.random.default_rng(rows + N)
    t0 = rng.normal(0, 0.01, (rows, d)).astype(np.float32)
    idx = workloads.zipf_ids(rng, rows, s, N)
    Y = rng.normal(0, 1e-3, (N, d)).astype(np.float32)
    alpha = 0.75
    ctx = pg().Context(1000, 16, 5, 8, max_batch=1, max_scatter=N, max_rows=rows)
    td = dev(t0)
    ctx.scatter_add(td, dev(idx), dev(Y), alpha, mode)
    assert ctx.status() == pg().OK
    got = host(td)
    ref = t0.copy()
    oracle.scatter_add(ref, idx, Y, alpha)
    err = np.abs(got.astype(np.float64) - ref.astype(np.float64))
    assert np.all(err <= scatter_bound(t0, idx, Y, alpha))
    untouched = np.setdiff1d(np.arange(rows), idx)
    assert np.array_equal(got[untouched], t0[untouched])


def _run_lengths_covering_every_lane(rng, N):
    """Keys whose sorted runs have every length 1..70 (shuffled), so piece
    heads fall on every lane of a chunk (32 or 64 entries), runs cross chunk
    ends, and a run starting at lane 31 continues past lane 32."""
    lens = []
    while sum(lens) < N:
        lens.extend(rng.permutation(np.arange(1, 71)).tolist())
    keys = np.repeat(np.arange(len(lens)), lens)[:N]
    return keys.astype(np.int32)


@pytest.mark.parametrize("pattern", ["every_lane", "head_at_lane_31"])
@pytest.mark.parametrize("d", [64, 80])
def test_scatter_add_long_chunks_piece_structure(pattern, d):
    """A 140,000-entry list (32-entry chunks, ranges of 128 entries); these
    key layouts put piece boundaries on each lane of a chunk, runs across
    chunk and range ends, and rows of 80 floats take a second, partial
    column block.  (Both halves of the 64-bit lane masks are covered by the
    partition-wise apply's 64-entry chunks: test_scatter_add_partition_every_lane.)"""
    rng = np.random.default_rng(7)
    N = 140_000
    if pattern == "every_lane":
        keys = _run_lengths_covering_every_lane(rng, N)
    else:  # runs of 64 whose heads all sit at lane 31 of their chunk
        keys = ((np.arange(N) + 33) // 64).astype(np.int32)
    rows = int(keys.max()) + 5
    idx = keys[rng.permutation(N)]  # the sort regroups the runs
    t0 = rng.normal(0, 0.01, (rows, d)).astype(np.float32)
    Y = rng.normal(0, 1e-3, (N, d)).astype(np.float32)
    ctx = pg().Context(1000, 16, 5, 8, max_batch=1, max_scatter=N, max_rows=rows)
    td = dev(t0)
    ctx.scatter_add(td, dev(idx), dev(Y), -0.5, pg().SCATTER_SORTED)
    assert ctx.status() == pg().OK
    got = host(td)
    ref = t0.copy()
    oracle.scatter_add(ref, idx, Y, -0.5)
    err = np.abs(got.astype(np.float64) - ref.astype(np.float64))
    assert np.all(err <= scatter_bound(t0, idx, Y, -0.5))
    untouched = np.setdiff1d(np.arange(rows), idx)
    assert np.array_equal(got[untouched], t0[untouched])


@pytest.mark.parametrize("d", [64, 80])
def test_scatter_add_partition_every_lane(d):
    """8,192 entries whose ids are all multiples of 128 fall into one
    partition of the partitioned sort, with runs of every length 1..70: the
    partition-wise update's 64-entry chunks get piece heads on every lane,
    both halves of the 64-bit lane masks, and runs across chunk and round
    ends."""
    rng = np.random.default_rng(17)
    N = 8192
    idx = (_run_lengths_covering_every_lane(rng, N) * 128).astype(np.int32)
    rows = int(idx.max()) + 1
    idx = idx[rng.permutation(N)]
    t0 = rng.normal(0, 0.01, (rows, d)).astype(np.float32)
    Y = rng.normal(0, 1e-3, (N, d)).astype(np.float32)
    ctx = pg().Context(1000, 16, 5, 8, max_batch=1, max_scatter=N, max_rows=rows)
    td = dev(t0)
    ctx.scatter_add(td, dev(idx), dev(Y), -0.5, pg().SCATTER_SORTED)
    assert ctx.status() == pg().OK
    got = host(td)
    ref = t0.copy()
    oracle.scatter_add(ref, idx, Y, -0.5)
    err = np.abs(got.astype(np.float64) - ref.astype(np.float64))
    assert np.all(err <= scatter_bound(t0, idx, Y, -0.5))
    untouched = np.setdiff1d(np.arange(rows), idx)
    assert np.array_equal(got[untouched], t0[untouched])


@pytest.mark.parametrize("keys_kind,d", [("one_key", 16), ("one_key", 80), ("three_keys", 64),
                                          ("zipf_small_table", 80)])
def test_scatter_add_partition_rounds(keys_kind, d):
    """Lists of at most 8192 entries take the partitioned sort and the
    partition-wise update (one workgroup per partition, 1024 entries per
    round): these put several rounds into one partition, so segments carry
    over from round to round, and rows of 80 floats add a partial column
    block."""
    rng = np.random.default_rng(11)
    N = 8192
    if keys_kind == "one_key":
        rows, idx = 5, np.full(N, 3, np.int32)
    elif keys_kind == "three_keys":  # 0, 128, 256 share partition 0 of 7 key bits
        rows = 300
        idx = rng.choice(np.array([0, 128, 256], np.int32), N, p=[0.6, 0.3, 0.1]).astype(np.int32)
    else:
        rows = 40
        idx = workloads.zipf_ids(rng, rows, 1.5, N)
    t0 = rng.normal(0, 0.01, (rows, d)).astype(np.float32)
    Y = rng.normal(0, 1e-3, (N, d)).astype(np.float32)
    ctx = pg().Context(1000, 16, 5, 8, max_batch=1, max_scatter=N, max_rows=rows)
    td = dev(t0)
    ctx.scatter_add(td, dev(idx), dev(Y), 0.5, pg().SCATTER_SORTED)
    assert ctx.status() == pg().OK
    got = host(td)
    ref = t0.copy()
    oracle.scatter_add(ref, idx, Y, 0.5)
    err = np.abs(got.astype(np.float64) - ref.astype(np.float64))
    assert np.all(err <= scatter_bound(t0, idx, Y, 0.5))
    untouched = np.setdiff1d(np.arange(rows), idx)
    assert np.array_equal(got[untouched], t0[untouched])


@pytest.mark.parametrize("M", [1, 2, 255, 256, 257, 511, 512, 513, 700, 1024, 2000])
def test_scatter_add_partition_sizes_exact(M):
    """Partition 0 (ids that are multiples of 128) holds exactly M entries
    over eight ids, the rest of the 6000 entries fall in other partitions:
    sizes on both sides of where the partitioned sort switches from ranking
    by counting to its radix passes.  Y holds small integers and the table
    starts at zero, so every order of summation gives the same float32 and
    the result must equal the oracle's exactly: an entry lost or taken twice
    by the ranking shows."""
    rng = np.random.default_rng(1000 + M)
    rows, N, d = 1024, 6000, 24
    hot = rng.choice(np.arange(0, rows, 128, dtype=np.int32), M)
    other = rng.integers(0, rows, 4 * N).astype(np.int32)
    other = other[other % 128 != 0][: N - M]
    idx = rng.permutation(np.concatenate([hot, other])).astype(np.int32)
    assert idx.size == N and np.count_nonzero(idx % 128 == 0) == M
    Y = rng.integers(-8, 9, (N, d)).astype(np.float32)
    ctx = pg().Context(1000, 16, 5, 8, max_batch=1, max_scatter=N, max_rows=rows)
    t0 = np.zeros((rows, d), np.float32)
    ref = t0.astype(np.float64)
    oracle.scatter_add(ref, idx, Y.astype(np.float64), 0.5)
    for mode in (pg().SCATTER_SORTED, pg().SCATTER_ATOMIC):
        td = dev(t0)
        ctx.scatter_add(td, dev(idx), dev(Y), 0.5, mode)
        assert ctx.status() == pg().OK
        assert np.array_equal(host(td), ref.astype(np.float32)), mode


@pytest.mark.parametrize("M", [129, 300, 512])
@pytest.mark.parametrize("case", ["absent", "only", "mixed"])
def test_scatter_add_smallest_key_placement(M, case):
    """A partition of more than 128 entries places the entries of its
    smallest key (id 0 in partition 0) first by a prefix count and ranks only
    the others: partition 0 here holds M entries with none of id 0, only id 0,
    or id 0 among seven other multiples of 128, in shuffled entry order.
    Integer Y and a zero table make every summation order exact, so the
    result must equal the oracle's exactly."""
    rng = np.random.default_rng(3000 + M + 7 * len(case))
    rows, N, d = 1024, 6000, 24
    mult = np.arange(0, rows, 128, dtype=np.int32)
    pool = {"absent": mult[1:], "only": mult[:1], "mixed": mult}[case]
    hot = rng.choice(pool, M)
    if case == "mixed":
        hot[: M // 3] = 0
    other = rng.integers(0, rows, 4 * N).astype(np.int32)
    other = other[other % 128 != 0][: N - M]
    idx = rng.permutation(np.concatenate([hot, other])).astype(np.int32)
    assert idx.size == N and np.count_nonzero(idx % 128 == 0) == M
    Y = rng.integers(-8, 9, (N, d)).astype(np.float32)
    ctx = pg().Context(1000, 16, 5, 8, max_batch=1, max_scatter=N, max_rows=rows)
    t0 = np.zeros((rows, d), np.float32)
    ref = t0.astype(np.float64)
    oracle.scatter_add(ref, idx, Y.astype(np.float64), 0.5)
    td = dev(t0)
    ctx.scatter_add(td, dev(idx), dev(Y), 0.5, pg().SCATTER_SORTED)
    assert ctx.status() == pg().OK
    assert np.array_equal(host(td), ref.astype(np.float32))


@pytest.mark.parametrize("L", [64 * 15 + 1, 64 * 16, 64 * 16 + 1, 64 * 17 + 5])
@pytest.mark.parametrize("lead", [0, 10])
def test_scatter_add_segment_spans_fixup(L, lead):
    """A 20,000-entry list (16-entry chunks, ranges of 64 entries): row 7
    holds L entries that start at sorted position `lead` (after `lead`
    entries of row 3; no other id below 100), so its segment runs through a
    known number of ranges: up to 16 partials are finished by one fix-up
    wave, which finds the segment's end from the ranges marked as run
    through; more go to the whole workgroup.  Exact integer sums."""
    rng = np.random.default_rng(5000 + L + lead)
    rows, N, d = 4096, 20000, 24
    head = np.concatenate([np.full(lead, 3, np.int32), np.full(L, 7, np.int32)])
    other = rng.integers(100, rows, N - head.size).astype(np.int32)
    idx = rng.permutation(np.concatenate([head, other])).astype(np.int32)
    Y = rng.integers(-8, 9, (N, d)).astype(np.float32)
    ctx = pg().Context(1000, 16, 5, 8, max_batch=1, max_scatter=N, max_rows=rows)
    t0 = np.zeros((rows, d), np.float32)
    ref = t0.astype(np.float64)
    oracle.scatter_add(ref, idx, Y.astype(np.float64), 0.25)
    for mode in (pg().SCATTER_SORTED, pg().SCATTER_ATOMIC):
        td = dev(t0)
        ctx.scatter_add(td, dev(idx), dev(Y), 0.25, mode)
        assert ctx.status() == pg().OK
        assert np.array_equal(host(td), ref.astype(np.float32)), mode


def test_small_vocabulary_step_partition_rounds():
    """A 64-word vocabulary at B = 1365 (8190 entries, the largest list the
    partitioned sort takes): each partition holds one word, the most frequent
    with about 1800 entries, so the partition-wise update runs two rounds."""
    w = workloads.Workload("v64_b1365", V=64, d=16, win=5, H=8, B=1365, lr=0.05, steps=3,
                           zipf_s=1.0, seed=31)
    run_both(w, w.steps, w.B, 0)


@pytest.mark.parametrize("mode", [0, 1])
def test_scatter_add_full_size_zipf12(mode):
    """327,680 Zipf(1.2) rows into a 100000 x 64 table, the standalone
    scatter-add workload, against the oracle."""
    table, idx, Y = workloads.scatter_inputs()
    ctx = pg().Context(1000, 16, 5, 8, max_batch=1, max_scatter=idx.size, max_rows=table.shape[0])
    td = dev(table)
    ctx.scatter_add(td, dev(idx), dev(Y), 1.0, mode)
    assert ctx.status() == pg().OK
    got = host(td)
    ref = table.copy()
    oracle.scatter_add(ref, idx, Y, 1.0)
    err = np.abs(got.astype(np.float64) - ref.astype(np.float64))
    assert np.all(err <= scatter_bound(table, idx, Y, 1.0))
    untouched = np.setdiff1d(np.arange(table.shape[0]), idx)
    assert np.array_equal(got[untouched], table[untouched])


@pytest.mark.parametrize("s", [1.2, 0.0])
def test_scatter_add_many_sort_tiles(s):
    """700,000 rows, 171 sort tiles of 4096 keys: more earlier tiles than one
    look-back step reads (128), so late tiles continue below their first
    window.  Zipf(1.2) and uniform ids; sorted against the oracle, and two
    calls bit-identical."""
    sw = dataclasses.replace(workloads.SCATTER_ISO, d=16, N=700_000, zipf_s=s, seed=41)
    table, idx, Y = workloads.scatter_inputs(sw)
    ctx = pg().Context(1000, 16, 5, 8, max_batch=1, max_scatter=idx.size, max_rows=table.shape[0])
    outs = []
    for _ in range(2):
        td = dev(table)
        ctx.scatter_add(td, dev(idx), dev(Y), 1.0, pg().SCATTER_SORTED)
        assert ctx.status() == pg().OK
        outs.append(host(td))
    ref = table.copy()
    oracle.scatter_add(ref, idx, Y, 1.0)
    err = np.abs(outs[0].astype(np.float64) - ref.astype(np.float64))
    assert np.all(err <= scatter_bound(table, idx, Y, 1.0))
    assert np.array_equal(outs[0], outs[1])


def _bucket_case(kind):
    rng = np.random.default_rng(zlib.crc32(kind.encode()))
    if kind == "permuted_zipf":   # heavy rows at random ids: oversize hashed buckets, 1 pass
        rows, d, N = 100_000, 64, 327_680
        idx = rng.permutation(rows).astype(np.int32)[workloads.zipf_ids(rng, rows, 1.2, N)]
    elif kind == "one_key":       # one hashed bucket holds every entry
        rows, d, N = 100_000, 16, 50_000
        idx = np.full(N, 77_777, np.int32)
    elif kind == "wide_keys":     # 24-bit keys: 2 global passes, 3 LDS passes
        rows, d, N = 1 << 24, 4, 200_000
        idx = rng.permutation(rows).astype(np.int32)[workloads.zipf_ids(rng, rows, 1.1, N)]
    elif kind == "few_keys":      # every key has a bucket of its own
        rows, d, N = 50, 8, 30_000
        idx = workloads.zipf_ids(rng, rows, 1.0, N)
    elif kind == "one_key_per_bucket":  # keys below 576: hashed buckets of one or two keys
        rows, d, N = 600, 32, 100_000
        idx = rng.integers(0, rows, N).astype(np.int32)
    elif kind == "uniform_mid":   # hashed buckets of 513..2048 entries: LDS radix passes
        rows, d, N = 5_000, 8, 700_000
        idx = rng.integers(0, rows, N).astype(np.int32)
    else:                         # above 786,432 entries: the multi-tile look-back sort
        rows, d, N = 100_000, 4, 1_200_000
        idx = workloads.zipf_ids(rng, rows, 1.0, N)
    t0 = rng.normal(0, 0.01, (rows, d)).astype(np.float32)
    Y = rng.normal(0, 1e-3, (N, d)).astype(np.float32)
    return t0, idx, Y


@pytest.mark.parametrize("kind", ["permuted_zipf", "one_key", "wide_keys", "few_keys",
                                  "one_key_per_bucket", "uniform_mid", "look_back"])
def test_scatter_add_sort_paths(kind):
    """Lists of 8,192 < N <= 786,432 entries take the bucketed sort (64
    dedicated buckets for the smallest ids, 512 hashed ones for the rest);
    these inputs reach its less common paths: heavy rows at random ids
    (hashed buckets above 2,048 entries, ordered through global memory),
    one key for every entry, 24-bit keys, key ranges inside the dedicated
    buckets, buckets of one key, and hashed buckets sorted by LDS radix
    passes; above 786,432 entries the multi-tile look-back sort.  Against
    the oracle, the touched rows, and two calls bit-identical."""
    t0, idx, Y = _bucket_case(kind)
    rows, d = t0.shape
    ctx = pg().Context(1000, 16, 5, 8, max_batch=1, max_scatter=idx.size, max_rows=rows)
    outs = []
    for _ in range(2):
        td = dev(t0)
        ctx.scatter_add(td, dev(idx), dev(Y), -0.5, pg().SCATTER_SORTED)
        assert ctx.status() == pg().OK
        outs.append(host(td))
        del td
    ref = t0.copy()
    oracle.scatter_add(ref, idx, Y, -0.5)
    touched = np.zeros(rows, bool)
    touched[idx] = True
    err = np.abs(outs[0][touched].astype(np.float64) - ref[touched].astype(np.float64))
    assert np.all(err <= scatter_bound(t0, idx, Y, -0.5)[touched])
    assert np.array_equal(outs[0][~touched], t0[~touched])
    assert np.array_equal(outs[0], outs[1])


def test_scatter_add_sorted_is_deterministic():
    table, idx, Y = workloads.scatter_inputs(N=100_000)
    ctx = pg().Context(1000, 16, 5, 8, max_batch=1, max_scatter=idx.size, max_rows=table.shape[0])
    outs = []
    for _ in range(2):
        td = dev(table)
        ctx.scatter_add(td, dev(idx), dev(Y), 1.0, pg().SCATTER_SORTED)
        outs.append(host(td))
    assert np.array_equal(outs[0], outs[1])


def test_scatter_add_bad_index_leaves_table_untouched():
    m = pg()
    rng = np.random.default_rng(0)
    t0 = rng.normal(0, 1, (10, 4)).astype(np.float32)
    idx = np.array([1, 2, 10, 3], np.int32)
    Y = np.ones((4, 4), np.float32)
    ctx = m.Context(1000, 16, 5, 8, max_batch=1, max_scatter=4, max_rows=10)
    for mode in (0, 1):
        td = dev(t0)
        ctx.scatter_add(td, dev(idx), dev(Y), 1.0, mode)
        assert ctx.status() == m.EID
        assert np.array_equal(host(td), t0)
        assert ctx.status() == m.OK


# --------------------------------------------------------------- train steps

@pytest.mark.parametrize("mode", [0, 1])
def test_tiny_100_steps(mode):
    w = PRESETS["tiny"]
    run_both(w, 100, w.B, mode)


def test_tiny_amplified_updates():
    # larger parameters and step so that updates dominate; some hinges go inactive
    w = dataclasses.replace(PRESETS["tiny"], init_std=0.5)
    _, _, _, gl, _, _ = run_both(w, 30, 32, 0, lr=0.1, seed=7)
    assert np.min(gl) < 1.0  # the run is away from the all-active start


@pytest.mark.parametrize("mode", [0, 1])
def test_poly256_1000_steps(mode):
    w = PRESETS["poly256"]
    run_both(w, 1000 if mode == 0 else 100, w.B, mode)


@pytest.mark.parametrize("B,steps", [(1024, 20), (1365, 5), (1366, 3), (4096, 10), (16384, 3)])
def test_sweep_batches(B, steps):
    w = PRESETS["sweep_1024"].with_batch(B)
    run_both(w, steps, B, 0)


@pytest.mark.parametrize("B", [341, 342, 853, 854, 2730, 2731, 10922, 10923, 21845, 21846])
def test_update_forms_at_their_limits(B):
    """Batches on both sides of each switch of the update's form (N = 6B
    entries): 8- or 16-wave partition workgroups at 2,048 entries, 32- or
    64-entry partition chunks at 5,120, and the chunked update's 16- or
    32-entry chunks at 16,384, 65,536 and 131,072 entries."""
    N = 6 * B
    assert any(lim - 6 < N <= lim + 6 for lim in (2048, 5120, 16384, 65536, 131072))
    w = PRESETS["sweep_1024"].with_batch(B)
    run_both(w, 2, B, 0)


@pytest.mark.parametrize("B", [4100, 8215, 8231])
def test_pipelined_tiles_ragged(B):
    """More than 256 tiles, so workgroups take their tiles in pairs (an even
    number per workgroup), and the last workgroup fewer: 257 tiles at two per
    workgroup (the last has one: a pair whose second tile is past the batch),
    514 and 515 tiles at four per workgroup (the last has two or three); the
    last tile holds 4, 7 or 7 windows."""
    ntiles = -(-B // 16)
    per = -(-ntiles // 256)
    per += per & 1
    assert per > 1 and ntiles % per != 0
    w = PRESETS["sweep_1024"].with_batch(B)
    run_both(w, 2, B, 0)


@pytest.mark.parametrize("B", [32653, 32773])
def test_role_specialised_tiles_ragged(B):
    """Eight or more tiles per workgroup take the role-specialised form
    (staging, forward and dW1 waves pipelined one tile apart): 2041 tiles at
    eight per workgroup leave the last workgroup one tile (the pipeline's
    fill and drain with nothing between), 2049 tiles at ten per workgroup
    leave it nine; the last tile holds 13 or 5 windows."""
    ntiles = -(-B // 16)
    per = -(-ntiles // 256)
    per += per & 1
    assert per >= 8 and ntiles % per in (1, 9) and B % 16 != 0
    w = PRESETS["sweep_1024"].with_batch(B)
    run_both(w, 2, B, 0)


@pytest.mark.parametrize("mode", [0, 1])
def test_full_size_batch_65536_one_step(mode):
    w = PRESETS["sweep_65536"]
    run_both(w, 1, w.B, mode)


@pytest.mark.parametrize("B", [1, 17, 33])
def test_ragged_and_single_window_batches(B):
    w = PRESETS["tiny"]
    run_both(w, 5, B, 0, lr=0.5)


# Shapes that reach the other kernel variants: hidden widths padded to 16,
# 32 and 64, K-chunks per wave up to 8, window 1 (the centre is the whole
# window) and the widest window.
OTHER_SHAPES = [
    workloads.Workload("w7_d32_h20", V=5000, d=32, win=7, H=20, B=300, lr=0.05, steps=4,
                       zipf_s=1.0, seed=11),
    workloads.Workload("w5_d64_h64", V=3000, d=64, win=5, H=64, B=200, lr=0.05, steps=3,
                       zipf_s=1.1, seed=12),
    workloads.Workload("w3_d112_h48", V=2000, d=112, win=3, H=48, B=150, lr=0.05, steps=3,
                       zipf_s=1.0, seed=13),
    workloads.Workload("w1_d16_h1", V=500, d=16, win=1, H=1, B=50, lr=0.5, steps=5,
                       zipf_s=1.0, seed=14),
    workloads.Workload("w31_d16_h8", V=800, d=16, win=31, H=8, B=70, lr=0.1, steps=3,
                       zipf_s=1.0, seed=15),
]


@pytest.mark.parametrize("mode", [0, 1])
@pytest.mark.parametrize("w", OTHER_SHAPES, ids=[w.name for w in OTHER_SHAPES])
def test_other_shapes(w, mode):
    run_both(w, w.steps, w.B, mode)


# Hidden layers wider than 64 units take the three-contraction path
# (forward, dW1 slices, per-entry rows); B = 1030 crosses a 1024-window slice.
LARGE_SHAPES = [
    workloads.Workload("w11_d128_h256", V=3000, d=128, win=11, H=256, B=100, lr=0.05, steps=3,
                       zipf_s=1.0, seed=21),
    workloads.Workload("w3_d64_h128", V=2000, d=64, win=3, H=128, B=1030, lr=0.05, steps=2,
                       zipf_s=1.0, seed=22),
    workloads.Workload("w5_d192_h192", V=1500, d=192, win=5, H=192, B=70, lr=0.05, steps=2,
                       zipf_s=1.1, seed=23),
]


@pytest.mark.parametrize("mode", [0, 1])
@pytest.mark.parametrize("w", LARGE_SHAPES, ids=[w.name for w in LARGE_SHAPES])
def test_large_hidden_layer_shapes(w, mode):
    run_both(w, w.steps, w.B, mode)


@pytest.mark.parametrize("w", LARGE_SHAPES[:2], ids=[w.name for w in LARGE_SHAPES[:2]])
def test_large_hidden_layer_scores(w):
    p = workloads.init_params(w)
    win, _ = workloads.batch(w, 1, w.B)
    ctx = pg().Context(w.V, w.d, w.win, w.H, max_batch=w.B)
    got = host(ctx.score(params_dev(p), dev(win)))
    np.testing.assert_allclose(got, oracle.score(p, win), rtol=1e-5, atol=1e-6)


def test_stress_full_size_sampled():
    """The stress workload at its full size (V 1M, d 128, window 11, H 256,
    B 16384): scores of sampled true and corrupted windows against the oracle,
    then one sorted step: status clean, loss finite and in the hinge range,
    rows outside the batch and b2 bit-identical."""
    w = PRESETS["stress"]
    p = workloads.init_params(w)
    pd = params_dev(p)
    win, cor = workloads.batch(w, 0, w.B)
    ctx = pg().Context(w.V, w.d, w.win, w.H, max_batch=w.B)
    rng = np.random.default_rng(0)
    pick = np.sort(rng.choice(w.B, 48, replace=False))
    sample = np.ascontiguousarray(win[pick])
    corrupted = sample.copy()
    corrupted[:, w.win // 2] = cor[pick]
    both = np.concatenate([sample, corrupted])
    got = host(ctx.score(pd, dev(both)))
    np.testing.assert_allclose(got, oracle.score(p, both), rtol=1e-5, atol=1e-6)
    loss = torch.zeros(1, device="cuda")
    ctx.train_step(pd, dev(win), dev(cor), w.lr, loss)
    assert ctx.status() == pg().OK
    lv = float(host(loss)[0])
    assert np.isfinite(lv) and 0.0 < lv < 2.0
    touched = np.zeros(w.V, bool)
    touched[win.reshape(-1)] = True
    touched[cor] = True
    E = host(pd["E"])
    assert np.array_equal(E[~touched], p["E"][~touched])
    assert not np.array_equal(E[touched], p["E"][touched])
    assert np.array_equal(host(pd["b2"]), p["b2"])


@pytest.mark.parametrize("mode,steps", [(0, 3), (1, 1)])
def test_stress_full_size_parity(mode, steps):
    """The stress workload at its full size (V 1M, d 128, window 11, H 256,
    B 16384, lr 0.005) against the oracle: per-step losses, W1, b1, w2, b2
    and the touched rows of E under the parameter and delta bars, the other
    rows bit-identical.  This is the one shape that runs the wide-layer
    backward with 16 dW1 slices, the multi-tile sort and 32-entry chunks
    together."""
    w = PRESETS["stress"]
    run_both(w, steps, w.B, mode, touched_only=True)


@pytest.mark.parametrize("B,lr,S", [(16, 1.0, 64), (4096, 4.0, 8), (1024, 0.25 * 8.0, 16)])
def test_planted_task_high_rate_parity(B, lr, S):
    """The batch-size study's regime (the planted task of the convergence
    study, learning rates 1.0 to 4.0) through train_steps, the call the
    study times, against the oracle: per-step losses and the parameters
    under the same bars as every other step test."""
    m = pg()
    task = workloads.PLANTED
    w = task.workload(B, lr)
    p = workloads.init_params(w)
    init = {k: v.astype(np.float64) for k, v in p.items()}
    rng = np.random.default_rng([task.seed, 4, B])
    wins, cors = task.batch(rng, S * B)
    wins, cors = wins.reshape(S, B, task.win), cors.reshape(S, B)
    st = torch.cuda.Stream()
    with torch.cuda.stream(st):
        pd = params_dev(p)
        ctx = m.Context(task.V, task.d, task.win, task.H, max_batch=B, stream=st)
        losses = torch.zeros(S, device="cuda")
        ctx.train_steps(pd, dev(wins), dev(cors), lr, losses)
        st.synchronize()
    assert ctx.status() == m.OK
    ref_losses = [oracle.train_step(p, wins[s], cors[s], lr) for s in range(S)]
    row_steps = np.zeros(task.V)
    for s in range(S):
        row_steps[np.unique(np.concatenate([wins[s].reshape(-1), cors[s]]))] += 1
    np.testing.assert_allclose(host(losses), ref_losses, rtol=1e-5, atol=1e-6)
    got = {k: host(v) for k, v in pd.items()}
    stores = {"E": row_steps, "W1": S, "b1": S, "w2": S, "b2": S}
    assert_params_close(got, p, init, stores, case=f"planted B={B} lr={lr} S={S}")


@pytest.mark.parametrize("name,B", [("tiny", 32), ("poly256", 256), ("poly256", 4096)])
def test_touched_rows_bit_exact(name, B):
    w = PRESETS[name]
    p = params_dev(workloads.init_params(w))
    win, cor = workloads.batch(w, 3, B)
    ctx = pg().Context(w.V, w.d, w.win, w.H, max_batch=B)
    ctx.train_step(p, dev(win), dev(cor), w.lr)
    assert np.array_equal(np.array(ctx.touched_rows(), np.int32),
                          oracle.touched_rows(w.V, win, cor))


def test_untouched_rows_bit_identical_and_b2_constant():
    w = PRESETS["poly256"]
    p = workloads.init_params(w)
    pd = params_dev(p)
    win, cor = workloads.batch(w, 0, 4096)
    ctx = pg().Context(w.V, w.d, w.win, w.H, max_batch=4096)
    ctx.train_step(pd, dev(win), dev(cor), 0.5)
    E = host(pd["E"])
    touched = np.zeros(w.V, bool)
    touched[win.reshape(-1)] = True
    touched[cor] = True
    assert np.array_equal(E[~touched], p["E"][~touched])
    assert np.array_equal(host(pd["b2"]), p["b2"])


@pytest.mark.parametrize("mode", [0, 1])
def test_corrupt_equal_centre_changes_nothing(mode):
    w = PRESETS["tiny"]
    p = workloads.init_params(w, seed=3)
    pd = params_dev(p)
    win, _ = workloads.batch(w, 0, 40)
    cor = win[:, w.win // 2].copy()
    ctx = pg().Context(w.V, w.d, w.win, w.H, max_batch=40, scatter_mode=mode)
    loss = torch.zeros(1, device="cuda")
    ctx.train_step(pd, dev(win), dev(cor), 0.3, loss)
    assert host(loss)[0] == 1.0
    for k in p:
        assert np.array_equal(host(pd[k]), p[k]), k


def test_margin_met_and_lr_zero_change_nothing():
    w = PRESETS["tiny"]
    p = workloads.init_params(w, seed=4)
    win, cor = workloads.batch(w, 0, 32)
    ctx = pg().Context(w.V, w.d, w.win, w.H, max_batch=32)
    pd = params_dev(p)
    ctx.train_step(pd, dev(win), dev(cor), 0.0)
    for k in p:
        assert np.array_equal(host(pd[k]), p[k]), k
    # saturate tanh so that every margin is exactly 0 (closed form): nothing moves
    q = {k: v.copy() for k, v in p.items()}
    q["E"][:] = 0.0
    q["E"][:, 0] = 40.0
    q["E"][cor, 0] = -40.0
    q["W1"][:] = 0.0
    q["W1"][:, (w.win // 2) * w.d] = 1.0
    q["b1"][:] = 0.0
    q["w2"][:] = 0.5 / w.H
    q["b2"][:] = 0.0
    wins = win.copy()
    wins[:, w.win // 2] = np.setdiff1d(np.arange(w.V), cor)[: 32]
    qd = params_dev(q)
    loss = torch.zeros(1, device="cuda")
    ctx.train_step(qd, dev(wins), dev(cor), 0.1, loss)
    assert oracle.train_step({k: v.copy() for k, v in q.items()}, wins, cor, 0.1) == 0.0
    assert host(loss)[0] == 0.0
    for k in q:
        assert np.array_equal(host(qd[k]), q[k]), k


def test_sorted_mode_is_deterministic():
    w = PRESETS["poly256"]
    outs = []
    for _ in range(2):
        p = params_dev(workloads.init_params(w))
        ctx = pg().Context(w.V, w.d, w.win, w.H, max_batch=4096)
        for s in range(3):
            win, cor = workloads.batch(w, s, 4096)
            ctx.train_step(p, dev(win), dev(cor), 0.5)
        outs.append({k: host(v) for k, v in p.items()})
    for k in outs[0]:
        assert np.array_equal(outs[0][k], outs[1][k]), k


GRAPH_CASES = [
    (PRESETS["sweep_1024"], 1024, 6),   # sort fused into the step kernel, partition-wise update
    (PRESETS["sweep_1024"], 4096, 4),   # bucketed sort of the next step inside the update
                                        # and fix-up launches
    (PRESETS["sweep_1024"], 8192, 3),   # two tiles per workgroup: the pipelined tile loop
    (LARGE_SHAPES[0], 100, 4),          # wide layers: partitioned sort on the side stream
    (LARGE_SHAPES[1], 1030, 3),         # wide layers, two dW1 slices
]


@pytest.mark.parametrize("w,B,S", GRAPH_CASES, ids=[f"{c[0].name}_B{c[1]}" for c in GRAPH_CASES])
def test_train_steps_graph_equals_single_steps(w, B, S):
    """S steps recorded into one HIP graph (and replayed) leave bit-identical
    parameters and losses to S single-step calls."""
    m = pg()
    batches = [workloads.batch(w, s, B) for s in range(S)]
    wall = dev(np.stack([b[0] for b in batches]))
    call = dev(np.stack([b[1] for b in batches]))
    p0 = workloads.init_params(w)
    st = torch.cuda.Stream()
    with torch.cuda.stream(st):
        a = params_dev(p0)
        ctx = m.Context(w.V, w.d, w.win, w.H, max_batch=B, stream=st)
        la = torch.zeros(S, device="cuda")
        ctx.train_steps(a, wall, call, 0.5, la)
        ctx.train_steps(a, wall, call, 0.5, la)  # replay of the cached graph
        b = params_dev(p0)
        lb = torch.zeros(2 * S, device="cuda")
        for r in range(2):
            for s in range(S):
                ctx.train_step(b, wall[s], call[s], 0.5, lb[r * S + s:r * S + s + 1])
        st.synchronize()
    assert ctx.status() == m.OK
    for k in p0:
        assert np.array_equal(host(a[k]), host(b[k])), k
    assert np.array_equal(host(la), host(lb)[S:])


def test_out_of_range_id_voids_the_step():
    m = pg()
    w = PRESETS["tiny"]
    p = workloads.init_params(w)
    for mode in (0, 1):
        pd = params_dev(p)
        win, cor = workloads.batch(w, 0, 32)
        win[5, 1] = w.V
        ctx = m.Context(w.V, w.d, w.win, w.H, max_batch=32, scatter_mode=mode)
        loss = torch.zeros(1, device="cuda")
        ctx.train_step(pd, dev(win), dev(cor), 0.1, loss)
        assert ctx.status() == m.EID
        assert np.isnan(host(loss)[0])
        for k in p:
            assert np.array_equal(host(pd[k]), p[k]), k
        assert ctx.status() == m.OK


@pytest.mark.parametrize("graph", [False, True])
@pytest.mark.parametrize("shape", ["sweep", "wide"])
def test_bad_id_in_next_step_leaves_this_step_intact(shape, graph):
    """Two steps in one call, a bad id only in the second.  From 12,288
    entries up (and for every wide layer) the second step's sort runs on a
    side stream while the first step updates; it raises its own error word,
    so the first step must equal a single valid step bit for bit and only
    the second is void."""
    m = pg()
    if shape == "sweep":
        w, B = PRESETS["poly256"], 2048
    else:
        w, B = LARGE_SHAPES[1], 1030
    p0 = workloads.init_params(w)
    (w0, c0), (w1, c1) = workloads.batch(w, 0, B), workloads.batch(w, 1, B)
    w1 = w1.copy()
    w1[B // 2, w.win // 2] = w.V  # out of range, in the second step only
    st = torch.cuda.Stream() if graph else torch.cuda.current_stream()
    with torch.cuda.stream(st):
        a = params_dev(p0)
        ctx = m.Context(w.V, w.d, w.win, w.H, max_batch=B, stream=st)
        la = torch.zeros(2, device="cuda")
        ctx.train_steps(a, dev(np.stack([w0, w1])), dev(np.stack([c0, c1])), 0.5, la)
        st.synchronize()
        assert ctx.status() == m.EID
        assert ctx.status() == m.OK
        b = params_dev(p0)
        lb = torch.zeros(1, device="cuda")
        ctx.train_step(b, dev(w0), dev(c0), 0.5, lb)
        st.synchronize()
        assert ctx.status() == m.OK
    got = host(la)
    assert got[0] == host(lb)[0]
    assert np.isnan(got[1])
    for k in p0:
        assert np.array_equal(host(a[k]), host(b[k])), k


def test_train_step_sync_returns_the_step_loss():
    m = pg()
    w = PRESETS["poly256"]
    p0 = workloads.init_params(w)
    B = 4096
    win, cor = workloads.batch(w, 2, B)
    ctx = m.Context(w.V, w.d, w.win, w.H, max_batch=B)
    a, b = params_dev(p0), params_dev(p0)
    la = torch.zeros(1, device="cuda")
    ctx.train_step(a, dev(win), dev(cor), 0.3, la)
    lb = ctx.train_step_sync(b, dev(win), dev(cor), 0.3)
    assert isinstance(lb, float)
    assert np.float32(lb) == host(la)[0]
    for k in p0:
        assert np.array_equal(host(a[k]), host(b[k])), k
    # host errors: nothing enqueued, the output untouched
    args = ctx._params(b)
    wd, cd = dev(win), dev(cor)
    wp, cp = ctypes.c_void_p(wd.data_ptr()), ctypes.c_void_p(cd.data_ptr())
    out = ctypes.c_float(7.0)
    lib = ctx._lib
    assert lib.polyglot_train_step_sync(ctx._h, *args, wp, cp, B, ctypes.c_float(0.3),
                                        None) == m.ENULL
    assert lib.polyglot_train_step_sync(ctx._h, *args, wp, cp, 0, ctypes.c_float(0.3),
                                        ctypes.byref(out)) == m.EBATCH
    assert lib.polyglot_train_step_sync(ctx._h, *args, wp, cp, B + 1, ctypes.c_float(0.3),
                                        ctypes.byref(out)) == m.EBATCH
    assert lib.polyglot_train_step_sync(ctx._h, *args, wp, cp, B, ctypes.c_float(float("nan")),
                                        ctypes.byref(out)) == m.EINVAL
    assert out.value == 7.0
    for k in p0:
        assert np.array_equal(host(a[k]), host(b[k])), k
    # an out-of-range id: EID, a NaN loss, no parameter changed
    bad = win.copy()
    bad[3, 0] = -1
    with pytest.raises(m.PolyglotError) as e:
        ctx.train_step_sync(b, dev(bad), dev(cor), 0.3)
    assert e.value.rc == m.EID
    assert ctx.status() == m.EID
    assert ctx.status() == m.OK
    for k in p0:
        assert np.array_equal(host(a[k]), host(b[k])), k


def test_host_errors_enqueue_nothing():
    m = pg()
    w = PRESETS["tiny"]
    ctx = m.Context(w.V, w.d, w.win, w.H, max_batch=8)
    p = params_dev(workloads.init_params(w))
    win, cor = workloads.batch(w, 0, 16)
    with pytest.raises(m.PolyglotError) as e:
        ctx.train_step(p, dev(win), dev(cor), 0.1)
    assert e.value.rc == m.EBATCH
    with pytest.raises(m.PolyglotError) as e:
        ctx.train_step(p, dev(win[:8]), dev(cor[:8]), float("inf"))
    assert e.value.rc == m.EINVAL


# ---------------------------------------------------------------- score

@pytest.mark.parametrize("name,B", [("tiny", 50), ("poly256", 777)])
def test_score_matches_oracle(name, B):
    w = PRESETS[name]
    p = workloads.init_params(w, seed=9)
    p["W1"] *= 30  # make the hidden layer leave the linear regime of tanh
    win, _ = workloads.batch(w, 1, B)
    ctx = pg().Context(w.V, w.d, w.win, w.H, max_batch=B)
    s = host(ctx.score(params_dev(p), dev(win)))
    r = oracle.score(p, win)
    np.testing.assert_allclose(s, r, rtol=1e-5, atol=1e-6 * np.max(np.abs(r)))


# --------------------------------------------- the general advanced-indexing op

_FMT = {"f32": (np.float32, 0), "bf16": (np.uint16, 1), "f16": (np.float16, 2)}


def _to_dev(a, fmt):
    t = torch.from_numpy(np.ascontiguousarray(a))
    if fmt == "bf16":
        t = t.view(torch.int16).view(torch.bfloat16)
    return t.cuda()


def _to_host(t, fmt):
    torch.cuda.synchronize()
    if fmt == "bf16":
        return t.view(torch.int16).cpu().numpy().view(np.uint16)
    return t.cpu().numpy()


def _format_inputs(rng, fmt, rows, d, N, s, idx_dtype):
    code = _FMT[fmt][1]
    t64 = rng.normal(0, 0.01, (rows, d))
    y64 = rng.normal(0, 1e-3, (N, d))
    if fmt == "f32":
        t0, Y = t64.astype(np.float32), y64.astype(np.float32)
    elif fmt == "f16":
        t0, Y = t64.astype(np.float16), y64.astype(np.float16)
    else:
        t0, Y = oracle.encode(t64, code), oracle.encode(y64, code)
    idx = workloads.zipf_ids(rng, rows, s, N).astype(idx_dtype)
    return t0, Y, idx


def _format_bound(fmt, t0, idx, Y, alpha, ref_vals):
    """One unit in the last place of the storage format at the reference
    value (the once-per-row rounding may land on the other side of a
    rounding boundary) plus the float32 accumulation bound of the sums."""
    code = _FMT[fmt][1]
    tv = oracle.decode(t0, code) if fmt == "bf16" else t0.astype(np.float64)
    yv = oracle.decode(Y, code) if fmt == "bf16" else Y.astype(np.float64)
    acc = scatter_bound(tv, idx, yv, alpha)
    a = np.abs(ref_vals).astype(np.float32)
    if fmt == "bf16":
        ulp = np.spacing(a).astype(np.float64) * 2.0 ** 16
    elif fmt == "f16":
        ulp = np.spacing(np.abs(ref_vals).astype(np.float16)).astype(np.float64)
    else:
        ulp = np.zeros_like(acc)
    return ulp + acc


@pytest.mark.parametrize("fmt", ["f32", "bf16", "f16"])
@pytest.mark.parametrize("op", [0, 1])
@pytest.mark.parametrize("rows,d,N,s,idx_dtype", [
    (50, 8, 400, 1.2, np.int32), (1000, 33, 5000, 1.2, np.int64), (100_000, 64, 20_000, 1.2, np.int32),
    (3, 4, 1, 1.0, np.int64), (7, 256, 3000, 1.5, np.int32), (100_000, 1, 9000, 1.1, np.int64),
    (20_000, 17, 140_000, 1.2, np.int64),
])
def test_scatter_update_matches_oracle(fmt, op, rows, d, N, s, idx_dtype):
    """Every storage format and op, int32 and int64 indices, widths that are
    not multiples of 4, the partition-sorted (N <= 8192) and the chunked list
    (32-entry chunks above 131072, with heavy rows in the fix-up)."""
    rng = np.random.default_rng(rows * 7 + N + d)
    t0, Y, idx = _format_inputs(rng, fmt, rows, d, N, s, idx_dtype)
    alpha = -0.75
    ctx = pg().Context(1000, 16, 5, 8, max_batch=1, max_scatter=N, max_rows=rows)
    td = _to_dev(t0, fmt)
    ctx.scatter_update(td, dev(idx), _to_dev(Y, fmt), alpha, op)
    assert ctx.status() == pg().OK
    got = _to_host(td, fmt)
    ref = t0.copy()
    oracle.scatter_add_ex(ref, idx, Y, alpha, op, bf16=fmt == "bf16")
    untouched = np.setdiff1d(np.arange(rows), idx)
    assert np.array_equal(got[untouched], t0[untouched])
    if op == 1:  # assignment copies bits
        assert np.array_equal(got, ref)
        return
    code = _FMT[fmt][1]
    gv = oracle.decode(got, code) if fmt == "bf16" else got.astype(np.float64)
    rv = oracle.decode(ref, code) if fmt == "bf16" else ref.astype(np.float64)
    assert np.all(np.abs(gv - rv) <= _format_bound(fmt, t0, idx, Y, alpha, rv))


def test_scatter_update_bf16_full_size_and_deterministic():
    """The standalone scatter-add workload (327,680 Zipf(1.2) rows into
    100000 x 64) on a bfloat16 table: against the oracle, and two calls
    bit-identical."""
    table, idx, Y = workloads.scatter_inputs()
    t0 = oracle.encode(table.astype(np.float64), 1)
    Yb = oracle.encode(Y.astype(np.float64), 1)
    ctx = pg().Context(1000, 16, 5, 8, max_batch=1, max_scatter=idx.size, max_rows=table.shape[0])
    outs = []
    for _ in range(2):
        td = _to_dev(t0, "bf16")
        ctx.scatter_update(td, dev(idx.astype(np.int64)), _to_dev(Yb, "bf16"), 1.0)
        assert ctx.status() == pg().OK
        outs.append(_to_host(td, "bf16"))
    assert np.array_equal(outs[0], outs[1])
    ref = t0.copy()
    oracle.scatter_add_ex(ref, idx, Yb, 1.0, 0, bf16=True)
    rv = oracle.decode(ref, 1)
    assert np.all(np.abs(oracle.decode(outs[0], 1) - rv) <= _format_bound("bf16", t0, idx, Yb, 1.0, rv))


def test_scatter_update_bad_int64_index_leaves_table_untouched():
    m = pg()
    rng = np.random.default_rng(3)
    t0 = rng.normal(0, 1, (10, 3)).astype(np.float16)
    Y = np.ones((3, 3), np.float16)
    ctx = m.Context(1000, 16, 5, 8, max_batch=1, max_scatter=3, max_rows=10)
    for bad in (10, -1, 1 << 33):
        for op in (m.OP_INC, m.OP_SET):
            td = _to_dev(t0, "f16")
            ctx.scatter_update(td, dev(np.array([1, bad, 2], np.int64)), _to_dev(Y, "f16"), 1.0, op)
            assert ctx.status() == m.EID
            assert np.array_equal(_to_host(td, "f16"), t0)
            assert ctx.status() == m.OK


def test_scatter_update_rejects_unsupported_combinations():
    m = pg()
    ctx = m.Context(1000, 16, 5, 8, max_batch=1, max_scatter=4, max_rows=10)
    idx = dev(np.zeros(4, np.int32))
    tb = torch.zeros(10, 8, dtype=torch.bfloat16, device="cuda")
    Yb = torch.zeros(4, 8, dtype=torch.bfloat16, device="cuda")
    with pytest.raises(m.PolyglotError):
        ctx.scatter_update(tb, idx, Yb, 1.0, m.OP_INC, m.SCATTER_ATOMIC)
    tf = torch.zeros(10, 8, dtype=torch.float32, device="cuda")
    Yf = torch.zeros(4, 8, dtype=torch.float32, device="cuda")
    with pytest.raises(m.PolyglotError):
        ctx.scatter_update(tf, idx, Yf, 1.0, m.OP_SET, m.SCATTER_ATOMIC)
    ctx.scatter_update(tf, idx, Yf, 1.0, m.OP_INC, m.SCATTER_ATOMIC)
    assert ctx.status() == m.OK


def test_scatter_update_host_validation_enqueues_nothing():
    """Bad storage format, index width, row width, op, mode, N, and
    misaligned pointers are refused on the host (EINVAL / EBATCH / ENULL)
    and leave the table untouched."""
    m = pg()
    lib = m.load_library()
    ctx = m.Context(1000, 16, 5, 8, max_batch=1, max_scatter=8, max_rows=10)
    t = torch.zeros(10 * 8 + 1, dtype=torch.float16, device="cuda")
    Y = torch.ones(8 * 8 + 1, dtype=torch.float16, device="cuda")
    idx = torch.zeros(9, dtype=torch.int64, device="cuda")
    tp, yp, ip = t.data_ptr(), Y.data_ptr(), idx.data_ptr()
    good = dict(table=tp, dtype=m.F16, rows=10, d=8, idx=ip, idx_bytes=8, Y=yp, N=8, alpha=1.0,
                op=m.OP_INC, mode=m.SCATTER_SORTED)
    bad = [({"dtype": 3}, m.EINVAL), ({"idx_bytes": 2}, m.EINVAL), ({"d": 0}, m.EINVAL),
           ({"d": 257}, m.EINVAL), ({"rows": 11}, m.EINVAL), ({"op": 2}, m.EINVAL),
           ({"mode": 2}, m.EINVAL), ({"N": 9}, m.EBATCH), ({"N": 0}, m.EBATCH),
           ({"table": tp + 1}, m.EINVAL), ({"Y": yp + 1}, m.EINVAL), ({"idx": ip + 4}, m.EINVAL),
           ({"alpha": float("inf")}, m.EINVAL), ({"table": None}, m.ENULL),
           ({"mode": m.SCATTER_ATOMIC}, m.EINVAL)]
    for change, code in bad:
        a = dict(good, **change)
        rc = lib.polyglot_scatter_update(ctx._h, a["table"], a["dtype"], a["rows"], a["d"], a["idx"],
                                         a["idx_bytes"], a["Y"], a["N"], a["alpha"], a["op"],
                                         a["mode"])
        assert rc == code, (change, rc)
    assert ctx.status() == m.OK
    assert torch.count_nonzero(t).item() == 0
    # the same arguments unchanged are accepted
    rc = lib.polyglot_scatter_update(ctx._h, tp, m.F16, 10, 8, ip, 8, yp, 8, 1.0, m.OP_INC,
                                     m.SCATTER_SORTED)
    assert rc == m.OK and ctx.status() == m.OK
    assert torch.count_nonzero(t).item() == 8


@pytest.mark.parametrize("fmt", ["bf16", "f16"])
def test_scatter_update_widest_rows_long_list(fmt):
    """d = 256 (four column blocks per row) on a 140,000-entry list: the
    32-entry-chunk apply and the fix-up of heavy rows, every column block."""
    rows, d, N = 3000, 256, 140_000
    rng = np.random.default_rng(77)
    t0, Y, idx = _format_inputs(rng, fmt, rows, d, N, 1.1, np.int32)
    ctx = pg().Context(1000, 16, 5, 8, max_batch=1, max_scatter=N, max_rows=rows)
    td = _to_dev(t0, fmt)
    ctx.scatter_update(td, dev(idx), _to_dev(Y, fmt), 0.5)
    assert ctx.status() == pg().OK
    got = _to_host(td, fmt)
    ref = t0.copy()
    oracle.scatter_add_ex(ref, idx, Y, 0.5, 0, bf16=fmt == "bf16")
    code = _FMT[fmt][1]
    gv = oracle.decode(got, code) if fmt == "bf16" else got.astype(np.float64)
    rv = oracle.decode(ref, code) if fmt == "bf16" else ref.astype(np.float64)
    assert np.all(np.abs(gv - rv) <= _format_bound(fmt, t0, idx, Y, 0.5, rv))
    untouched = np.setdiff1d(np.arange(rows), idx)
    assert np.array_equal(got[untouched], t0[untouched])


def _offset_view(a, fmt):
    """The array on the device one element past a 4-byte boundary: rows are
    no longer whole 32-bit words, so 16-bit increments take the one-row walk
    instead of the packed one."""
    flat = np.concatenate([np.zeros(1, a.dtype), np.ascontiguousarray(a).reshape(-1)])
    t = _to_dev(flat, fmt)[1:].view(a.shape)
    assert t.data_ptr() % 4 == 2
    return t


@pytest.mark.parametrize("fmt", ["bf16", "f16"])
@pytest.mark.parametrize("rows,d,N", [(100_000, 64, 327_680), (3000, 128, 20_000), (500, 2, 6000)])
def test_scatter_update_packed_and_one_row_walks(fmt, rows, d, N):
    """Even widths from 4-byte aligned pointers (two rows per load and store)
    and the same inputs one element off that alignment (one row per load),
    chunked and partition-sorted lists: both against the oracle."""
    rng = np.random.default_rng(d * 31 + N)
    t0, Y, idx = _format_inputs(rng, fmt, rows, d, N, 1.2, np.int32)
    ref = t0.copy()
    oracle.scatter_add_ex(ref, idx, Y, -0.5, 0, bf16=fmt == "bf16")
    code = _FMT[fmt][1]
    rv = oracle.decode(ref, code) if fmt == "bf16" else ref.astype(np.float64)
    bound = _format_bound(fmt, t0, idx, Y, -0.5, rv)
    untouched = np.setdiff1d(np.arange(rows), idx)
    ctx = pg().Context(1000, 16, 5, 8, max_batch=1, max_scatter=N, max_rows=rows)
    for aligned in (True, False):
        td = _to_dev(t0, fmt) if aligned else _offset_view(t0, fmt)
        Yd = _to_dev(Y, fmt) if aligned else _offset_view(Y, fmt)
        ctx.scatter_update(td, dev(idx), Yd, -0.5)
        assert ctx.status() == pg().OK
        got = _to_host(td.contiguous(), fmt)
        gv = oracle.decode(got, code) if fmt == "bf16" else got.astype(np.float64)
        assert np.all(np.abs(gv - rv) <= bound), aligned
        assert np.array_equal(got[untouched], t0[untouched]), aligned


def _shifted(a, fmt, k):
    """The array on the device k elements past a 256-byte boundary."""
    flat = np.concatenate([np.zeros(k, a.dtype), np.ascontiguousarray(a).reshape(-1)])
    return _to_dev(flat, fmt)[k:].view(a.shape)


@pytest.mark.parametrize("fmt", ["f32", "bf16", "f16"])
@pytest.mark.parametrize("rows,d,N", [(100_000, 64, 327_680), (700, 6, 3000), (5000, 24, 40_000)])
def test_scatter_update_assignment_word_widths(fmt, rows, d, N):
    """The assignment copies rows in the widest words that divide a row and
    both pointers' alignment: pointers 0, 1, 2 and 4 elements past a 256-byte
    boundary give 16-, 2-, 4- and 8-byte words (16-bit formats) or 16-, 4-,
    8- and 16-byte words (float32), the last entry of each row winning,
    bit-exact against the oracle."""
    rng = np.random.default_rng(d * 7 + N)
    t0, Y, idx = _format_inputs(rng, fmt, rows, d, N, 1.2, np.int32)
    ref = t0.copy()
    oracle.scatter_add_ex(ref, idx, Y, 1.0, 1, bf16=fmt == "bf16")
    ctx = pg().Context(1000, 16, 5, 8, max_batch=1, max_scatter=N, max_rows=rows)
    for k in (0, 1, 2, 4):
        td, Yd = _shifted(t0, fmt, k), _shifted(Y, fmt, k)
        ctx.scatter_update(td, dev(idx), Yd, 1.0, pg().OP_SET)
        assert ctx.status() == pg().OK
        assert np.array_equal(_to_host(td.contiguous(), fmt), ref), k


@pytest.mark.parametrize("fmt", ["bf16", "f16"])
def test_scatter_update_int64_ids_lookback_sort(fmt):
    """int64 ids are narrowed and range-checked by the sort's own key loads
    in every sort form; 1,200,000 entries take the look-back sort (beyond the
    bucketed sort's 786,432): against the oracle, then the same call with
    one id out of range (past the first tile) leaves the table untouched."""
    rows, d, N = 200_000, 8, 1_200_000
    rng = np.random.default_rng(1200)
    t0, Y, idx = _format_inputs(rng, fmt, rows, d, N, 1.1, np.int64)
    ctx = pg().Context(1000, 16, 5, 8, max_batch=1, max_scatter=N, max_rows=rows)
    td = _to_dev(t0, fmt)
    ctx.scatter_update(td, dev(idx), _to_dev(Y, fmt), -0.5)
    assert ctx.status() == pg().OK
    got = _to_host(td, fmt)
    ref = t0.copy()
    oracle.scatter_add_ex(ref, idx, Y, -0.5, 0, bf16=fmt == "bf16")
    code = _FMT[fmt][1]
    gv = oracle.decode(got, code) if fmt == "bf16" else got.astype(np.float64)
    rv = oracle.decode(ref, code) if fmt == "bf16" else ref.astype(np.float64)
    assert np.all(np.abs(gv - rv) <= _format_bound(fmt, t0, idx, Y, -0.5, rv))
    untouched = np.setdiff1d(np.arange(rows), idx)
    assert np.array_equal(got[untouched], t0[untouched])
    bad = idx.copy()
    bad[N - 7] = rows
    td = _to_dev(t0, fmt)
    ctx.scatter_update(td, dev(bad), _to_dev(Y, fmt), -0.5)
    assert ctx.status() == pg().EID
    assert np.array_equal(_to_host(td, fmt), t0)
    assert ctx.status() == pg().OK
