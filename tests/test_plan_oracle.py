"""Pins of the plan oracle: hand-computed plans and closed-form properties."""
import numpy as np
import pytest

import oracle
from synth import configs, generate as G
from golden_io import load_plan
from plan_checks import check_plan


@pytest.mark.parametrize("name", ["plan_small_w3.txt", "plan_small_w3_exact.txt", "plan_small_w8.txt"])
def test_golden_plan(name):
    c = load_plan(name)
    p = oracle.plan(list(c["dims"]), c["dtypes"], c["out_dtype"], c["offsets"], c["batch"], c["total_ids"],
                    c["chunk_rows"], c["item_cost"], c["waves"], c["flags"])
    for key in ("header", "col_base", "id_base", "bag_item_base", "bag_cost_base", "wave_item_begin",
                "wave_bag", "wave_bag_base", "head_first", "split_pieces", "split_last"):
        assert np.array_equal(p[key], c[key]), key


def _rand_plan_case(rng):
    T = int(rng.integers(1, 6))
    B = int(rng.integers(0, 10))
    dims = [int(rng.choice([1, 2, 4, 6, 8, 16, 64])) for _ in range(T)]
    dtypes = [int(rng.integers(0, 2)) if d % 2 == 0 else 0 for d in dims]
    lengths = rng.integers(0, 71, size=(T, B)) * (rng.random((T, B)) < 0.8)
    return T, B, dims, dtypes, lengths.astype(np.int64)


@pytest.mark.parametrize("seed", range(60))
def test_random_small_plans(seed):
    rng = np.random.default_rng(seed)
    T, B, dims, dtypes, lengths = _rand_plan_case(rng)
    offs = G.offsets_from_lengths(lengths) if B else np.zeros((T, 1), np.int32)
    total = int(lengths.sum())
    N_est = max(1, T * B + total)
    for C in (1, 3, 32):
        for K in (1, 64):
            for Wr in (1, 2, 7, N_est, N_est + 5):
                for flags in (0, 2):
                    out_dtype = int(rng.integers(0, 2))
                    p = oracle.plan(dims, dtypes, out_dtype, offs, B, total, C, K, Wr, flags)
                    check_plan(p, dims, dtypes, out_dtype, lengths.reshape(T, B), C, K, Wr, flags, total)


def test_brute_force_partition_tiny():
    """Enumerate items one by one and search targets linearly (Python ints)."""
    rng = np.random.default_rng(11)
    for _ in range(200):
        T, B, dims, dtypes, lengths = _rand_plan_case(rng)
        if B == 0:
            continue
        offs = G.offsets_from_lengths(lengths)
        C, K, Wr = int(rng.integers(1, 9)), int(rng.integers(1, 100)), int(rng.integers(1, 40))
        flags = int(rng.choice([0, 2]))
        out_dtype = int(rng.integers(0, 2))
        p = oracle.plan(dims, dtypes, out_dtype, offs, B, int(lengths.sum()), C, K, Wr, flags)
        items = []                      # (bag, cost, is_first_of_bag)
        for t in range(T):
            rb = dims[t] * (2 if dtypes[t] else 4)
            ob = dims[t] * (2 if out_dtype else 4)
            for b in range(B):
                L = int(lengths[t, b])
                j = 0
                while True:
                    rows = max(0, min(L, (j + 1) * C) - j * C)
                    items.append((t * B + b, rows * rb + (ob if j == 0 else 0) + K, j == 0))
                    j += 1
                    if j * C >= L:
                        break
        N = len(items)
        E = [0]
        for it in items:
            E.append(E[-1] + it[1])
        S = E[-1]
        W = min(Wr, N)
        bag_end = {}
        for i, it in enumerate(items):
            bag_end[it[0]] = i + 1
        expect = []
        for w in range(W + 1):
            c = -(-w * S // W)
            i = next(k for k in range(N + 1) if E[k] >= c)
            if i < N and not items[i][2] and not (flags & 2):
                e = bag_end[items[i][0]]
                if E[e] - c <= S // (2 * W):
                    i = e
            expect.append(i)
        assert list(p["wave_item_begin"]) == expect


@pytest.mark.parametrize("key,batch", [(1, None), (2, None), (3, None), (4, None),
                                       (5, 1), (5, 16), (5, 128), (5, 512), (5, 4096)])
def test_config_plans(key, batch):
    cfg = configs.get(key, batch=batch)
    lengths = G.bag_lengths(cfg)
    offs = None if cfg.all_onehot else G.offsets_from_lengths(lengths)
    dims = [cfg.dim(t) for t in range(cfg.num_tables)]
    dtypes = [1 if cfg.dtype == configs.F16 else 0] * cfg.num_tables
    out_dtype = 1 if cfg.out_dtype == configs.F16 else 0
    total = int(lengths.sum())
    for Wr in (2048, 100000):
        p = oracle.plan(dims, dtypes, out_dtype, offs, cfg.batch, total, 32, 64, Wr, 0)
        check_plan(p, dims, dtypes, out_dtype, lengths, 32, 64, Wr, 0, total)


def test_bad_offsets_rejected():
    dims, dtypes = [4, 4], [0, 0]
    good = np.array([[0, 1, 3], [0, 2, 2]], np.int32)
    oracle.plan(dims, dtypes, 0, good, 2, 5, 32, 64, 8)
    for bad, total in ((np.array([[1, 1, 3], [0, 2, 2]], np.int32), 5),
                       (np.array([[0, 3, 1], [0, 2, 2]], np.int32), 3),
                       (good, 6)):
        with pytest.raises(oracle.OracleError) as e:
            oracle.plan(dims, dtypes, 0, bad, 2, total, 32, 64, 8)
        assert e.value.code == oracle.BAD_OFFSETS


def test_empty_batch_plan():
    p = oracle.plan([4], [0], 0, np.zeros((1, 1), np.int32), 0, 0, 32, 64, 8)
    assert p["header"][3] == 0 and p["header"][9] == 0 and list(p["wave_item_begin"]) == [0]


def waves_from_items(bib, wib):
    """The per-wave arrays by brute force: every item is assigned to the wave whose
    range holds it, and every bag to the set of waves holding its items.  A bag held
    by several waves is split: its first wave records the last one and how many
    waves hold items of it, and every boundary after the first wave up to the last
    one starts inside the bag and points back to the first wave."""
    bib = [int(x) for x in bib]
    wib = [int(x) for x in wib]
    TB, W, N = len(bib) - 1, len(wib) - 1, bib[-1]
    item_bag = []
    for bag in range(TB):
        item_bag += [bag] * (bib[bag + 1] - bib[bag])
    item_wave = []
    for i in range(N):
        item_wave.append(next(w for w in range(W) if wib[w] <= i < wib[w + 1]))
    wave_bag = [item_bag[wib[w]] if wib[w] < N else TB for w in range(W + 1)]
    wave_bag_base = [bib[b] for b in wave_bag]
    hf, sp, sl = [-1] * W, [0] * W, [-1] * W
    for bag in range(TB):
        held = sorted({item_wave[i] for i in range(bib[bag], bib[bag + 1])})
        if len(held) > 1:
            first, last = held[0], held[-1]
            sp[first], sl[first] = len(held), last
            for w in range(first + 1, last + 1):
                hf[w] = first
    return {"wave_bag": wave_bag, "wave_bag_base": wave_bag_base, "head_first": hf, "split_pieces": sp,
            "split_last": sl}


def test_wave_arrays_brute_force():
    """The oracle's per-wave arrays (closed forms of the wave starts) against the
    item-by-item assignment, on random small plans of every kind: snapped and
    exact boundaries, empty waves (W close to or above N), one-row chunks."""
    rng = np.random.default_rng(23)
    checked = 0
    for _ in range(300):
        T, B, dims, dtypes, lengths = _rand_plan_case(rng)
        offs = G.offsets_from_lengths(lengths) if B else np.zeros((T, 1), np.int32)
        total = int(lengths.sum())
        C, K = int(rng.choice([1, 2, 5, 32])), int(rng.choice([1, 7, 64]))
        Wr = int(rng.choice([1, 2, 3, 9, 40, 400]))
        flags = int(rng.choice([0, 2]))
        p = oracle.plan(dims, dtypes, int(rng.integers(0, 2)), offs, B, total, C, K, Wr, flags)
        ref = waves_from_items(p["bag_item_base"], p["wave_item_begin"])
        for k, v in ref.items():
            assert list(p[k]) == v, (k, list(p[k]), v)
        checked += int(np.count_nonzero(p["split_pieces"]))
    assert checked > 100     # many split bags were exercised
