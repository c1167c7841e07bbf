"""Closed-form checks of a work plan (any producer), vectorised with numpy."""
import numpy as np


def item_prefix(bib, bcb, lengths_flat, rb_bag, orow_bag, C, K, items):
    """Cost prefix E at the given item indices, from the bag arrays in closed form."""
    items = np.asarray(items, dtype=np.int64)
    N = bib[-1]
    out = np.empty(items.shape, dtype=np.int64)
    end = items >= N
    out[end] = bcb[-1]
    it = items[~end]
    bag = np.searchsorted(bib, it, side="right") - 1
    j = it - bib[bag]
    L = lengths_flat[bag]
    rows = np.minimum(L, j * C)
    out[~end] = bcb[bag] + rows * rb_bag[bag] + np.where(j > 0, orow_bag[bag], 0) + j * K
    return out


def check_plan(p, dims, dtypes, out_dtype, lengths, C, K, W_req, flags, total_ids):
    """Assert every closed-form property of the plan ``p`` (dict of int64 arrays)."""
    T, B = lengths.shape
    dims = np.asarray(dims, dtype=np.int64)
    esize = np.where(np.asarray(dtypes) == 1, 2, 4)
    osize = 2 if out_dtype == 1 else 4
    rb = dims * esize
    orow = dims * osize
    hdr = p["header"]
    assert list(hdr[[1, 2, 4, 5, 6, 7]]) == [T, B, C, K, out_dtype, flags]
    assert np.array_equal(p["col_base"], np.concatenate([[0], np.cumsum(dims)]))
    nnz = lengths.sum(axis=1)
    assert np.array_equal(p["id_base"], np.concatenate([[0], np.cumsum(nnz)]))
    assert p["id_base"][-1] == total_ids == hdr[11]
    L = lengths.reshape(-1).astype(np.int64)
    n = np.maximum(1, (L + C - 1) // C)
    rb_bag = np.repeat(rb, B)
    orow_bag = np.repeat(orow, B)
    cost = L * rb_bag + orow_bag + n * K
    bib, bcb = p["bag_item_base"], p["bag_cost_base"]
    assert np.array_equal(bib, np.concatenate([[0], np.cumsum(n)]))
    assert np.array_equal(bcb, np.concatenate([[0], np.cumsum(cost)]))
    N, S = int(bib[-1]), int(bcb[-1])
    assert hdr[9] == N and hdr[10] == S and hdr[8] == dims.sum()
    W = min(W_req, N)
    assert hdr[3] == W and hdr[13] == W_req
    wib = p["wave_item_begin"]
    assert len(wib) == W + 1
    if W == 0:
        assert wib[0] == 0 and hdr[12] == 0
        return
    assert wib[0] == 0 and wib[-1] == N
    assert np.all(np.diff(wib) >= 0)
    w = np.arange(W + 1, dtype=object)
    target = np.array([(int(x) * S + W - 1) // W for x in w], dtype=np.int64)
    E_at = item_prefix(bib, bcb, L, rb_bag, orow_bag, C, K, wib)
    E_before = item_prefix(bib, bcb, L, rb_bag, orow_bag, C, K, np.maximum(wib - 1, 0))
    bag_of = np.searchsorted(bib, np.minimum(wib, N - 1), side="right") - 1
    at_bag_start = (wib >= N) | (bib[bag_of] == wib)
    # every boundary reaches its target; an unmoved boundary is the first such item
    assert np.all(E_at >= target)
    slack = -1 if flags & 2 else S // (2 * W)
    moved = E_before >= target
    moved[0] = False
    # a moved boundary sits at a bag start and the move stayed within the slack
    assert np.all(at_bag_start[moved])
    if slack < 0:
        assert not moved.any()
    else:
        assert np.all(E_at[moved] - target[moved] <= slack)
    # an unmoved boundary strictly inside a bag was not allowed to move
    inside = ~at_bag_start
    if slack >= 0 and inside.any():
        rest = bcb[bag_of[inside] + 1] - target[inside]
        assert np.all(rest > slack)
    # per-wave cost stays within target spacing + largest item + slack
    max_item = int(np.max(np.minimum(L, C) * rb_bag + orow_bag + K))
    spacing = -(-S // W)
    assert np.all(np.diff(E_at) <= spacing + max_item + max(slack, 0))
    # split bags: bags cut by an inner boundary
    inner = wib[1:-1]
    inner_in = inner[(inner < N)]
    bags = np.searchsorted(bib, inner_in, side="right") - 1
    cut = bags[bib[bags] < inner_in]
    assert hdr[12] == len(np.unique(cut))
