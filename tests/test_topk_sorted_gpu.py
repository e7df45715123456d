"""htam_topk_sorted: the row merge that reads sorted lists only as far as they
can reach the top-k. On lists sorted as htam_attend_transitions returns them
(descending score, ties to the lower id, padding at the end) its outputs must
equal htam_topk's bit for bit: ids, scores, weights, row statistics, counts.
The cases cover padding (short and empty lists, empty rows), exact score ties,
lists without ids (ids are positions), top_k above lists x k_in (no bound),
more than 64 lists (merged by the unsorted kernel) and rows without softmax
statistics."""
import numpy as np
import pytest
import torch

from gpu_cases import say, to_np

pytestmark = pytest.mark.gpu


def sorted_lists(rng, rows, lists, k_in, ties, with_ids, pad):
    """[rows][lists][k_in] scores and ids, each list sorted by descending score
    then ascending id, its padding (-inf, -1) at the end."""
    if ties:
        sc = rng.integers(-6, 6, size=(rows, lists, k_in)).astype(np.float32) / 4
    else:
        sc = rng.standard_normal((rows, lists, k_in)).astype(np.float32)
    if not with_ids:                    # ids are positions: scores descending along each list
        return -np.sort(-sc, axis=2), None
    ids = np.stack([rng.permutation(lists * k_in).reshape(lists, k_in) for _ in range(rows)])
    ids = ids.astype(np.int32)
    valid = np.full((rows, lists), k_in)
    if pad:
        valid = rng.integers(0, k_in + 1, size=(rows, lists))
        valid[0] = 0                    # an empty row
    for r in range(rows):
        for l in range(lists):
            order = np.lexsort((ids[r, l], -sc[r, l]))     # score descending, then id ascending
            sc[r, l], ids[r, l] = sc[r, l][order], ids[r, l][order]
            sc[r, l, valid[r, l]:] = -np.inf
            ids[r, l, valid[r, l]:] = -1
    return sc, ids


def stats(rng, sc, ids, tau):
    rows, lists, _ = sc.shape
    ok = np.isfinite(sc) if ids is None else ids >= 0
    m = np.where(ok, sc, -np.inf).max(2).astype(np.float32)
    z = np.where(np.isfinite(m), rng.uniform(1.0, 50.0, size=m.shape), 0.0).astype(np.float32)
    return m, z


CASES = [
    # rows, lists, k_in, top_k, ties, ids, pad, stats
    (300, 16, 128, 128, False, True, False, True),    # the before_after shape
    (300, 32, 64, 64, False, True, True, True),       # zipf_large's, padded
    (257, 16, 32, 32, True, True, True, True),        # ties and padding
    (100, 8, 16, 16, True, True, False, True),        # zipf_bf16's
    (64, 5, 40, 24, True, True, True, False),         # lists not a multiple of four, no statistics
    (64, 3, 7, 100, False, True, True, True),         # top_k above lists x k_in: no bound
    (64, 1, 300, 200, True, True, True, True),        # one long list
    (64, 64, 17, 256, False, True, True, True),       # 64 lists, ragged chunks
    (40, 70, 20, 64, False, True, True, True),        # more than 64 lists
    (64, 12, 50, 30, True, False, False, False),      # no ids: positions
]


@pytest.mark.parametrize("rows,lists,k_in,top_k,ties,with_ids,pad,with_stats", CASES)
def test_sorted_merge_equals_general(rows, lists, k_in, top_k, ties, with_ids, pad, with_stats):
    from paper_2605_29734_amd import htam
    say(f"[case] htam_topk_sorted rows={rows} lists={lists} k_in={k_in} top_k={top_k} "
        f"ties={ties} ids={with_ids} pad={pad} stats={with_stats}")
    rng = np.random.default_rng(rows * 1000 + lists * 10 + k_in)
    tau = 0.4
    sc, ids = sorted_lists(rng, rows, lists, k_in, ties, with_ids, pad)
    dev = torch.device("cuda:0")
    t = lambda a: None if a is None else torch.from_numpy(np.ascontiguousarray(a)).to(dev)  # noqa: E731
    sm = sz = None
    if with_stats:
        sm, sz = stats(rng, sc, ids, tau)
    ref = htam.htam_topk(t(sc), t(ids), top_k, t(sm), t(sz), tau)
    got = htam.htam_topk(t(sc), t(ids), top_k, t(sm), t(sz), tau, sorted_lists=True)
    torch.cuda.synchronize()
    for name, a, b in zip(("id", "score", "weight", "row_max", "row_sum", "count"), ref, got):
        if a is None:
            assert b is None
            continue
        np.testing.assert_array_equal(to_np(a), to_np(b), err_msg=name)
