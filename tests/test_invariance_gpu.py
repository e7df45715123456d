"""Permutation invariance of GPU retrieval (the result is a function of the
memory's content, not of how it is stored or of the batch order):

  * relabelling the clusters (coarse keys and parent ids permuted together)
    changes only the selected ids, by the same permutation; everything else
    is the same bits;
  * reordering the build input, or shuffling the records inside their
    segments, leaves the ids, the scores and the maxima the same bits (every
    score is one MFMA inner product over d, whose order does not depend on
    the record's position); the softmax sums Z, and so the weights, add the
    same terms in another order and agree to the rounding of an fp32 sum;
  * permuting the queries permutes every per-query output, bit for bit: a
    query's results do not depend on its place in its clusters' lists (and
    so on which pass, query tile or kernel instantiation computed them).

Each case runs the one-block and the multi-block routing and the LDS-staged
stream kernel, with segments of several chunks (merged partials)."""
import numpy as np
import pytest
import torch

from gpu_cases import say, to_np
from paper_2605_29734_amd import synth

pytestmark = pytest.mark.gpu
U = 2.0 ** -24

ROW_KEYS = ("id", "score", "m", "count")
SLOT_KEYS = ("slot_max", "slot_score", "slot_id")


def _spec(B):
    # d = 256 (LDS-staged kernel); ~625-row segments cut into 128-row chunks
    return synth.Spec("invariance", B=B, d=256, G=64, N=40000, top_c=4, top_k=32, tau=0.3,
                      storage="bf16", compute="bf16", sizes="zipf", zipf_s=0.8, min_size=50)


def _run(cluster_of, keys_in, coarse, q, spec, bank=None):
    from paper_2605_29734_amd import htam
    if bank is None:
        bank = htam.build_bank(cluster_of, keys_in, coarse, spec.compute)
    out = htam.Retriever(bank, q.shape[0], spec.top_c, spec.top_k, spec.tau).run(q)
    torch.cuda.synchronize()
    return {k: to_np(v) for k, v in out.items()}, bank


def _z_bound(spec, sizes):
    """Relative difference allowed between two fp32 sums of the same positive
    terms in different orders: each sum is within (n_lane + 64) u of the exact
    one, n_lane being the terms one lane adds in sequence (a lane sees 4 of
    every 64 rows of a chunk; 4096 rows is the longest chunk) and 64 bounding
    the depth of the lane, wave, chunk and slot merges after it."""
    n_lane = min(int(sizes.max()), 4096) // 16 + 4
    return 2 * (n_lane + 64) * U


def _same(a, b, keys, what):
    for k in keys:
        np.testing.assert_array_equal(a[k], b[k], err_msg=f"{what}: {k}")


def _same_ids_up_to_ties(a, b, what):
    """Ids in rows whose scores are the same bits. Equal scores are ordered by
    caller id, and reordering the build input renames the records, so among
    records of exactly equal score (they occur: bf16 operands give a coarse
    grid of fp32 sums) the ids may differ; elsewhere they must match."""
    for ik, sk in (("id", "score"), ("slot_id", "slot_score")):
        ia, ib = a[ik].reshape(-1, a[ik].shape[-1]), b[ik].reshape(-1, b[ik].shape[-1])
        sc = a[sk].reshape(ia.shape)
        tied = np.zeros(sc.shape, dtype=bool)
        tied[:, 1:] |= sc[:, 1:] == sc[:, :-1]
        tied[:, :-1] |= sc[:, :-1] == sc[:, 1:]
        # a tie group at the end of the list may continue past the k-th entry
        tied |= (sc == sc[:, -1:]) & np.isfinite(sc)
        diff = (ia != ib) & ~tied
        assert not diff.any(), f"{what}: {ik} differs outside exact ties at {np.argwhere(diff)[:5]}"
        assert (ia != ib).sum() <= tied.sum()


def _close_z(a, b, tol, what):
    for k in ("Z", "slot_sum"):
        x, y = a[k].astype(np.float64), b[k].astype(np.float64)
        zero = x == 0
        assert np.array_equal(zero, y == 0), f"{what}: empty {k} differ"
        rel = np.abs(x[~zero] - y[~zero]) / x[~zero]
        assert rel.max(initial=0) <= tol, f"{what}: {k} differs by {rel.max()} > {tol}"
    w = a["weight"].astype(np.float64)
    rel = np.abs(w - b["weight"]) / np.where(w > 0, w, 1)
    assert rel.max() <= tol + 4 * U, f"{what}: weights differ by {rel.max()}"


@pytest.mark.parametrize("B", [200, 4200])         # one-block and multi-block routing
def test_permutation_invariance(B):
    from paper_2605_29734_amd import htam
    spec = _spec(B)
    say(f"[case] permutation invariance B={B}")
    w = synth.make(spec, device="cuda", seed=11)
    cl, kin, ck, q = w.cluster_of, w.keys_in, w.coarse_keys, w.queries
    base, bank = _run(cl, kin, ck, q, spec)
    tol = _z_bound(spec, w.sizes)
    rng = np.random.default_rng(7)

    say("[step] relabelled clusters")
    pi = rng.permutation(spec.G)
    pit = torch.from_numpy(pi).to("cuda")
    ck2 = torch.empty_like(ck)
    ck2[pit] = ck                                   # cluster g is now called pi[g]
    out, _ = _run(pit[cl.long()].to(torch.int32), kin, ck2, q, spec)
    np.testing.assert_array_equal(out["sel"], pi[base["sel"]])
    _same(out, base, ROW_KEYS + SLOT_KEYS + ("sel_score", "Z", "slot_sum", "weight"),
          "relabelled clusters")

    say("[step] reordered build input")
    sigma = torch.from_numpy(rng.permutation(spec.N)).to("cuda")
    out, _ = _run(cl[sigma], kin[sigma], ck, q, spec)
    sg = to_np(sigma)
    for k in ("id", "slot_id"):                     # ids name input records: map back
        out[k] = np.where(out[k] >= 0, sg[np.maximum(out[k], 0)], -1)
    _same(out, base, ("score", "m", "count", "slot_max", "slot_score", "sel", "sel_score"),
          "reordered build input")
    _same_ids_up_to_ties(out, base, "reordered build input")
    _close_z(out, base, tol, "reordered build input")

    say("[step] records shuffled inside their segments")
    off = to_np(bank.seg_offsets)
    perm = np.arange(spec.N)
    for g in range(spec.G):
        a, b = int(off[g]), int(off[g + 1])
        perm[a:b] = a + rng.permutation(b - a)
    pt = torch.from_numpy(perm).to("cuda")
    shuffled = htam.Bank(coarse_keys=ck, fine_keys=bank.fine_keys[pt].contiguous(),
                         seg_offsets=bank.seg_offsets, transition_id=bank.transition_id[pt].contiguous(),
                         compute=spec.compute)
    out, _ = _run(None, None, None, q, spec, bank=shuffled)
    _same(out, base, ROW_KEYS + SLOT_KEYS + ("sel", "sel_score"), "shuffled segments")
    _close_z(out, base, tol, "shuffled segments")

    say("[step] permuted queries")
    rho = rng.permutation(B)
    out, _ = _run(None, None, None, q[torch.from_numpy(rho).to("cuda")].contiguous(), spec,
                  bank=bank)
    for k in base:
        np.testing.assert_array_equal(out[k], base[k][rho], err_msg=f"permuted queries: {k}")
