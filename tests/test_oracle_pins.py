"""Pins of the CPU oracle against facts that do not come from the oracle itself.

Each test fixes the oracle to something independent: a hand-derived worked
example, closed forms of the temperature softmax, a brute-force flat retrieval
(the top_c = G special case, computed with numpy's own sort), numpy's stable
argsort for the memory build, bit-level bf16 rounding cases, torch's bf16
conversion, planted matches and invariances. A plausible slip in the oracle
(a dropped term, a wrong sign or index, a transposed operand, a missing mask)
fails at least one of them.
"""
import json
import math
import os
from fractions import Fraction

import numpy as np
import pytest
import torch

import oracle

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _num(x):
    if isinstance(x, str):
        if x == "-inf":
            return -math.inf
        return float(Fraction(x))
    return float(x)


def _arr(x):
    return np.vectorize(_num, otypes=[np.float64])(np.array(x, dtype=object))


def _unit(rng, n, d):
    x = rng.standard_normal((n, d))
    return (x / np.linalg.norm(x, axis=1, keepdims=True)).astype(np.float32)


def _bank(rng, G, sizes, d):
    """Random segment-contiguous bank: offsets, keys, and shuffled caller ids."""
    off = np.zeros(G + 1, dtype=np.int64)
    off[1:] = np.cumsum(sizes)
    N = int(off[-1])
    keys = _unit(rng, N, d) if N else np.zeros((0, d), np.float32)
    tid = rng.permutation(N).astype(np.int32)
    return off, keys, tid


# ---------------------------------------------------------------------------
# hand-derived worked example (tests/golden/worked_example.json)
# ---------------------------------------------------------------------------
def test_worked_example_exact():
    ex = json.load(open(os.path.join(GOLDEN, "worked_example.json")))
    G = len(ex["coarse_keys"])
    off, tid = oracle.build_bank(ex["cluster_of"], G)
    keys = np.asarray(ex["keys"], np.float32)[tid]
    r = oracle.retrieve(np.asarray(ex["queries"], np.float32), np.asarray(ex["coarse_keys"], np.float32),
                        off, ex["top_c"], ex["top_k"], ex["tau"], "f32", keys=keys,
                        transition_id=tid)
    e = ex["expect"]
    np.testing.assert_array_equal(r["own_sel"], e["sel"])
    np.testing.assert_allclose(r["own_sel_score"], _arr(e["sel_score"]), rtol=0, atol=1e-12)
    np.testing.assert_array_equal(r["id"], e["id"])
    np.testing.assert_allclose(r["score"], _arr(e["score"]), rtol=0, atol=1e-12)
    np.testing.assert_allclose(r["weight"], _arr(e["weight"]), rtol=1e-12, atol=1e-15)
    np.testing.assert_allclose(r["m"], _arr(e["m"]), rtol=0, atol=1e-12)
    np.testing.assert_allclose(r["Z"], _arr(e["Z"]), rtol=1e-12)
    np.testing.assert_array_equal(r["count"], e["count"])
    np.testing.assert_array_equal(r["slot_id"], e["slot_id"])
    np.testing.assert_allclose(r["slot_score"], _arr(e["slot_score"]), rtol=0, atol=1e-12)
    np.testing.assert_allclose(r["slot_m"], _arr(e["slot_m"]), rtol=0, atol=1e-12)
    np.testing.assert_allclose(r["slot_Z"], _arr(e["slot_Z"]), rtol=1e-12)


# ---------------------------------------------------------------------------
# O0: bf16 rounding
# ---------------------------------------------------------------------------
@pytest.mark.parametrize("bits,expect", [
    (0x3F800000, 0x3F800000),   # exact
    (0x3F808000, 0x3F800000),   # halfway, even below -> down
    (0x3F818000, 0x3F820000),   # halfway, odd below -> up
    (0x3F808001, 0x3F810000),   # above halfway -> up
    (0x3F807FFF, 0x3F800000),   # below halfway -> down
    (0xBF818000, 0xBF820000),   # negative, halfway, odd -> away from zero
    (0xBF808000, 0xBF800000),   # negative, halfway, even -> toward zero
    (0x7F7FFFFF, 0x7F800000),   # largest float rounds to +inf
    (0x00008000, 0x00000000),   # subnormal halfway, even -> zero
    (0x00018000, 0x00020000),   # subnormal halfway, odd -> up
    (0x80000000, 0x80000000),   # -0 stays -0
])
def test_bf16_rounding_bits(bits, expect):
    x = np.array([bits], dtype=np.uint32).view(np.float32)
    y = oracle.round_bf16(x).view(np.uint32)[0]
    assert int(y) == expect, f"{bits:#x} -> {int(y):#x}, expected {expect:#x}"


def test_bf16_rounding_matches_torch():
    rng = np.random.default_rng(1)
    x = (rng.standard_normal(1 << 16) * np.exp2(rng.integers(-20, 20, 1 << 16))).astype(np.float32)
    ref = torch.from_numpy(x).to(torch.bfloat16).to(torch.float32).numpy()
    np.testing.assert_array_equal(oracle.round_bf16(x).view(np.uint32), ref.view(np.uint32))


# ---------------------------------------------------------------------------
# O1 + O2: coarse selection
# ---------------------------------------------------------------------------
def test_coarse_matches_full_sort():
    rng = np.random.default_rng(2)
    B, G, d, c = 9, 37, 24, 5
    q, C = _unit(rng, B, d), _unit(rng, G, d)
    C[7] = C[3]                       # exact duplicate keys -> exact ties
    sel, sc = oracle.coarse(q, C, c)
    S = q.astype(np.float64) @ C.astype(np.float64).T
    for b in range(B):
        order = np.lexsort((np.arange(G), -S[b]))      # -score, then id
        np.testing.assert_array_equal(sel[b], order[:c])
        np.testing.assert_allclose(sc[b], S[b, order[:c]], rtol=0, atol=1e-12)


def test_coarse_argmax_and_ties_to_lower_id():
    rng = np.random.default_rng(3)
    d = 16
    C = _unit(rng, 6, d)
    C[4] = C[1]
    q = C[[1, 2]].copy()              # query 0 ties clusters 1 and 4 exactly
    sel, _ = oracle.coarse(q, C, 1)
    assert sel[0, 0] == 1
    assert sel[1, 0] == int(np.argmax(q[1].astype(np.float64) @ C.astype(np.float64).T))
    sel2, _ = oracle.coarse(q, C, 2)
    np.testing.assert_array_equal(sel2[0], [1, 4])


# ---------------------------------------------------------------------------
# O5: closed forms of the temperature softmax
# ---------------------------------------------------------------------------
def test_softmax_single_candidate():
    r = oracle.attend([0.3], [7], 0.07, 3)
    assert r["Z"] == 1.0 and r["m"] == 0.3
    np.testing.assert_array_equal(r["id"], [7, -1, -1])
    np.testing.assert_array_equal(r["weight"], [1.0, 0.0, 0.0])
    assert r["score"][1] == -np.inf and r["count"] == 1


def test_softmax_equal_scores_uniform():
    n = 11
    r = oracle.attend(np.full(n, 0.25), np.arange(n)[::-1], 0.5, n, full_weights=True)
    np.testing.assert_allclose(r["w_full"], 1.0 / n, rtol=1e-14)
    np.testing.assert_array_equal(r["id"], np.arange(n))    # ties: ascending id


@pytest.mark.parametrize("tau", [0.07, 1.0, 3.0])
def test_softmax_two_candidates_logistic(tau):
    s1, s2 = 0.41, 0.17
    r = oracle.attend([s2, s1], [0, 1], tau, 2)
    w1 = 1.0 / (1.0 + math.exp(-(s1 - s2) / tau))
    np.testing.assert_allclose(r["weight"], [w1, 1 - w1], rtol=1e-13)
    np.testing.assert_array_equal(r["id"], [1, 0])


def test_softmax_scale_invariance_and_large_tau():
    rng = np.random.default_rng(4)
    s = rng.standard_normal(50)
    ids = np.arange(50)
    a = oracle.attend(s, ids, 0.3, 50, full_weights=True)
    b = oracle.attend(4.0 * s, ids, 1.2, 50, full_weights=True)
    np.testing.assert_allclose(a["w_full"], b["w_full"], rtol=1e-12)
    u = oracle.attend(s, ids, 1e12, 50, full_weights=True)
    np.testing.assert_allclose(u["w_full"], 1 / 50, rtol=1e-9)
    np.testing.assert_allclose(a["w_full"].sum(), 1.0, rtol=1e-13)
    # ordering by weight agrees with ordering by score for tau > 0
    assert np.all(np.diff(a["weight"]) <= 0)


def test_empty_row():
    r = oracle.attend([], [], 1.0, 4)
    assert r["m"] == -np.inf and r["Z"] == 0.0 and r["count"] == 0
    np.testing.assert_array_equal(r["id"], [-1] * 4)
    np.testing.assert_array_equal(r["weight"], [0.0] * 4)


# ---------------------------------------------------------------------------
# whole path: brute-force flat retrieval when every cluster is selected
# ---------------------------------------------------------------------------
@pytest.mark.parametrize("tau", [0.07, 1.0])
def test_top_c_equal_G_is_flat_retrieval(tau):
    rng = np.random.default_rng(5)
    B, G, d, k = 7, 6, 32, 9
    sizes = rng.integers(0, 12, G)
    off, keys, tid = _bank(rng, G, sizes, d)
    q, C = _unit(rng, B, d), _unit(rng, G, d)
    r = oracle.retrieve(q, C, off, G, k, tau, "f32", keys=keys, transition_id=tid)
    S = q.astype(np.float64) @ keys.astype(np.float64).T       # every record
    N = keys.shape[0]
    for b in range(B):
        order = np.lexsort((tid, -S[b]))
        m = S[b].max()
        e = np.exp((S[b] - m) / tau)
        w = e / e.sum()
        kk = min(k, N)
        np.testing.assert_array_equal(r["id"][b, :kk], tid[order[:kk]])
        np.testing.assert_allclose(r["score"][b, :kk], S[b, order[:kk]], rtol=0, atol=1e-12)
        np.testing.assert_allclose(r["weight"][b, :kk], w[order[:kk]], rtol=1e-12)
        np.testing.assert_allclose(r["Z"][b], e.sum(), rtol=1e-12)
        assert r["m"][b] == pytest.approx(m, abs=1e-12)


@pytest.mark.parametrize("tau,compute", [(0.07, "f32"), (1.0, "bf16")])
def test_flat_is_brute_force(tau, compute):
    """oracle.flat against a full numpy sort and softmax over every record."""
    rng = np.random.default_rng(21)
    B, N, d, k = 6, 50, 24, 11
    q, keys = _unit(rng, B, d), _unit(rng, N, d)
    keys[7] = keys[3]                                  # an exact tie: lower caller id first
    tid = rng.permutation(N).astype(np.int32)
    r = oracle.flat(q, keys, tau, k, compute, transition_id=tid)
    qq, kq = (oracle.round_bf16(q), oracle.round_bf16(keys)) if compute == "bf16" else (q, keys)
    S = qq.astype(np.float64) @ kq.astype(np.float64).T
    for b in range(B):
        order = np.lexsort((tid, -S[b]))[:k]
        e = np.exp((S[b] - S[b].max()) / tau)
        np.testing.assert_array_equal(r["id"][b], tid[order])
        np.testing.assert_allclose(r["score"][b], S[b, order], rtol=0, atol=1e-12)
        np.testing.assert_allclose(r["weight"][b], e[order] / e.sum(), rtol=1e-12)
        assert r["Z"][b] == pytest.approx(e.sum(), rel=1e-12) and r["count"][b] == k


def test_flat_ties_go_to_the_lower_id():
    """Two records equal to the query tie at the top: the lower caller id comes
    first, with row indices as ids when the caller gives none."""
    rng = np.random.default_rng(23)
    q, keys = _unit(rng, 2, 16), _unit(rng, 12, 16)
    keys[3] = keys[7] = q[0]
    keys[9] = keys[2] = q[1]
    r = oracle.flat(q, keys, 0.5, 2, "f32")
    np.testing.assert_array_equal(r["id"], [[3, 7], [2, 9]])
    tid = np.array([50, 40, 30, 20, 10, 0, 1, 2, 3, 4, 5, 6], np.int32)
    r = oracle.flat(q, keys, 0.5, 2, "f32", transition_id=tid)
    np.testing.assert_array_equal(r["id"], [[2, 20], [4, 30]])


def test_flat_equals_hierarchy_with_every_cluster():
    """Selecting every cluster (top_c = G) leaves the hierarchy nothing to
    exclude: its row outputs are flat retrieval's, and with fewer clusters
    selected the flat top-1 can only be at least as good."""
    rng = np.random.default_rng(22)
    B, G, d, k = 5, 7, 16, 6
    off, keys, tid = _bank(rng, G, rng.integers(1, 9, G), d)
    q, C = _unit(rng, B, d), _unit(rng, G, d)
    f = oracle.flat(q, keys, 0.5, k, "f32", transition_id=tid)
    h = oracle.retrieve(q, C, off, G, k, 0.5, "f32", keys=keys, transition_id=tid)
    for key in ("id", "count"):
        np.testing.assert_array_equal(f[key], h[key])
    for key in ("score", "weight", "m", "Z"):        # sums taken in another order
        np.testing.assert_allclose(f[key], h[key], rtol=1e-12, atol=1e-300)
    h2 = oracle.retrieve(q, C, off, 2, k, 0.5, "f32", keys=keys, transition_id=tid)
    assert np.all(f["score"][:, 0] >= h2["score"][:, 0])


def test_hierarchy_masks_unselected_clusters():
    """The best record overall sits in a cluster that is not selected: it must not appear."""
    rng = np.random.default_rng(6)
    d = 16
    q = _unit(rng, 1, d)
    C = np.stack([q[0], -q[0], _unit(rng, 1, d)[0]]).astype(np.float32)
    keys = _unit(rng, 9, d)
    keys[7] = q[0]                    # perfect match, placed in cluster 1 (anti-aligned key)
    off = np.array([0, 4, 8, 9], dtype=np.int64)
    r = oracle.retrieve(q, C, off, 1, 9, 1.0, "f32", keys=keys)
    assert r["own_sel"][0, 0] == 0
    assert 7 not in r["id"][0]
    np.testing.assert_array_equal(np.sort(r["id"][0, :4]), [0, 1, 2, 3])
    assert r["count"][0] == 4
    S = (q.astype(np.float64) @ keys[:4].astype(np.float64).T)[0]
    w = np.exp(S - S.max())
    np.testing.assert_allclose(r["weight"][0, :4], np.sort(w / w.sum())[::-1], rtol=1e-12)


def test_planted_match_is_top1():
    rng = np.random.default_rng(7)
    B, G, d = 5, 10, 64
    sizes = rng.integers(3, 9, G)
    off, keys, tid = _bank(rng, G, sizes, d)
    C = _unit(rng, G, d)
    q = _unit(rng, B, d)
    clusters = rng.choice(G, B, replace=False)      # one planted record per distinct cluster
    targets = [int(off[g] + rng.integers(0, off[g + 1] - off[g])) for g in clusters]
    for b, j in enumerate(targets):
        g = int(np.searchsorted(off, j, side="right") - 1)
        q[b] = keys[j]
        C[g] = keys[j]                # the cluster key equals the query: score 1 (unit norm)
    r = oracle.retrieve(q, C, off, 2, 4, 0.07, "f32", keys=keys, transition_id=tid)
    for b, j in enumerate(targets):
        g = int(np.searchsorted(off, j, side="right") - 1)
        assert r["own_sel"][b, 0] == g
        assert r["id"][b, 0] == tid[j]
        exact = float(np.dot(keys[j].astype(np.float64), keys[j].astype(np.float64)))
        assert r["score"][b, 0] == pytest.approx(exact, abs=1e-12)


def test_permutation_invariance():
    """Relabelling clusters and reordering records inside segments leaves every output unchanged."""
    rng = np.random.default_rng(8)
    B, G, d, c, k = 6, 12, 48, 3, 10
    sizes = rng.integers(0, 15, G)
    off, keys, tid = _bank(rng, G, sizes, d)
    q, C = _unit(rng, B, d), _unit(rng, G, d)
    base = oracle.retrieve(q, C, off, c, k, 0.5, "bf16", keys=keys, transition_id=tid)

    perm = rng.permutation(G)                          # new cluster i = old cluster perm[i]
    new_keys, new_tid, new_sizes = [], [], []
    for g in perm:
        a, b = off[g], off[g + 1]
        inner = rng.permutation(b - a)
        new_keys.append(keys[a:b][inner])
        new_tid.append(tid[a:b][inner])
        new_sizes.append(b - a)
    off2 = np.zeros(G + 1, dtype=np.int64)
    off2[1:] = np.cumsum(new_sizes)
    r = oracle.retrieve(q, C[perm], off2, c, k, 0.5, "bf16", keys=np.concatenate(new_keys),
                        transition_id=np.concatenate(new_tid))
    np.testing.assert_array_equal(perm[r["own_sel"]], base["own_sel"])
    for f in ("id", "count"):
        np.testing.assert_array_equal(r[f], base[f])
    for f in ("score", "weight", "m", "Z"):
        np.testing.assert_allclose(r[f], base[f], rtol=1e-12, atol=1e-15)


def test_rows_are_independent():
    rng = np.random.default_rng(9)
    B, G, d = 10, 8, 32
    off, keys, tid = _bank(rng, G, rng.integers(1, 20, G), d)
    q, C = _unit(rng, B, d), _unit(rng, G, d)
    full = oracle.retrieve(q, C, off, 3, 5, 1.0, "f32", keys=keys, transition_id=tid)
    sub = oracle.retrieve(q, C, off, 3, 5, 1.0, "f32", keys=keys, transition_id=tid,
                          rows=[7, 2, 5])
    for f in ("id", "score", "weight", "m", "Z", "count"):
        np.testing.assert_array_equal(sub[f], full[f][[7, 2, 5]])


def test_empty_clusters_and_short_rows():
    rng = np.random.default_rng(10)
    d = 16
    C = _unit(rng, 4, d)
    q = C[[0, 2]].copy()
    keys = _unit(rng, 3, d)
    off = np.array([0, 0, 3, 3, 3], dtype=np.int64)   # only cluster 1 holds records
    r = oracle.retrieve(q, C, off, 1, 4, 1.0, "f32", keys=keys)
    assert r["own_sel"][0, 0] == 0 and r["own_sel"][1, 0] == 2
    for b in range(2):                                  # both rows select an empty cluster
        assert r["count"][b] == 0 and r["m"][b] == -np.inf and r["Z"][b] == 0
        np.testing.assert_array_equal(r["id"][b], [-1] * 4)
    r2 = oracle.retrieve(q, C, off, 2, 4, 1.0, "f32", keys=keys, sel=[[0, 1], [1, 2]])
    np.testing.assert_array_equal(r2["count"], [3, 3])
    assert r2["id"][0, 3] == -1 and r2["weight"][0, 3] == 0.0
    np.testing.assert_allclose(r2["weight"][0, :3].sum(), 1.0, rtol=1e-13)


def test_weights_sum_to_one_and_slots_combine():
    """Row weights sum to 1 over the candidate set; slot (m, Z) combine to the row's (m, Z)."""
    rng = np.random.default_rng(11)
    B, G, d, c = 8, 10, 40, 4
    sizes = rng.integers(1, 30, G)
    off, keys, tid = _bank(rng, G, sizes, d)
    q, C = _unit(rng, B, d), _unit(rng, G, d)
    N = keys.shape[0]
    r = oracle.retrieve(q, C, off, c, N, 0.07, "bf16", keys=keys, transition_id=tid)
    for b in range(B):
        n = r["count"][b]
        assert n == sum(sizes[g] for g in r["own_sel"][b])
        np.testing.assert_allclose(r["weight"][b, :n].sum(), 1.0, rtol=1e-12)
        M = r["slot_m"][b].max()
        Z = np.sum(r["slot_Z"][b] * np.exp((r["slot_m"][b] - M) / 0.07))
        assert r["m"][b] == M
        np.testing.assert_allclose(r["Z"][b], Z, rtol=1e-12)


def test_bf16_compute_quantises_every_operand():
    rng = np.random.default_rng(12)
    B, G, d = 4, 5, 24
    off, keys, tid = _bank(rng, G, np.full(G, 6), d)
    q, C = _unit(rng, B, d), _unit(rng, G, d)
    r = oracle.retrieve(q, C, off, 2, 3, 1.0, "bf16", keys=keys, transition_id=tid)
    qb = torch.from_numpy(q).bfloat16().double().numpy()
    kb = torch.from_numpy(keys).bfloat16().double().numpy()
    for b in range(B):
        for t in range(3):
            j = int(np.nonzero(tid == r["id"][b, t])[0][0])
            assert r["score"][b, t] == pytest.approx(float(qb[b] @ kb[j]), abs=1e-12)


# ---------------------------------------------------------------------------
# memory build
# ---------------------------------------------------------------------------
def test_build_is_stable_counting_sort():
    rng = np.random.default_rng(13)
    G = 17
    cl = rng.integers(0, G, 500).astype(np.int32)
    cl[cl == 5] = 6                     # an empty cluster
    off, tid = oracle.build_bank(cl, G)
    np.testing.assert_array_equal(tid, np.argsort(cl, kind="stable"))
    np.testing.assert_array_equal(np.diff(off), np.bincount(cl, minlength=G))
    assert off[0] == 0 and off[-1] == cl.size


def test_build_rejects_bad_cluster_id():
    with pytest.raises(ValueError):
        oracle.build_bank([0, 3, 1], 3)


# ---------------------------------------------------------------------------
# prefix-aware transition scoring (Eq. score, Eq. prefix_weight)
# ---------------------------------------------------------------------------
def _prefix_inputs(rng, B, G, d, Lmax):
    q, C = _unit(rng, B, d), _unit(rng, G, d)
    E = (rng.standard_normal((G, G, d)) / np.sqrt(d)).astype(np.float32)
    lengths = rng.integers(0, Lmax + 1, B)
    P = np.full((B, Lmax), -1, dtype=np.int32)
    for b in range(B):
        P[b, :lengths[b]] = rng.integers(0, G, lengths[b])
    return q, C, E, P, lengths


def test_prefix_worked_example_exact():
    ex = json.load(open(os.path.join(GOLDEN, "prefix_example.json")))
    sel, ss, S = oracle.coarse_prefix(np.asarray(ex["queries"], np.float32),
                                      np.asarray(ex["coarse_keys"], np.float32),
                                      np.asarray(ex["edge_keys"], np.float32),
                                      np.asarray(ex["prefix"]), math.log(2.0), ex["top_c"], "f32")
    np.testing.assert_allclose(S, _arr(ex["scores"]), rtol=1e-15, atol=1e-15)
    np.testing.assert_array_equal(sel, ex["sel"])


def test_prefix_weights_closed_form():
    a = oracle.prefix_weights(4, math.log(3.0))
    np.testing.assert_allclose(a, [1 / 27, 1 / 9, 1 / 3, 1], rtol=1e-14)
    assert oracle.prefix_weights(0, 1.0).size == 0
    np.testing.assert_array_equal(oracle.prefix_weights(3, 0.0), [1, 1, 1])


def test_prefix_one_term_with_node_edges_is_plain_coarse():
    """Edge keys that repeat the node keys, E[s][g] = c_g, and a one-term
    prefix (alpha = 1): the prefix score is the one-term score <q, c_g>."""
    rng = np.random.default_rng(31)
    B, G, d = 9, 12, 16
    q, C = _unit(rng, B, d), _unit(rng, G, d)
    E = np.broadcast_to(C, (G, G, d)).copy()
    P = rng.integers(0, G, (B, 1)).astype(np.int32)
    sel, ss, S = oracle.coarse_prefix(q, C, E, P, 0.7, 4, "f32")
    sel0, ss0 = oracle.coarse(q, C, 4)
    np.testing.assert_array_equal(sel, sel0)
    np.testing.assert_allclose(ss, ss0, rtol=1e-13, atol=1e-15)


@pytest.mark.parametrize("compute", ["f32", "bf16"])
def test_prefix_against_direct_sums(compute):
    """lam = 0 adds every term with weight 1; a large lam keeps only the most
    recent term; an empty prefix scores the node keys; ids outside [0, G)
    end a prefix."""
    rng = np.random.default_rng(32)
    B, G, d, L = 10, 7, 24, 4
    q, C, E, P, lengths = _prefix_inputs(rng, B, G, d, L)
    P[0] = [3, 5, G, 1]                                 # ends after two entries
    lengths[0] = 2
    qq, cq, eq = ((oracle.round_bf16(q), oracle.round_bf16(C), oracle.round_bf16(E))
                  if compute == "bf16" else (q, C, E))
    qq, cq, eq = (x.astype(np.float64) for x in (qq, cq, eq))
    for lam in (0.0, 60.0):
        _, _, S = oracle.coarse_prefix(q, C, E, P, lam, 3, compute)
        for b in range(B):
            L_b = lengths[b]
            if L_b == 0:
                ref = cq @ qq[b]
            elif lam == 0.0:
                ref = sum(eq[P[b, i]] @ qq[b] for i in range(L_b))
            else:
                ref = eq[P[b, L_b - 1]] @ qq[b]
            np.testing.assert_allclose(S[b], ref, rtol=1e-12, atol=1e-20)


def test_prefix_relabel_invariance():
    """Renaming the global directions (node keys, both edge axes and the
    prefixes permuted together) renames the selection and nothing else."""
    rng = np.random.default_rng(33)
    B, G, d = 8, 9, 12
    q, C, E, P, _ = _prefix_inputs(rng, B, G, d, 3)
    pi = rng.permutation(G)
    C2 = np.empty_like(C)
    C2[pi] = C
    E2 = np.empty_like(E)
    E2[np.ix_(pi, pi)] = E
    P2 = np.where(P >= 0, pi[np.maximum(P, 0)], -1)
    sel, ss, S = oracle.coarse_prefix(q, C, E, P, 0.5, 4, "f32")
    sel2, ss2, S2 = oracle.coarse_prefix(q, C2, E2, P2, 0.5, 4, "f32")
    np.testing.assert_array_equal(sel2, pi[sel])
    np.testing.assert_allclose(ss2, ss, rtol=1e-13)
    np.testing.assert_allclose(S2[:, pi], S, rtol=1e-13)


# ---------------------------------------------------------------------------
# the sampled direction policy (Eq. global direction, Gumbel-top-k)
# ---------------------------------------------------------------------------
def test_policy_limits():
    """eps = 0 is the softmax (scipy's), eps = 1 the uniform distribution, and
    every row sums to 1."""
    from scipy.special import softmax
    rng = np.random.default_rng(41)
    S = rng.standard_normal((5, 13))
    np.testing.assert_allclose(oracle.policy(S, 0.0, 0.3), softmax(S / 0.3, axis=1), rtol=1e-13)
    np.testing.assert_allclose(oracle.policy(S, 1.0, 0.3), np.full((5, 13), 1 / 13), rtol=1e-13)
    np.testing.assert_allclose(oracle.policy(S, 0.25, 2.0).sum(axis=1), 1.0, rtol=1e-13)


def test_gumbel_of_bits():
    """u = 1/2 gives -log(log 2); the variates of evenly spread words have the
    Gumbel mean (Euler's constant) and variance pi^2/6."""
    assert oracle.gumbel_of_bits(np.uint32(2 ** 31) - 1)[()] == pytest.approx(
        -math.log(-math.log(0.5 - 0.5 / 2 ** 32)), rel=1e-15)
    # the extreme words: u = 2^-33 and u = 1 - 2^-33
    assert oracle.gumbel_of_bits(np.uint32(0))[()] == pytest.approx(-math.log(33 * math.log(2)), rel=1e-15)
    assert oracle.gumbel_of_bits(np.uint32(2 ** 32 - 1))[()] == pytest.approx(
        -math.log(-math.log1p(-2.0 ** -33)), rel=1e-6)
    x = (np.arange(1 << 20, dtype=np.uint64) << 12).astype(np.uint32)
    g = oracle.gumbel_of_bits(x)
    assert g.mean() == pytest.approx(np.euler_gamma, abs=2e-3)
    assert g.var() == pytest.approx(math.pi ** 2 / 6, rel=5e-3)


def test_philox_known_answers():
    """The oracle's Philox4x32-10 reproduces the published known-answer vectors
    (tests/golden/philox_kat.json), and the word layout of philox_words puts
    output word g % 4 of counter (g / 4, b, offset) at (b, g)."""
    with open(os.path.join(GOLDEN, "philox_kat.json")) as f:
        kat = json.load(f)["vectors"]
    h = lambda v: np.array([int(x, 16) for x in v], dtype=np.uint64)   # noqa: E731
    for v in kat:
        got = oracle.philox4x32_10(h(v["counter"]), h(v["key"]))
        np.testing.assert_array_equal(got, h(v["output"]).astype(np.uint32))
    seed, off = 0x0123456789ABCDEF, (5 << 32) | 7
    W = oracle.philox_words(seed, off, 3, 10)
    for b, g in [(0, 0), (2, 9), (1, 4), (2, 3)]:
        one = oracle.philox4x32_10(np.array([g // 4, b, 7, 5]), np.array([0x89ABCDEF, 0x01234567]))
        assert W[b, g] == one[g % 4]
    # Weyl key schedule: the words of a different seed share nothing
    assert not np.any(oracle.philox_words(seed + 1, off, 3, 10) == W)


def test_sampled_ties_go_to_the_lower_id():
    """Equal scores and equal noise make every key equal: the draw is the
    clusters in id order."""
    q = np.zeros((3, 8))
    q[:, 0] = 1.0
    C = np.zeros((9, 8))
    C[:, 1] = 1.0                                    # every score 0
    noise = np.full((3, 9), 77, dtype=np.uint32)
    sel, _, keys, _ = oracle.coarse_sampled(q, C, 4, 0.3, 0.7, noise, "f32")
    assert np.all(keys == keys[0, 0])
    np.testing.assert_array_equal(sel, np.tile(np.arange(4), (3, 1)))


def test_sampled_with_constant_noise_is_greedy():
    """Equal noise for every cluster leaves the order of log mu, which is the
    order of the scores: the greedy top-c."""
    rng = np.random.default_rng(42)
    q, C = _unit(rng, 7, 16), _unit(rng, 30, 16)
    noise = np.full((7, 30), 123456789, dtype=np.uint32)
    sel, ss, _, _ = oracle.coarse_sampled(q, C, 5, 0.2, 0.5, noise, "f32")
    sel0, ss0 = oracle.coarse(q, C, 5)
    np.testing.assert_array_equal(sel, sel0)
    np.testing.assert_allclose(ss, ss0, rtol=1e-13)


def test_sampled_frequencies_follow_the_policy():
    """Many independent draws for one query: the first pick is distributed as
    mu, and the ordered pair of the first two picks as sequential sampling
    without replacement, mu(a) mu(b) / (1 - mu(a)) (chi-square, 1e-4 level)."""
    from scipy.stats import chi2
    rng = np.random.default_rng(43)
    G, n = 6, 60000
    q, C = _unit(rng, 1, 8), _unit(rng, G, 8)
    Q = np.repeat(q, n, axis=0)
    noise = rng.integers(0, 2 ** 32, (n, G), dtype=np.uint64).astype(np.uint32)
    sel, _, _, S = oracle.coarse_sampled(Q, C, 2, 0.3, 0.1, noise, "f32")
    mu = oracle.policy(S[:1], 0.3, 0.1)[0]
    obs = np.bincount(sel[:, 0], minlength=G)
    stat = ((obs - n * mu) ** 2 / (n * mu)).sum()
    assert stat < chi2.ppf(1 - 1e-4, G - 1)
    pair = sel[:, 0] * G + sel[:, 1]
    exp2 = np.array([mu[a] * mu[b] / (1 - mu[a]) if a != b else 0.0
                     for a in range(G) for b in range(G)]) * n
    obs2 = np.bincount(pair, minlength=G * G)
    m = exp2 > 0
    assert np.all(obs2[~m] == 0)
    stat2 = ((obs2[m] - exp2[m]) ** 2 / exp2[m]).sum()
    assert stat2 < chi2.ppf(1 - 1e-4, m.sum() - 1)


# ---------------------------------------------------------------------------
# online memory update: feedback statistics and the rule-based scorer
# ---------------------------------------------------------------------------
def _empty_stats(G, NB):
    W = oracle.STATS_WORDS
    return (np.zeros((G, W), np.int64), np.zeros((G, G, W), np.int64),
            np.zeros((G, G, NB, W), np.int64))


def test_feedback_worked_example_exact():
    ex = json.load(open(os.path.join(GOLDEN, "feedback_example.json")))
    G, NB, mc = ex["G"], ex["n_buckets"], ex["min_count"]
    node, edge, eb = oracle.feedback_update(G, NB, ex["src"], ex["dst"], ex["bucket"],
                                            ex["features"], *_empty_stats(G, NB))
    np.testing.assert_array_equal(node[:, 0], ex["node_count"])
    assert edge[0, 1, 0] == ex["edge_count_0_1"]
    np.testing.assert_array_equal(eb[0, 1, :, 0], ex["edge_bucket_count_0_1"])
    w = np.asarray(ex["w"], np.float64)
    for k, key in ((0, "phi_0_1_bucket0"), (1, "phi_0_1_bucket1")):
        assert oracle.transition_utility(edge, eb, 0, 1, k, mc, w) == pytest.approx(_num(ex[key]), abs=1e-12)
    assert oracle.transition_utility(edge, eb, 1, 0, 0, mc, w) == _num(ex["phi_1_0_bucket0"])
    S = oracle.transition_scores(np.full((1, 2), -1), [0], 0.5, w, mc, node, edge, eb)
    np.testing.assert_allclose(S[0], [_num(x) for x in ex["node_score"]], atol=1e-12)
    # distinct weights: each entry of z sits at its place in App. B.6's order
    w = np.asarray(ex["w_distinct"], np.float64)
    for k, key in ((0, "phi_0_1_bucket0_w_distinct"), (1, "phi_0_1_bucket1_w_distinct")):
        assert oracle.transition_utility(edge, eb, 0, 1, k, mc, w) == pytest.approx(_num(ex[key]), abs=1e-12)
    S = oracle.transition_scores(np.full((1, 2), -1), [0], 0.5, w, mc, node, edge, eb)
    np.testing.assert_allclose(S[0], [_num(x) for x in ex["node_score_w_distinct"]], atol=1e-12)


def test_feedback_sums_are_order_free_and_exact():
    """The statistics are integer sums: any order of the events gives the
    same bits, and the counts are the bincounts."""
    rng = np.random.default_rng(51)
    G, NB, n = 5, 3, 400
    src = rng.integers(-1, G, n)
    dst = rng.integers(0, G, n)
    bk = rng.integers(0, NB, n)
    feat = rng.standard_normal((n, oracle.FEEDBACK_FEATURES)).astype(np.float32)
    a = oracle.feedback_update(G, NB, src, dst, bk, feat, *_empty_stats(G, NB))
    p = rng.permutation(n)
    b = oracle.feedback_update(G, NB, src[p], dst[p], bk[p], feat[p], *_empty_stats(G, NB))
    for x, y in zip(a, b):
        np.testing.assert_array_equal(x, y)
    np.testing.assert_array_equal(a[0][:, 0], np.bincount(dst, minlength=G))
    fx = np.rint(feat.astype(np.float64) * oracle.FIXED_ONE).astype(np.int64)
    np.testing.assert_array_equal(a[0][2, 1:], fx[dst == 2].sum(axis=0))


def test_transition_scores_prefix_and_fallback():
    """Prefix weighting as in Eq. prefix_weight over phi; a bucket below
    min_count falls back to the edge aggregate."""
    rng = np.random.default_rng(52)
    G, NB, n = 4, 2, 300
    src, dst, bk = rng.integers(0, G, n), rng.integers(0, G, n), rng.integers(0, NB, n)
    feat = rng.random((n, oracle.FEEDBACK_FEATURES)).astype(np.float32)
    node, edge, eb = oracle.feedback_update(G, NB, src, dst, bk, feat, *_empty_stats(G, NB))
    w = rng.standard_normal(oracle.STATS_WORDS)
    P = np.array([[2, 0, 3], [1, -1, -1]])
    S = oracle.transition_scores(P, [1, 0], 0.7, w, 5, node, edge, eb)
    a = oracle.prefix_weights(3, 0.7)
    for g in range(G):
        ref = sum(a[i] * oracle.transition_utility(edge, eb, P[0, i], g, 1, 5, w) for i in range(3))
        assert S[0, g] == pytest.approx(ref, rel=1e-13)
    huge = 10 ** 6                                   # no bucket qualifies: the aggregate
    S2 = oracle.transition_scores(P[1:], [0], 0.7, w, huge, node, edge, eb)
    for g in range(G):
        assert S2[0, g] == pytest.approx(w @ oracle.feature_vector(edge[1, g], 0.0), rel=1e-13)
