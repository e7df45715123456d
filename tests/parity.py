"""Tie-aware comparison of GPU retrieval outputs with the CPU oracle.

Floating point decides which clusters and which records are selected, so an
index may legitimately differ from the oracle's when two candidates are closer
than the rounding error of an fp32 inner product. The window used here is the
standard bound for a dot product accumulated in fp32 in any order
(|error| <= gamma_n * sum |q_i k_i|, gamma_n = n u / (1 - n u), u = 2^-24), doubled
for safety, plus one ulp of the score itself; n = d for bf16 operands (their
products are exact in fp32) and d + 1 for fp32 operands.

Protocol:
  P1 coarse: the GPU's clusters must be the oracle's, except for clusters whose
     oracle score lies within the window of the oracle's c-th score;
  P2 fine: the oracle is re-run on the GPU's selection; the kept ids must match
     except at the k-th boundary within the window; shared ids keep the oracle's
     order except among near-ties;
  P3 values: scores within rtol * |s| plus the window of s, weights within rtol
     relative, slot and row max within rtol * |m| plus the window of the
     top-1 record's score, log Z within rtol; counts exact;
  P4 rows whose coarse selection needed no tie acceptance match the oracle's own
     selection.
"""
from __future__ import annotations

import numpy as np

import oracle

U = 2.0 ** -24


def gamma(n: int) -> float:
    return n * U / (1 - n * U)


def window(absdot: np.ndarray, s: np.ndarray, n: int) -> np.ndarray:
    return 2.0 * gamma(n) * absdot + U * np.abs(s)


class Report(dict):
    def bump(self, key, v=1):
        self[key] = self.get(key, 0) + v

    def worst(self, key, v):
        self[key] = max(self.get(key, 0.0), float(v))


def check(gpu: dict, q, c, seg_offsets, top_c: int, top_k: int, tau: float, compute: str,
          fetch_keys, gather_keys, transition_id=None, rows=None, rtol=None) -> Report:
    """Compare GPU outputs (numpy, rows already selected) with the oracle; raise on mismatch.

    fetch_keys(a, b) returns bank rows a..b-1 and gather_keys(rows) the given bank
    rows, both as fp32 arrays in storage precision.
    """
    if rtol is None:
        rtol = 2e-2 if compute == "bf16" else 1e-5
    n_acc = q.shape[1] if compute == "bf16" else q.shape[1] + 1
    rows = np.arange(q.shape[0]) if rows is None else np.asarray(rows)
    R = rows.size
    rep = Report(rows=R)

    ref = oracle.retrieve(q, c, seg_offsets, top_c, top_k, tau, compute, fetch_keys=fetch_keys,
                          transition_id=transition_id, sel=gpu["sel"], rows=rows)
    qh = ref["qh"]
    ch = oracle.round_bf16(c) if compute == "bf16" else np.asarray(c, np.float32)

    # ---- P1: coarse selection --------------------------------------------------
    S = oracle.scores(qh, ch)
    A = np.abs(qh).astype(np.float64) @ np.abs(ch).astype(np.float64).T
    W = window(A, S, n_acc)
    tie_rows = np.zeros(R, dtype=bool)
    for r in range(R):
        g_gpu = gpu["sel"][r]
        g_ref = ref["own_sel"][r]
        assert len(set(g_gpu.tolist())) == top_c, f"row {r}: duplicate clusters {g_gpu}"
        theta = S[r, g_ref[-1]]
        diff = set(g_gpu.tolist()) ^ set(g_ref.tolist())
        for g in diff:
            assert abs(S[r, g] - theta) <= W[r, g] + W[r, g_ref[-1]], \
                f"row {r}: cluster {g} selected differently (score {S[r, g]}, c-th {theta})"
        if diff:
            tie_rows[r] = True
            rep.bump("coarse_tie_events", len(diff) // 2)
        # scores of the GPU's clusters and their order
        sg = gpu["sel_score"][r].astype(np.float64)
        err = np.abs(sg - S[r, g_gpu])
        allow = rtol * np.abs(S[r, g_gpu]) + W[r, g_gpu]
        assert np.all(err <= allow), f"row {r}: coarse scores {sg} vs {S[r, g_gpu]}"
        rep.worst("coarse_score_err", (err / allow).max())
        assert np.all(np.diff(sg) <= 0), f"row {r}: coarse scores not descending {sg}"
        if not diff:
            # same set: the order may only differ among oracle near-ties
            for a in range(top_c):
                if g_gpu[a] != g_ref[a]:
                    assert abs(S[r, g_gpu[a]] - S[r, g_ref[a]]) <= W[r, g_gpu[a]] + W[r, g_ref[a]]
                    rep.bump("coarse_order_ties")
    # P4
    exact = ~tie_rows
    assert np.array_equal(np.sort(gpu["sel"][exact], axis=1), np.sort(ref["own_sel"][exact], axis=1))

    # ---- P2 + P3: per-slot and per-row outputs on the GPU's selection ----------
    inv = None
    if transition_id is not None:
        tid = np.asarray(transition_id)
        inv = np.empty(tid.size, dtype=np.int64)
        inv[tid] = np.arange(tid.size)

    kmap = {}

    def load_row_keys(r):
        """Quantised keys of every id that row r's outputs mention, in one gather."""
        ids = np.concatenate([gpu["slot_id"][r].ravel(), gpu["id"][r].ravel(),
                              ref["slot_id"][r].ravel(), ref["id"][r].ravel()])
        ids = np.unique(ids[ids >= 0])
        kmap.clear()
        if ids.size == 0:
            return
        brow = ids if inv is None else inv[ids]
        kr = np.asarray(gather_keys(brow), dtype=np.float32)
        kr = oracle.round_bf16(kr) if compute == "bf16" else kr
        for i, v in zip(ids.tolist(), kr):
            kmap[i] = v

    def key_row(i):
        return kmap[int(i)]

    def compare_list(tag, r, ids_g, sc_g, cnt_ref, ids_r, sc_r):
        qv = qh[r].astype(np.float64)
        kept = int(cnt_ref)
        assert np.all(ids_g[kept:] == -1) and np.all(np.isneginf(sc_g[kept:])), \
            f"{tag} row {r}: padding {ids_g[kept:]}"
        ids_g, sc_g, ids_r, sc_r = ids_g[:kept], sc_g[:kept].astype(np.float64), ids_r[:kept], sc_r[:kept]
        assert np.all(ids_g >= 0) and len(set(ids_g.tolist())) == kept, f"{tag} row {r}: ids {ids_g}"
        assert np.all(np.diff(sc_g) <= 0), f"{tag} row {r}: scores not descending"
        ref_score = dict(zip(ids_r.tolist(), sc_r.tolist()))
        kvecs = {}
        for i in ids_g.tolist():
            if i not in ref_score:
                kvecs[i] = key_row(i)
                ref_score[i] = float(kvecs[i].astype(np.float64) @ qv)
        # window of every id involved
        def win(i):
            kv = kvecs.get(i)
            if kv is None:
                kv = kvecs[i] = key_row(i)
            return window(np.abs(qv) @ np.abs(kv.astype(np.float64)), ref_score[i], n_acc)
        diff = set(ids_g.tolist()) ^ set(ids_r.tolist())
        if diff:
            kth = sc_r[-1]
            kth_w = win(int(ids_r[-1]))
            for i in diff:
                assert abs(ref_score[i] - kth) <= win(i) + kth_w, \
                    f"{tag} row {r}: id {i} (score {ref_score[i]}) vs k-th {kth}"
            rep.bump(f"{tag}_tie_events", len(diff) // 2)
        # values of every GPU id: within rtol of the score plus its window
        for i, sg in zip(ids_g.tolist(), sc_g.tolist()):
            allow = rtol * abs(ref_score[i]) + win(i)
            e = abs(sg - ref_score[i])
            assert e <= allow, f"{tag} row {r}: id {i} score {sg} vs {ref_score[i]}"
            rep.worst(f"{tag}_score_err", e / allow)
        # order: consecutive GPU entries must be ordered by the oracle up to the window
        for a in range(kept - 1):
            i0, i1 = int(ids_g[a]), int(ids_g[a + 1])
            if ref_score[i0] < ref_score[i1]:
                assert ref_score[i1] - ref_score[i0] <= win(i0) + win(i1), \
                    f"{tag} row {r}: order of ids {i0}, {i1}"
                rep.bump(f"{tag}_order_ties")

    def max_allow(r, top_id, m_ref):
        # the maximum is the top-1 record's score: rtol * |m| plus its window
        kv = key_row(top_id).astype(np.float64)
        qv = qh[r].astype(np.float64)
        return rtol * abs(m_ref) + float(window(np.abs(qv) @ np.abs(kv), m_ref, n_acc))

    for r in range(R):
        if r and r % 128 == 0:
            print(f"[parity] {r} of {R} rows checked", flush=True)
        load_row_keys(r)
        for s in range(top_c):
            compare_list("slot", r, gpu["slot_id"][r, s], gpu["slot_score"][r, s],
                         ref["slot_count"][r, s], ref["slot_id"][r, s], ref["slot_score"][r, s])
            mr, zr = ref["slot_m"][r, s], ref["slot_Z"][r, s]
            mg, zg = float(gpu["slot_max"][r, s]), float(gpu["slot_sum"][r, s])
            if ref["slot_count"][r, s] == 0:
                assert mg == -np.inf and zg == 0.0
            else:
                assert abs(mg - mr) <= max_allow(r, ref["slot_id"][r, s, 0], mr), \
                    f"slot max {mg} vs {mr}"
                e = abs(np.log(zg) - np.log(zr))
                assert e <= rtol, f"slot row {r}: log Z {np.log(zg)} vs {np.log(zr)}"
                rep.worst("slot_logZ_err", e)
        compare_list("row", r, gpu["id"][r], gpu["score"][r], ref["count"][r], ref["id"][r],
                     ref["score"][r])
        assert gpu["count"][r] == ref["count"][r], f"row {r}: count {gpu['count'][r]} vs {ref['count'][r]}"
        if ref["count"][r] == 0:
            assert gpu["m"][r] == -np.inf and gpu["Z"][r] == 0.0
            assert np.all(gpu["weight"][r] == 0.0)
            continue
        mr, zr = ref["m"][r], ref["Z"][r]
        assert abs(gpu["m"][r] - mr) <= max_allow(r, ref["id"][r, 0], mr), \
            f"row {r}: max {gpu['m'][r]} vs {mr}"

        e = abs(np.log(float(gpu["Z"][r])) - np.log(zr))
        assert e <= rtol, f"row {r}: log Z {np.log(float(gpu['Z'][r]))} vs {np.log(zr)}"
        rep.worst("row_logZ_err", e)
        # weights: exact softmax over the candidate set at the GPU's ids
        n = int(ref["count"][r])
        for a in range(n):
            i = int(gpu["id"][r, a])
            qv = qh[r].astype(np.float64)
            kv = key_row(i).astype(np.float64)
            w_ref = np.exp((kv @ qv - mr) / tau) / zr
            wg = float(gpu["weight"][r, a])
            e = abs(wg - w_ref) / max(w_ref, 1e-30)
            assert e <= rtol, f"row {r}: weight of id {i} {wg} vs {w_ref}"
            rep.worst("weight_err", e)
        assert np.all(gpu["weight"][r, n:] == 0.0)
    return rep


def check_rows(gpu: dict, ref: dict, qh, key_rows, tau: float, compute: str, rtol=None,
               tag: str = "row") -> Report:
    """Row outputs (id, score, weight, m, Z, count) of a GPU retrieval against the
    oracle's over the same candidates, by the P2/P3 rules: ids match except at
    the k-th boundary within the window, scores within rtol * |s| plus the
    window, weights within rtol, max within rtol * |m| plus the top-1 window,
    log Z within rtol, counts exact. key_rows(ids) returns the quantised keys
    of caller ids (fp32, [len][d])."""
    if rtol is None:
        rtol = 2e-2 if compute == "bf16" else 1e-5
    n_acc = qh.shape[1] if compute == "bf16" else qh.shape[1] + 1
    rep = Report(rows=gpu["id"].shape[0])
    for r in range(gpu["id"].shape[0]):
        kept = int(ref["count"][r])
        assert int(gpu["count"][r]) == kept, f"{tag} {r}: count {gpu['count'][r]} vs {kept}"
        ig, sg = gpu["id"][r], gpu["score"][r].astype(np.float64)
        assert np.all(ig[kept:] == -1) and np.all(np.isneginf(sg[kept:])), f"{tag} {r}: padding"
        if kept == 0:
            assert gpu["m"][r] == -np.inf and gpu["Z"][r] == 0.0 and np.all(gpu["weight"][r] == 0)
            continue
        ig, sg = ig[:kept], sg[:kept]
        ir = ref["id"][r, :kept]
        assert len(set(ig.tolist())) == kept and np.all(np.diff(sg) <= 0), f"{tag} {r}: ids/order"
        ids = np.unique(np.concatenate([ig, ir]))
        kv = dict(zip(ids.tolist(), np.asarray(key_rows(ids), dtype=np.float64)))
        qv = qh[r].astype(np.float64)
        s_ref = {i: float(kv[i] @ qv) for i in ids.tolist()}
        win = {i: float(window(np.abs(qv) @ np.abs(kv[i]), s_ref[i], n_acc)) for i in ids.tolist()}
        diff = set(ig.tolist()) ^ set(ir.tolist())
        kth = int(ir[-1])
        for i in diff:
            assert abs(s_ref[i] - s_ref[kth]) <= win[i] + win[kth], \
                f"{tag} {r}: id {i} ({s_ref[i]}) vs k-th {s_ref[kth]}"
        if diff:
            rep.bump("tie_events", len(diff) // 2)
        for i, s in zip(ig.tolist(), sg.tolist()):
            allow = rtol * abs(s_ref[i]) + win[i]
            assert abs(s - s_ref[i]) <= allow, f"{tag} {r}: id {i} score {s} vs {s_ref[i]}"
            rep.worst("score_err", abs(s - s_ref[i]) / allow)
        mr, zr = float(ref["m"][r]), float(ref["Z"][r])
        top = int(ir[0])
        assert abs(float(gpu["m"][r]) - mr) <= rtol * abs(mr) + win[top], f"{tag} {r}: max"
        e = abs(np.log(float(gpu["Z"][r])) - np.log(zr))
        assert e <= rtol, f"{tag} {r}: log Z {np.log(float(gpu['Z'][r]))} vs {np.log(zr)}"
        rep.worst("logZ_err", e)
        for a, i in enumerate(ig.tolist()):
            w_ref = np.exp((s_ref[i] - mr) / tau) / zr
            e = abs(float(gpu["weight"][r, a]) - w_ref) / max(w_ref, 1e-30)
            assert e <= rtol, f"{tag} {r}: weight of {i}: {gpu['weight'][r, a]} vs {w_ref}"
            rep.worst("weight_err", e)
        assert np.all(gpu["weight"][r, kept:] == 0.0)
    return rep
