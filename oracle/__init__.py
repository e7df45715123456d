"""Plain CPU oracle for HTAM's hierarchical transition-attended retrieval.

TEST INFRASTRUCTURE ONLY: only ``tests/``, ``__graft_entry__.smoke()`` and the
CPU-baseline leg of ``bench.py`` may import this package. The GPU library never
calls it, and it shares no code with the GPU library.

The arithmetic lives in ``htam_oracle.c`` (fp64, OpenMP over rows); this module
loads it with ctypes and composes its steps in the order the paper gives them
(arXiv 2605.29734, Sec. 4.3 and Alg. 1):

  O0  bf16 operand quantisation when the bank computes in bf16;
  O1  coarse scores <q, c_g>          (Eq. score with a one-term prefix and the
                                       linear scorer of App. B.6);
  O2  top-c clusters, ties to the lower id (greedy limit of Eq. global direction);
  O3  candidates = the selected clusters' segments (Eq. local nodes);
  O4  fine scores <q, k_j>            (Eq. local policy with an inner product);
  O5  temperature softmax over the candidates;
  O6  top-k by (-score, caller id), padded with (-1, -inf, 0).

Every result here is computed in double from the stored fp32 / bf16 values.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "htam_oracle.c")
_LIB = os.path.join(_HERE, "liboracle.so")
_lib = None


def build(force: bool = False) -> str:
    """Compile the C oracle with gcc (OpenMP) into oracle/liboracle.so."""
    if force or not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
        tmp = _LIB + ".tmp"
        subprocess.check_call(["gcc", "-O2", "-fopenmp", "-fPIC", "-shared", "-std=c11",
                               "-o", tmp, _SRC, "-lm"])
        os.replace(tmp, _LIB)
    return _LIB


def _load():
    global _lib
    if _lib is None:
        build()
        lib = ctypes.CDLL(_LIB)
        P = ctypes.c_void_p
        i32, i64, f64 = ctypes.c_int32, ctypes.c_int64, ctypes.c_double
        lib.htam_oracle_round_bf16.argtypes = [P, P, i64]
        lib.htam_oracle_scores.argtypes = [i32, i64, i32, P, P, P]
        lib.htam_oracle_coarse.argtypes = [i32, i32, i32, P, P, i32, P, P]
        lib.htam_oracle_attend.argtypes = [i64, P, P, f64, i32, P, P, P, P, P, P]
        lib.htam_oracle_attend_rows.argtypes = [i64, P, P, P, f64, i32, P, P, P, P, P]
        lib.htam_oracle_build.argtypes = [i64, i32, P, P, P]
        lib.htam_oracle_build.restype = ctypes.c_int
        _lib = lib
    return _lib


def _p(a: np.ndarray):
    return a.ctypes.data_as(ctypes.c_void_p)


def _f32(a) -> np.ndarray:
    return np.ascontiguousarray(np.asarray(a, dtype=np.float32))


# ---------------------------------------------------------------------------
# single steps
# ---------------------------------------------------------------------------
def round_bf16(x) -> np.ndarray:
    """O0: fp32 -> bf16 (round to nearest, ties to even), returned as fp32 values."""
    x = _f32(x)
    y = np.empty_like(x)
    _load().htam_oracle_round_bf16(_p(x), _p(y), x.size)
    return y


def scores(q, k) -> np.ndarray:
    """O1/O4: double inner products, out[i][j] = <q_i, k_j>."""
    q, k = _f32(q), _f32(k)
    nq, d = q.shape
    nk = k.shape[0]
    out = np.empty((nq, nk), dtype=np.float64)
    if nq and nk:
        _load().htam_oracle_scores(nq, nk, d, _p(q), _p(k), _p(out))
    return out


def coarse(q, c, top_c: int):
    """O1 + O2: the top_c clusters per query by (-score, cluster id)."""
    q, c = _f32(q), _f32(c)
    B, d = q.shape
    G = c.shape[0]
    sel = np.empty((B, top_c), dtype=np.int32)
    sel_score = np.empty((B, top_c), dtype=np.float64)
    if B:
        _load().htam_oracle_coarse(B, G, d, _p(q), _p(c), top_c, _p(sel), _p(sel_score))
    return sel, sel_score


def attend(s, ids, tau: float, top_k: int, full_weights: bool = False) -> dict:
    """O5 + O6 over one candidate set (scores s, caller ids)."""
    s = np.ascontiguousarray(np.asarray(s, dtype=np.float64))
    ids = np.ascontiguousarray(np.asarray(ids, dtype=np.int32))
    n = s.size
    out_id = np.empty(top_k, dtype=np.int32)
    out_s = np.empty(top_k, dtype=np.float64)
    out_w = np.empty(top_k, dtype=np.float64)
    m = np.zeros(1, dtype=np.float64)
    Z = np.zeros(1, dtype=np.float64)
    w_full = np.empty(max(n, 1), dtype=np.float64) if full_weights else None
    _load().htam_oracle_attend(n, _p(s), _p(ids), float(tau), top_k, _p(out_id), _p(out_s),
                               _p(out_w), _p(m), _p(Z),
                               _p(w_full) if full_weights else None)
    r = dict(id=out_id, score=out_s, weight=out_w, m=float(m[0]), Z=float(Z[0]),
             count=min(top_k, n))
    if full_weights:
        r["w_full"] = w_full[:n]
    return r


def attend_rows(offsets, s, ids, tau: float, top_k: int) -> dict:
    """O5 + O6 over many independent candidate sets (rows r = s[off[r]:off[r+1]])."""
    off = np.ascontiguousarray(np.asarray(offsets, dtype=np.int64))
    s = np.ascontiguousarray(np.asarray(s, dtype=np.float64))
    ids = np.ascontiguousarray(np.asarray(ids, dtype=np.int32))
    rows = off.size - 1
    out_id = np.empty((rows, top_k), dtype=np.int32)
    out_s = np.empty((rows, top_k), dtype=np.float64)
    out_w = np.empty((rows, top_k), dtype=np.float64)
    m = np.empty(rows, dtype=np.float64)
    Z = np.empty(rows, dtype=np.float64)
    if rows:
        _load().htam_oracle_attend_rows(rows, _p(off), _p(s), _p(ids), float(tau), top_k,
                                        _p(out_id), _p(out_s), _p(out_w), _p(m), _p(Z))
    count = np.minimum(np.diff(off), top_k).astype(np.int32)
    return dict(id=out_id, score=out_s, weight=out_w, m=m, Z=Z, count=count)


def build_bank(cluster_of, n_clusters: int):
    """Memory build: stable counting sort of records by parent cluster.

    Returns (seg_offsets int64 [G+1], transition_id int32 [N]).
    """
    cl = np.ascontiguousarray(np.asarray(cluster_of, dtype=np.int32))
    off = np.empty(n_clusters + 1, dtype=np.int64)
    tid = np.empty(cl.size, dtype=np.int32)
    rc = _load().htam_oracle_build(cl.size, n_clusters, _p(cl), _p(off), _p(tid))
    if rc != 0:
        raise ValueError("cluster id out of range")
    return off, tid


# ---------------------------------------------------------------------------
# flat memory retrieval (the baseline without a hierarchy)
# ---------------------------------------------------------------------------
def flat(q, keys, tau: float, top_k: int, compute: str, transition_id=None,
         chunk_rows: int = 65536) -> dict:
    """Flat memory retrieval: every record of the memory is a candidate of
    every query, with no coarse level (the "Flat Memory Retrieval" baseline
    of Table 1 and App. C.4; the "w/o hierarchy" ablation of Sec. 5.5).
    O0 quantisation, O4 scores <q_b, k_j> over all N records, O5 the
    temperature softmax over all N, O6 the top-k by (-score, caller id).

    q [B][d], keys [N][d] (fp32 arrays; bf16 storage passed widened),
    transition_id [N] (None = row index). Returns id, score, weight, m, Z,
    count per query, like the row outputs of retrieve().
    """
    q = _f32(q)
    kk = _f32(keys)
    if compute == "bf16":
        quant = round_bf16
    elif compute == "f32":
        def quant(x):
            return _f32(x)
    else:
        raise ValueError(compute)
    qh = quant(q)
    N = kk.shape[0]
    parts = [scores(qh, quant(kk[a:min(N, a + chunk_rows)])) for a in range(0, N, chunk_rows)]
    S = np.concatenate(parts, axis=1) if parts else np.zeros((q.shape[0], 0))
    ids = (np.arange(N) if transition_id is None else np.asarray(transition_id)).astype(np.int32)
    B = q.shape[0]
    off = np.arange(B + 1, dtype=np.int64) * N
    r = attend_rows(off, S.reshape(-1), np.tile(ids, B), tau, top_k)
    r["qh"] = qh
    return r


# ---------------------------------------------------------------------------
# the whole retrieval, composed in the paper's order
# ---------------------------------------------------------------------------
def retrieve(q, c, seg_offsets, top_c: int, top_k: int, tau: float, compute: str,
             fetch_keys=None, keys=None, transition_id=None, sel=None, rows=None,
             chunk_rows: int = 65536) -> dict:
    """Hierarchical retrieval for the queries ``rows`` (default: all).

    q [B][d], c [G][d]: stored query / coarse-key values (fp32 arrays; bf16
    storage is passed widened to fp32, which is exact).
    seg_offsets [G+1]: segment bounds of the segment-contiguous bank.
    keys [N][d] or fetch_keys(start, stop) -> fp32 array [stop-start][d]: the
    bank rows (the callback lets a caller stream a large bank cluster by cluster).
    transition_id [N]: bank position -> caller id (None = identity).
    compute: "f32" or "bf16" (O0 applies to q, c and the keys for "bf16").
    sel: if given ([len(rows)][top_c]), the coarse selection to use instead of
    the oracle's own O2 (used to check a fine stage on another implementation's
    selection); the oracle's own selection is returned too.

    Returns per-row outputs (id, score, weight, m, Z, count) over the union of
    the selected segments, and per-slot outputs (slot_m, slot_Z, slot_id,
    slot_score, slot_count) over each selected segment alone.
    """
    q = _f32(q)
    c = _f32(c)
    off = np.asarray(seg_offsets, dtype=np.int64)
    if rows is None:
        rows = np.arange(q.shape[0])
    rows = np.asarray(rows, dtype=np.int64)
    if compute == "bf16":
        quant = round_bf16
    elif compute == "f32":
        def quant(x):
            return _f32(x)
    else:
        raise ValueError(compute)
    if fetch_keys is None:
        kk = _f32(keys)

        def fetch_keys(a, b):
            return kk[a:b]

    qh = quant(q[rows])
    ch = quant(c)
    own_sel, own_sel_score = coarse(qh, ch, top_c)                    # O1, O2
    use_sel = own_sel if sel is None else np.asarray(sel, dtype=np.int32)
    R = rows.size

    # O3 + O4, cluster-major so that a large bank is streamed once.
    slot_s = [[None] * top_c for _ in range(R)]
    slot_ids = [[None] * top_c for _ in range(R)]
    users = {}
    for r in range(R):
        for j in range(top_c):
            users.setdefault(int(use_sel[r, j]), []).append((r, j))
    for g, lst in users.items():
        a, b = int(off[g]), int(off[g + 1])
        rr = np.array([u[0] for u in lst], dtype=np.int64)
        parts = []
        for s0 in range(a, b, chunk_rows):
            s1 = min(b, s0 + chunk_rows)
            kh = quant(fetch_keys(s0, s1))
            parts.append(scores(qh[rr], kh))
        sc = np.concatenate(parts, axis=1) if parts else np.zeros((rr.size, 0))
        ids = (np.arange(a, b, dtype=np.int64) if transition_id is None
               else np.asarray(transition_id[a:b], dtype=np.int64)).astype(np.int32)
        for t, (r, j) in enumerate(lst):
            slot_s[r][j] = sc[t]
            slot_ids[r][j] = ids

    # O5 + O6 per slot (one selected segment) and per row (union of segments).
    def pack(seq_s, seq_i):
        lens = [x.size for x in seq_s]
        o = np.zeros(len(lens) + 1, dtype=np.int64)
        o[1:] = np.cumsum(lens)
        s_all = np.concatenate(seq_s) if seq_s else np.zeros(0)
        i_all = np.concatenate(seq_i) if seq_i else np.zeros(0, dtype=np.int32)
        return o, s_all, i_all

    o, s_all, i_all = pack([slot_s[r][j] for r in range(R) for j in range(top_c)],
                           [slot_ids[r][j] for r in range(R) for j in range(top_c)])
    per_slot = attend_rows(o, s_all, i_all, tau, top_k)
    o, s_all, i_all = pack([np.concatenate(slot_s[r]) for r in range(R)],
                           [np.concatenate(slot_ids[r]) for r in range(R)])
    per_row = attend_rows(o, s_all, i_all, tau, top_k)

    out = dict(rows=rows, sel=use_sel, own_sel=own_sel, own_sel_score=own_sel_score,
               slot_m=per_slot["m"].reshape(R, top_c), slot_Z=per_slot["Z"].reshape(R, top_c),
               slot_id=per_slot["id"].reshape(R, top_c, top_k),
               slot_score=per_slot["score"].reshape(R, top_c, top_k),
               slot_count=per_slot["count"].reshape(R, top_c))
    out.update(per_row)
    out["qh"] = qh
    return out


# ---------------------------------------------------------------------------
# prefix-aware transition scoring of the global directions
# ---------------------------------------------------------------------------
def prefix_weights(length: int, lam: float) -> np.ndarray:
    """Position-aware weights of a prefix of `length` directions (Eq. prefix_weight):
    alpha_i = exp(-lam * (length - i)) for i = 1..length; the most recent
    direction (i = length) has weight 1."""
    i = np.arange(1, length + 1, dtype=np.float64)
    return np.exp(-float(lam) * (length - i))


def coarse_prefix(q, c, edge_keys, prefix, lam: float, top_c: int, compute: str):
    """Prefix-aware coarse scores and top-c selection (Sec. 4.3, Eq. score with
    Eq. prefix_weight; App. A.1 and App. B.2 for the edge memories).

    The score of direction g for query b with prefix p_b = (g_1, ..., g_L) is
    sum_{i=1..L} alpha_i * phi(g_i, g), alpha_i = exp(-lam (L - i)), where the
    state-conditioned transition utility read from edge E_G(g_i, g) is the
    inner product <q_b, E[g_i][g]> (the linear scorer of App. B.6 in embedding
    space). A query with an empty prefix (the first step, which reads no edge)
    is scored by its node keys, <q_b, c_g>.

    q [B][d], c [G][d], edge_keys [G][G][d] (edge_keys[src][dst]), prefix
    [B][Lmax] int (a row's prefix ends at its first entry outside [0, G)).
    Returns (sel [B][top_c], sel_score, S [B][G]) with the selection ordered by
    (-score, g). Computed in double over the (bf16-quantised) operands.
    """
    quant = round_bf16 if compute == "bf16" else _f32
    qh = quant(q).astype(np.float64)
    ch = quant(c).astype(np.float64)
    eh = quant(edge_keys).astype(np.float64)
    G = ch.shape[0]
    prefix = np.asarray(prefix)
    B = qh.shape[0]
    S = np.empty((B, G))
    for b in range(B):
        row = prefix[b]
        L = 0
        while L < row.size and 0 <= row[L] < G:
            L += 1
        if L == 0:
            S[b] = ch @ qh[b]
        else:
            alpha = prefix_weights(L, lam)
            S[b] = sum(alpha[i] * (eh[row[i]] @ qh[b]) for i in range(L))
    sel = np.empty((B, top_c), dtype=np.int32)
    sel_score = np.empty((B, top_c))
    for b in range(B):
        order = np.lexsort((np.arange(G), -S[b]))[:top_c]
        sel[b], sel_score[b] = order, S[b, order]
    return sel, sel_score, S


# ---------------------------------------------------------------------------
# the stochastic direction policy mu_g, sampled c times without replacement
# ---------------------------------------------------------------------------
def policy(S, eps: float, tau_g: float) -> np.ndarray:
    """The direction policy of Eq. global direction over every cluster:
    mu(g) = eps / G + (1 - eps) exp(S[g] / tau_g) / sum_g' exp(S[g'] / tau_g),
    row by row, in double."""
    S = np.asarray(S, dtype=np.float64)
    z = (S - S.max(axis=-1, keepdims=True)) / tau_g
    soft = np.exp(z) / np.exp(z).sum(axis=-1, keepdims=True)
    return eps / S.shape[-1] + (1.0 - eps) * soft


def gumbel_of_bits(x) -> np.ndarray:
    """Standard Gumbel variate of a uniform 32-bit word x: u = (x + 1/2) / 2^32
    in (0, 1), G = -log(-log u)."""
    u = (np.asarray(x, dtype=np.float64) + 0.5) / 4294967296.0
    return -np.log(-np.log(u))


_MASK32 = np.uint64(0xFFFFFFFF)


def philox4x32_10(counter, key) -> np.ndarray:
    """Philox4x32 with ten rounds, as Salmon, Moraes, Dror and Shaw define it
    (SC'11, Sec. 3): counter [..., 4] and key [..., 2] of 32-bit words. A round
    takes the full 64-bit products of counter words 0 and 2 with the two
    multipliers; the new counter is (hi(M1 x2) ^ x1 ^ k0, lo(M1 x2),
    hi(M0 x0) ^ x3 ^ k1, lo(M0 x0)), and the key grows by the two Weyl
    constants between rounds. Returns the [..., 4] output words."""
    m0, m1 = np.uint64(0xD2511F53), np.uint64(0xCD9E8D57)
    w0, w1 = np.uint64(0x9E3779B9), np.uint64(0xBB67AE85)
    x = [np.asarray(counter, dtype=np.uint64)[..., i] & _MASK32 for i in range(4)]
    k0 = np.asarray(key, dtype=np.uint64)[..., 0] & _MASK32
    k1 = np.asarray(key, dtype=np.uint64)[..., 1] & _MASK32
    for r in range(10):
        if r:
            k0, k1 = (k0 + w0) & _MASK32, (k1 + w1) & _MASK32
        p0, p1 = m0 * x[0], m1 * x[2]          # < 2^64: exact in uint64
        x = [(p1 >> np.uint64(32)) ^ x[1] ^ k0, p1 & _MASK32,
             (p0 >> np.uint64(32)) ^ x[3] ^ k1, p0 & _MASK32]
    return np.stack(x, axis=-1).astype(np.uint32)


def philox_words(seed: int, offset: int, B: int, G: int) -> np.ndarray:
    """The uniform words [B][G] that htam_retrieve_coarse_sampled draws when the
    caller passes none: the word of (b, g) is output word g % 4 of Philox4x32-10
    at counter (g / 4, b, offset low, offset high) under key (seed low, seed
    high), so a draw depends only on (seed, offset, b, g)."""
    n4 = (G + 3) // 4
    ctr = np.zeros((B, n4, 4), dtype=np.uint64)
    ctr[..., 0] = np.arange(n4, dtype=np.uint64)[None, :]
    ctr[..., 1] = np.arange(B, dtype=np.uint64)[:, None]
    ctr[..., 2] = offset & 0xFFFFFFFF
    ctr[..., 3] = (offset >> 32) & 0xFFFFFFFF
    key = np.array([seed & 0xFFFFFFFF, (seed >> 32) & 0xFFFFFFFF], dtype=np.uint64)
    return philox4x32_10(ctr, key).reshape(B, n4 * 4)[:, :G]


def coarse_sampled(q, c, top_c: int, eps: float, tau_g: float, noise, compute: str):
    """Direction choice by sampling the policy mu_g (Eq. global direction;
    Alg. 1 Step 2, g_t ~ mu_g) top_c times without replacement, by the
    Gumbel-top-k construction (Kool et al., ICML 2019): perturb log mu(g) with
    independent standard Gumbel variates and keep the top_c, which is a draw
    of top_c clusters one after another without replacement from mu.

    Scores are the one-term coarse scores <q_b, c_g> (O0/O1). noise [B][G]
    uint32 supplies the uniform words (one per query and cluster). Returns
    (sel [B][top_c] ordered by descending perturbed key, ties to the lower
    cluster id; their raw scores; the keys [B][G]; S [B][G])."""
    quant = round_bf16 if compute == "bf16" else _f32
    qh, ch = quant(q), quant(c)
    S = scores(qh, ch)
    keys = np.log(policy(S, eps, tau_g)) + gumbel_of_bits(noise)
    B, G = S.shape
    sel = np.empty((B, top_c), dtype=np.int32)
    for b in range(B):
        sel[b] = np.lexsort((np.arange(G), -keys[b]))[:top_c]
    return sel, np.take_along_axis(S, sel, axis=1), keys, S


# ---------------------------------------------------------------------------
# online memory update, statistics side (Eq. memory_update; App. B.6)
# ---------------------------------------------------------------------------
FEEDBACK_FEATURES = 11     # r_imm, r_fut, pos, succ, comp, corr, safe, cfail, corfail, neg, risk
STATS_WORDS = 12           # count, then the fixed-point sum of each feature
FIXED_ONE = 1 << 24        # fixed-point scale of the sums


def feedback_update(G: int, n_buckets: int, src, dst, bucket, feat, node, edge, edge_bucket):
    """Rule-based aggregation of step outcomes into the memory's statistics
    (Eq. memory_update refreshes the node statistics of V_G(g_t) and the
    transition-edge feedback of E_G(g_{t-1}, g_t), t > 1; App. B.2 and B.6).
    Event e adds one observation with features feat[e] (the outcome's
    r_imm, r_fut and indicator/rate values, App. B.6) to node dst[e], and,
    when src[e] >= 0 (not the first step), to edge (src[e], dst[e]) and to
    that edge's state bucket bucket[e]. Sums are kept in fixed point
    (round-to-nearest-even of x * 2^24, exact int64 additions), so they do not
    depend on the order of the events. Events with dst or bucket out of range
    are skipped. Returns updated copies of node [G][12], edge [G][G][12],
    edge_bucket [G][G][n_buckets][12]."""
    node, edge, edge_bucket = (np.array(x, dtype=np.int64, copy=True) for x in
                               (node, edge, edge_bucket))
    fx = np.rint(np.asarray(feat, dtype=np.float32).astype(np.float64) * FIXED_ONE).astype(np.int64)
    for e in range(len(dst)):
        s, d, k = int(src[e]), int(dst[e]), int(bucket[e])
        if not (0 <= d < G and 0 <= k < n_buckets and s < G):
            continue
        rec = np.concatenate([[1], fx[e]])
        node[d] += rec
        if s >= 0:
            edge[s, d] += rec
            edge_bucket[s, d, k] += rec
    return node, edge, edge_bucket


def feature_vector(stats, h_ctx: float) -> np.ndarray:
    """z of App. B.6 (Eq. transition_feature_vector) from one statistics record:
    [r_imm, r_fut, p_pos | p_succ, p_comp, p_corr, p_safe, h_ctx |
     -p_cfail, -p_corfail, -p_neg, -rho_risk], means over the observations;
    no observation gives the zero prior."""
    stats = np.asarray(stats, dtype=np.int64)
    n = int(stats[0])
    if n == 0:
        return np.zeros(STATS_WORDS)
    m = stats[1:].astype(np.float64) / (n * FIXED_ONE)
    return np.concatenate([m[:7], [h_ctx], -m[7:]])


def transition_utility(edge, edge_bucket, s: int, g: int, k: int, min_count: int, w) -> float:
    """phi(s -> g | state bucket k) = w^T z: the bucket's statistics when it has
    at least min_count observations (h_ctx = 1), else the edge's aggregate
    statistics (h_ctx = 0) (App. B.6, Eq. transition_phi)."""
    eb = np.asarray(edge_bucket)[s, g, k]
    if eb[0] >= min_count and eb[0] > 0:
        z = feature_vector(eb, 1.0)
    else:
        z = feature_vector(np.asarray(edge)[s, g], 0.0)
    return float(np.dot(np.asarray(w, dtype=np.float64), z))


def transition_scores(prefix, bucket, lam: float, w, min_count: int, node, edge, edge_bucket):
    """Scores of every direction by the rule-based scorer: for a query with
    prefix (g_1..g_L) and state bucket k, score(g) = sum_i alpha_i
    phi(g_i -> g | k) with alpha_i = exp(-lam (L - i)) (Eq. score,
    Eq. prefix_weight); an empty prefix uses the node statistics of g
    (w^T z with h_ctx = 0). Returns [B][G] in double."""
    node = np.asarray(node)
    G = node.shape[0]
    prefix = np.asarray(prefix)
    B = prefix.shape[0]
    S = np.zeros((B, G))
    for b in range(B):
        L = 0
        while L < prefix.shape[1] and 0 <= prefix[b, L] < G:
            L += 1
        for g in range(G):
            if L == 0:
                S[b, g] = float(np.dot(w, feature_vector(node[g], 0.0)))
            else:
                a = prefix_weights(L, lam)
                S[b, g] = sum(a[i] * transition_utility(edge, edge_bucket, int(prefix[b, i]), g,
                                                        int(bucket[b]), min_count, w)
                              for i in range(L))
    return S
