"""Prefix-aware coarse scoring (htam_retrieve_coarse_prefix) through the C ABI
against the oracle: the selected clusters and their scores, by the tie-window
protocol of the coarse stage, with the window of a weighted sum of inner
products; and its reduction to htam_retrieve_coarse for a one-term prefix
over edge keys that repeat the node keys."""
import numpy as np
import pytest
import torch

import oracle
import parity
from gpu_cases import say, to_np
from paper_2605_29734_amd import synth

pytestmark = pytest.mark.gpu
U = 2.0 ** -24


def _inputs(spec, lmax, seed):
    from paper_2605_29734_amd import htam
    w = synth.make(spec, device="cuda", seed=seed)
    E, P = synth.make_prefix(spec, w.coarse_keys, lmax, device="cuda", seed=seed)
    dt = w.coarse_keys.dtype
    bank = htam.Bank(coarse_keys=w.coarse_keys, fine_keys=torch.zeros(1, spec.d, dtype=dt, device="cuda"),
                     seg_offsets=torch.zeros(spec.G + 1, dtype=torch.int64, device="cuda"),
                     transition_id=None, compute=spec.compute)
    return bank, w.queries, E, P


def _check(spec, q, C, E, P, lam, sel, ss):
    ref_sel, _, S = oracle.coarse_prefix(q, C, E, P, lam, spec.top_c, spec.compute)
    quant = oracle.round_bf16 if spec.compute == "bf16" else (lambda x: np.asarray(x, np.float32))
    qh, ch, eh = (quant(x).astype(np.float64) for x in (q, C, E))
    d = q.shape[1]
    n_acc = d if spec.compute == "bf16" else d + 1
    B, G = S.shape
    W = np.empty((B, G))
    for b in range(B):                  # window of each oracle score
        L = 0
        while L < P.shape[1] and 0 <= P[b, L] < G:
            L += 1
        if L == 0:
            W[b] = parity.window(np.abs(ch) @ np.abs(qh[b]), S[b], n_acc)
        else:
            a = oracle.prefix_weights(L, lam)
            absdot = sum(a[i] * (np.abs(eh[P[b, i]]) @ np.abs(qh[b])) for i in range(L))
            terms = sum(a[i] * np.abs(eh[P[b, i]] @ qh[b]) for i in range(L))
            W[b] = 2 * parity.gamma(n_acc) * absdot + 2 * (L + 2) * U * terms + U * np.abs(S[b])
    rtol = 2e-2 if spec.compute == "bf16" else 1e-5
    ties = 0
    for b in range(B):
        assert len(set(sel[b].tolist())) == spec.top_c
        theta = S[b, ref_sel[b, -1]]
        for g in set(sel[b].tolist()) ^ set(ref_sel[b].tolist()):
            assert abs(S[b, g] - theta) <= W[b, g] + W[b, ref_sel[b, -1]], f"row {b}: cluster {g}"
            ties += 1
        err = np.abs(ss[b] - S[b, sel[b]])
        assert np.all(err <= rtol * np.abs(S[b, sel[b]]) + W[b, sel[b]]), f"row {b}: scores"
        assert np.all(np.diff(ss[b]) <= 0)
    return ties


@pytest.mark.parametrize("storage,compute,B,G,d,lmax,lam,c", [
    ("bf16", "bf16", 200, 96, 256, 5, 0.5, 8),
    ("f32", "bf16", 64, 40, 128, 3, 1.0, 5),
    ("f32", "f32", 50, 33, 72, 4, 0.0, 4),
    ("bf16", "bf16", 300, 8, 64, 6, 2.0, 3),       # many pairs per source: several groups
])
def test_prefix_against_oracle(storage, compute, B, G, d, lmax, lam, c):
    from paper_2605_29734_amd import htam
    spec = synth.Spec("prefix", B=B, d=d, G=G, N=G, top_c=c, top_k=1, tau=1.0, storage=storage,
                      compute=compute, sizes="uniform")
    say(f"[case] prefix B={B} G={G} d={d} lmax={lmax} lambda={lam} {storage}/{compute}")
    bank, q, E, P = _inputs(spec, lmax, seed=B + G)
    sel, ss = htam.htam_retrieve_coarse_prefix(bank, E, P, lam, q, c)
    torch.cuda.synchronize()
    ties = _check(spec, to_np(q), to_np(bank.coarse_keys), to_np(E), to_np(P), lam, to_np(sel),
                  to_np(ss).astype(np.float64))
    say(f"[ok] prefix: tie events {ties}")


def test_one_term_prefix_over_node_edges_is_coarse():
    from paper_2605_29734_amd import htam
    spec = synth.Spec("prefix1", B=500, d=256, G=300, N=300, top_c=10, top_k=1, tau=1.0,
                      storage="bf16", compute="bf16", sizes="uniform")
    say("[case] one-term prefix over node-key edges")
    bank, q, _, _ = _inputs(spec, 1, seed=3)
    E = bank.coarse_keys.unsqueeze(0).expand(spec.G, -1, -1).contiguous()
    P = torch.randint(0, spec.G, (spec.B, 1), dtype=torch.int32, device="cuda")
    sel, ss = htam.htam_retrieve_coarse_prefix(bank, E, P, 0.9, q, spec.top_c)
    sel0, ss0 = htam.htam_retrieve_coarse(bank, q, spec.top_c)
    torch.cuda.synchronize()
    # alpha = exp(0) = 1 and the same MFMA inner products: the same bits
    np.testing.assert_array_equal(to_np(sel), to_np(sel0))
    np.testing.assert_array_equal(to_np(ss), to_np(ss0))
