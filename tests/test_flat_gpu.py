"""Flat memory retrieval (htam_retrieve_flat: every record a candidate, no
coarse level) through the C ABI against the oracle's flat retrieval, and
against the hierarchical path with every cluster selected (which leaves it
nothing to exclude)."""
import numpy as np
import pytest
import torch

import oracle
import parity
from gpu_cases import say, to_np
from paper_2605_29734_amd import synth

pytestmark = pytest.mark.gpu


def _flat_case(spec, seed=0, identity_ids=False, rows=None):
    from paper_2605_29734_amd import htam
    say(f"[case] flat {spec.name} B={spec.B} d={spec.d} N={spec.N} k={spec.top_k} "
        f"tau={spec.tau} storage={spec.storage} compute={spec.compute}")
    w = synth.make(spec, device="cuda", seed=seed)
    bank = htam.build_bank(w.cluster_of, w.keys_in, w.coarse_keys, spec.compute)
    if identity_ids:
        bank = htam.Bank(coarse_keys=bank.coarse_keys, fine_keys=bank.fine_keys,
                         seg_offsets=bank.seg_offsets, transition_id=None, compute=spec.compute)
    out = htam.htam_retrieve_flat(bank, w.queries, spec.tau, spec.top_k)
    torch.cuda.synchronize()
    names = ("id", "score", "weight", "m", "Z", "count")
    gpu = {k: to_np(v) for k, v in zip(names, out)}
    rows = np.arange(spec.B) if rows is None else np.asarray(rows)
    gpu = {k: v[rows] for k, v in gpu.items()}
    keys = to_np(bank.fine_keys)
    tid = None if identity_ids else to_np(bank.transition_id)
    ref = oracle.flat(to_np(w.queries)[rows], keys, spec.tau, spec.top_k, spec.compute,
                      transition_id=tid)
    inv = None
    if tid is not None:
        inv = np.empty(tid.size, dtype=np.int64)
        inv[tid] = np.arange(tid.size)
    kq = oracle.round_bf16(keys) if spec.compute == "bf16" else keys

    def key_rows(ids):
        return kq[ids if inv is None else inv[ids]]

    rep = parity.check_rows(gpu, ref, ref["qh"], key_rows, spec.tau, spec.compute, tag="flat")
    say(f"[ok] flat {spec.name}: {dict(rep)}")
    return rep


@pytest.mark.parametrize("storage,compute,d,N,k,tau,ident", [
    ("bf16", "bf16", 256, 5000, 32, 1.0, False),      # GEMM tiles, 3 segments (ragged)
    ("f32", "bf16", 512, 3000, 20, 0.3, False),       # fp32 storage rounded to bf16
    ("f32", "f32", 72, 1000, 7, 0.07, True),          # fp32 arithmetic, d % 32 != 0, row ids
    ("bf16", "bf16", 64, 40, 64, 1.0, False),         # fewer records than k (padding)
    ("bf16", "bf16", 96, 9000, 256, 0.5, False),      # the largest k, small-tile GEMM
])
def test_flat_against_oracle(storage, compute, d, N, k, tau, ident):
    spec = synth.Spec("flat", B=70, d=d, G=8, N=N, top_c=1, top_k=k, tau=tau, storage=storage,
                      compute=compute, sizes="zipf", zipf_s=1.0, min_size=1)
    _flat_case(spec, identity_ids=ident)


def test_flat_several_bands():
    """4096 queries cap the score band at 16,384 records: 40,000 records take
    three GEMM launches, whose segment lists are merged."""
    spec = synth.Spec("flat_bands", B=4096, d=64, G=16, N=40000, top_c=1, top_k=16, tau=0.2,
                      storage="bf16", compute="bf16", sizes="uniform")
    _flat_case(spec, rows=np.sort(np.random.default_rng(0).choice(4096, 96, replace=False)))


def test_hierarchy_with_every_cluster_equals_flat():
    from paper_2605_29734_amd import htam
    spec = synth.Spec("allclusters", B=96, d=256, G=64, N=20000, top_c=64, top_k=32, tau=0.5,
                      storage="bf16", compute="bf16", sizes="zipf", zipf_s=1.0, min_size=10)
    say("[case] hierarchy with top_c = G vs flat")
    w = synth.make(spec, device="cuda", seed=4)
    bank = htam.build_bank(w.cluster_of, w.keys_in, w.coarse_keys, spec.compute)
    h = htam.retrieve(bank, w.queries, spec.top_c, spec.top_k, spec.tau)
    f = htam.htam_retrieve_flat(bank, w.queries, spec.tau, spec.top_k)
    torch.cuda.synchronize()
    hn = {k: to_np(h[k]) for k in ("id", "score", "weight", "m", "Z", "count")}
    fn = dict(zip(("id", "score", "weight", "m", "Z", "count"), (to_np(x) for x in f)))
    np.testing.assert_array_equal(hn["count"], fn["count"])
    # the same MFMA inner products: the same scores, maxima and (up to exact
    # ties, ordered by id either way) the same ids
    np.testing.assert_array_equal(hn["score"], fn["score"])
    np.testing.assert_array_equal(hn["m"], fn["m"])
    np.testing.assert_array_equal(hn["id"], fn["id"])
    # the sums add the same terms in another order
    np.testing.assert_allclose(hn["Z"], fn["Z"], rtol=1e-5)
    np.testing.assert_allclose(hn["weight"], fn["weight"], rtol=1e-5)
