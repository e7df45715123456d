"""Shared driver of the GPU parity tests: draw a workload, build the bank and run
retrieval through the C ABI, then compare with the CPU oracle (tests/parity.py)."""
from __future__ import annotations

import sys

import numpy as np
import torch

import oracle
import parity
from paper_2605_29734_amd import synth


def say(msg: str):
    print(msg, flush=True)
    sys.stdout.flush()


def to_np(t: torch.Tensor) -> np.ndarray:
    if t.dtype == torch.bfloat16:
        t = t.float()
    return t.detach().cpu().numpy()


def run_case(spec, seed=0, rows=None, tau=None, gen_device="cpu", check_build=True,
             determinism=False, identity_ids=False, tiled=False):
    from paper_2605_29734_amd import htam
    dev = torch.device("cuda:0")
    tau = spec.tau if tau is None else tau
    say(f"[case] {spec.name} B={spec.B} d={spec.d} G={spec.G} N={spec.N} c={spec.top_c} "
        f"k={spec.top_k} tau={tau} storage={spec.storage} compute={spec.compute} seed={seed}")
    w = synth.make(spec, device=gen_device, seed=seed)
    q = w.queries.to(dev)
    ck = w.coarse_keys.to(dev)
    cl = w.cluster_of.to(dev)
    kin = w.keys_in.to(dev)
    say("[step] htam_memory_build")
    bank = htam.build_bank(cl, kin, ck, spec.compute)
    torch.cuda.synchronize()
    off = to_np(bank.seg_offsets)
    tid = to_np(bank.transition_id)
    if check_build:
        say("[step] build parity")
        ref_off, ref_tid = oracle.build_bank(to_np(cl), spec.G)
        assert np.array_equal(off, ref_off), "seg_offsets differ from the oracle's build"
        assert np.array_equal(tid, ref_tid), "transition ids differ from the oracle's build"
        if spec.N <= (1 << 20):
            assert torch.equal(bank.fine_keys, kin[bank.transition_id.long()]), "key gather"
    del kin
    if identity_ids:        # the bank without a transition id array: ids are bank rows
        bank = htam.Bank(coarse_keys=bank.coarse_keys, fine_keys=bank.fine_keys,
                         seg_offsets=bank.seg_offsets, transition_id=None, compute=bank.compute)
        tid = None
    plain = None
    if tiled:               # the same bank read through its prepared copies
        say("[step] retrieve without the prepared copies")
        plain = {k: to_np(v) for k, v in
                 htam.Retriever(bank, spec.B, spec.top_c, spec.top_k, tau).run(q).items()}
        torch.cuda.synchronize()
        say("[step] htam_memory_tile, htam_coarse_keys_bf16")
        bank = htam.prepared(bank)
    say("[step] retrieve (coarse, attend, topk)")
    r = htam.Retriever(bank, spec.B, spec.top_c, spec.top_k, tau)
    out = r.run(q)
    torch.cuda.synchronize()
    gpu = {k: to_np(v) for k, v in out.items()}
    if plain is not None:
        for k in gpu:       # only where keys are read from changes: the same bits
            assert np.array_equal(gpu[k], plain[k], equal_nan=True), f"{k}: prepared bank differs"
        del plain
    if determinism:
        say("[step] second run for bitwise determinism")
        again = {k: to_np(v) for k, v in r.run(q).items()}
        torch.cuda.synchronize()
        for k in gpu:
            assert np.array_equal(gpu[k], again[k], equal_nan=True), f"{k} differs between runs"
    if callable(rows):      # rows chosen after the GPU run, from its full outputs
        rows = rows(gpu, np.diff(off))
    if rows is not None:
        rows = np.asarray(rows)
        gpu = {k: v[rows] for k, v in gpu.items()}

    def fetch(a, b):
        return to_np(bank.fine_keys[a:b])

    def gather(brow):
        idx = torch.from_numpy(np.asarray(brow, dtype=np.int64)).to(dev)
        return to_np(bank.fine_keys.index_select(0, idx))

    say("[step] oracle comparison")
    rep = parity.check(gpu, to_np(q), to_np(ck), off, spec.top_c, spec.top_k, tau, spec.compute,
                       fetch, gather, transition_id=tid, rows=rows)
    say(f"[ok] {spec.name}: {dict(rep)}")
    rep["sel"] = gpu["sel"]
    rep["sizes"] = np.diff(off)
    return rep
