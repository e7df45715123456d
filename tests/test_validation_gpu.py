"""Malformed banks through the C ABI: segment offsets that are not a partition
of the bank's rows, a tiled copy of the keys whose header does not match
them, and selected cluster ids out of range.

The first kernel that reads the offsets (the routing's planning step) checks
them before any record is indexed through them, so such a call reads no bank
row and leaves every slot empty. With HTAM_VALIDATE set the call waits for
that check and returns HTAM_ERR_VALUE. Both routing paths are covered: the
one-block routing (few (query, slot) pairs) and the multi-block routing."""
import numpy as np
import pytest
import torch

from gpu_cases import say, to_np
from paper_2605_29734_amd import synth

pytestmark = pytest.mark.gpu


def _bank_and_queries(B, G=16, N=2000, d=64, seed=5):
    from paper_2605_29734_amd import htam
    spec = synth.Spec("validate", B=B, d=d, G=G, N=N, top_c=4, top_k=8, tau=1.0, storage="bf16",
                      compute="bf16", sizes="uniform")
    w = synth.make(spec, device="cuda", seed=seed)
    bank = htam.build_bank(w.cluster_of, w.keys_in, w.coarse_keys, "bf16")
    torch.cuda.synchronize()
    return spec, bank, w.queries


def _malformed(off: torch.Tensor, how: str) -> torch.Tensor:
    o = off.clone()
    G = o.numel() - 1
    if how == "end_past_rows":        # off[G] > N: the last segment would run off the bank
        o[G] += 1000
    elif how == "start_not_zero":
        o[0] = 5
    elif how == "decreasing":         # a negative segment length
        o[3] = o[4] + 7
    elif how == "negative":
        o[1] = -64
    return o


@pytest.mark.parametrize("B", [40, 4200])          # one-block and multi-block routing
@pytest.mark.parametrize("how", ["end_past_rows", "start_not_zero", "decreasing", "negative"])
def test_malformed_offsets(B, how, monkeypatch):
    from paper_2605_29734_amd import htam
    say(f"[case] malformed offsets ({how}), B={B}")
    spec, bank, q = _bank_and_queries(B)
    bad = htam.Bank(coarse_keys=bank.coarse_keys, fine_keys=bank.fine_keys,
                    seg_offsets=_malformed(bank.seg_offsets, how),
                    transition_id=bank.transition_id, compute="bf16")
    sel, _ = htam.htam_retrieve_coarse(bank, q, spec.top_c)
    monkeypatch.delenv("HTAM_VALIDATE", raising=False)
    smax, ssum, cs, ci = (to_np(x) for x in htam.htam_attend_transitions(bad, q, sel, spec.tau,
                                                                           spec.top_k))
    torch.cuda.synchronize()
    assert np.all(smax == -np.inf) and np.all(ssum == 0.0)
    assert np.all(ci == -1) and np.all(cs == -np.inf)
    monkeypatch.setenv("HTAM_VALIDATE", "1")
    with pytest.raises(htam.HtamError) as ei:
        htam.htam_attend_transitions(bad, q, sel, spec.tau, spec.top_k)
    assert ei.value.status == -4 and "seg_offsets" in str(ei.value)


@pytest.mark.parametrize("B", [40, 4200])
def test_validate_mode_passes_good_banks_and_flags_bad_selections(B, monkeypatch):
    from paper_2605_29734_amd import htam
    say(f"[case] validate mode, B={B}")
    spec, bank, q = _bank_and_queries(B)
    sel, _ = htam.htam_retrieve_coarse(bank, q, spec.top_c)
    monkeypatch.delenv("HTAM_VALIDATE", raising=False)
    plain = [to_np(x) for x in htam.htam_attend_transitions(bank, q, sel, spec.tau, spec.top_k)]
    monkeypatch.setenv("HTAM_VALIDATE", "1")
    checked = [to_np(x) for x in htam.htam_attend_transitions(bank, q, sel, spec.tau, spec.top_k)]
    for a, b in zip(plain, checked):
        np.testing.assert_array_equal(a, b)
    bad_sel = sel.clone()
    bad_sel[3, 1] = spec.G
    with pytest.raises(htam.HtamError) as ei:
        htam.htam_attend_transitions(bank, q, bad_sel, spec.tau, spec.top_k)
    assert ei.value.status == -4 and "outside" in str(ei.value)


@pytest.mark.parametrize("B", [40, 4200])          # one-block and multi-block routing
@pytest.mark.parametrize("how", ["shifted_segment", "start_not_zero"])
def test_tiled_copy_header_mismatch(B, how, monkeypatch):
    """A tiled copy whose header of segment starts does not match the bank's
    offsets (a stale copy): checked with the offsets, before any row is read
    through it; a matching copy passes and gives the row-major results."""
    import dataclasses
    from paper_2605_29734_amd import htam
    say(f"[case] tiled copy header ({how}), B={B}")
    spec, bank, q = _bank_and_queries(B)
    tb = htam.with_tiled_keys(bank)
    sel, _ = htam.htam_retrieve_coarse(bank, q, spec.top_c)
    monkeypatch.setenv("HTAM_VALIDATE", "1")
    plain = [to_np(x) for x in htam.htam_attend_transitions(bank, q, sel, spec.tau, spec.top_k)]
    tiled = [to_np(x) for x in htam.htam_attend_transitions(tb, q, sel, spec.tau, spec.top_k)]
    for a, b in zip(plain, tiled):
        np.testing.assert_array_equal(a, b)
    raw = tb.fine_keys_tiled.clone()
    head = raw.view(torch.uint8)[:(spec.G + 1) * 8].view(torch.int64)
    if how == "shifted_segment":
        head[3:] += 16
    else:
        head[0] = 16
    bad = dataclasses.replace(tb, fine_keys_tiled=raw)
    monkeypatch.delenv("HTAM_VALIDATE", raising=False)
    smax, ssum, cs, ci = (to_np(x) for x in htam.htam_attend_transitions(bad, q, sel, spec.tau,
                                                                           spec.top_k))
    torch.cuda.synchronize()
    assert np.all(smax == -np.inf) and np.all(ssum == 0.0)
    assert np.all(ci == -1) and np.all(cs == -np.inf)
    monkeypatch.setenv("HTAM_VALIDATE", "1")
    with pytest.raises(htam.HtamError) as ei:
        htam.htam_attend_transitions(bad, q, sel, spec.tau, spec.top_k)
    assert ei.value.status == -4 and "fine_keys_tiled" in str(ei.value)
