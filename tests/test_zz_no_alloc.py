"""htam_attend_transitions_noalloc (workspace in the library's own device
array) against htam_attend_transitions (caller workspace), through the C ABI:
the same kernels on the same inputs, so the outputs must be the same bits.
Two calls in a row, the second with fewer queries and other sizes (the array
keeps the first call's contents, which the kernels must not depend on), and
a call too large for the array, which is refused before anything runs."""
import numpy as np
import pytest
import torch

from gpu_cases import say, to_np
from paper_2605_29734_amd import synth

pytestmark = pytest.mark.gpu


def _case(spec, seed):
    from paper_2605_29734_amd import htam
    w = synth.make(spec, device="cuda", seed=seed)
    bank = htam.build_bank(w.cluster_of, w.keys_in, w.coarse_keys, spec.compute)
    sel, _ = htam.htam_retrieve_coarse(bank, w.queries, spec.top_c)
    torch.cuda.synchronize()
    return bank, w.queries, sel


def _compare(spec, bank, q, sel):
    from paper_2605_29734_amd import htam
    ref = htam.htam_attend_transitions(bank, q, sel, spec.tau, spec.top_k)
    got = htam.htam_attend_transitions_noalloc(bank, q, sel, spec.tau, spec.top_k)
    torch.cuda.synchronize()
    for name, a, b in zip(("slot_max", "slot_sum", "cand_score", "cand_id"), got, ref):
        np.testing.assert_array_equal(to_np(a), to_np(b), err_msg=name)
    assert int((to_np(got[3]) >= 0).sum()) > 0


def test_noalloc_matches_workspace_entry_point():
    from paper_2605_29734_amd import htam
    first = synth.scaled(synth.SPECS["mixture_bf16"], B=512, G=256, N=262144)   # ~8 MiB of workspace
    say(f"[case] noalloc call 1: B={first.B} G={first.G} N={first.N}")
    _compare(first, *_case(first, seed=1))
    second = synth.scaled(synth.SPECS["zipf_bf16"], B=100, G=64, N=20000, top_k=24)
    say(f"[case] noalloc call 2: B={second.B} G={second.G} N={second.N}")
    _compare(second, *_case(second, seed=2))

    say("[case] noalloc call beyond the scratch array")
    big = synth.scaled(synth.SPECS["zipf_bf16"], B=8192, G=64, N=20000, top_c=16, top_k=256)
    bank, q, _ = _case(synth.scaled(big, B=4), seed=3)
    qq = q.repeat(big.B // 4, 1).contiguous()
    sel = torch.zeros(big.B, big.top_c, dtype=torch.int32, device="cuda")
    out = [torch.full((big.B, big.top_c), 7.0, device="cuda") for _ in range(2)]
    with pytest.raises(htam.HtamError) as ei:
        htam.htam_attend_transitions_noalloc(bank, qq, sel, big.tau, big.top_k,
                                             out=(out[0], out[1],
                                                  torch.empty(big.B, big.top_c, big.top_k,
                                                              device="cuda"),
                                                  torch.empty(big.B, big.top_c, big.top_k,
                                                              dtype=torch.int32, device="cuda")))
    assert ei.value.status == -5 and "scratch" in str(ei.value)
    torch.cuda.synchronize()
    assert torch.all(out[0] == 7.0) and torch.all(out[1] == 7.0)      # nothing ran
