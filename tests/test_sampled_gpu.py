"""The sampled direction choice (htam_retrieve_coarse_sampled) through the C
ABI: with caller-supplied uniform words against the oracle's Gumbel-top-k
over the same words, and with the library's Philox draws against the policy
by chi-square frequencies, plus determinism per (seed, offset)."""
import numpy as np
import pytest
import torch
from scipy.stats import chi2

import oracle
import parity
from gpu_cases import say, to_np
from paper_2605_29734_amd import synth

pytestmark = pytest.mark.gpu
U = 2.0 ** -24


def _bank(spec, seed):
    from paper_2605_29734_amd import htam
    w = synth.make(spec, device="cuda", seed=seed)
    dt = w.coarse_keys.dtype
    bank = htam.Bank(coarse_keys=w.coarse_keys, fine_keys=torch.zeros(1, spec.d, dtype=dt, device="cuda"),
                     seg_offsets=torch.zeros(spec.G + 1, dtype=torch.int64, device="cuda"),
                     transition_id=None, compute=spec.compute)
    return bank, w.queries


@pytest.mark.parametrize("storage,compute,B,G,d,c,eps,tau", [
    ("bf16", "bf16", 300, 500, 256, 8, 0.2, 0.1),
    ("f32", "bf16", 64, 3000, 128, 16, 0.0, 0.05),    # segmented selection (G > 2048)
    ("f32", "f32", 40, 33, 72, 4, 1.0, 1.0),          # uniform: the words decide
    ("bf16", "bf16", 100, 64, 64, 64, 0.5, 0.3),      # every cluster drawn (a full order)
])
@pytest.mark.parametrize("source", ["words", "philox"])
def test_sampled_against_oracle(storage, compute, B, G, d, c, eps, tau, source):
    """source "words": the caller's uniform words; "philox": the library's own
    draws, against the oracle fed with Philox4x32-10 words of the same (seed,
    offset), its implementation pinned by the published known answers."""
    from paper_2605_29734_amd import htam
    spec = synth.Spec("sampled", B=B, d=d, G=G, N=G, top_c=c, top_k=1, tau=1.0, storage=storage,
                      compute=compute, sizes="uniform")
    say(f"[case] sampled B={B} G={G} d={d} c={c} eps={eps} tau_g={tau} {storage}/{compute} {source}")
    bank, q = _bank(spec, seed=G + c)
    if source == "words":
        noise = torch.randint(-2 ** 31, 2 ** 31, (B, G), dtype=torch.int32, device="cuda",
                              generator=torch.Generator(device="cuda").manual_seed(B))
        sel, ss = htam.htam_retrieve_coarse_sampled(bank, q, c, eps, tau, noise=noise)
        words = to_np(noise).view(np.uint32)
    else:
        seed, offset = 0xDEADBEEF00000000 + G, (3 << 32) + B
        sel, ss = htam.htam_retrieve_coarse_sampled(bank, q, c, eps, tau, seed=seed, offset=offset)
        words = oracle.philox_words(seed, offset, B, G)
    torch.cuda.synchronize()
    sel, ss = to_np(sel), to_np(ss).astype(np.float64)
    ref_sel, _, keys, S = oracle.coarse_sampled(to_np(q), to_np(bank.coarse_keys), c, eps, tau,
                                                words, compute)
    quant = oracle.round_bf16 if compute == "bf16" else (lambda x: np.asarray(x, np.float32))
    qh = quant(to_np(q)).astype(np.float64)
    ch = quant(to_np(bank.coarse_keys)).astype(np.float64)
    n_acc = d if compute == "bf16" else d + 1
    W = parity.window(np.abs(qh) @ np.abs(ch).T, S, n_acc)
    gum = oracle.gumbel_of_bits(words)
    m = S.max(axis=1, keepdims=True)
    lz = 2 * G * U if 0.0 < eps < 1.0 else 0.0
    # window of each key: the scores' windows through 1/tau, fp32 rounding of
    # (s - m)/tau, the Gumbel variate and the log-sum, and of log Z (eps in (0, 1))
    Wk = ((W + W[np.arange(B), S.argmax(axis=1)][:, None]) / tau
          + 4 * U * (np.abs(S - m) / tau + np.abs(gum) + np.abs(keys) + 2) + lz)
    rtol = 2e-2 if compute == "bf16" else 1e-5
    ties = 0
    for b in range(B):
        assert len(set(sel[b].tolist())) == c
        kth = ref_sel[b, -1]
        for g in set(sel[b].tolist()) ^ set(ref_sel[b].tolist()):
            assert abs(keys[b, g] - keys[b, kth]) <= Wk[b, g] + Wk[b, kth], f"row {b}: cluster {g}"
            ties += 1
        for a in range(c - 1):                       # draw order = descending key
            g0, g1 = sel[b, a], sel[b, a + 1]
            assert keys[b, g0] >= keys[b, g1] - Wk[b, g0] - Wk[b, g1], f"row {b}: order"
        np.testing.assert_allclose(ss[b], S[b, sel[b]], rtol=rtol, atol=W[b, sel[b]].max())
    say(f"[ok] sampled: key-window events {ties}")


def _repeat_query(G, n, d=64, seed=5):
    from paper_2605_29734_amd import htam
    spec = synth.Spec("freq", B=1, d=d, G=G, N=G, top_c=2, top_k=1, tau=1.0, storage="bf16",
                      compute="bf16", sizes="uniform")
    bank, q = _bank(spec, seed)
    S = oracle.scores(oracle.round_bf16(to_np(q)), oracle.round_bf16(to_np(bank.coarse_keys)))
    return bank, q.repeat(n, 1).contiguous(), S


@pytest.mark.parametrize("eps,tau", [(0.3, 0.1), (1.0, 1.0), (0.0, 0.05)])
def test_philox_draws_follow_the_policy(eps, tau):
    """65,536 independent draws (one query repeated; each row has its own
    counter): the first pick has the policy's distribution, and the ordered
    first two picks that of sampling without replacement, chi-square at the
    1e-4 level."""
    from paper_2605_29734_amd import htam
    G, n = 8, 65536
    say(f"[case] Philox draws eps={eps} tau_g={tau}")
    bank, Q, S = _repeat_query(G, n)
    sel, _ = htam.htam_retrieve_coarse_sampled(bank, Q, 2, eps, tau, seed=20261202, offset=7)
    torch.cuda.synchronize()
    sel = to_np(sel)
    mu = oracle.policy(S, eps, tau)[0]
    exp1 = n * mu
    m1 = exp1 > 5
    obs = np.bincount(sel[:, 0], minlength=G)
    assert np.all(obs[~m1] <= 5 * (~m1).sum() + 5)
    stat = ((obs[m1] - exp1[m1]) ** 2 / exp1[m1]).sum()
    assert stat < chi2.ppf(1 - 1e-4, max(m1.sum() - 1, 1)), f"first pick chi2 {stat}"
    exp2 = n * np.array([mu[a] * mu[b] / (1 - mu[a]) if a != b else 0.0
                         for a in range(G) for b in range(G)])
    obs2 = np.bincount(sel[:, 0] * G + sel[:, 1], minlength=G * G)
    assert np.all(obs2[exp2 == 0] == 0)
    m2 = exp2 > 5
    stat2 = ((obs2[m2] - exp2[m2]) ** 2 / exp2[m2]).sum()
    assert stat2 < chi2.ppf(1 - 1e-4, max(m2.sum() - 1, 1)), f"pair chi2 {stat2}"
    say(f"[ok] chi2 first {stat:.1f} pairs {stat2:.1f}")


def test_philox_draws_are_reproducible():
    from paper_2605_29734_amd import htam
    bank, Q, _ = _repeat_query(64, 4096)
    a, _ = htam.htam_retrieve_coarse_sampled(bank, Q, 4, 0.5, 0.5, seed=1, offset=0)
    b, _ = htam.htam_retrieve_coarse_sampled(bank, Q, 4, 0.5, 0.5, seed=1, offset=0)
    c, _ = htam.htam_retrieve_coarse_sampled(bank, Q, 4, 0.5, 0.5, seed=1, offset=1)
    d, _ = htam.htam_retrieve_coarse_sampled(bank, Q, 4, 0.5, 0.5, seed=2, offset=0)
    torch.cuda.synchronize()
    assert torch.equal(a, b)
    assert (a != c).any(dim=1).float().mean() > 0.5
    assert (a != d).any(dim=1).float().mean() > 0.5
    assert (a[1:] != a[:-1]).any(dim=1).float().mean() > 0.5      # rows draw independently
