"""The seeded input generator: reproducible, shaped as specified."""
import numpy as np
import pytest
import torch

from paper_2605_29734_amd import synth


def test_zipf_sizes_rank_law_and_sum():
    rng = np.random.default_rng(0)
    sizes = synth.zipf_sizes(65536, 256, 1.2, 8, rng)
    assert sizes.sum() == 65536 and sizes.min() >= 8 and sizes.size == 256
    ranked = np.sort(sizes)[::-1].astype(np.float64)
    # size_r ~ r^-s: the log-log slope over ranks 1..256 is about -1.2
    slope = np.polyfit(np.log(np.arange(1, 257)), np.log(ranked), 1)[0]
    assert -1.25 < slope < -1.15
    big = synth.zipf_sizes(8388608, 4096, 1.1, 8, np.random.default_rng(0))
    assert big.sum() == 8388608 and big.min() >= 8


def test_zipf_min_clamp():
    sizes = synth.zipf_sizes(1000, 100, 2.0, 5, np.random.default_rng(1))
    assert sizes.sum() == 1000 and sizes.min() >= 5


@pytest.mark.parametrize("name", ["paper_htg", "tiny_f32"])
def test_small_workloads_shapes(name):
    w = synth.make(name)
    s = w.spec
    assert w.queries.shape == (s.B, s.d) and w.coarse_keys.shape == (s.G, s.d)
    assert w.keys_in.shape == (s.N, s.d) and w.cluster_of.shape == (s.N,)
    assert int(w.sizes.sum()) == s.N
    np.testing.assert_array_equal(np.bincount(w.cluster_of.numpy(), minlength=s.G), w.sizes)
    np.testing.assert_allclose(w.keys_in.norm(dim=1).numpy(), 1.0, rtol=1e-5)
    if name == "paper_htg":
        np.testing.assert_array_equal(w.sizes, [4, 3, 3, 3, 3])


def test_reproducible_and_seeded():
    a = synth.make(synth.scaled(synth.SPECS["zipf_bf16"], N=4096, G=32, B=16, d=64))
    b = synth.make(synth.scaled(synth.SPECS["zipf_bf16"], N=4096, G=32, B=16, d=64))
    c = synth.make(synth.scaled(synth.SPECS["zipf_bf16"], N=4096, G=32, B=16, d=64), seed=1)
    assert torch.equal(a.keys_in, b.keys_in) and torch.equal(a.cluster_of, b.cluster_of)
    assert not torch.equal(a.keys_in, c.keys_in)
    assert a.keys_in.dtype == torch.bfloat16


def test_mixture_and_before_after_draws():
    m = synth.make(synth.scaled(synth.SPECS["mixture_bf16"], B=32, d=256, G=16, N=1024))
    k = m.keys_in.float()
    cen = m.coarse_keys.float()
    # every record lies close to its own centre (sigma = 0.1 noise)
    cos = (k * cen[m.cluster_of.long()]).sum(1)
    assert cos.min() > 0.95
    ba = synth.make(synth.scaled(synth.SPECS["before_after_f32"], B=8, d=128, G=8, N=64))
    half = ba.keys_in[:, :64].norm(dim=1)
    np.testing.assert_allclose(half.numpy(), 0.5 ** 0.5, rtol=1e-5)
    assert ba.keys_in.dtype == torch.float32 and ba.spec.compute == "bf16"
