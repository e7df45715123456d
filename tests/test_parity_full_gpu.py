"""GPU parity at the full workload sizes, in the launch configuration the bench
times: the whole batch runs on the GPU, and a seeded sample of queries is
checked against the CPU oracle (rows are independent, so a sample is exact
for the rows it covers). The oracle streams the sampled rows' segments from
the device cluster by cluster."""
import numpy as np
import pytest
import torch

from gpu_cases import run_case
from paper_2605_29734_amd import synth

pytestmark = pytest.mark.gpu
S = synth.SPECS


def _rows(spec, n, seed=0):
    return np.sort(np.random.default_rng(seed).choice(spec.B, size=n, replace=False))


@pytest.mark.parametrize("name,n_rows", [
    ("zipf_bf16", 256),             # every query of the benchmarked workload
    ("mixture_bf16", 48),
    ("zipf_large_bf16", 24),
    ("before_after_f32", 24),
])
def test_full_size_sampled(name, n_rows):
    spec = S[name]
    run_case(spec, rows=_rows(spec, min(n_rows, spec.B)), gen_device="cuda",
             check_build=name == "zipf_bf16")
    torch.cuda.empty_cache()
