"""Seeded synthetic inputs for hierarchical transition-attended retrieval.

This module only draws inputs (queries, coarse keys, transition records and
their parent clusters); it holds none of the retrieval arithmetic, and both the
GPU library's tests and the CPU oracle are fed from it.

The paper (arXiv 2605.29734) stores its memory as text and measures only
search outcomes, so there is no dataset of embeddings to load: every workload
below is synthetic, with the shape of a two-level memory (coarse cluster keys,
and transition records grouped under a parent cluster, Sec. 4.1, Eq. HTG).

Workloads (name -> shape):
  paper_htg        the paper's initial memory shape: 5 global nodes holding
                   4/3/3/3/3 local records (App. B.1 global-node table and the
                   local-node catalogue), d = 64, 6 queries (T = 6 steps), c = 1,
                   k = 1, fp32.
  tiny_f32         16 queries, d = 128, 32 clusters x 64 records (contiguous),
                   c = 4, k = 8, fp32.
  zipf_bf16        256 queries, d = 512, 256 clusters, 65,536 records, cluster
                   sizes by a Zipf(1.2) rank law (min 8), c = 8, k = 16, bf16.
  mixture_bf16     1,024 queries, d = 1,024, 1,024 clusters x 1,024 records, keys
                   drawn around 1,024 Gaussian centres (sigma = 0.1), c = 16,
                   k = 32, bf16.
  zipf_large_bf16  4,096 queries, d = 1,024, 4,096 clusters, 8,388,608 records,
                   Zipf(1.1) sizes (min 8), tau = 0.07, c = 32, k = 64, bf16.
  before_after_f32 8,192 queries, d = 2,048 (before-state and after-state halves
                   of 1,024), 16,384 clusters x 256 records, c = 16, k = 128,
                   fp32 storage with bf16 arithmetic.

Draw rules:
  * unit Gaussian rows: x ~ N(0, I_d), divided by its L2 norm;
  * Zipf rank law: size_r proportional to r^-s for r = 1..G, floored, clamped
    to the minimum, corrected to sum exactly to N (largest fractional parts
    first), and assigned to cluster ids by a seeded permutation;
  * mixture: centres mu_g = unit Gaussian; a record or query of centre g is
    (mu_g + sigma * e / sqrt(d)) / norm with e ~ N(0, I_d); coarse keys = centres;
  * before/after: [e_before; e_after], each half a unit Gaussian row of d/2
    scaled by 1/sqrt(2), so that the whole row has unit norm;
  * records are stored in a seeded shuffled order (cluster_of gives each
    record's parent), except tiny_f32 and paper_htg whose records come grouped
    by cluster; building the bank sorts them.

All draws use one torch.Generator per (seed, workload, role) on the target
device, so a workload is reproducible on a given device type.
"""
from __future__ import annotations

import dataclasses
import zlib

import numpy as np
import torch


@dataclasses.dataclass(frozen=True)
class Spec:
    name: str
    B: int            # queries per batch
    d: int            # embedding width
    G: int            # clusters (coarse keys)
    N: int            # transition records
    top_c: int
    top_k: int
    tau: float
    storage: str      # "f32" | "bf16"  (stored dtype of queries and keys)
    compute: str      # "f32" | "bf16"  (arithmetic dtype of the scores)
    sizes: str        # "uniform" | "zipf" | "fixed"
    zipf_s: float = 0.0
    min_size: int = 0
    keys: str = "gauss"   # "gauss" | "mixture" | "before_after"
    sigma: float = 0.0
    shuffled: bool = True
    fixed_sizes: tuple = ()


SPECS = {
    "paper_htg": Spec("paper_htg", B=6, d=64, G=5, N=16, top_c=1, top_k=1, tau=1.0,
                      storage="f32", compute="f32", sizes="fixed", fixed_sizes=(4, 3, 3, 3, 3),
                      shuffled=False),
    "tiny_f32": Spec("tiny_f32", B=16, d=128, G=32, N=2048, top_c=4, top_k=8, tau=1.0,
                     storage="f32", compute="f32", sizes="uniform", shuffled=False),
    "zipf_bf16": Spec("zipf_bf16", B=256, d=512, G=256, N=65536, top_c=8, top_k=16, tau=1.0,
                      storage="bf16", compute="bf16", sizes="zipf", zipf_s=1.2, min_size=8),
    "mixture_bf16": Spec("mixture_bf16", B=1024, d=1024, G=1024, N=1048576, top_c=16, top_k=32,
                         tau=1.0, storage="bf16", compute="bf16", sizes="uniform",
                         keys="mixture", sigma=0.1),
    "zipf_large_bf16": Spec("zipf_large_bf16", B=4096, d=1024, G=4096, N=8388608, top_c=32,
                            top_k=64, tau=0.07, storage="bf16", compute="bf16", sizes="zipf",
                            zipf_s=1.1, min_size=8),
    "before_after_f32": Spec("before_after_f32", B=8192, d=2048, G=16384, N=4194304, top_c=16,
                             top_k=128, tau=1.0, storage="f32", compute="bf16", sizes="uniform",
                             keys="before_after"),
}


def scaled(spec: Spec, **changes) -> Spec:
    """A copy of ``spec`` with some fields changed (for small parity cases)."""
    return dataclasses.replace(spec, **changes)


def zipf_sizes(N: int, G: int, s: float, min_size: int, rng: np.random.Generator) -> np.ndarray:
    """Cluster sizes by the Zipf rank law, summing exactly to N, in seeded cluster order."""
    if G * min_size > N:
        raise ValueError("N too small for the minimum cluster size")
    r = np.arange(1, G + 1, dtype=np.float64)
    w = r ** (-s)
    raw = N * w / w.sum()
    base = np.maximum(np.floor(raw).astype(np.int64), min_size)
    delta = N - int(base.sum())
    if delta > 0:
        frac = raw - np.floor(raw)
        order = np.lexsort((r, -frac))          # largest remainder first, then rank
        base[order[:delta]] += 1
    elif delta < 0:
        need = -delta
        i = 0
        while need > 0:                          # take the excess from the largest ranks
            take = min(need, int(base[i]) - min_size)
            base[i] -= take
            need -= take
            i += 1
    perm = rng.permutation(G)
    sizes = np.empty(G, dtype=np.int64)
    sizes[perm] = base                           # rank r goes to cluster perm[r]
    return sizes


def _seed(seed: int, name: str, role: str) -> int:
    return (seed * 1000003 + zlib.crc32(f"{name}/{role}".encode())) & 0x7FFFFFFFFFFF


def _gen(device, seed: int, name: str, role: str) -> torch.Generator:
    g = torch.Generator(device=device)
    g.manual_seed(_seed(seed, name, role))
    return g


def _unit(x: torch.Tensor) -> torch.Tensor:
    return x / x.norm(dim=1, keepdim=True)


def _store(x: torch.Tensor, storage: str) -> torch.Tensor:
    return x.to(torch.bfloat16) if storage == "bf16" else x.to(torch.float32)


def _rows(spec: Spec, n: int, gen, device, centres=None, centre_of=None) -> torch.Tensor:
    d = spec.d
    if spec.keys == "gauss":
        return _unit(torch.randn(n, d, generator=gen, device=device))
    if spec.keys == "before_after":
        h = d // 2
        a = _unit(torch.randn(n, h, generator=gen, device=device))
        b = _unit(torch.randn(n, h, generator=gen, device=device))
        return torch.cat([a, b], dim=1) * (0.5 ** 0.5)
    if spec.keys == "mixture":
        e = torch.randn(n, d, generator=gen, device=device)
        return _unit(centres[centre_of] + spec.sigma * e / (d ** 0.5))
    raise ValueError(spec.keys)


@dataclasses.dataclass
class Workload:
    spec: Spec
    queries: torch.Tensor       # [B][d]  storage dtype
    coarse_keys: torch.Tensor   # [G][d]  storage dtype
    cluster_of: torch.Tensor    # [N] int32, parent cluster of each record (record order)
    keys_in: torch.Tensor       # [N][d]  storage dtype, record order
    sizes: np.ndarray           # [G] int64 segment lengths


def make(spec, device="cpu", seed: int = 0, chunk_rows: int = 1 << 20) -> Workload:
    """Draw one workload on ``device`` (records in their stored, possibly shuffled order)."""
    if isinstance(spec, str):
        spec = SPECS[spec]
    device = torch.device(device)
    rng = np.random.default_rng(_seed(seed, spec.name, "host"))
    if spec.sizes == "fixed":
        sizes = np.asarray(spec.fixed_sizes, dtype=np.int64)
    elif spec.sizes == "uniform":
        sizes = np.full(spec.G, spec.N // spec.G, dtype=np.int64)
        sizes[: spec.N - int(sizes.sum())] += 1
    elif spec.sizes == "zipf":
        sizes = zipf_sizes(spec.N, spec.G, spec.zipf_s, spec.min_size, rng)
    else:
        raise ValueError(spec.sizes)
    assert sizes.size == spec.G and int(sizes.sum()) == spec.N

    cluster_sorted = np.repeat(np.arange(spec.G, dtype=np.int32), sizes)
    if spec.shuffled:
        cluster_of_np = cluster_sorted[rng.permutation(spec.N)]
    else:
        cluster_of_np = cluster_sorted
    cluster_of = torch.from_numpy(np.ascontiguousarray(cluster_of_np)).to(device)

    centres = None
    q_centre = None
    if spec.keys == "mixture":
        centres = _unit(torch.randn(spec.G, spec.d, generator=_gen(device, seed, spec.name, "centres"),
                                    device=device))
        coarse = centres
        q_centre = torch.from_numpy(rng.integers(0, spec.G, size=spec.B)).to(device)
    else:
        coarse = _rows(spec, spec.G, _gen(device, seed, spec.name, "coarse"), device)
    queries = _rows(spec, spec.B, _gen(device, seed, spec.name, "queries"), device,
                    centres=centres, centre_of=q_centre)

    dt = torch.bfloat16 if spec.storage == "bf16" else torch.float32
    keys_in = torch.empty(spec.N, spec.d, dtype=dt, device=device)
    gk = _gen(device, seed, spec.name, "keys")
    for a in range(0, spec.N, chunk_rows):
        b = min(spec.N, a + chunk_rows)
        cof = cluster_of[a:b].long() if centres is not None else None
        keys_in[a:b] = _store(_rows(spec, b - a, gk, device, centres=centres, centre_of=cof),
                              spec.storage)
    return Workload(spec=spec, queries=_store(queries, spec.storage).contiguous(),
                    coarse_keys=_store(coarse, spec.storage).contiguous(),
                    cluster_of=cluster_of, keys_in=keys_in, sizes=sizes)


def make_prefix(spec, coarse_keys: torch.Tensor, lmax: int, device="cpu", seed: int = 0,
                sigma: float = 0.5):
    """Edge keys and prefixes for prefix-aware coarse scoring (the edge
    memories E_G(g_src, g_dst) over the complete directed pair space, and each
    query's recent global directions).

    edge_keys [G][G][d] in the storage dtype: E[src][dst] = normalise(c_dst +
    sigma * e / sqrt(d)), e ~ N(0, I_d) drawn per (src, dst), so an edge key is
    its destination's node key perturbed per source. prefix [B][lmax] int32:
    each query's prefix length is uniform on 0..lmax (0: the first step) and
    its entries uniform over the G directions; rows are padded with -1."""
    if isinstance(spec, str):
        spec = SPECS[spec]
    device = torch.device(device)
    G, d = spec.G, spec.d
    ck = coarse_keys.to(device=device, dtype=torch.float32)
    gen = _gen(device, seed, spec.name, "edges")
    dt = torch.bfloat16 if spec.storage == "bf16" else torch.float32
    E = torch.empty(G, G, d, dtype=dt, device=device)
    for s0 in range(G):
        e = torch.randn(G, d, generator=gen, device=device)
        E[s0] = _store(_unit(ck + sigma * e / (d ** 0.5)), spec.storage)
    rng = np.random.default_rng(_seed(seed, spec.name, "prefix"))
    lengths = rng.integers(0, lmax + 1, spec.B)
    P = np.full((spec.B, lmax), -1, dtype=np.int32)
    for b in range(spec.B):
        P[b, :lengths[b]] = rng.integers(0, G, lengths[b])
    return E, torch.from_numpy(P).to(device)

