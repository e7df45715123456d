"""GPU parity: the HIP path through the C ABI against the CPU oracle, on seeded
workloads small enough for the oracle to finish in seconds, spanning several
tiles, chunks and ragged tails, plus the method's degenerate cases."""
import numpy as np
import pytest
import torch

import oracle
from gpu_cases import run_case, say, to_np
from paper_2605_29734_amd import synth

pytestmark = pytest.mark.gpu
S = synth.SPECS


@pytest.mark.parametrize("tau", [1.0, 0.07])
def test_paper_shaped_memory(tau):
    """Five global nodes with 4/3/3/3/3 children, one direction, the best child (k = 1)."""
    run_case(S["paper_htg"], tau=tau, determinism=True)


def test_tiny_f32():
    run_case(S["tiny_f32"], determinism=True)


@pytest.mark.parametrize("tiled", [False, True])
def test_zipf_bf16_full(tiled):
    run_case(S["zipf_bf16"], tiled=tiled)


@pytest.mark.parametrize("tiled", [False, True])
def test_mixture_bf16_reduced(tiled):
    run_case(synth.scaled(S["mixture_bf16"], B=128, G=64, N=65536), tiled=tiled)


@pytest.mark.parametrize("tiled", [False, True])
def test_zipf_large_bf16_reduced(tiled):
    run_case(synth.scaled(S["zipf_large_bf16"], B=256, G=256, N=262144), tiled=tiled)


@pytest.mark.parametrize("tiled", [False, True])
def test_before_after_reduced(tiled):
    run_case(synth.scaled(S["before_after_f32"], B=96, G=256, N=65536), tiled=tiled)


@pytest.mark.parametrize("tiled", [False, True])
@pytest.mark.parametrize("storage,B,G,N,top_k,min_size", [
    ("f32", 512, 512, 200000, 128, 20),   # Zipf segments (mean 390 rows, 1024-row chunks):
    ("bf16", 512, 512, 200000, 64, 20),   # long ones of several four-step row groups per chunk
    ("f32", 128, 64, 6000, 128, 1),       # short and ragged segments: groups under four steps
])
def test_split_stream_kernel(storage, B, G, N, top_k, min_size, tiled):
    """The two-blocks-per-CU stream kernel that stages half of d's query
    fragments at a time (d = 2048, short segments on average, one query tile
    per pass: at most about eight queries per selected cluster); with the
    tiled copy of the keys (segments start anywhere in a 16-row tile) its
    outputs must equal those of the row-major bank bit for bit."""
    run_case(synth.Spec("split", B=B, d=2048, G=G, N=N, top_c=4, top_k=top_k, tau=0.5,
                        storage=storage, compute="bf16", sizes="zipf", zipf_s=1.0,
                        min_size=min_size), gen_device="cuda", check_build=False, tiled=tiled)


@pytest.mark.parametrize("dtype", [torch.float32, torch.bfloat16])
@pytest.mark.parametrize("sizes,d", [([1000], 64), ([16], 32), ([37, 0, 5, 16, 0, 33], 96),
                                     ([0, 0], 32)])
def test_tiled_copy_layout(sizes, d, dtype):
    """htam_memory_tile against the layout written out in numpy: the header
    of padded segment starts, then element 32 s + 8 c + e of copy row
    16 t + i at block (t, s), piece (e // P) * 64 + c * 16 + i, offset e % P;
    segment g's record j at copy row toff[g] + j, padding rows zero (empty
    segments, segments that end inside a tile). Bit-exact."""
    from paper_2605_29734_amd import htam
    say(f"[case] tiled copy sizes={sizes} d={d} dtype={dtype}")
    dev = torch.device("cuda:0")
    G, N = len(sizes), sum(sizes)
    off = np.concatenate([[0], np.cumsum(sizes)]).astype(np.int64)
    g = torch.Generator().manual_seed(N + d + G)
    keys = torch.randn(max(N, 1), d, generator=g).to(dtype)[:N]
    bank = htam.Bank(coarse_keys=torch.zeros(G, d, dtype=dtype, device=dev),
                     fine_keys=keys.to(dev) if N else torch.zeros(1, d, dtype=dtype, device=dev),
                     seg_offsets=torch.from_numpy(off).to(dev), transition_id=None,
                     compute="bf16")
    bank.struct.n_transitions = N
    out = htam.htam_memory_tile(bank)
    torch.cuda.synchronize()
    raw = out.view(torch.uint8).cpu().numpy()
    head = ((G + 1) * 8 + 255) // 256 * 256
    toff = raw[:(G + 1) * 8].view(np.int64)
    pad = [(n + 15) // 16 * 16 for n in sizes]
    assert np.array_equal(toff, np.concatenate([[0], np.cumsum(pad)]).astype(np.int64))
    P = 16 // keys.element_size()
    T, S = int(toff[-1]) // 16, d // 32
    ref = np.zeros((T, S, 8 // P, 4, 16, P), dtype=np.float32)
    k = keys.float().numpy()
    for gi in range(G):
        for j in range(sizes[gi]):
            t, i = divmod(int(toff[gi]) + j, 16)
            for s_ in range(S):
                for c in range(4):
                    for e in range(8):
                        ref[t, s_, e // P, c, i, e % P] = k[off[gi] + j, 32 * s_ + 8 * c + e]
    if T == 0:
        return
    tiles = torch.from_numpy(raw[head:head + T * 16 * d * keys.element_size()].copy())
    got = tiles.view(dtype).float().numpy()
    np.testing.assert_array_equal(got, ref.reshape(-1))


@pytest.mark.parametrize("compute", ["bf16", "f32"])
def test_ragged_shapes_and_tail_dim(compute):
    """B, G not multiples of a tile; d not a multiple of the MFMA K step."""
    st = "bf16" if compute == "bf16" else "f32"
    run_case(synth.Spec("ragged", B=37, d=72, G=13, N=1000, top_c=3, top_k=7, tau=0.5, storage=st,
                        compute=compute, sizes="zipf", zipf_s=1.0, min_size=1), determinism=True)


def test_many_queries_per_cluster():
    """More queries select one cluster than one pass over a chunk holds."""
    run_case(synth.Spec("crowded", B=300, d=128, G=4, N=4000, top_c=2, top_k=16, tau=1.0,
                        storage="bf16", compute="bf16", sizes="uniform"))


def test_flat_retrieval_top_c_equals_G():
    run_case(synth.Spec("flat", B=24, d=64, G=6, N=3000, top_c=6, top_k=32, tau=0.2,
                        storage="bf16", compute="bf16", sizes="zipf", zipf_s=1.5, min_size=2))


def test_short_and_empty_segments():
    """k larger than most segments; empty clusters selected; one segment > half the bank."""
    sizes = tuple([1100] + [0] * 10 + [30] * 29)
    spec = synth.Spec("sparse", B=50, d=64, G=len(sizes), N=sum(sizes), top_c=4, top_k=100,
                      tau=1.0, storage="f32", compute="f32", sizes="fixed", fixed_sizes=sizes,
                      shuffled=True)
    run_case(spec)


@pytest.mark.parametrize("d", [256, 512])
def test_large_k(d):
    """k = 256 (the largest top-k buffers); d = 512 runs the LDS-staged kernel, d = 256 the generic one."""
    run_case(synth.Spec("bigk", B=20, d=d, G=8, N=20000, top_c=3, top_k=256, tau=1.0,
                        storage="bf16", compute="bf16", sizes="uniform"))


@pytest.mark.parametrize("storage", ["bf16", "f32"])
def test_many_queries_per_cluster_lds_kernel(storage):
    """More queries per cluster than one pass of the LDS-staged kernel holds (several passes)."""
    run_case(synth.Spec("crowded_lds", B=400, d=512, G=4, N=6000, top_c=2, top_k=32, tau=0.3,
                        storage=storage, compute="bf16", sizes="zipf", zipf_s=0.5, min_size=100),
             determinism=True)


@pytest.mark.parametrize("storage,compute,d", [("bf16", "bf16", 512), ("f32", "bf16", 512),
                                               ("f32", "f32", 96)])
def test_identity_transition_ids(storage, compute, d):
    """A bank without a transition id array reports bank rows as ids (LDS and generic kernels)."""
    run_case(synth.Spec("identity", B=96, d=d, G=24, N=12000, top_c=3, top_k=20, tau=0.5,
                        storage=storage, compute=compute, sizes="zipf", zipf_s=1.0, min_size=4),
             identity_ids=True)


def test_topk_merge_standalone():
    """htam_topk on unsorted lists with padding and exact ties, against the oracle's sort."""
    from paper_2605_29734_amd import htam
    say("[case] htam_topk standalone")
    rng = np.random.default_rng(0)
    rows, lists, kin, k, tau = 33, 5, 40, 24, 0.3
    sc = rng.standard_normal((rows, lists, kin)).astype(np.float32)
    sc[:, 1, :10] = sc[:, 0, :10]                      # exact score ties, distinct ids
    ids = rng.permutation(rows * lists * kin).reshape(rows, lists, kin).astype(np.int32) % 100000
    ids[:, 2, 5:] = -1                                 # padding
    ids[3] = -1                                        # an empty row
    sm = np.where(ids >= 0, sc, -np.inf).max(2).astype(np.float32)   # max over real entries
    ss = np.array([[np.exp((sc[r, l][ids[r, l] >= 0] - sm[r, l]) / tau).sum() if np.isfinite(sm[r, l])
                    else 0.0 for l in range(lists)] for r in range(rows)], np.float32)
    dev = torch.device("cuda:0")
    t = lambda a: torch.from_numpy(a).to(dev)           # noqa: E731
    out = htam.htam_topk(t(sc), t(ids), k, t(sm), t(ss), tau)
    torch.cuda.synchronize()
    oid, osc, ow, om, oz, oc = (to_np(x) for x in out)
    for r in range(rows):
        m = ids[r] >= 0
        ref = oracle.attend(sc[r][m].astype(np.float64), ids[r][m], tau, k)
        assert oc[r] == ref["count"]
        np.testing.assert_array_equal(oid[r], ref["id"])          # fp32 inputs: exact ranking
        np.testing.assert_array_equal(osc[r], ref["score"].astype(np.float32))
        if ref["count"]:
            np.testing.assert_allclose(ow[r], ref["weight"], rtol=1e-5, atol=1e-30)
            np.testing.assert_allclose(np.log(oz[r]), np.log(ref["Z"]), rtol=0, atol=1e-5)
            assert om[r] == np.float32(ref["m"])
        else:
            assert om[r] == -np.inf and oz[r] == 0 and np.all(ow[r] == 0)
    # dense rows with implicit ids (the coarse selection path)
    dense = rng.standard_normal((17, 1000)).astype(np.float32)
    dense[:, 500] = dense[:, 20]
    o2 = htam.htam_topk(t(dense), None, 50)
    torch.cuda.synchronize()
    for r in range(17):
        order = np.lexsort((np.arange(1000), -dense[r].astype(np.float64)))[:50]
        np.testing.assert_array_equal(to_np(o2[0])[r], order)


def test_attend_out_of_range_selection_is_empty():
    """Selected cluster ids outside [0, G) give empty slots; the other slots are unaffected."""
    from paper_2605_29734_amd import htam
    spec = synth.scaled(synth.SPECS["tiny_f32"], B=8)
    say("[case] attend with out-of-range selections")
    w = synth.make(spec, device="cpu", seed=3)
    dev = torch.device("cuda:0")
    bank = htam.build_bank(w.cluster_of.to(dev), w.keys_in.to(dev), w.coarse_keys.to(dev),
                           spec.compute)
    q = w.queries.to(dev)
    sel = torch.tensor([[0, 5, -1, 7]] * 4 + [[spec.G, 1, 2, 3]] * 4, dtype=torch.int32,
                       device=dev)
    good = torch.tensor([[0, 5, 6, 7]] * 4 + [[4, 1, 2, 3]] * 4, dtype=torch.int32, device=dev)
    out = htam.htam_attend_transitions(bank, q, sel, spec.tau, spec.top_k)
    ref = htam.htam_attend_transitions(bank, q, good, spec.tau, spec.top_k)
    torch.cuda.synchronize()
    out = [to_np(x) for x in out]
    ref = [to_np(x) for x in ref]
    bad = (to_np(sel) < 0) | (to_np(sel) >= spec.G)
    smax, ssum, cscore, cid = out
    assert np.all(smax[bad] == -np.inf) and np.all(ssum[bad] == 0)
    assert np.all(cscore[bad] == -np.inf) and np.all(cid[bad] == -1)
    for a, b in zip(out, ref):
        np.testing.assert_array_equal(a[~bad], b[~bad])


@pytest.mark.parametrize("B,G,d,c,storage", [
    (4096, 4096, 64, 256, "bf16"),     # 256 x 256-tile GEMM: one tile per CU, two K stages
    (4000, 4099, 160, 256, "bf16"),    # ragged tiles, G % 4 != 0, five K stages
    (300, 1000, 200, 256, "bf16"),     # 32 x 32-tile GEMM, d % 32 != 0, ragged B and G
    (300, 1000, 200, 5, "bf16"),       # the same with many radix-select cuts per row
    (70, 4099, 64, 100, "f32"),        # fp32 storage rounded to bf16
    (64, 20000, 128, 40, "bf16"),      # long rows for the row top-k
    (100, 300, 200, 50, "bf16"),       # 16 x 16-tile GEMM (few tiles), ragged, d % 32 != 0
    (50, 500, 96, 20, "f32"),          # the same with fp32 storage
    (2048, 8192, 64, 16, "bf16"),      # 256 x 256 tiles with tile maxima: selection reads the
    (2100, 9000, 96, 5, "bf16"),       # tiles that reach the bound (ragged rows and last tile)
    (2048, 8300, 64, 33, "f32"),
])
def test_coarse_every_row(B, G, d, c, storage):
    """Coarse retrieval over every row against the oracle's full score matrix
    over the same bf16-rounded operands, for each kernel path (chosen by the
    shape): the ids are distinct clusters, each score is the oracle's score of
    its id, and the sorted scores are the oracle's c largest, all within 1e-4
    (fp32 accumulation of at most 200 products of unit rows)."""
    from paper_2605_29734_amd import htam
    say(f"[case] coarse B={B} G={G} d={d} c={c} storage={storage}")
    rng = np.random.default_rng(B + G + d + c)
    unit = lambda n: (lambda x: x / np.linalg.norm(x, axis=1, keepdims=True))(   # noqa: E731
        rng.standard_normal((n, d)))
    dev = torch.device("cuda:0")
    dt = torch.bfloat16 if storage == "bf16" else torch.float32
    q = torch.from_numpy(unit(B).astype(np.float32)).to(dev).to(dt)
    ck = torch.from_numpy(unit(G).astype(np.float32)).to(dev).to(dt)
    bank = htam.Bank(coarse_keys=ck, fine_keys=torch.zeros(1, d, dtype=dt, device=dev),
                     seg_offsets=torch.zeros(G + 1, dtype=torch.int64, device=dev),
                     transition_id=None, compute="bf16")
    sel, ss = htam.htam_retrieve_coarse(bank, q, c)
    torch.cuda.synchronize()
    sel, ss = to_np(sel), to_np(ss)
    ref = oracle.scores(oracle.round_bf16(to_np(q)), oracle.round_bf16(to_np(ck)))
    assert sel.min() >= 0 and sel.max() < G
    assert all(len(np.unique(row)) == c for row in sel)
    rows = np.arange(B)[:, None]
    np.testing.assert_allclose(ss, ref[rows, sel], rtol=0, atol=1e-4)
    assert np.all(np.diff(ss, axis=1) <= 0)
    top = -np.sort(-ref, axis=1)[:, :c]
    np.testing.assert_allclose(ss, top, rtol=0, atol=1e-4)


@pytest.mark.parametrize("B,G,d,c", [(2048, 8300, 64, 33), (1024, 4096, 96, 16)])
def test_coarse_with_bf16_coarse_keys(B, G, d, c):
    """An fp32 bank with its coarse keys rounded to bf16 once
    (htam_coarse_keys_bf16): the 256 x 256-tile GEMM then rounds only the
    queries, and the selection and scores equal those of the bank without
    the copy bit for bit (the same rounding, done earlier)."""
    import dataclasses
    from paper_2605_29734_amd import htam
    say(f"[case] coarse with a bf16 coarse-key copy B={B} G={G} d={d} c={c}")
    rng = np.random.default_rng(B + G + d)
    dev = torch.device("cuda:0")
    q = torch.from_numpy(rng.standard_normal((B, d)).astype(np.float32)).to(dev)
    ck = torch.from_numpy(rng.standard_normal((G, d)).astype(np.float32)).to(dev)
    bank = htam.Bank(coarse_keys=ck, fine_keys=torch.zeros(1, d, device=dev),
                     seg_offsets=torch.zeros(G + 1, dtype=torch.int64, device=dev),
                     transition_id=None, compute="bf16")
    c16 = htam.htam_coarse_keys_bf16(bank)
    assert torch.equal(c16, ck.to(torch.bfloat16))          # round to nearest even
    a = [to_np(x) for x in htam.htam_retrieve_coarse(bank, q, c)]
    b = [to_np(x) for x in htam.htam_retrieve_coarse(
        dataclasses.replace(bank, coarse_keys_bf16=c16), q, c)]
    torch.cuda.synchronize()
    for x, y in zip(a, b):
        np.testing.assert_array_equal(x, y)


def test_level_one_merge_groups():
    """A bank large enough for two merge levels (level-one groups of chunk
    partials): one 1.5M-row cluster next to 15 of 33K rows, k = 128. The
    partial buffer (4 B c entries) sets the chunk at 65,536 rows, so the large
    cluster is 23 chunks whose partials (23 x 128 keys) exceed what one merge
    level reads. Every query against the oracle."""
    sizes = tuple([1_500_000] + [33_000] * 15)
    spec = synth.Spec("groups", B=128, d=64, G=len(sizes), N=sum(sizes), top_c=2, top_k=128,
                      tau=0.5, storage="bf16", compute="bf16", sizes="fixed", fixed_sizes=sizes)
    run_case(spec, gen_device="cuda", check_build=False)


def test_chunk_choice_many_blocks():
    """The multi-block routing (more than 8,192 (query, slot) pairs) choosing
    a chunk past its first candidates: one 200K-row cluster next to 15 of 10K
    rows, 4,200 queries, c = 2. At the shortest candidate chunk the partial
    results would exceed the buffer (4 B c of them; asserted here from the
    selection), so the chunk comes from the length-bit counts at a later
    candidate. Every row that selected the large cluster (up to 256) and 256
    seeded others are checked against the oracle."""
    sizes = tuple([200_000] + [10_000] * 15)
    spec = synth.Spec("chunks", B=4200, d=64, G=len(sizes), N=sum(sizes), top_c=2, top_k=128,
                      tau=0.5, storage="bf16", compute="bf16", sizes="fixed", fixed_sizes=sizes)
    n_cu = torch.cuda.get_device_properties(0).multi_processor_count
    chunk_min = 64
    while chunk_min * 2 <= spec.N // n_cu and chunk_min * 2 <= 4096:
        chunk_min *= 2

    def pick(gpu, seg):
        sel = gpu["sel"]
        parts = int(np.sum(-(-seg[sel] // chunk_min)))
        assert parts > 4 * sel.size, "the shortest chunk must not fit the partial buffer"
        big = np.flatnonzero((sel == 0).any(axis=1))
        assert big.size >= 16, "the large cluster must be selected"
        rest = np.setdiff1d(np.arange(spec.B), big)
        rng = np.random.default_rng(0)
        return np.sort(np.concatenate([big[:256], rng.choice(rest, 256, replace=False)]))

    run_case(spec, gen_device="cuda", check_build=False, rows=pick)


def test_level_one_merge_groups_selected():
    """The workload above selects its large cluster (so the two-level merge ran)."""
    from paper_2605_29734_amd import htam
    sizes = tuple([1_500_000] + [33_000] * 15)
    spec = synth.Spec("groups", B=128, d=64, G=len(sizes), N=sum(sizes), top_c=2, top_k=128,
                      tau=0.5, storage="bf16", compute="bf16", sizes="fixed", fixed_sizes=sizes)
    w = synth.make(spec, device="cuda", seed=0)
    bank = htam.Bank(coarse_keys=w.coarse_keys, fine_keys=torch.zeros(1, spec.d, dtype=torch.bfloat16,
                                                                       device="cuda"),
                     seg_offsets=torch.zeros(spec.G + 1, dtype=torch.int64, device="cuda"),
                     transition_id=None, compute="bf16")
    sel, _ = htam.htam_retrieve_coarse(bank, w.queries, spec.top_c)
    torch.cuda.synchronize()
    assert int((sel == 0).sum()) >= 4
