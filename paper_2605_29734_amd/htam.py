"""Python binding of libhtam.so (the C ABI of include/htam.h).

Argument marshalling only: every step of retrieval runs in the library's HIP
kernels. PyTorch supplies device memory (outputs and workspaces are torch
tensors on the queries' device) and the stream (the current torch stream).
If the library has not been built, importing this module raises ImportError:
there is no fallback path.
"""
from __future__ import annotations

import ctypes
import dataclasses
import os

import torch

_LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libhtam.so")

HTAM_F32 = 0
HTAM_BF16 = 1
HTAM_MAX_TOP_K = 256
HTAM_MAX_TOP_C = 256
HTAM_MAX_DIM = 8192
HTAM_NOALLOC_SCRATCH_MIB = 64
HTAM_MAX_PREFIX = 16

HTAM_KERNEL_COARSE = 0
HTAM_KERNEL_STREAM = 1

STATUS = {0: "HTAM_OK", -1: "HTAM_ERR_NULL", -2: "HTAM_ERR_SHAPE", -3: "HTAM_ERR_DTYPE",
          -4: "HTAM_ERR_VALUE", -5: "HTAM_ERR_WORKSPACE", -6: "HTAM_ERR_ALIGN",
          -7: "HTAM_ERR_DEVICE"}


class HtamError(RuntimeError):
    def __init__(self, where: str, status: int, message: str):
        super().__init__(f"{where}: {STATUS.get(status, status)}: {message}")
        self.status = status


class BankStruct(ctypes.Structure):
    """Mirror of struct htam_bank."""
    _fields_ = [("d", ctypes.c_int32), ("n_clusters", ctypes.c_int32),
                ("n_transitions", ctypes.c_int64), ("key_dtype", ctypes.c_int32),
                ("compute_dtype", ctypes.c_int32), ("coarse_keys", ctypes.c_void_p),
                ("fine_keys", ctypes.c_void_p), ("seg_offsets", ctypes.c_void_p),
                ("transition_id", ctypes.c_void_p), ("fine_keys_tiled", ctypes.c_void_p),
                ("coarse_keys_bf16", ctypes.c_void_p)]


def _load():
    if not os.path.exists(_LIB_PATH):
        raise ImportError(f"{_LIB_PATH} is missing: build it with "
                          "`python -m paper_2605_29734_amd.build_lib` (hipcc, gfx950)")
    lib = ctypes.CDLL(_LIB_PATH)
    P, i32, i64, f32, sz = (ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_float,
                            ctypes.c_size_t)
    u64 = ctypes.c_uint64
    BP = ctypes.POINTER(BankStruct)
    sig = {
        "htam_memory_build": ([i64, i32, i32, i32, P, P, P, P, P, P, sz, P], i32),
        "htam_memory_build_workspace_size": ([i64, i32], sz),
        "htam_memory_tile": ([BP, P, P], i32),
        "htam_memory_tile_bytes": ([BP], sz),
        "htam_coarse_keys_bf16": ([BP, P, P], i32),
        "htam_retrieve_coarse": ([BP, P, i32, i32, i32, P, P, P, sz, P], i32),
        "htam_retrieve_coarse_workspace_size": ([BP, i32, i32], sz),
        "htam_attend_transitions": ([BP, P, i32, i32, P, i32, f32, i32, P, P, P, P, P, sz, P], i32),
        "htam_attend_transitions_workspace_size": ([BP, i32, i32, i32], sz),
        "htam_feedback_update": ([i32, i32, i32, P, P, P, P, P, P, P, P], i32),
        "htam_transition_scores": ([i32, i32, i32, P, i32, P, f32, P, i32, P, P, P, P, P], i32),
        "htam_memory_merge": ([i32, i32, i32, P, P, P, i64, P, P, P, i64, P, P, P, P, sz, P], i32),
        "htam_memory_merge_workspace_size": ([], sz),
        "htam_retrieve_coarse_sampled": ([BP, P, i32, i32, i32, f32, f32, P, u64, u64, P, P, P, sz, P], i32),
        "htam_retrieve_coarse_sampled_workspace_size": ([BP, i32, i32], sz),
        "htam_retrieve_coarse_prefix": ([BP, P, P, i32, f32, P, i32, i32, i32, P, P, P, sz, P], i32),
        "htam_retrieve_coarse_prefix_workspace_size": ([BP, i32, i32, i32], sz),
        "htam_retrieve_flat": ([BP, P, i32, i32, f32, i32, P, P, P, P, P, P, P, sz, P], i32),
        "htam_retrieve_flat_workspace_size": ([BP, i32, i32], sz),
        "htam_attend_transitions_noalloc": ([BP, P, i32, i32, P, i32, f32, i32, P, P, P, P, P], i32),
        "htam_topk": ([i32, i32, i32, P, P, P, P, f32, i32, P, P, P, P, P, P, P], i32),
        "htam_topk_sorted": ([i32, i32, i32, P, P, P, P, f32, i32, P, P, P, P, P, P, P], i32),
        "htam_set_kernel_events": ([i32, P, P], i32),
        "htam_status_string": ([i32], ctypes.c_char_p),
        "htam_last_error": ([], ctypes.c_char_p),
    }
    for name, (args, res) in sig.items():
        fn = getattr(lib, name)
        fn.argtypes = args
        fn.restype = res
    return lib


lib = _load()


def _check(where: str, status: int):
    if status < 0:
        raise HtamError(where, status, lib.htam_last_error().decode())
    return status


def _ptr(t):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _stream(device) -> ctypes.c_void_p:
    return ctypes.c_void_p(torch.cuda.current_stream(device).cuda_stream)


def dtype_code(dt: torch.dtype) -> int:
    if dt == torch.float32:
        return HTAM_F32
    if dt == torch.bfloat16:
        return HTAM_BF16
    raise TypeError(f"unsupported dtype {dt}")


def _workspace(nbytes: int, device) -> torch.Tensor:
    # torch's caching allocator returns blocks aligned to at least 512 bytes
    return torch.empty(max(int(nbytes), 256), dtype=torch.uint8, device=device)


@dataclasses.dataclass
class Bank:
    """A built two-level memory bank (device tensors) and its descriptor."""
    coarse_keys: torch.Tensor       # [G][d]
    fine_keys: torch.Tensor         # [N][d], segment-contiguous
    seg_offsets: torch.Tensor       # [G+1] int64
    transition_id: torch.Tensor | None   # [N] int32 or None (= row index)
    compute: str = "bf16"           # "f32" | "bf16"
    fine_keys_tiled: torch.Tensor | None = None   # htam_memory_tile's copy, or None
    coarse_keys_bf16: torch.Tensor | None = None  # htam_coarse_keys_bf16's copy, or None

    def __post_init__(self):
        self._s = BankStruct(
            d=self.coarse_keys.shape[1], n_clusters=self.coarse_keys.shape[0],
            n_transitions=self.fine_keys.shape[0], key_dtype=dtype_code(self.fine_keys.dtype),
            compute_dtype=HTAM_BF16 if self.compute == "bf16" else HTAM_F32,
            coarse_keys=self.coarse_keys.data_ptr(), fine_keys=self.fine_keys.data_ptr(),
            seg_offsets=self.seg_offsets.data_ptr(),
            transition_id=None if self.transition_id is None else self.transition_id.data_ptr(),
            fine_keys_tiled=None if self.fine_keys_tiled is None else self.fine_keys_tiled.data_ptr(),
            coarse_keys_bf16=None if self.coarse_keys_bf16 is None else self.coarse_keys_bf16.data_ptr())

    @property
    def struct(self) -> BankStruct:
        return self._s

    @property
    def device(self):
        return self.fine_keys.device


# ---------------------------------------------------------------------------
# the four calls
# ---------------------------------------------------------------------------
def htam_memory_build(cluster_of: torch.Tensor, keys_in: torch.Tensor | None, n_clusters: int):
    """Group records by parent cluster. Returns (keys_out, seg_offsets, transition_id)."""
    dev = cluster_of.device
    n = cluster_of.numel()
    keys_out = None if keys_in is None else torch.empty_like(keys_in)
    off = torch.empty(n_clusters + 1, dtype=torch.int64, device=dev)
    tid = torch.empty(n, dtype=torch.int32, device=dev)
    ws = _workspace(lib.htam_memory_build_workspace_size(n, n_clusters), dev)
    d = 0 if keys_in is None else keys_in.shape[1]
    kd = HTAM_F32 if keys_in is None else dtype_code(keys_in.dtype)
    _check("htam_memory_build",
           lib.htam_memory_build(n, n_clusters, d, kd, _ptr(cluster_of), _ptr(keys_in),
                                 _ptr(keys_out), _ptr(off), _ptr(tid), _ptr(ws), ws.numel(),
                                 _stream(dev)))
    return keys_out, off, tid


def htam_retrieve_coarse(bank: Bank, q: torch.Tensor, top_c: int, out=None, ws=None):
    """Top-c clusters per query. Returns (sel_cluster int32 [B][c], sel_score fp32 [B][c])."""
    B = q.shape[0]
    dev = q.device
    if out is None:
        out = (torch.empty(B, top_c, dtype=torch.int32, device=dev),
               torch.empty(B, top_c, dtype=torch.float32, device=dev))
    if ws is None:
        ws = _workspace(lib.htam_retrieve_coarse_workspace_size(ctypes.byref(bank.struct), B,
                                                                top_c), dev)
    _check("htam_retrieve_coarse",
           lib.htam_retrieve_coarse(ctypes.byref(bank.struct), _ptr(q), dtype_code(q.dtype), B,
                                    top_c, _ptr(out[0]), _ptr(out[1]), _ptr(ws), ws.numel(),
                                    _stream(dev)))
    return out


def htam_attend_transitions(bank: Bank, q: torch.Tensor, sel: torch.Tensor, tau: float,
                            top_k: int, out=None, ws=None):
    """Per (query, slot): (slot_max, slot_sum, cand_score [B][c][k], cand_id [B][c][k])."""
    B, c = sel.shape
    dev = q.device
    if out is None:
        out = (torch.empty(B, c, dtype=torch.float32, device=dev),
               torch.empty(B, c, dtype=torch.float32, device=dev),
               torch.empty(B, c, top_k, dtype=torch.float32, device=dev),
               torch.empty(B, c, top_k, dtype=torch.int32, device=dev))
    if ws is None:
        ws = _workspace(lib.htam_attend_transitions_workspace_size(ctypes.byref(bank.struct), B,
                                                                   c, top_k), dev)
    _check("htam_attend_transitions",
           lib.htam_attend_transitions(ctypes.byref(bank.struct), _ptr(q), dtype_code(q.dtype), B,
                                       _ptr(sel), c, float(tau), top_k, _ptr(out[0]), _ptr(out[1]),
                                       _ptr(out[2]), _ptr(out[3]), _ptr(ws), ws.numel(),
                                       _stream(dev)))
    return out


def htam_retrieve_coarse_sampled(bank: Bank, q: torch.Tensor, top_c: int, eps: float, tau_g: float,
                                 noise: torch.Tensor | None = None, seed: int = 0, offset: int = 0,
                                 out=None, ws=None):
    """Draw top_c clusters per query from the policy mu_g without replacement.
    noise: [B][G] uint32 words as int32 tensor, or None (Philox from seed, offset).
    Returns (sel_cluster int32 [B][c], sel_score fp32 [B][c])."""
    B = q.shape[0]
    dev = q.device
    if out is None:
        out = (torch.empty(B, top_c, dtype=torch.int32, device=dev),
               torch.empty(B, top_c, dtype=torch.float32, device=dev))
    if ws is None:
        ws = _workspace(lib.htam_retrieve_coarse_sampled_workspace_size(
            ctypes.byref(bank.struct), B, top_c), dev)
    _check("htam_retrieve_coarse_sampled",
           lib.htam_retrieve_coarse_sampled(ctypes.byref(bank.struct), _ptr(q), dtype_code(q.dtype), B,
                                            top_c, float(eps), float(tau_g), _ptr(noise), int(seed),
                                            int(offset), _ptr(out[0]), _ptr(out[1]), _ptr(ws),
                                            ws.numel(), _stream(dev)))
    return out


def htam_retrieve_coarse_prefix(bank: Bank, edge_keys: torch.Tensor, prefix: torch.Tensor,
                                lam: float, q: torch.Tensor, top_c: int, out=None, ws=None):
    """Prefix-aware top-c clusters per query. edge_keys [G][G][d]; prefix [B][Lmax] int32
    (-1 padded). Returns (sel_cluster int32 [B][c], sel_score fp32 [B][c])."""
    B, lmax = prefix.shape
    dev = q.device
    if out is None:
        out = (torch.empty(B, top_c, dtype=torch.int32, device=dev),
               torch.empty(B, top_c, dtype=torch.float32, device=dev))
    if ws is None:
        ws = _workspace(lib.htam_retrieve_coarse_prefix_workspace_size(
            ctypes.byref(bank.struct), B, lmax, top_c), dev)
    _check("htam_retrieve_coarse_prefix",
           lib.htam_retrieve_coarse_prefix(ctypes.byref(bank.struct), _ptr(edge_keys), _ptr(prefix),
                                           lmax, float(lam), _ptr(q), dtype_code(q.dtype), B, top_c,
                                           _ptr(out[0]), _ptr(out[1]), _ptr(ws), ws.numel(),
                                           _stream(dev)))
    return out


def htam_retrieve_flat(bank: Bank, q: torch.Tensor, tau: float, top_k: int, out=None, ws=None):
    """Flat retrieval over every record. Returns (id, score, weight, row_max, row_sum, count)."""
    B = q.shape[0]
    dev = q.device
    if out is None:
        out = (torch.empty(B, top_k, dtype=torch.int32, device=dev),
               torch.empty(B, top_k, dtype=torch.float32, device=dev),
               torch.empty(B, top_k, dtype=torch.float32, device=dev),
               torch.empty(B, dtype=torch.float32, device=dev),
               torch.empty(B, dtype=torch.float32, device=dev),
               torch.empty(B, dtype=torch.int32, device=dev))
    if ws is None:
        ws = _workspace(lib.htam_retrieve_flat_workspace_size(ctypes.byref(bank.struct), B, top_k),
                        dev)
    _check("htam_retrieve_flat",
           lib.htam_retrieve_flat(ctypes.byref(bank.struct), _ptr(q), dtype_code(q.dtype), B,
                                  float(tau), top_k, _ptr(out[0]), _ptr(out[1]), _ptr(out[2]),
                                  _ptr(out[3]), _ptr(out[4]), _ptr(out[5]), _ptr(ws), ws.numel(),
                                  _stream(dev)))
    return out


def htam_attend_transitions_noalloc(bank: Bank, q: torch.Tensor, sel: torch.Tensor, tau: float,
                                    top_k: int, out=None):
    """htam_attend_transitions with the library's own scratch array as workspace."""
    B, c = sel.shape
    dev = q.device
    if out is None:
        out = (torch.empty(B, c, dtype=torch.float32, device=dev),
               torch.empty(B, c, dtype=torch.float32, device=dev),
               torch.empty(B, c, top_k, dtype=torch.float32, device=dev),
               torch.empty(B, c, top_k, dtype=torch.int32, device=dev))
    _check("htam_attend_transitions_noalloc",
           lib.htam_attend_transitions_noalloc(ctypes.byref(bank.struct), _ptr(q),
                                               dtype_code(q.dtype), B, _ptr(sel), c, float(tau),
                                               top_k, _ptr(out[0]), _ptr(out[1]), _ptr(out[2]),
                                               _ptr(out[3]), _stream(dev)))
    return out


def htam_topk(cand_score: torch.Tensor, cand_id: torch.Tensor | None, top_k: int,
              slot_max: torch.Tensor | None = None, slot_sum: torch.Tensor | None = None,
              tau: float = 1.0, out=None, sorted_lists: bool = False):
    """Merge [rows][lists][k_in] candidates. Returns (id, score, weight, row_max, row_sum, count);
    the softmax outputs are None without slot statistics. sorted_lists: every list is sorted
    as htam_attend_transitions returns them (htam_topk_sorted)."""
    if cand_score.dim() == 2:
        cand_score = cand_score.unsqueeze(1)
        cand_id = None if cand_id is None else cand_id.unsqueeze(1)
    rows, lists, k_in = cand_score.shape
    dev = cand_score.device
    stats = slot_max is not None
    if out is None:
        out = (torch.empty(rows, top_k, dtype=torch.int32, device=dev),
               torch.empty(rows, top_k, dtype=torch.float32, device=dev),
               torch.empty(rows, top_k, dtype=torch.float32, device=dev) if stats else None,
               torch.empty(rows, dtype=torch.float32, device=dev) if stats else None,
               torch.empty(rows, dtype=torch.float32, device=dev) if stats else None,
               torch.empty(rows, dtype=torch.int32, device=dev))
    fn = lib.htam_topk_sorted if sorted_lists else lib.htam_topk
    _check("htam_topk_sorted" if sorted_lists else "htam_topk",
           fn(rows, lists, k_in, _ptr(cand_score), _ptr(cand_id), _ptr(slot_max),
              _ptr(slot_sum), float(tau), top_k, _ptr(out[0]), _ptr(out[1]),
              _ptr(out[2]), _ptr(out[3]), _ptr(out[4]), _ptr(out[5]), _stream(dev)))
    return out


# ---------------------------------------------------------------------------
# a whole retrieval with preallocated buffers
# ---------------------------------------------------------------------------
class Retriever:
    """Preallocates outputs and workspaces for a fixed (bank, batch, top_c, top_k, tau),
    so that ``run`` only enqueues the three retrieval calls on the current stream."""

    def __init__(self, bank: Bank, n_queries: int, top_c: int, top_k: int, tau: float):
        self.bank, self.B, self.c, self.k, self.tau = bank, n_queries, top_c, top_k, tau
        dev = bank.device
        e = lambda *s, dt=torch.float32: torch.empty(*s, dtype=dt, device=dev)  # noqa: E731
        self.sel = (e(n_queries, top_c, dt=torch.int32), e(n_queries, top_c))
        self.slots = (e(n_queries, top_c), e(n_queries, top_c), e(n_queries, top_c, top_k),
                      e(n_queries, top_c, top_k, dt=torch.int32))
        self.rows = (e(n_queries, top_k, dt=torch.int32), e(n_queries, top_k),
                     e(n_queries, top_k), e(n_queries), e(n_queries),
                     e(n_queries, dt=torch.int32))
        bs = ctypes.byref(bank.struct)
        self.ws_coarse = _workspace(lib.htam_retrieve_coarse_workspace_size(bs, n_queries, top_c), dev)
        self.ws_attend = _workspace(
            lib.htam_attend_transitions_workspace_size(bs, n_queries, top_c, top_k), dev)

    def run(self, q: torch.Tensor) -> dict:
        htam_retrieve_coarse(self.bank, q, self.c, out=self.sel, ws=self.ws_coarse)
        htam_attend_transitions(self.bank, q, self.sel[0], self.tau, self.k, out=self.slots,
                                ws=self.ws_attend)
        htam_topk(self.slots[2], self.slots[3], self.k, self.slots[0], self.slots[1], self.tau,
                  out=self.rows, sorted_lists=True)
        return self.outputs()

    def outputs(self) -> dict:
        return dict(sel=self.sel[0], sel_score=self.sel[1], slot_max=self.slots[0],
                    slot_sum=self.slots[1], slot_score=self.slots[2], slot_id=self.slots[3],
                    id=self.rows[0], score=self.rows[1], weight=self.rows[2], m=self.rows[3],
                    Z=self.rows[4], count=self.rows[5])


def htam_memory_merge(main: Bank, delta: Bank) -> Bank:
    """Compact a delta bank into the main bank (both with transition ids)."""
    dev = main.device
    G = main.coarse_keys.shape[0]
    na, nb = main.fine_keys.shape[0], delta.fine_keys.shape[0]
    keys = torch.empty(na + nb, main.fine_keys.shape[1], dtype=main.fine_keys.dtype, device=dev)
    off = torch.empty(G + 1, dtype=torch.int64, device=dev)
    ids = torch.empty(na + nb, dtype=torch.int32, device=dev)
    ws = _workspace(lib.htam_memory_merge_workspace_size(), dev)
    _check("htam_memory_merge",
           lib.htam_memory_merge(G, main.fine_keys.shape[1], dtype_code(main.fine_keys.dtype),
                                 _ptr(main.fine_keys), _ptr(main.seg_offsets),
                                 _ptr(main.transition_id), na, _ptr(delta.fine_keys),
                                 _ptr(delta.seg_offsets), _ptr(delta.transition_id), nb,
                                 _ptr(keys), _ptr(off), _ptr(ids), _ptr(ws), ws.numel(),
                                 _stream(dev)))
    return Bank(coarse_keys=main.coarse_keys, fine_keys=keys, seg_offsets=off, transition_id=ids,
                compute=main.compute)


HTAM_FEEDBACK_FEATURES = 11
HTAM_STATS_WORDS = 12


def empty_stats(G: int, n_buckets: int, device):
    """Zeroed (node, edge, edge_bucket) statistics of an empty memory."""
    W = HTAM_STATS_WORDS
    z = lambda *s: torch.zeros(*s, W, dtype=torch.int64, device=device)  # noqa: E731
    return z(G), z(G, G), z(G, G, n_buckets)


def htam_feedback_update(stats, src, dst, bucket, features):
    """Add step outcomes to (node, edge, edge_bucket) statistics in place."""
    node, edge, eb = stats
    G, NB = node.shape[0], eb.shape[2]
    _check("htam_feedback_update",
           lib.htam_feedback_update(G, NB, dst.numel(), _ptr(src), _ptr(dst), _ptr(bucket),
                                    _ptr(features), _ptr(node), _ptr(edge), _ptr(eb),
                                    _stream(node.device)))
    return stats


def htam_transition_scores(stats, prefix, bucket, lam: float, w, min_count: int, out=None):
    """Rule-based direction scores [B][G] over the feedback statistics."""
    node, edge, eb = stats
    G, NB = node.shape[0], eb.shape[2]
    B, lmax = prefix.shape
    if out is None:
        out = torch.empty(B, G, dtype=torch.float32, device=node.device)
    _check("htam_transition_scores",
           lib.htam_transition_scores(G, NB, B, _ptr(prefix), lmax, _ptr(bucket), float(lam),
                                      _ptr(w), int(min_count), _ptr(node), _ptr(edge), _ptr(eb),
                                      _ptr(out), _stream(node.device)))
    return out


def retrieve_two_banks(main: Bank, delta: Bank, q: torch.Tensor, top_c: int, top_k: int,
                       tau: float) -> dict:
    """Retrieval over a main bank and a delta bank of recent records (same
    clusters and coarse keys): one coarse selection, the fine stage on each
    bank, then each slot's two lists merged and every row's 2 * top_c lists
    merged by htam_topk -- the result over the union of the two banks."""
    B = q.shape[0]
    sel, ss = htam_retrieve_coarse(main, q, top_c)
    a = htam_attend_transitions(main, q, sel, tau, top_k)
    b = htam_attend_transitions(delta, q, sel, tau, top_k)
    # per slot: the two lists of (query, slot) merged
    sc = torch.stack([a[2], b[2]], dim=2).reshape(B * top_c, 2, top_k).contiguous()
    si = torch.stack([a[3], b[3]], dim=2).reshape(B * top_c, 2, top_k).contiguous()
    sm = torch.stack([a[0], b[0]], dim=2).reshape(B * top_c, 2).contiguous()
    sz = torch.stack([a[1], b[1]], dim=2).reshape(B * top_c, 2).contiguous()
    slot = htam_topk(sc, si, top_k, sm, sz, tau)
    row = htam_topk(slot[1].reshape(B, top_c, top_k), slot[0].reshape(B, top_c, top_k), top_k,
                    slot[3].reshape(B, top_c), slot[4].reshape(B, top_c), tau)
    return dict(sel=sel, sel_score=ss, slot_id=slot[0].reshape(B, top_c, top_k),
                slot_score=slot[1].reshape(B, top_c, top_k), slot_max=slot[3].reshape(B, top_c),
                slot_sum=slot[4].reshape(B, top_c), id=row[0], score=row[1], weight=row[2],
                m=row[3], Z=row[4], count=row[5])


def htam_memory_tile(bank: Bank) -> torch.Tensor:
    """The tiled copy of bank.fine_keys (htam_memory_tile), same dtype, flat."""
    nbytes = lib.htam_memory_tile_bytes(ctypes.byref(bank.struct))
    if nbytes == 0:
        raise HtamError("htam_memory_tile", -2,
                        f"no tiled copy for d = {bank.fine_keys.shape[1]} (needs d % 32 == 0)")
    dev = bank.fine_keys.device
    out = torch.empty(nbytes // bank.fine_keys.element_size(), dtype=bank.fine_keys.dtype, device=dev)
    _check("htam_memory_tile", lib.htam_memory_tile(ctypes.byref(bank.struct), _ptr(out), _stream(dev)))
    return out


def with_tiled_keys(bank: Bank) -> Bank:
    """The same bank with the tiled copy of its fine keys attached."""
    return dataclasses.replace(bank, fine_keys_tiled=htam_memory_tile(bank))


def htam_coarse_keys_bf16(bank: Bank) -> torch.Tensor:
    """The bank's fp32 coarse keys rounded to bf16 (htam_coarse_keys_bf16)."""
    out = torch.empty(bank.coarse_keys.shape, dtype=torch.bfloat16, device=bank.coarse_keys.device)
    _check("htam_coarse_keys_bf16", lib.htam_coarse_keys_bf16(ctypes.byref(bank.struct), _ptr(out),
                                                              _stream(out.device)))
    return out


def prepared(bank: Bank) -> Bank:
    """The bank with the copies the retrieval calls read when present: the
    tiled fine keys (d % 32 == 0) and, for fp32 keys, the bf16 coarse keys."""
    if bank.fine_keys.shape[1] % 32 == 0 and bank.fine_keys_tiled is None:
        bank = with_tiled_keys(bank)
    if bank.fine_keys.dtype == torch.float32 and bank.coarse_keys_bf16 is None:
        bank = dataclasses.replace(bank, coarse_keys_bf16=htam_coarse_keys_bf16(bank))
    return bank


def build_bank(cluster_of: torch.Tensor, keys_in: torch.Tensor, coarse_keys: torch.Tensor,
               compute: str, tiled: bool = False) -> Bank:
    """Run htam_memory_build on records in arrival order and wrap the result as a
    Bank (with the tiled copy of the keys when tiled is set)."""
    keys_out, off, tid = htam_memory_build(cluster_of, keys_in, coarse_keys.shape[0])
    bank = Bank(coarse_keys=coarse_keys, fine_keys=keys_out, seg_offsets=off, transition_id=tid,
                compute=compute)
    return with_tiled_keys(bank) if tiled else bank


def retrieve(bank: Bank, q: torch.Tensor, top_c: int, top_k: int, tau: float) -> dict:
    """One hierarchical retrieval: coarse top-c, segment attention, top-k."""
    return Retriever(bank, q.shape[0], top_c, top_k, tau).run(q)
