"""The C ABI library: it loads, exports every declared entry point, and rejects
bad arguments on the host before touching a GPU (no compute call is made here)."""
import ctypes
import math
import os
import re

import pytest

from paper_2605_29734_amd import htam

HEADER = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))), "include",
                      "htam.h")
FAKE = 1 << 20          # a 16- and 256-byte aligned non-null address that is never dereferenced


def declared():
    text = open(HEADER).read()
    return sorted(set(re.findall(r"\b(htam_[a-z_]+)\s*\(", text)))


def test_every_declared_symbol_is_exported():
    names = declared()
    assert "htam_memory_build" in names and "htam_topk" in names and len(names) >= 9
    lib = ctypes.CDLL(htam._LIB_PATH)
    for n in names:
        assert hasattr(lib, n), n


def test_status_strings():
    for code, name in htam.STATUS.items():
        assert htam.lib.htam_status_string(code).decode() == name


def _bank(d=64, G=8, N=100, kd=htam.HTAM_BF16, cd=htam.HTAM_BF16, ptr=FAKE):
    return htam.BankStruct(d=d, n_clusters=G, n_transitions=N, key_dtype=kd, compute_dtype=cd,
                           coarse_keys=ptr, fine_keys=ptr, seg_offsets=ptr, transition_id=None)


def _coarse(bank, q=FAKE, qd=htam.HTAM_BF16, B=4, c=2, ws=FAKE, wsb=1 << 40):
    return htam.lib.htam_retrieve_coarse(ctypes.byref(bank) if bank is not None else None, q, qd,
                                         B, c, FAKE, FAKE, ws, wsb, None)


def _attend(bank, B=4, c=2, tau=1.0, k=8, ws=FAKE, wsb=1 << 40, qd=htam.HTAM_BF16):
    return htam.lib.htam_attend_transitions(ctypes.byref(bank), FAKE, qd, B, FAKE, c, tau, k,
                                            FAKE, FAKE, FAKE, FAKE, ws, wsb, None)


@pytest.mark.parametrize("bank,status", [
    (None, -1),
    (_bank(d=12), -2), (_bank(d=4), -2), (_bank(d=16384), -2), (_bank(G=0), -2),
    (_bank(N=-1), -2), (_bank(N=1 << 31), -2),
    (_bank(kd=htam.HTAM_BF16, cd=htam.HTAM_F32), -3), (_bank(kd=7), -3),
    (_bank(ptr=None), -1), (_bank(ptr=FAKE + 8), -6),
])
def test_coarse_rejects_bad_bank(bank, status):
    assert _coarse(bank) == status
    assert htam.lib.htam_last_error()


def test_coarse_rejects_bad_arguments():
    b = _bank()
    assert _coarse(b, qd=htam.HTAM_F32) == -3          # q dtype differs from the keys
    assert _coarse(b, q=None) == -1
    assert _coarse(b, q=FAKE + 4) == -6
    assert _coarse(b, B=-1) == -2
    assert _coarse(b, c=0) == -2
    assert _coarse(b, c=9) == -2                       # top_c > G
    assert _coarse(b, ws=None) == -5
    assert _coarse(b, wsb=16) == -5
    assert _coarse(b, ws=FAKE + 64) == -6
    assert _coarse(b, B=0) == 0                        # empty batch: nothing to do


def test_attend_rejects_bad_arguments():
    b = _bank()
    assert _attend(b, tau=0.0) == -4
    assert _attend(b, tau=-1.0) == -4
    assert _attend(b, tau=math.nan) == -4
    assert _attend(b, tau=math.inf) == -4
    assert _attend(b, k=0) == -2
    assert _attend(b, k=htam.HTAM_MAX_TOP_K + 1) == -2
    assert _attend(b, c=0) == -2
    assert _attend(b, wsb=100) == -5
    assert _attend(b, qd=htam.HTAM_F32) == -3
    assert _attend(b, B=0) == 0


@pytest.mark.parametrize("name", ["htam_topk", "htam_topk_sorted"])
def test_topk_rejects_bad_arguments(name):
    t = getattr(htam.lib, name)
    assert t(4, 2, 8, FAKE, FAKE, None, None, 1.0, 0, FAKE, FAKE, None, None, None, None, None) == -2
    assert t(4, 0, 8, FAKE, FAKE, None, None, 1.0, 4, FAKE, FAKE, None, None, None, None, None) == -2
    assert t(4, 2, 8, FAKE, FAKE, FAKE, None, 1.0, 4, FAKE, FAKE, None, None, None, None, None) == -1
    assert t(4, 2, 8, FAKE, FAKE, None, None, 1.0, 4, FAKE, FAKE, FAKE, None, None, None, None) == -4
    assert t(4, 2, 8, FAKE, FAKE, FAKE, FAKE, 0.0, 4, FAKE, FAKE, FAKE, None, None, None, None) == -4
    assert t(4, 2, 8, None, FAKE, None, None, 1.0, 4, FAKE, FAKE, None, None, None, None, None) == -1
    assert t(0, 2, 8, None, None, None, None, 1.0, 4, None, None, None, None, None, None, None) == 0


def test_build_rejects_bad_arguments():
    mb = htam.lib.htam_memory_build
    assert mb(-1, 4, 64, 1, FAKE, None, None, FAKE, FAKE, FAKE, 1 << 40, None) == -2
    assert mb(10, 0, 64, 1, FAKE, None, None, FAKE, FAKE, FAKE, 1 << 40, None) == -2
    assert mb(10, 4, 64, 1, None, None, None, FAKE, FAKE, FAKE, 1 << 40, None) == -1
    assert mb(10, 4, 64, 1, FAKE, FAKE, None, FAKE, FAKE, FAKE, 1 << 40, None) == -1
    assert mb(10, 4, 60, 1, FAKE, FAKE, FAKE * 2, FAKE, FAKE, FAKE, 1 << 40, None) == -2
    assert mb(10, 4, 64, 1, FAKE, FAKE, FAKE + 64, FAKE, FAKE, FAKE, 1 << 40, None) == -4   # overlap
    assert mb(10, 4, 64, 1, FAKE, FAKE, FAKE * 4, FAKE, FAKE, FAKE, 8, None) == -5


def test_tiled_copy_rejects_bad_arguments():
    """htam_memory_tile and a bank carrying a tiled copy: validated on the host
    (the tiled copy needs d % 32 == 0 and 16-byte alignment)."""
    tile = htam.lib.htam_memory_tile
    b = _bank(d=64, N=100, kd=htam.HTAM_F32, cd=htam.HTAM_BF16)
    # header of G + 1 = 9 int64 (256 bytes), then at most N / 16 + G = 7 + 8 tiles of 16 rows
    assert htam.lib.htam_memory_tile_bytes(ctypes.byref(b)) == 256 + 15 * 16 * 64 * 4
    assert htam.lib.htam_memory_tile_bytes(ctypes.byref(_bank(d=40))) == 0
    assert tile(None, FAKE, None) == -1
    assert tile(ctypes.byref(_bank(d=40)), FAKE, None) == -2
    assert tile(ctypes.byref(b), None, None) == -1
    assert tile(ctypes.byref(b), FAKE + 8, None) == -6
    assert tile(ctypes.byref(b), FAKE + 64, None) == -4            # overlaps fine_keys
    bad = _bank(d=40)
    bad.fine_keys_tiled = FAKE * 2
    assert _coarse(bad) == -2 and _attend(bad) == -2
    mis = _bank(d=64)
    mis.fine_keys_tiled = FAKE * 2 + 8
    assert _attend(mis) == -6
    ck = _bank(d=64, kd=htam.HTAM_F32, cd=htam.HTAM_BF16)
    ck.coarse_keys_bf16 = FAKE * 2 + 8
    assert _coarse(ck, qd=htam.HTAM_F32) == -6
    c16 = htam.lib.htam_coarse_keys_bf16
    assert c16(None, FAKE, None) == -1
    assert c16(ctypes.byref(_bank(d=64)), FAKE * 2, None) == -3        # bf16 keys: nothing to round
    assert c16(ctypes.byref(ck), None, None) == -1
    assert c16(ctypes.byref(ck), FAKE * 2 + 8, None) == -6
    assert c16(ctypes.byref(ck), FAKE + 16, None) == -4                # overlaps coarse_keys


def test_workspace_sizes():
    b = _bank(d=1024, G=4096, N=8388608)
    assert htam.lib.htam_memory_build_workspace_size(8388608, 4096) > 2048 * 4096 * 4
    assert htam.lib.htam_retrieve_coarse_workspace_size(ctypes.byref(b), 4096, 32) > 0
    a = htam.lib.htam_attend_transitions_workspace_size(ctypes.byref(b), 4096, 32, 64)
    assert a > 4 * 4096 * 32 * 64 * 8                  # partial top-k lists dominate
    assert htam.lib.htam_attend_transitions_workspace_size(ctypes.byref(b), 4096, 0, 64) == 0
    assert htam.lib.htam_memory_build_workspace_size(-1, 4) == 0


def test_flat_rejects_bad_arguments():
    f = htam.lib.htam_retrieve_flat
    b = _bank()
    args = lambda **kw: dict(dict(B=4, tau=1.0, k=8, ws=FAKE, wsb=1 << 40, qd=htam.HTAM_BF16), **kw)  # noqa: E731

    def call(**kw):
        a = args(**kw)
        return f(ctypes.byref(b), FAKE, a["qd"], a["B"], a["tau"], a["k"], FAKE, FAKE, None, None,
                 None, None, a["ws"], a["wsb"], None)
    assert call(tau=0.0) == -4
    assert call(k=0) == -2
    assert call(k=htam.HTAM_MAX_TOP_K + 1) == -2
    assert call(qd=htam.HTAM_F32) == -3
    assert call(wsb=64) == -5
    assert call(B=0) == 0
    assert htam.lib.htam_retrieve_flat_workspace_size(ctypes.byref(b), 4, 8) > 0


def test_prefix_rejects_bad_arguments():
    f = htam.lib.htam_retrieve_coarse_prefix
    b = _bank()

    def call(edges=FAKE, prefix=FAKE, lmax=4, lam=0.5, B=4, c=2, wsb=1 << 40):
        return f(ctypes.byref(b), edges, prefix, lmax, lam, FAKE, htam.HTAM_BF16, B, c, FAKE, FAKE,
                 FAKE, wsb, None)
    assert call(edges=None) == -1
    assert call(edges=FAKE + 8) == -6
    assert call(lmax=0) == -2
    assert call(lmax=htam.HTAM_MAX_PREFIX + 1) == -2
    assert call(lam=-1.0) == -4
    assert call(lam=math.inf) == -4
    assert call(c=9) == -2
    assert call(prefix=None) == -1
    assert call(wsb=64) == -5
    assert call(B=0) == 0
    assert htam.lib.htam_retrieve_coarse_prefix_workspace_size(ctypes.byref(b), 4, 4, 2) > 0


def test_sampled_rejects_bad_arguments():
    f = htam.lib.htam_retrieve_coarse_sampled
    b = _bank()

    def call(eps=0.1, tau=1.0, B=4, c=2, wsb=1 << 40, sel=FAKE):
        return f(ctypes.byref(b), FAKE, htam.HTAM_BF16, B, c, eps, tau, None, 1, 0, sel, FAKE,
                 FAKE, wsb, None)
    assert call(eps=-0.1) == -4
    assert call(eps=1.5) == -4
    assert call(eps=math.nan) == -4
    assert call(tau=0.0) == -4
    assert call(c=0) == -2
    assert call(sel=None) == -1
    assert call(wsb=64) == -5
    assert call(B=0) == 0
    assert htam.lib.htam_retrieve_coarse_sampled_workspace_size(ctypes.byref(b), 4, 2) > 0



def test_merge_rejects_bad_arguments():
    f = htam.lib.htam_memory_merge

    def call(G=4, d=64, kd=htam.HTAM_BF16, na=10, nb=5, ka=FAKE, kout=FAKE * 4, ida=FAKE, wsb=256):
        return f(G, d, kd, ka, FAKE, ida, na, FAKE * 2, FAKE, FAKE, nb, kout, FAKE, FAKE, FAKE,
                 wsb, None)
    assert call(G=0) == -2
    assert call(d=12) == -2
    assert call(kd=5) == -3
    assert call(na=-1) == -2
    assert call(ida=None) == -1
    assert call(ka=FAKE + 8) == -6
    assert call(kout=FAKE) == -4                         # output overlaps an input
    assert call(wsb=4) == -5


def test_feedback_and_transition_scores_reject_bad_arguments():
    f = htam.lib.htam_feedback_update
    assert f(0, 2, 5, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, None) == -2
    assert f(4, 2, 5, FAKE, FAKE, FAKE, FAKE, None, FAKE, FAKE, None) == -1
    assert f(4, 2, 5, None, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, None) == -1
    assert f(4, 2, 0, None, None, None, None, FAKE, FAKE, FAKE, None) == 0
    s = htam.lib.htam_transition_scores
    assert s(4, 2, 3, FAKE, 0, FAKE, 0.5, FAKE, 1, FAKE, FAKE, FAKE, FAKE, None) == -2
    assert s(4, 2, 3, FAKE, 4, FAKE, -0.5, FAKE, 1, FAKE, FAKE, FAKE, FAKE, None) == -4
    assert s(4, 2, 3, FAKE, 4, FAKE, 0.5, FAKE, -1, FAKE, FAKE, FAKE, FAKE, None) == -4
    assert s(4, 2, 3, FAKE, 4, FAKE, 0.5, None, 1, FAKE, FAKE, FAKE, FAKE, None) == -1
