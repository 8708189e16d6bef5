"""C-ABI contract of libvecattn on the host: the library loads, exports every
entry point include/vecattn.h declares, and rejects bad arguments with the
documented status before any launch (so no GPU is touched here: every call
below fails validation).
"""
import ctypes
import os
import re

import pytest

import paper_2603_29494_amd as va
from paper_2603_29494_amd import _lib

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "vecattn.h")

OK, INVALID, UNSUPPORTED, CAPACITY = 0, 1, 2, 3
FAKE = 0x100000   # 16-byte aligned address that validation rejects before any use


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(vecattn_[a-z_0-9]+)\s*\(", text)))


def test_library_exports_every_declared_entry_point():
    lib = _lib.load()
    names = declared_functions()
    assert {"vecattn_select", "vecattn_sparse_attn", "vecattn_pool"} <= set(names)
    for n in names:
        assert hasattr(lib, n), n
    assert lib.vecattn_version() >= 100


def test_status_strings():
    for s, text in ((0, "ok"), (1, "invalid argument"), (2, "unsupported"), (3, "capacity"),
                    (4, "device error")):
        assert text in _lib.status_string(s)


def test_max_count_matches_workloads():
    assert va.max_count(1024, 64, False, "topk", 0.125) == 128
    assert va.max_count(32768, 64, True, "topk", 0.10) == 3277
    assert va.max_count(75600, 64, False, "topk", 0.15) == 11340
    assert va.max_count(131072, 64, True, "topp", 0.95) == 131072
    assert va.max_count(118800, 128, False, "topp", 0.9) == 118800
    assert va.max_count(100, 64, True, "topp", 0.5) == 100        # last block ragged
    with pytest.raises(va.VecattnError):
        va.max_count(100, 64, False, "topk", 1.5)
    with pytest.raises(va.VecattnError):
        va.max_count(100, 0, False, "topk", 0.5)


def desc(B, H, N, D, sN=None):
    sN = D if sN is None else sN
    return _lib.TDesc(B, H, N, D, H * N * sN, N * sN, sN)


def attn(q=FAKE, qd=None, k=FAKE, kd=None, v=FAKE, vd=None, idx=FAKE, cap=16, cnt=FAKE, block=64,
         causal=0, scale=0.0, o=FAKE, od=None):
    lib = _lib.load()
    qd = qd or desc(1, 4, 128, 128)
    kd = kd or desc(1, 2, 128, 128)
    vd = vd or desc(1, 2, 128, 128)
    od = od or desc(1, 4, 128, 128)
    return lib.vecattn_sparse_attn(q, ctypes.byref(qd), k, ctypes.byref(kd), v, ctypes.byref(vd),
                                   idx, cap, cnt, block, causal, scale, o, ctypes.byref(od), None,
                                   None)


def test_sparse_attn_rejects_bad_arguments():
    assert attn(q=None) == INVALID
    assert attn(idx=None) == INVALID
    assert attn(cnt=None) == INVALID
    assert attn(block=0) == INVALID
    assert attn(cap=0) == INVALID
    assert attn(scale=-1.0) == INVALID
    assert attn(scale=float("nan")) == INVALID
    assert attn(q=FAKE + 2) == INVALID                                   # misaligned
    assert attn(kd=desc(1, 3, 128, 128), vd=desc(1, 3, 128, 128)) == INVALID   # 4 % 3
    assert attn(kd=desc(1, 2, 127, 128)) == INVALID                     # N mismatch
    assert attn(vd=desc(1, 1, 128, 128)) == INVALID                     # v != k
    assert attn(od=desc(1, 4, 128, 64)) == INVALID
    assert attn(qd=desc(1, 4, 128, 128, sN=132)) == INVALID              # row not 16-B aligned
    d96 = desc(1, 4, 128, 96)
    assert attn(qd=d96, kd=desc(1, 2, 128, 96), vd=desc(1, 2, 128, 96), od=d96) == UNSUPPORTED


def select(q=FAKE, qd=None, k=FAKE, kd=None, block=64, causal=0, mode=0, param=0.25, idx=FAKE,
           cap=64, cnt=FAKE, ws=FAKE, ws_bytes=1 << 40):
    lib = _lib.load()
    qd = qd or desc(1, 4, 256, 128)
    kd = kd or desc(1, 2, 256, 128)
    return lib.vecattn_select(q, ctypes.byref(qd), k, ctypes.byref(kd), block, causal, mode, param,
                              idx, cap, cnt, None, ws, ws_bytes, None)


def test_select_rejects_bad_arguments():
    assert select(q=None) == INVALID
    assert select(k=None) == INVALID
    assert select(idx=None) == INVALID
    assert select(cnt=None) == INVALID
    assert select(block=0) == INVALID
    assert select(param=0.0) == INVALID
    assert select(param=1.01) == INVALID
    assert select(mode=1, param=-0.1) == INVALID
    assert select(mode=7) == INVALID
    assert select(kd=desc(1, 3, 256, 128)) == INVALID
    assert select(kd=desc(1, 2, 255, 128)) == INVALID
    assert select(mode=2, param=-0.5) == INVALID           # minS: alpha >= 0
    assert select(mode=2, param=float('nan')) == INVALID
    assert select(mode=3, param=-0.5) == INVALID           # cross-tile minS: alpha >= 0
    assert select(mode=3, param=float('nan')) == INVALID
    assert select(cap=63) == CAPACITY                      # topK 25% of 256 keys = 64
    assert select(ws=None) == CAPACITY
    assert select(ws_bytes=16) == CAPACITY
    d64 = desc(1, 4, 256, 96)
    assert select(qd=d64, kd=desc(1, 2, 256, 96)) == UNSUPPORTED


def select_tiled(q=FAKE, qd=None, k=FAKE, kd=None, block=64, causal=0, alpha=0.5, tile=16,
                 group_tiles=16, idx=FAKE, cap=256, cnt=FAKE, ws=FAKE, ws_bytes=1 << 40):
    lib = _lib.load()
    qd = qd or desc(1, 4, 256, 128)
    kd = kd or desc(1, 2, 256, 128)
    return lib.vecattn_select_mins_tiled(q, ctypes.byref(qd), k, ctypes.byref(kd), block, causal,
                                         alpha, tile, group_tiles, idx, cap, cnt, None, ws,
                                         ws_bytes, None)


def test_select_mins_tiled_rejects_bad_arguments():
    assert select_tiled(q=None) == INVALID
    assert select_tiled(idx=None) == INVALID
    assert select_tiled(alpha=-1.0) == INVALID
    assert select_tiled(alpha=float("nan")) == INVALID
    for tile in (0, 8, 24, 64):
        assert select_tiled(tile=tile) == INVALID
    for gt in (0, -4, 3, 12):
        assert select_tiled(group_tiles=gt) == INVALID
    assert select_tiled(group_tiles=1 << 27) == INVALID     # 2^30 keys per group at most
    assert select_tiled(block=0) == INVALID
    assert select_tiled(cap=0) == INVALID
    assert select_tiled(ws=None) == CAPACITY                 # otherwise valid
    d96 = desc(1, 4, 256, 96)
    assert select_tiled(qd=d96, kd=desc(1, 2, 256, 96)) == UNSUPPORTED
    assert va.max_count(75600, 64, False, "mins_tiled", 0.5) == 75600
    assert va.max_count(1000, 64, True, "mins_tiled", 0.5) == 1000


def select_per_head(params, q=FAKE, qd=None, k=FAKE, kd=None, mode=0, cap=256, H=4):
    lib = _lib.load()
    qd = qd or desc(1, H, 256, 128)
    kd = kd or desc(1, 2, 256, 128)
    arr = None if params is None else (ctypes.c_double * len(params))(*params)
    return lib.vecattn_select_per_head(q, ctypes.byref(qd), k, ctypes.byref(kd), 64, 0, mode,
                                       arr, 16, 16, FAKE, cap, FAKE, None, None, 1 << 40, None)


def test_select_per_head_rejects_bad_arguments():
    assert select_per_head(None) == INVALID
    assert select_per_head([0.5, 0.5, 1.5, 0.5]) == INVALID            # topK ratio > 1
    assert select_per_head([0.5, 0.5, 0.5, 0.0]) == INVALID
    assert select_per_head([0.1, 0.2, 0.5, 0.3], cap=100) == CAPACITY  # head 2 keeps 128
    assert select_per_head([1.0, -1.0, 1.0, 1.0], mode=2) == INVALID   # minS alpha < 0
    assert select_per_head([0.5] * 4, mode=9) == INVALID
    assert select_per_head([0.5] * 130, qd=desc(1, 130, 256, 128), kd=desc(1, 130, 256, 128),
                           H=130) == UNSUPPORTED
    assert select_per_head([0.5] * 4, q=None) == INVALID
    # otherwise valid: the missing workspace is reported before any launch
    assert select_per_head([0.1, 0.2, 0.5, 0.3], cap=128) == CAPACITY


def test_keep_diag_flag():
    # topK with the diagonal: block i keeps k_i + its own rows (at most L_i)
    assert va.max_count(1024, 64, False, "topk", 0.125, keep_diag=True) == 192
    assert va.max_count(1024, 64, True, "topk", 0.125, keep_diag=True) == 192
    assert va.max_count(100, 64, True, "topk", 0.5, keep_diag=True) == 86   # 50 + 36 rows
    assert va.max_count(1000, 64, True, "topp", 0.5, keep_diag=True) == 1000
    assert select(mode=0, param=0.25, cap=64, causal=8) == INVALID        # unknown bit
    assert select(mode=0, param=0.25, cap=127, causal=2) == CAPACITY       # 64 + 64 needed
    assert select(mode=1, param=0.5, cap=255, causal=2) == CAPACITY        # no clamping
    assert select(mode=1, param=0.5, cap=256, causal=3, ws=None) == CAPACITY   # valid flags
    assert attn(causal=8) == INVALID


def test_varlen_rejects_bad_offsets():
    lib = _lib.load()
    qd, kd = desc(1, 4, 256, 128), desc(1, 2, 256, 128)

    def sel(cu, n=None, qd_=qd, cap=256):
        arr = None if cu is None else (ctypes.c_int64 * len(cu))(*cu)
        return lib.vecattn_select_varlen(FAKE, ctypes.byref(qd_), FAKE, ctypes.byref(kd), arr,
                                         len(cu) - 1 if n is None else n, 64, 0, 0, 0.25, FAKE,
                                         cap, FAKE, None, None, 1 << 40, None)

    assert sel(None, n=1) == INVALID
    assert sel([0]) == INVALID                        # no sequence
    assert sel([1, 256]) == INVALID                   # must start at row 0
    assert sel([0, 100, 50, 256]) == INVALID          # decreasing
    assert sel([0, 100, 200]) == INVALID              # must end at N
    assert sel([0, 100, 256], qd_=desc(2, 4, 256, 128)) == INVALID   # packed: B = 1
    assert sel([0, 100, 256], cap=24) == CAPACITY     # topK 25% of 156 keys = 39
    assert sel([0, 100, 256], cap=64) == CAPACITY     # valid: the missing workspace is reported

    def att(cu):
        arr = (ctypes.c_int64 * len(cu))(*cu)
        return lib.vecattn_sparse_attn_varlen(FAKE, ctypes.byref(qd), FAKE, ctypes.byref(kd), FAKE,
                                              ctypes.byref(kd), arr, len(cu) - 1, FAKE, 16, FAKE,
                                              64, 0, 0.0, FAKE, ctypes.byref(qd), None, None)
    assert att([0, 300]) == INVALID
    assert att([0, 200, 100]) == INVALID


def test_check_lists_rejects_bad_arguments():
    lib = _lib.load()

    def chk(idx=FAKE, rows=10, cap=16, cnt=FAKE, n=256, out=FAKE):
        return lib.vecattn_check_lists(idx, rows, cap, cnt, n, out, None)

    assert chk(idx=None) == INVALID
    assert chk(cnt=None) == INVALID
    assert chk(out=None) == INVALID
    assert chk(rows=-1) == INVALID
    assert chk(rows=1 << 31) == INVALID
    assert chk(cap=0) == INVALID
    assert chk(cap=(1 << 30) + 1) == INVALID
    assert chk(n=0) == INVALID
    assert chk(n=(1 << 30) + 1) == INVALID
    assert chk(rows=0, idx=None, cnt=None, n=0) == INVALID         # still validated when empty


def test_workspace_size_query():
    qd, kd = desc(1, 40, 75600, 128), desc(1, 40, 75600, 128)
    n = ctypes.c_size_t(0)
    lib = _lib.load()
    assert lib.vecattn_select_workspace_size(ctypes.byref(qd), ctypes.byref(kd), 64, 0, 0, 11340,
                                             ctypes.byref(n)) == OK
    assert n.value > 0
    assert lib.vecattn_select_workspace_size(None, ctypes.byref(kd), 64, 0, 0, 11340,
                                             ctypes.byref(n)) == INVALID


def test_pool_rejects_bad_arguments():
    lib = _lib.load()
    qd, pd = desc(1, 2, 100, 64), desc(1, 2, 2, 64)
    assert lib.vecattn_pool(None, ctypes.byref(qd), 64, FAKE, ctypes.byref(pd), None) == INVALID
    assert lib.vecattn_pool(FAKE, ctypes.byref(qd), 0, FAKE, ctypes.byref(pd), None) == INVALID
    bad = desc(1, 2, 3, 64)
    assert lib.vecattn_pool(FAKE, ctypes.byref(qd), 64, FAKE, ctypes.byref(bad), None) == INVALID


def test_sparse_attn_rejects_heads_beyond_32bit_gather_offsets():
    # The gathers address a head's K/V rows with 32-bit byte offsets (24-bit
    # row products): N >= 2^24, a row stride of 2^24 bytes or more, or rows
    # spanning 2^31 bytes or more are rejected before any launch.
    def big(N, sN, H=2):
        return _lib.TDesc(1, H, N, 128, H * N * sN, N * sN, sN)
    # a packed [B, N, 3, 40, 128] QKV view: K rows 30720 bytes apart
    packed = lambda N: _lib.TDesc(1, 40, N, 128, N * 15360, 128, 15360)
    N_ok = 69906          # (N - 1) * 30720 + 256 < 2^31
    assert (N_ok - 1) * 30720 + 256 < 2 ** 31 <= N_ok * 30720 + 256
    q_ok, q_bad = desc(1, 40, N_ok, 128), desc(1, 40, N_ok + 1, 128)
    # valid shapes otherwise: these fail only later, on the FAKE pointers' data
    # (never reached: the call below returns before any launch when rejected)
    assert attn(qd=q_bad, kd=packed(N_ok + 1), vd=packed(N_ok + 1), od=q_bad) == UNSUPPORTED
    assert attn(qd=q_bad, kd=desc(1, 40, N_ok + 1, 128), vd=packed(N_ok + 1), od=q_bad) == UNSUPPORTED
    n24 = 1 << 24
    d24 = desc(1, 1, n24, 64)
    assert attn(qd=d24, kd=desc(1, 1, n24, 64), vd=desc(1, 1, n24, 64), od=d24) == UNSUPPORTED
    wide = _lib.TDesc(1, 1, 2, 64, 2 * (1 << 23), 2 * (1 << 23), 1 << 23)   # 2^24-byte rows
    q2 = desc(1, 1, 2, 64)
    assert attn(qd=q2, kd=wide, vd=desc(1, 1, 2, 64), od=q2) == UNSUPPORTED
    assert attn(qd=q2, kd=desc(1, 1, 2, 64), vd=wide, od=q2) == UNSUPPORTED
    assert q_ok.N == N_ok


def test_varlen_attention_checks_every_tensor_before_launching():
    # K, V and O must cover Q's rows (each sequence's view is cut from them).
    lib = _lib.load()
    qd = desc(1, 4, 256, 128)

    def att(kd=None, vd=None, od=None, cu=(0, 100, 256)):
        kd, vd, od = kd or desc(1, 2, 256, 128), vd or desc(1, 2, 256, 128), od or qd
        arr = (ctypes.c_int64 * len(cu))(*cu)
        return lib.vecattn_sparse_attn_varlen(FAKE, ctypes.byref(qd), FAKE, ctypes.byref(kd), FAKE,
                                              ctypes.byref(vd), arr, len(cu) - 1, FAKE, 16, FAKE,
                                              64, 0, 0.0, FAKE, ctypes.byref(od), None, None)
    assert att(kd=desc(1, 2, 200, 128)) == INVALID
    assert att(vd=desc(1, 2, 200, 128)) == INVALID
    assert att(od=desc(1, 4, 200, 128)) == INVALID
    assert att(kd=desc(1, 3, 256, 128), vd=desc(1, 3, 256, 128)) == INVALID   # 4 % 3
    assert att(vd=desc(1, 2, 256, 64)) == INVALID
    assert att(od=desc(1, 4, 256, 64)) == INVALID


def test_workspace_counts_kv_heads_once():
    # The K operand copy is one per key/value head: a GQA layer (28 / 4 heads)
    # needs less than the same layer with 28 key/value heads.
    lib = _lib.load()
    q = desc(1, 28, 32768, 128)
    n_gqa, n_mha = ctypes.c_size_t(0), ctypes.c_size_t(0)
    assert lib.vecattn_select_workspace_size(ctypes.byref(q), ctypes.byref(desc(1, 4, 32768, 128)),
                                             64, 1, 0, 3277, ctypes.byref(n_gqa)) == OK
    assert lib.vecattn_select_workspace_size(ctypes.byref(q), ctypes.byref(desc(1, 28, 32768, 128)),
                                             64, 1, 0, 3277, ctypes.byref(n_mha)) == OK
    kop = 32768 * 128 * 2      # one head's K in operand order
    assert n_mha.value - n_gqa.value >= 24 * kop
    # the size-returning form agrees, and returns 0 on bad arguments
    assert lib.vecattn_select_workspace_bytes(ctypes.byref(q), ctypes.byref(desc(1, 4, 32768, 128)),
                                              64, 0, 3277) == n_gqa.value
    assert lib.vecattn_select_workspace_bytes(ctypes.byref(q), ctypes.byref(desc(1, 3, 32768, 128)),
                                              64, 0, 3277) == 0
    assert lib.vecattn_select_workspace_bytes(None, ctypes.byref(q), 64, 0, 3277) == 0
    assert lib.vecattn_select_workspace_bytes(ctypes.byref(q), ctypes.byref(q), 0, 0, 3277) == 0


def test_head_sparsity_and_recall_reject_bad_arguments():
    lib = _lib.load()

    def hs(cnt=FAKE, B=1, H=4, N=256, block=64, causal=0, out=FAKE):
        return lib.vecattn_head_sparsity(cnt, B, H, N, block, causal, out, None)
    assert hs(cnt=None) == INVALID and hs(out=None) == INVALID
    assert hs(B=0) == INVALID and hs(H=0) == INVALID and hs(N=0) == INVALID
    assert hs(N=(1 << 30) + 1) == INVALID and hs(block=0) == INVALID and hs(causal=8) == INVALID

    def rc(q=FAKE, qd=None, k=FAKE, kd=None, idx=FAKE, cap=16, cnt=FAKE, block=64, causal=0,
           scale=0.0, kept=FAKE):
        qd = qd or desc(1, 4, 256, 128)
        kd = kd or desc(1, 2, 256, 128)
        return lib.vecattn_recall(q, ctypes.byref(qd), k, ctypes.byref(kd), idx, cap, cnt, block,
                                  causal, scale, kept, None)
    assert rc(q=None) == INVALID and rc(k=None) == INVALID and rc(idx=None) == INVALID
    assert rc(cnt=None) == INVALID and rc(kept=None) == INVALID
    assert rc(block=0) == INVALID and rc(cap=0) == INVALID and rc(causal=8) == INVALID
    assert rc(scale=-1.0) == INVALID and rc(scale=float("nan")) == INVALID
    assert rc(kd=desc(1, 3, 256, 128)) == INVALID and rc(kd=desc(1, 2, 255, 128)) == INVALID
    assert rc(q=FAKE + 2) == INVALID
    assert rc(qd=desc(1, 4, 256, 96), kd=desc(1, 2, 256, 96)) == UNSUPPORTED
    n = (1 << 18) + 1
    assert rc(qd=desc(1, 4, n, 128), kd=desc(1, 2, n, 128)) == UNSUPPORTED


def test_select_noalloc_checks_before_any_device_call():
    # Every argument error, and a workspace need above the library's 64 MiB,
    # is reported before the call touches a device (FAKE pointers here).
    lib = _lib.load()

    def sel(qd=None, kd=None, block=64, causal=0, mode=0, param=0.25, idx=FAKE, cap=64, cnt=FAKE):
        qd = qd or desc(1, 4, 256, 128)
        kd = kd or desc(1, 2, 256, 128)
        return lib.vecattn_select_noalloc(FAKE, ctypes.byref(qd), FAKE, ctypes.byref(kd), block,
                                          causal, mode, param, idx, cap, cnt, None, None)
    assert sel(idx=None) == INVALID and sel(cnt=None) == INVALID and sel(block=0) == INVALID
    assert sel(param=1.5) == INVALID and sel(mode=9) == INVALID and sel(causal=8) == INVALID
    assert sel(kd=desc(1, 3, 256, 128)) == INVALID
    assert sel(cap=63) == CAPACITY
    big_q, big_k = desc(1, 40, 75600, 128), desc(1, 40, 75600, 128)
    assert lib.vecattn_select_workspace_bytes(ctypes.byref(big_q), ctypes.byref(big_k), 64, 0,
                                              11340) > _lib.STATIC_WORKSPACE_BYTES
    assert sel(qd=big_q, kd=big_k, cap=11340, param=0.15) == CAPACITY


def test_attn_order_and_ordered_attention_reject_bad_arguments():
    lib = _lib.load()

    def order(idx=FAKE, cap=16, cnt=FAKE, B=1, H=4, N=256, block=64, out=FAKE):
        return lib.vecattn_attn_order(idx, cap, cnt, B, H, N, block, out, None)
    assert order(idx=None) == INVALID and order(cnt=None) == INVALID and order(out=None) == INVALID
    assert order(B=0) == INVALID and order(H=0) == INVALID and order(N=0) == INVALID
    assert order(block=0) == INVALID and order(cap=0) == INVALID
    assert order(cap=(1 << 30) + 1) == INVALID and order(N=(1 << 30) + 1) == INVALID
    assert order(B=1 << 20, H=1 << 12) == INVALID                      # B * Hq > 2^31 - 1

    def oattn(q=FAKE, idx=FAKE, cnt=FAKE, order=FAKE, block=64, cap=16, scale=0.0, kd=None):
        qd, od = desc(1, 4, 128, 128), desc(1, 4, 128, 128)
        kd = kd or desc(1, 2, 128, 128)
        vd = desc(1, 2, 128, 128)
        return lib.vecattn_sparse_attn_ordered(q, ctypes.byref(qd), FAKE, ctypes.byref(kd), FAKE,
                                               ctypes.byref(vd), idx, cap, cnt, order, block, 0,
                                               scale, FAKE, ctypes.byref(od), None, None)
    # the checks of vecattn_sparse_attn apply unchanged (a NULL order is allowed)
    assert oattn(q=None) == INVALID and oattn(idx=None) == INVALID and oattn(cnt=None) == INVALID
    assert oattn(block=0) == INVALID and oattn(cap=0) == INVALID and oattn(scale=-1.0) == INVALID
    assert oattn(order=None, q=None) == INVALID
    assert oattn(kd=desc(1, 2, 127, 128)) == INVALID
    assert oattn(kd=desc(1, 2, 1 << 24, 128)) == INVALID                # N mismatch before size
