"""C ABI checks that need no GPU: the library loads, exports every symbol the
header declares, sizes its workspace, and rejects bad arguments before any
launch (every call here returns before touching device memory)."""
import ctypes
import os
import re

import numpy as np
import pytest
import torch

import paper_2608_19758_amd as fp2

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def header_symbols():
    text = open(os.path.join(ROOT, "include", "fp2.h")).read()
    return sorted(set(re.findall(r"\b(fp2_[a-z_]+)\s*\(", text)))


def test_exports_every_declared_symbol():
    lib = fp2.lib()
    syms = header_symbols()
    assert set(syms) == set(fp2.EXPORTS)
    for s in syms:
        assert hasattr(lib, s), s


def base(**kw):
    d = dict(batch=2, num_q_heads=32, num_kv_heads=8, max_seq_len=4096, page_size=64,
             max_pages_per_seq=64, alpha=0.1)
    d.update(kw)
    return fp2.make_params(**d)


def test_workspace_bytes():
    # the pooled means, lists and counts: the bulk of the workspace, by formula
    p = base(kv_splits=1)
    nb = 32
    rows = 2 * 8 * nb
    want = rows * 128 * 2 * 2 + rows * nb * 4 + rows * 4 + 256   # + the work counters
    got = fp2.workspace_bytes(p)
    assert want <= got <= want + rows * 2 * 16 + rows * 8 + 8 * 256   # + item table and unit info
    assert fp2.workspace_bytes(base(head_dim=64)) == 0
    assert fp2.workspace_bytes(base(batch=0)) == 0
    # prefix KV: pooled rows and list columns per key block, list rows per query block
    pk = base(max_kv_len=3 * 4096, max_pages_per_seq=192, kv_splits=1)
    nq, nk = 32, 96
    want = 2 * 8 * (nk * 128 * 2 * 2 + nq * nk * 4 + nq * 4) + 256
    assert want <= fp2.workspace_bytes(pk) <= want + rows * 2 * 16 + rows * 8 + 8 * 256
    # the cost-balanced plan adds 65536 packed rows of partial outputs (520 B each)
    assert fp2.workspace_bytes(base()) - got >= 65536 * 520


FAKE = ctypes.c_void_p(0x100000)   # never dereferenced: validation fails first


def call_prefill(p, **over):
    args = dict(q=FAKE, cu=FAKE, cuh=None, cuk=None, cukh=None, k=FAKE, v=FAKE, bt=FAKE, qs=None,
                ks=None, vs=None, out=FAKE, lse=None, mask=FAKE, ws=None, wsb=0)
    args.update(over)
    return fp2.lib().fp2_prefill(ctypes.byref(p), args["q"], args["cu"], args["cuh"], args["cuk"],
                                 args["cukh"], args["k"], args["v"], args["bt"], args["qs"],
                                 args["ks"], args["vs"], args["out"], args["lse"], args["mask"],
                                 args["ws"], args["wsb"], None)


@pytest.mark.parametrize("kw,status", [
    (dict(num_kv_heads=0), fp2.EINVAL),
    (dict(num_kv_heads=2048, num_q_heads=2048), fp2.EUNSUPPORTED),
    (dict(num_q_heads=30), fp2.EINVAL),
    (dict(num_q_heads=48, num_kv_heads=8), fp2.EUNSUPPORTED),      # g = 6
    (dict(num_q_heads=128, num_kv_heads=8), fp2.EUNSUPPORTED),     # g = 16
    (dict(head_dim=64), fp2.EUNSUPPORTED),
    (dict(score_splits=-1), fp2.EINVAL),
    (dict(score_splits=65), fp2.EINVAL),
    (dict(head_dim=0), fp2.EINVAL),
    (dict(block_size=64), fp2.EUNSUPPORTED),
    (dict(page_size=-1), fp2.EINVAL),
    (dict(max_pages_per_seq=10), fp2.EINVAL),
    (dict(max_seq_len=(1 << 20) + 1, max_pages_per_seq=1 << 15), fp2.EUNSUPPORTED),
    (dict(alpha=-0.5), fp2.EINVAL),
    (dict(alpha=float("nan")), fp2.EINVAL),
    (dict(alpha=float("inf")), fp2.EINVAL),
    (dict(sink_blocks=-1), fp2.EINVAL),
    (dict(mean_correction=2), fp2.EINVAL),
    (dict(dtype=7), fp2.EINVAL),
    (dict(batch=-1), fp2.EINVAL),
    (dict(max_kv_len=-1), fp2.EINVAL),
    (dict(max_kv_len=2048), fp2.EINVAL),                           # < max_seq_len
    (dict(max_kv_len=8192), fp2.EINVAL),                           # needs 128 pages
    (dict(max_kv_len=(1 << 20) + 1, max_pages_per_seq=1 << 15), fp2.EUNSUPPORTED),
    (dict(kv_splits=-1), fp2.EINVAL),
    (dict(kv_splits=33), fp2.EINVAL),
    (dict(query_tile_rows=64), fp2.EUNSUPPORTED),
    (dict(query_tile_rows=-1), fp2.EUNSUPPORTED),
])
def test_invalid_params(kw, status):
    assert call_prefill(base(**kw)) == status
    assert fp2.last_error() != ""


def test_null_and_workspace_errors():
    p = base()
    assert call_prefill(p, q=None) == fp2.EINVAL
    assert call_prefill(p, cu=None) == fp2.EINVAL
    assert call_prefill(p, bt=None) == fp2.EINVAL
    assert call_prefill(p, out=None) == fp2.EINVAL
    assert call_prefill(p, mask=None) == fp2.EINVAL
    assert call_prefill(p, q=ctypes.c_void_p(0x100008)) == fp2.EINVAL    # misaligned
    assert call_prefill(base(dtype="fp8")) == fp2.EINVAL                 # scales missing
    assert call_prefill(p) == fp2.EWORKSPACE
    need = fp2.workspace_bytes(p)
    assert call_prefill(p, ws=FAKE, wsb=need - 1) == fp2.EWORKSPACE
    assert call_prefill(p, ws=ctypes.c_void_p(0x100010), wsb=need) == fp2.EWORKSPACE  # alignment
    assert "workspace" in fp2.last_error()


def test_host_lengths_checked():
    p = base()
    bad = np.array([0, 5000, 6000], dtype=np.int32)       # 5000 > max_seq_len
    assert call_prefill(p, cuh=ctypes.c_void_p(bad.ctypes.data)) == fp2.EINVAL
    bad2 = np.array([1, 2, 3], dtype=np.int32)
    assert call_prefill(p, cuh=ctypes.c_void_p(bad2.ctypes.data)) == fp2.EINVAL
    bad3 = np.array([0, 10, 5], dtype=np.int32)
    assert call_prefill(p, cuh=ctypes.c_void_p(bad3.ctypes.data)) == fp2.EINVAL


def ws_parts(p):
    """Workspace bytes predicted from the documented sections (each 256-aligned)."""
    al = lambda x: (x + 255) // 256 * 256
    g = p.num_q_heads // p.num_kv_heads
    rows = p.batch * p.num_kv_heads * fp2.num_blocks(p)
    krows = p.batch * p.num_kv_heads * fp2.num_key_blocks(p)
    rpu = g * fp2.tile_positions(p)
    wpu = max(1, rpu // 256)
    if p.kv_splits == 0:
        slots = 65536 // rpu
        items = wpu * (rows + slots)
    else:
        slots = rows * p.kv_splits if p.kv_splits > 1 else 0
        items = wpu * rows * p.kv_splits
    n = 2 * al(krows * 256) + al(rows * fp2.num_key_blocks(p) * 4) + al(rows * 4)
    if p.dtype == fp2.FP8_E4M3:
        n += 2 * al(krows * 128)   # e4m3 code means of K and V (the fp8 correction)
    n += al(items * 16) + al(rows * 8) + al((slots // 2 + 1) * 4) + 256
    if slots:
        n += al(slots * rpu * 512) + al(slots * rpu * 8)
    return n


@pytest.mark.parametrize("kw", [dict(), dict(kv_splits=1), dict(kv_splits=4),
                                dict(num_q_heads=64, kv_splits=0), dict(num_q_heads=8),
                                dict(max_kv_len=12288, max_pages_per_seq=192, kv_splits=3),
                                dict(query_tile_rows=128), dict(query_tile_rows=128, kv_splits=2),
                                dict(num_q_heads=64, query_tile_rows=128), dict(dtype="fp8"),
                                dict(dtype="fp8", max_kv_len=12288, max_pages_per_seq=192)])
def test_workspace_sections(kw):
    p = base(**kw)
    assert fp2.workspace_bytes(p) == ws_parts(p)


def test_host_kv_lengths_checked():
    p = base(max_kv_len=8192, max_pages_per_seq=128)
    cu = np.array([0, 300, 1000], dtype=np.int32)
    host = lambda a: ctypes.c_void_p(a.ctypes.data)
    good = np.array([0, 300 + 256, 556 + 700 + 384], dtype=np.int32)  # prefixes 256 and 384
    assert call_prefill(p, cuh=host(cu), cuk=FAKE, cukh=host(good)) == fp2.EWORKSPACE
    # host KV lengths without the device array
    assert call_prefill(p, cuh=host(cu), cukh=host(good)) == fp2.EINVAL
    # a prefix that is not a multiple of the block size is accepted
    odd = np.array([0, 300 + 100, 400 + 700 + 1], dtype=np.int32)    # prefixes 100 and 1
    assert call_prefill(p, cuh=host(cu), cuk=FAKE, cukh=host(odd)) == fp2.EWORKSPACE
    # fewer keys than queries
    bad = np.array([0, 200, 900], dtype=np.int32)                    # 200 keys < 300 queries
    assert call_prefill(p, cuh=host(cu), cuk=FAKE, cukh=host(bad)) == fp2.EINVAL
    assert "KV length < query length" in fp2.last_error()
    # a KV length over max_kv_len
    bad = np.array([0, 300 + 8192, 8492 + 700], dtype=np.int32)
    assert call_prefill(p, cuh=host(cu), cuk=FAKE, cukh=host(bad)) == fp2.EINVAL
    assert "max_kv_len" in fp2.last_error()


def test_noop_problems_return_ok():
    assert call_prefill(base(batch=0), q=None, cu=None, k=None, v=None, out=None, mask=None) == fp2.OK
    assert call_prefill(base(max_seq_len=0), q=None, k=None, v=None, out=None, mask=None) == fp2.OK


def test_status_strings():
    for s in range(5):
        assert fp2.status_str(s)
    assert fp2.status_str(99) == "unknown status"


def test_mask_to_csr_validation():
    p = base(query_tile_rows=128)
    lib = fp2.lib()
    cap = fp2.csr_capacity(p)
    # 2 * 8 heads * 128 tiles of 32 positions * 2 * 32 key blocks
    assert cap == 2 * 8 * (4096 // 32) * 2 * 32
    call = lambda **o: lib.fp2_mask_to_csr(
        ctypes.byref(p), o.get("cu", FAKE), None, None, None, o.get("mask", FAKE),
        o.get("off", FAKE), o.get("idx", FAKE), o.get("cap", cap), o.get("ws", None),
        o.get("wsb", 0), None)
    assert call(cap=cap - 1) == fp2.EINVAL and "capacity" in fp2.last_error()
    assert call(mask=None) == fp2.EINVAL
    assert call(cu=None) == fp2.EINVAL
    assert call() == fp2.EWORKSPACE
    assert fp2.csr_capacity(base(query_tile_rows=7)) == 0


def test_means_cache_slots_and_validation():
    """Slot counts of the block-means cache, and the cached prefill's checks
    of its cache argument (all before any launch)."""
    p = base()                                   # page 64: one slot per page
    assert fp2.means_cache_slots(p, 1000) == 1000
    assert fp2.means_cache_slots(base(page_size=200, max_pages_per_seq=21), 10) == 20
    assert fp2.means_cache_slots(base(page_size=128, max_pages_per_seq=32), 10) == 10
    assert fp2.means_cache_slots(base(page_size=0, max_kv_len=5000), 0) == 2 * 40
    assert fp2.means_cache_slots(p, -1) == 0
    assert fp2.means_cache_slots(base(head_dim=64), 10) == 0
    L = fp2.lib()
    ws_need = fp2.workspace_bytes(p)
    ws = ctypes.c_void_p(0x200000)

    def cached(cache):
        return L.fp2_prefill_cached(ctypes.byref(p), FAKE, FAKE, None, None, None, FAKE, FAKE,
                                    FAKE, None, None, None, cache, FAKE, None, FAKE, ws, ws_need,
                                    None)
    assert cached(None) == fp2.EINVAL
    assert cached(ctypes.byref(fp2.MeansCache(None, FAKE.value, FAKE.value))) == fp2.EINVAL
    assert cached(ctypes.byref(fp2.MeansCache(FAKE.value, FAKE.value, None))) == fp2.EINVAL
    assert "pooled_blocks" in fp2.last_error()
    assert cached(ctypes.byref(fp2.MeansCache(0x100008, FAKE.value, FAKE.value))) == fp2.EINVAL
    assert "aligned" in fp2.last_error()


def test_calibrate_rejects_bad_arguments():
    L = fp2.lib()
    ops = ctypes.c_double(0.0)
    sink = ctypes.c_void_p(16)   # never dereferenced: every call below fails validation
    for kind, iters, s, o in [(3, 10, sink, ctypes.byref(ops)), (-1, 10, sink, ctypes.byref(ops)),
                              (0, 0, sink, ctypes.byref(ops)), (1, (1 << 24) + 1, sink, ctypes.byref(ops)),
                              (2, 10, None, ctypes.byref(ops)), (0, 10, sink, None)]:
        assert L.fp2_calibrate(kind, iters, s, o, None) == fp2.EINVAL
        assert fp2.last_error()
    with pytest.raises(ValueError):
        fp2.calibrate("mfma_fp4", 10)
    with pytest.raises(ValueError):   # a host tensor never reaches the kernel
        fp2.calibrate("exp", 10, sink=torch.zeros(1))


def test_means_cache_tensors_checked_before_the_call():
    """A means cache that is not a CUDA bf16 [slots, H_kv, 128] pair is refused
    by the binding (host tensors here: nothing reaches the library)."""
    p = base(batch=1)
    q = torch.zeros(4, 32, 128, dtype=torch.bfloat16)
    cu = torch.tensor([0, 4], dtype=torch.int32)
    kh = torch.zeros(8, 8, 128, dtype=torch.bfloat16)
    pooled = torch.zeros(1, dtype=torch.int32)
    with pytest.raises(ValueError):
        fp2.prefill(p, q, q, q, cu, cu, means_cache=(kh, kh.clone(), pooled))


def test_host_tensors_refused_as_device_arguments():
    """Device arguments must be CUDA tensors: a host tensor raises in the
    binding (its address never reaches a kernel)."""
    p = base(batch=1, page_size=0)
    q = torch.zeros(4, 32, 128, dtype=torch.bfloat16)
    kv = torch.zeros(4, 8, 128, dtype=torch.bfloat16)
    cu = torch.tensor([0, 4], dtype=torch.int32)
    with pytest.raises(ValueError, match="CUDA"):
        fp2.pool(p, kv, kv, cu)


def test_time_kernels_pairs():
    lib = fp2.lib()
    assert lib.fp2_time_kernels(None, None, None, None) == fp2.OK
    assert lib.fp2_time_kernels(ctypes.c_void_p(16), None, None, None) == fp2.EINVAL
    assert lib.fp2_time_kernels(None, None, None, ctypes.c_void_p(16)) == fp2.EINVAL
    assert "pairs" in fp2.last_error()


def test_noalloc_limits_checked_before_any_device_call():
    """The no-allocation prefill refuses a call whose scratch need exceeds the
    static array (a host-side check, no GPU touched), and validates params as
    fp2_prefill does; the 128K-token workloads with 8 KV heads fit."""
    lib = fp2.lib()
    for hq in (32, 64):
        p = fp2.make_params(batch=1, num_q_heads=hq, num_kv_heads=8, max_seq_len=131072,
                            page_size=64, max_pages_per_seq=2048, alpha=0.98, dtype="fp8")
        assert 0 < fp2.workspace_bytes(p) <= fp2.NOALLOC_SCRATCH_BYTES
    big = fp2.make_params(batch=4, num_q_heads=32, num_kv_heads=8, max_seq_len=131072,
                          page_size=64, max_pages_per_seq=2048, alpha=0.98)
    assert fp2.workspace_bytes(big) > fp2.NOALLOC_SCRATCH_BYTES
    st = lib.fp2_prefill_noalloc(ctypes.byref(big), *([None] * 14), None)
    assert st == fp2.EWORKSPACE
    assert "static array" in fp2.last_error()
    bad = fp2.make_params(batch=1, num_q_heads=3, num_kv_heads=2, max_seq_len=128)
    assert lib.fp2_prefill_noalloc(ctypes.byref(bad), *([None] * 14), None) == fp2.EINVAL
    # nothing to compute: OK without touching the device
    empty = fp2.make_params(batch=0, num_q_heads=4, num_kv_heads=1, max_seq_len=128)
    assert lib.fp2_prefill_noalloc(ctypes.byref(empty), *([None] * 14), None) == fp2.OK
