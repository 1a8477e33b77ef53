"""Python binding of libfp2 (block-sparse causal GQA prefill attention for
MI355X / gfx950): argument marshalling over the C ABI of ``include/fp2.h``.

Every step of the computation runs in the library's HIP kernels; torch only
provides device memory and the current stream. The library must be built
(``python paper_2608_19758_amd/build.py`` or ``__graft_entry__.build()``);
importing works without it, but every call raises until it is built.
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional

import torch

_DIR = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_DIR, "libfp2.so")
_lib = None

OK, EINVAL, EUNSUPPORTED, EWORKSPACE, EHIP = 0, 1, 2, 3, 4
BF16, FP8_E4M3 = 0, 1
HEAD_DIM = 128
BLOCK = 128


class Fp2Error(RuntimeError):
    def __init__(self, fn, status, msg):
        super().__init__("%s failed: %s (%s)" % (fn, status_str(status), msg))
        self.status = status


class Params(ctypes.Structure):
    """Mirror of fp2_params_t."""
    _fields_ = [
        ("batch", ctypes.c_int32), ("num_q_heads", ctypes.c_int32),
        ("num_kv_heads", ctypes.c_int32), ("head_dim", ctypes.c_int32),
        ("block_size", ctypes.c_int32), ("page_size", ctypes.c_int32),
        ("max_seq_len", ctypes.c_int32), ("max_pages_per_seq", ctypes.c_int32),
        ("alpha", ctypes.c_float),
        ("sink_blocks", ctypes.c_int32), ("window_blocks", ctypes.c_int32),
        ("recent_blocks", ctypes.c_int32), ("mean_correction", ctypes.c_int32),
        ("softmax_scale", ctypes.c_float), ("dtype", ctypes.c_int32),
        ("max_kv_len", ctypes.c_int32), ("kv_splits", ctypes.c_int32),
        ("query_tile_rows", ctypes.c_int32),
        ("score_splits", ctypes.c_int32),
    ]


EXPORTS = ["fp2_workspace_bytes", "fp2_prefill", "fp2_estimate", "fp2_attend", "fp2_pool",
           "fp2_csr_capacity", "fp2_mask_to_csr", "fp2_means_cache_slots", "fp2_prefill_cached",
           "fp2_calibrate", "fp2_time_kernels", "fp2_prefill_noalloc", "fp2_status_str",
           "fp2_last_error"]

CALIB_KINDS = {"mfma_bf16": 0, "mfma_fp8": 1, "exp": 2}


class MeansCache(ctypes.Structure):
    """fp2_means_cache_t: device pointers of a caller-owned block-means cache."""
    _fields_ = [("khat", ctypes.c_void_p), ("vbar", ctypes.c_void_p),
                ("pooled_blocks", ctypes.c_void_p)]


def lib():
    """The loaded libfp2.so; raises if it has not been built."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError("libfp2.so is not built (%s); run paper_2608_19758_amd/build.py"
                               % LIB_PATH)
        L = ctypes.CDLL(LIB_PATH)
        vp, P = ctypes.c_void_p, ctypes.POINTER(Params)
        L.fp2_workspace_bytes.restype = ctypes.c_size_t
        L.fp2_workspace_bytes.argtypes = [P]
        L.fp2_prefill.restype = ctypes.c_int
        L.fp2_prefill.argtypes = [P] + [vp] * 15 + [ctypes.c_size_t, vp]
        L.fp2_estimate.restype = ctypes.c_int
        L.fp2_estimate.argtypes = [P] + [vp] * 13 + [ctypes.c_size_t, vp]
        L.fp2_attend.restype = ctypes.c_int
        L.fp2_attend.argtypes = [P] + [vp] * 15 + [ctypes.c_size_t, vp]
        L.fp2_pool.restype = ctypes.c_int
        L.fp2_pool.argtypes = [P] + [vp] * 10
        L.fp2_csr_capacity.restype = ctypes.c_size_t
        L.fp2_csr_capacity.argtypes = [P]
        L.fp2_mask_to_csr.restype = ctypes.c_int
        L.fp2_mask_to_csr.argtypes = [P] + [vp] * 7 + [ctypes.c_size_t, vp, ctypes.c_size_t, vp]
        L.fp2_means_cache_slots.restype = ctypes.c_size_t
        L.fp2_means_cache_slots.argtypes = [P, ctypes.c_int64]
        L.fp2_prefill_cached.restype = ctypes.c_int
        L.fp2_prefill_cached.argtypes = [P] + [vp] * 11 + [ctypes.POINTER(MeansCache)] + \
            [vp] * 4 + [ctypes.c_size_t, vp]
        L.fp2_calibrate.restype = ctypes.c_int
        L.fp2_calibrate.argtypes = [ctypes.c_int, ctypes.c_int32, vp, ctypes.POINTER(ctypes.c_double), vp]
        L.fp2_time_kernels.restype = ctypes.c_int
        L.fp2_time_kernels.argtypes = [vp] * 4
        L.fp2_prefill_noalloc.restype = ctypes.c_int
        L.fp2_prefill_noalloc.argtypes = [P] + [vp] * 15
        L.fp2_status_str.restype = ctypes.c_char_p
        L.fp2_status_str.argtypes = [ctypes.c_int]
        L.fp2_last_error.restype = ctypes.c_char_p
        L.fp2_last_error.argtypes = []
        _lib = L
    return _lib


def status_str(st: int) -> str:
    return lib().fp2_status_str(st).decode()


def last_error() -> str:
    return lib().fp2_last_error().decode()


def _check(fn: str, st: int) -> None:
    if st != OK:
        raise Fp2Error(fn, st, last_error())


def make_params(*, batch, num_q_heads, num_kv_heads, max_seq_len, page_size=0,
                max_pages_per_seq=0, alpha=0.0, sink_blocks=1, window_blocks=2,
                recent_blocks=0, mean_correction=1, softmax_scale=0.0, dtype="bf16",
                head_dim=HEAD_DIM, block_size=BLOCK, max_kv_len=0, kv_splits=0,
                query_tile_rows=0, score_splits=0) -> Params:
    """fp2_params_t; max_kv_len bounds the KV lengths with a prefix (0: max_seq_len);
    kv_splits: 0 = cost-balanced KV splits planned on the device, n = n parts per unit
    (1 = none); query_tile_rows: 0 = query blocks of 128 positions x g heads,
    128 = tiles of 128 packed rows (128 / g positions x g heads); score_splits:
    0 = the scoring splits the rows of units over several workgroups in calls
    with few units, n = at most n parts (1 = none)."""
    dt = {"bf16": BF16, "fp8": FP8_E4M3}.get(dtype, dtype)
    return Params(batch=batch, num_q_heads=num_q_heads, num_kv_heads=num_kv_heads,
                  head_dim=head_dim, block_size=block_size, page_size=page_size,
                  max_seq_len=max_seq_len, max_pages_per_seq=max_pages_per_seq,
                  alpha=alpha, sink_blocks=sink_blocks, window_blocks=window_blocks,
                  recent_blocks=recent_blocks, mean_correction=int(mean_correction),
                  softmax_scale=softmax_scale, dtype=dt, max_kv_len=max_kv_len,
                  kv_splits=kv_splits, query_tile_rows=query_tile_rows,
                  score_splits=score_splits)


def tile_positions(p: Params) -> int:
    """Positions per query tile (block_size, or 128 / g for 128-row tiles)."""
    if p.query_tile_rows > 0:
        return p.query_tile_rows // (p.num_q_heads // p.num_kv_heads)
    return p.block_size


def num_blocks(p: Params) -> int:
    """Query tiles per sequence bound (block_mask rows)."""
    return (p.max_seq_len + tile_positions(p) - 1) // tile_positions(p)


def num_key_blocks(p: Params) -> int:
    """Key blocks per sequence bound (block_mask columns, pooled rows)."""
    kv = p.max_kv_len if p.max_kv_len > 0 else p.max_seq_len
    return (kv + p.block_size - 1) // p.block_size


def alloc_mask(p: Params, device="cuda") -> torch.Tensor:
    return torch.empty((p.batch, p.num_kv_heads, max(1, num_blocks(p)), max(1, num_key_blocks(p))),
                       dtype=torch.uint8, device=device)


def workspace_bytes(p: Params) -> int:
    return int(lib().fp2_workspace_bytes(ctypes.byref(p)))



def _ptr(t: Optional[torch.Tensor]):
    """Device pointer of a CUDA tensor (None passes NULL). A host tensor is
    refused here: its address would reach a kernel as a device pointer."""
    if t is None:
        return None
    if not t.is_cuda:
        raise ValueError("expected a CUDA tensor, got one on %s" % t.device)
    return ctypes.c_void_p(t.data_ptr())


_ESZ = {BF16: 2, FP8_E4M3: 1}


def _need(t, name, *, dtypes=None, esz=None, min_numel=None, divisible=None, contiguous=True):
    """Refuse a tensor the library would misread: wrong dtype (or element
    size), a non-contiguous view (the library reads dense rows at fixed
    strides), or too few elements. The device is checked by the caller."""
    if t is None:
        return
    if not isinstance(t, torch.Tensor):
        raise ValueError("%s must be a torch tensor" % name)
    if dtypes is not None and t.dtype not in dtypes:
        raise ValueError("%s must have dtype in %s, got %s" % (name, dtypes, t.dtype))
    if esz is not None and t.element_size() != esz:
        raise ValueError("%s must have %d-byte elements, got %s" % (name, esz, t.dtype))
    if contiguous and not t.is_contiguous():
        raise ValueError("%s must be contiguous" % name)
    if min_numel is not None and t.numel() < min_numel:
        raise ValueError("%s holds %d elements, needs at least %d" % (name, t.numel(), min_numel))
    if divisible is not None and t.numel() % divisible:
        raise ValueError("%s: %d elements is not a multiple of %d" % (name, t.numel(), divisible))


_INT32 = (torch.int32,)
_F32 = (torch.float32,)


def _check_inputs(p: Params, q=None, k_cache=None, v_cache=None, cu_seqlens=None,
                  block_table=None, cu_seqlens_k=None, q_scale=None, k_scale=None,
                  v_scale=None, out=None, lse=None, block_mask=None, workspace=None,
                  mask_in=None):
    """Dtype, contiguity and size of every device tensor handed to the library
    (the C ABI sees only pointers)."""
    esz = _ESZ.get(p.dtype)
    row_q = p.num_q_heads * p.head_dim
    row_kv = p.num_kv_heads * p.head_dim
    _need(q, "q", esz=esz, divisible=row_q)
    _need(k_cache, "k_cache", esz=esz, divisible=row_kv)
    _need(v_cache, "v_cache", esz=esz, divisible=row_kv)
    if k_cache is not None and v_cache is not None and k_cache.numel() != v_cache.numel():
        raise ValueError("k_cache and v_cache differ in size")
    _need(cu_seqlens, "cu_seqlens", dtypes=_INT32, min_numel=p.batch + 1)
    _need(cu_seqlens_k, "cu_seqlens_k", dtypes=_INT32, min_numel=p.batch + 1)
    if p.page_size > 0 and block_table is not None:
        # the library reads row b at b * max_pages_per_seq: the table must be
        # exactly that wide (a wider one would shift every row after the first)
        if block_table.dim() != 2 or block_table.shape[1] != p.max_pages_per_seq \
                or block_table.shape[0] < p.batch:
            raise ValueError("block_table must be int32 [>= batch, max_pages_per_seq = %d], got %s"
                             % (p.max_pages_per_seq, tuple(block_table.shape)))
        _need(block_table, "block_table", dtypes=_INT32)
    if p.dtype == FP8_E4M3:
        g = p.num_q_heads
        _need(q_scale, "q_scale", dtypes=_F32, min_numel=g)
        _need(k_scale, "k_scale", dtypes=_F32, min_numel=p.num_kv_heads)
        _need(v_scale, "v_scale", dtypes=_F32, min_numel=p.num_kv_heads)
    rows = None if q is None else q.numel() // row_q
    if out is not None:
        _need(out, "out", dtypes=(torch.bfloat16,), min_numel=(rows or 0) * row_q)
    if lse is not None:
        _need(lse, "lse", dtypes=_F32, min_numel=(rows or 0) * p.num_q_heads)
    nmask = p.batch * p.num_kv_heads * max(1, num_blocks(p)) * max(1, num_key_blocks(p))
    _need(block_mask, "block_mask", dtypes=(torch.uint8,), min_numel=nmask)
    _need(mask_in, "block_mask", dtypes=(torch.uint8, torch.bool), min_numel=nmask)
    _need(workspace, "workspace", esz=1)
    named = (("q", q), ("k_cache", k_cache), ("v_cache", v_cache), ("cu_seqlens", cu_seqlens),
             ("block_table", block_table if p.page_size > 0 else None),
             ("cu_seqlens_k", cu_seqlens_k), ("q_scale", q_scale), ("k_scale", k_scale),
             ("v_scale", v_scale), ("out", out), ("lse", lse), ("block_mask", block_mask),
             ("workspace", workspace), ("block_mask", mask_in))
    for name, t in named:
        if t is not None and not t.is_cuda:
            raise ValueError("%s must be a CUDA tensor" % name)


def _host_ptr(a):
    if a is None:
        return None
    return ctypes.c_void_p(a.ctypes.data) if hasattr(a, "ctypes") else ctypes.c_void_p(a.data_ptr())


def _stream(stream):
    if stream is None:
        stream = torch.cuda.current_stream()
    return ctypes.c_void_p(stream.cuda_stream)


def alloc_workspace(p: Params, device="cuda") -> torch.Tensor:
    n = max(1, workspace_bytes(p))
    return torch.empty(n, dtype=torch.uint8, device=device)


def alloc_outputs(p: Params, total_tokens: int, device="cuda", want_lse=False):
    out = torch.empty((total_tokens, p.num_q_heads, p.head_dim), dtype=torch.bfloat16,
                      device=device)
    mask = alloc_mask(p, device)
    lse = (torch.empty((total_tokens, p.num_q_heads), dtype=torch.float32, device=device)
           if want_lse else None)
    return out, mask, lse


def prefill(p: Params, q, k_cache, v_cache, cu_seqlens, block_table=None, *, cu_seqlens_host=None,
            cu_seqlens_k=None, cu_seqlens_k_host=None, q_scale=None, k_scale=None, v_scale=None,
            out=None, lse=None, block_mask=None, workspace=None, want_lse=False, stream=None,
            means_cache=None):
    """fp2_prefill: returns (out [total, Hq, 128] bf16, block_mask uint8, lse or None).

    cu_seqlens_k (device) gives the KV lengths when the queries are the last
    tokens of longer sequences (a prefix KV); None means no prefix.
    means_cache = (khat, vbar, pooled_blocks) device tensors calls
    fp2_prefill_cached (block means kept across calls)."""
    if means_cache is not None:
        kh, vb, pooled = means_cache
        for name, t in (("khat", kh), ("vbar", vb)):
            if not (t.is_cuda and t.dtype == torch.bfloat16 and t.dim() == 3
                    and tuple(t.shape[1:]) == (p.num_kv_heads, p.head_dim) and t.is_contiguous()):
                raise ValueError("means cache %s must be a contiguous CUDA bf16 tensor "
                                 "[slots, num_kv_heads, head_dim]" % name)
        if kh.shape[0] != vb.shape[0]:
            raise ValueError("means cache khat and vbar hold different slot counts")
        if not (pooled.is_cuda and pooled.dtype == torch.int32 and pooled.numel() >= p.batch):
            raise ValueError("pooled_blocks must be a CUDA int32 tensor of batch entries")
    if out is None or block_mask is None:
        o2, m2, l2 = alloc_outputs(p, q.shape[0], q.device, want_lse and lse is None)
        out = o2 if out is None else out
        block_mask = m2 if block_mask is None else block_mask
        lse = l2 if lse is None else lse
    if workspace is None:
        workspace = alloc_workspace(p, q.device)
    _check_inputs(p, q, k_cache, v_cache, cu_seqlens, block_table, cu_seqlens_k, q_scale,
                  k_scale, v_scale, out, lse, block_mask, workspace)
    head = (ctypes.byref(p), _ptr(q), _ptr(cu_seqlens), _host_ptr(cu_seqlens_host),
            _ptr(cu_seqlens_k), _host_ptr(cu_seqlens_k_host), _ptr(k_cache), _ptr(v_cache),
            _ptr(block_table), _ptr(q_scale), _ptr(k_scale), _ptr(v_scale))
    tail = (_ptr(out), _ptr(lse), _ptr(block_mask), _ptr(workspace), workspace.numel(),
            _stream(stream))
    if means_cache is None:
        _check("fp2_prefill", lib().fp2_prefill(*head, *tail))
    else:
        kh, vb, pooled = means_cache
        mc = MeansCache(_ptr(kh), _ptr(vb), _ptr(pooled))
        _check("fp2_prefill_cached", lib().fp2_prefill_cached(*head, ctypes.byref(mc), *tail))
    return out, block_mask, lse


NOALLOC_SCRATCH_BYTES = 96 << 20   # FP2_NOALLOC_SCRATCH_BYTES


def prefill_noalloc(p: Params, q, k_cache, v_cache, cu_seqlens, block_table=None, *,
                    cu_seqlens_host=None, cu_seqlens_k=None, cu_seqlens_k_host=None,
                    q_scale=None, k_scale=None, v_scale=None, out=None, lse=None,
                    block_mask=None, stream=None):
    """fp2_prefill_noalloc: fp2_prefill with the library's static scratch array
    instead of a workspace (the library allocates nothing; out, lse and
    block_mask are allocated here when not given). Returns (out, block_mask,
    lse)."""
    if out is None:
        out = torch.empty((q.shape[0], p.num_q_heads, p.head_dim), dtype=torch.bfloat16,
                          device=q.device)
    if block_mask is None:
        block_mask = alloc_mask(p, q.device)
    _check_inputs(p, q, k_cache, v_cache, cu_seqlens, block_table, cu_seqlens_k, q_scale,
                  k_scale, v_scale, out, lse, block_mask)
    st = lib().fp2_prefill_noalloc(ctypes.byref(p), _ptr(q), _ptr(cu_seqlens),
                                   _host_ptr(cu_seqlens_host), _ptr(cu_seqlens_k),
                                   _host_ptr(cu_seqlens_k_host), _ptr(k_cache), _ptr(v_cache),
                                   _ptr(block_table), _ptr(q_scale), _ptr(k_scale),
                                   _ptr(v_scale), _ptr(out), _ptr(lse), _ptr(block_mask),
                                   _stream(stream))
    _check("fp2_prefill_noalloc", st)
    return out, block_mask, lse


def time_kernels(estimate=None, attend=None):
    """fp2_time_kernels: estimate / attend are (begin, end) pairs of recorded
    torch.cuda.Event(enable_timing=True) (or None); later calls on this host
    thread record them around the estimation kernels / the attention kernel.
    time_kernels() stops."""
    def h(ev):
        if ev is None:
            return None
        if not ev.cuda_event:
            raise ValueError("record each event once before handing it to the library")
        return ctypes.c_void_p(ev.cuda_event)
    eb, ee = (None, None) if estimate is None else estimate
    ab, ae = (None, None) if attend is None else attend
    _check("fp2_time_kernels", lib().fp2_time_kernels(h(eb), h(ee), h(ab), h(ae)))


def means_cache_slots(p: Params, num_pages: int) -> int:
    """fp2_means_cache_slots: slots of a block-means cache for this params and
    a pool of num_pages pages."""
    return int(lib().fp2_means_cache_slots(ctypes.byref(p), int(num_pages)))


def alloc_means_cache(p: Params, num_pages: int, device="cuda"):
    """(khat, vbar) bf16 [slots, Hkv, 128] for fp2_prefill_cached."""
    import torch
    n = means_cache_slots(p, num_pages)
    if n == 0:
        raise ValueError("no means-cache slots for this configuration: " + last_error())
    shape = (n, p.num_kv_heads, p.head_dim)
    return (torch.zeros(shape, dtype=torch.bfloat16, device=device),
            torch.zeros(shape, dtype=torch.bfloat16, device=device))


def estimate(p: Params, q, k_cache, v_cache, cu_seqlens, block_table=None, *,
             cu_seqlens_host=None, cu_seqlens_k=None, cu_seqlens_k_host=None, q_scale=None,
             k_scale=None, v_scale=None, block_mask=None, workspace=None, stream=None):
    """fp2_estimate: returns (block_mask, workspace)."""
    if block_mask is None:
        block_mask = alloc_mask(p, q.device)
    if workspace is None:
        workspace = alloc_workspace(p, q.device)
    _check_inputs(p, q, k_cache, v_cache, cu_seqlens, block_table, cu_seqlens_k, q_scale,
                  k_scale, v_scale, block_mask=block_mask, workspace=workspace)
    st = lib().fp2_estimate(ctypes.byref(p), _ptr(q), _ptr(cu_seqlens), _host_ptr(cu_seqlens_host),
                            _ptr(cu_seqlens_k), _host_ptr(cu_seqlens_k_host), _ptr(k_cache),
                            _ptr(v_cache), _ptr(block_table), _ptr(q_scale), _ptr(k_scale),
                            _ptr(v_scale), _ptr(block_mask), _ptr(workspace),
                            workspace.numel(), _stream(stream))
    _check("fp2_estimate", st)
    return block_mask, workspace


def attend(p: Params, q, k_cache, v_cache, cu_seqlens, block_mask, block_table=None, *,
           cu_seqlens_host=None, cu_seqlens_k=None, cu_seqlens_k_host=None, q_scale=None,
           k_scale=None, v_scale=None, out=None, lse=None, workspace=None, want_lse=False,
           stream=None):
    """fp2_attend under ``block_mask`` (bit 0 = kept): returns (out, lse or None)."""
    if out is None:
        out = torch.empty((q.shape[0], p.num_q_heads, p.head_dim), dtype=torch.bfloat16,
                          device=q.device)
    if lse is None and want_lse:
        lse = torch.empty((q.shape[0], p.num_q_heads), dtype=torch.float32, device=q.device)
    if workspace is None:
        workspace = alloc_workspace(p, q.device)
    _check_inputs(p, q, k_cache, v_cache, cu_seqlens, block_table, cu_seqlens_k, q_scale,
                  k_scale, v_scale, out, lse, workspace=workspace, mask_in=block_mask)
    st = lib().fp2_attend(ctypes.byref(p), _ptr(q), _ptr(cu_seqlens), _host_ptr(cu_seqlens_host),
                          _ptr(cu_seqlens_k), _host_ptr(cu_seqlens_k_host), _ptr(k_cache),
                          _ptr(v_cache), _ptr(block_table), _ptr(q_scale), _ptr(k_scale),
                          _ptr(v_scale), _ptr(block_mask), _ptr(out), _ptr(lse),
                          _ptr(workspace), workspace.numel(), _stream(stream))
    _check("fp2_attend", st)
    return out, lse


def pool(p: Params, k_cache, v_cache, cu_seqlens, block_table=None, *, cu_seqlens_host=None,
         k_scale=None, v_scale=None, stream=None):
    """fp2_pool over the KV lengths cu_seqlens: returns (khat, vbar) as bf16
    [batch, Hkv, nbk, 128]."""
    nb = max(1, num_key_blocks(p))
    shape = (p.batch, p.num_kv_heads, nb, p.head_dim)
    khat = torch.empty(shape, dtype=torch.bfloat16, device=k_cache.device)
    vbar = torch.empty(shape, dtype=torch.bfloat16, device=k_cache.device)
    _check_inputs(p, k_cache=k_cache, v_cache=v_cache, cu_seqlens=cu_seqlens,
                  block_table=block_table, k_scale=k_scale, v_scale=v_scale)
    st = lib().fp2_pool(ctypes.byref(p), _ptr(cu_seqlens), _host_ptr(cu_seqlens_host),
                        _ptr(k_cache), _ptr(v_cache), _ptr(block_table), _ptr(k_scale),
                        _ptr(v_scale), _ptr(khat), _ptr(vbar), _stream(stream))
    _check("fp2_pool", st)
    return khat, vbar


def csr_capacity(p: Params) -> int:
    return int(lib().fp2_csr_capacity(ctypes.byref(p)))


def calibrate(kind: str, iters: int, sink=None, stream=None) -> float:
    """fp2_calibrate: enqueue one rate-calibration loop ("mfma_bf16",
    "mfma_fp8" or "exp") and return the operations it performs (FLOP or
    exps); time it on the stream to get the rate. sink: a device float32
    tensor of at least one element (allocated when None)."""
    if kind not in CALIB_KINDS:
        raise ValueError("calibration kind %r not in %s" % (kind, sorted(CALIB_KINDS)))
    if sink is None:
        sink = torch.zeros(1, dtype=torch.float32, device="cuda")
    if not (isinstance(sink, torch.Tensor) and sink.is_cuda and sink.dtype == torch.float32
            and sink.numel() >= 1):
        raise ValueError("sink must be a CUDA float32 tensor of at least one element")
    ops = ctypes.c_double(0.0)
    st = lib().fp2_calibrate(CALIB_KINDS[kind], int(iters), _ptr(sink), ctypes.byref(ops),
                             _stream(stream))
    _check("fp2_calibrate", st)
    return ops.value


def mask_to_csr(p: Params, block_mask, cu_seqlens, *, cu_seqlens_k=None, cu_seqlens_host=None,
                cu_seqlens_k_host=None, workspace=None, stream=None):
    """fp2_mask_to_csr: returns (offsets int32 [nseg + 1], indices int32 [capacity]);
    the index has offsets[-1] valid entries."""
    nseg = p.batch * p.num_kv_heads * max(1, num_blocks(p))
    offsets = torch.empty(nseg + 1, dtype=torch.int32, device=block_mask.device)
    cap = max(1, csr_capacity(p))
    indices = torch.empty(cap, dtype=torch.int32, device=block_mask.device)
    if workspace is None:
        workspace = alloc_workspace(p, block_mask.device)
    st = lib().fp2_mask_to_csr(ctypes.byref(p), _ptr(cu_seqlens), _host_ptr(cu_seqlens_host),
                               _ptr(cu_seqlens_k), _host_ptr(cu_seqlens_k_host), _ptr(block_mask),
                               _ptr(offsets), _ptr(indices), cap, _ptr(workspace),
                               workspace.numel(), _stream(stream))
    _check("fp2_mask_to_csr", st)
    return offsets, indices
