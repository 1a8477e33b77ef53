"""CPU oracle (fp64, plain C) for block-sparse causal GQA prefill attention.

TEST INFRASTRUCTURE ONLY: the tests, ``__graft_entry__.smoke()`` and the CPU
baseline leg of ``bench.py`` use it to judge the GPU library. The product path
never imports it. The C source is ``oracle.c``; its header comment states,
step by step, what is computed and which passage of the paper each step
follows (Sec. 3.1 Eq. (1)-(2), Eq. select, Sec. 3.2 Eq. correction, Sec. 3.3
Eq. page and Eq. fp8).

Pinned by the ``-m "not gpu"`` tests in ``tests/test_oracle_*.py``.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_DIR = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_DIR, "oracle.c")
_LIB = os.path.join(_DIR, "liboracle.so")
_lib = None


def build(force: bool = True) -> str:
    """Compile ``liboracle.so`` with gcc (plain -O2, no fast-math)."""
    if force or not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
        tmp = _LIB + ".tmp%d" % os.getpid()
        subprocess.check_call(["gcc", "-O2", "-std=c11", "-fPIC", "-shared", "-pthread",
                               "-Wall", "-Wextra", "-Wno-unused-parameter",
                               _SRC, "-o", tmp, "-lm"])
        os.replace(tmp, _LIB)
    return _LIB


class Params(ctypes.Structure):
    _fields_ = [
        ("batch", ctypes.c_int32), ("num_q_heads", ctypes.c_int32),
        ("num_kv_heads", ctypes.c_int32), ("head_dim", ctypes.c_int32),
        ("block_size", ctypes.c_int32), ("page_size", ctypes.c_int32),
        ("max_seq_len", ctypes.c_int32), ("max_pages_per_seq", ctypes.c_int32),
        ("alpha", ctypes.c_double),
        ("sink_blocks", ctypes.c_int32), ("window_blocks", ctypes.c_int32),
        ("recent_blocks", ctypes.c_int32), ("mean_correction", ctypes.c_int32),
        ("softmax_scale", ctypes.c_double),
        ("dtype", ctypes.c_int32), ("nthreads", ctypes.c_int32),
        ("max_kv_len", ctypes.c_int32), ("tile_rows", ctypes.c_int32),
    ]


def _load():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
            build(force=True)
        lib = ctypes.CDLL(_LIB)
        vp = ctypes.c_void_p
        lib.oracle_bf16_decode.restype = ctypes.c_double
        lib.oracle_bf16_decode.argtypes = [ctypes.c_uint16]
        lib.oracle_bf16_encode_rne.restype = ctypes.c_uint16
        lib.oracle_bf16_encode_rne.argtypes = [ctypes.c_double]
        lib.oracle_e4m3_decode.restype = ctypes.c_double
        lib.oracle_e4m3_decode.argtypes = [ctypes.c_uint8]
        P = ctypes.POINTER(Params)
        lib.oracle_pool.argtypes = [P] + [vp] * 9
        lib.oracle_estimate.argtypes = [P] + [vp] * 9 + [vp, ctypes.c_int, vp, vp, vp]
        lib.oracle_attend.argtypes = [P] + [vp] * 9 + [vp, vp, ctypes.c_int, vp, vp]
        for f in (lib.oracle_pool, lib.oracle_estimate, lib.oracle_attend):
            f.restype = ctypes.c_int
        _lib = lib
    return _lib


def nthreads_default() -> int:
    try:
        n = len(os.sched_getaffinity(0))
    except AttributeError:  # pragma: no cover
        n = os.cpu_count() or 1
    return max(1, min(16, n))


def bf16_decode(bits: int) -> float:
    return _load().oracle_bf16_decode(int(bits))


def bf16_encode_rne(x: float) -> int:
    return int(_load().oracle_bf16_encode_rne(float(x)))


def e4m3_decode(bits: int) -> float:
    return _load().oracle_e4m3_decode(int(bits))


def _ptr(a):
    return None if a is None else a.ctypes.data_as(ctypes.c_void_p)


class Inputs:
    """Host arrays in the layout the oracle reads (see oracle.c)."""

    def __init__(self, wl, compact=True):
        sp = wl.spec
        self.spec = sp
        self.q = np.ascontiguousarray(wl.q)
        k, bt = wl.host_pool("k", compact=compact)
        v, _ = wl.host_pool("v", compact=compact)
        self.k = np.ascontiguousarray(k)
        self.v = np.ascontiguousarray(v)
        self.bt = np.ascontiguousarray(bt, dtype=np.int32)
        self.cu = np.ascontiguousarray(wl.cu_seqlens, dtype=np.int32)
        self.cu_k = np.ascontiguousarray(wl.cu_seqlens_k, dtype=np.int32)
        self.qs = np.ascontiguousarray(wl.q_scale, dtype=np.float32)
        self.ks = np.ascontiguousarray(wl.k_scale, dtype=np.float32)
        self.vs = np.ascontiguousarray(wl.v_scale, dtype=np.float32)

    def params(self, alpha, sink=None, window=None, recent=None, correction=None,
               softmax_scale=0.0, nthreads=None, tile_rows=0) -> Params:
        """tile_rows: packed rows per query tile (0: a query block of B
        positions with all g heads)."""
        sp = self.spec
        return Params(
            batch=sp.batch, num_q_heads=sp.num_q_heads, num_kv_heads=sp.num_kv_heads,
            head_dim=sp.head_dim, block_size=sp.block_size, page_size=sp.page_size,
            max_seq_len=sp.max_seq_len, max_pages_per_seq=int(self.bt.shape[1]),
            alpha=float(alpha),
            sink_blocks=sp.sink_blocks if sink is None else sink,
            window_blocks=sp.window_blocks if window is None else window,
            recent_blocks=sp.recent_blocks if recent is None else recent,
            mean_correction=sp.mean_correction if correction is None else int(correction),
            softmax_scale=float(softmax_scale),
            dtype=1 if sp.dtype == "fp8" else 0,
            nthreads=nthreads_default() if nthreads is None else nthreads,
            max_kv_len=sp.max_kv_len, tile_rows=int(tile_rows))

    @property
    def nbmax(self):
        """Query blocks (mask rows with the default tile)."""
        sp = self.spec
        return (sp.max_seq_len + sp.block_size - 1) // sp.block_size

    def tile_positions(self, p: Params) -> int:
        """Positions per query tile under ``p``."""
        sp = self.spec
        g = sp.num_q_heads // sp.num_kv_heads
        return p.tile_rows // g if p.tile_rows > 0 else sp.block_size

    def ntiles(self, p: Params) -> int:
        """Query tiles per sequence bound (mask rows) under ``p``."""
        pt = self.tile_positions(p)
        return (self.spec.max_seq_len + pt - 1) // pt

    @property
    def nbk(self):
        """Key blocks (mask columns, pooled rows)."""
        sp = self.spec
        return (sp.max_kv_len + sp.block_size - 1) // sp.block_size

    def _args(self):
        return [_ptr(self.q), _ptr(self.cu), _ptr(self.cu_k), _ptr(self.k), _ptr(self.v),
                _ptr(self.bt), _ptr(self.qs), _ptr(self.ks), _ptr(self.vs)]


def _units_arr(units):
    if units is None:
        return None, 0
    u = np.ascontiguousarray(np.asarray(units, dtype=np.int32).reshape(-1, 3))
    return u, int(u.shape[0])


def pool(inp: Inputs, p: Params):
    """Block means kbar, vbar (fp64) and the bf16 scoring key bits khat."""
    sp = inp.spec
    shape = (sp.batch, sp.num_kv_heads, max(1, inp.nbk), sp.head_dim)
    kbar = np.zeros(shape, np.float64)
    vbar = np.zeros(shape, np.float64)
    khat = np.zeros(shape, np.uint16)
    rc = _load().oracle_pool(ctypes.byref(p), _ptr(inp.k), _ptr(inp.v), _ptr(inp.bt),
                             _ptr(inp.cu_k), _ptr(inp.ks), _ptr(inp.vs), _ptr(kbar), _ptr(vbar),
                             _ptr(khat))
    assert rc == 0
    return kbar, vbar, khat


def estimate(inp: Inputs, p: Params, units=None, want_scores=False):
    """Mask [b, Hkv, nbq, nbk] (uint8: bit0 kept, bit1 forced) and optionally
    ell [b, Hkv, nbq, nbk] (block log-energies, NaN past the diagonal) and
    mu [b, Hkv, nbq] (row maxima). Without a prefix nbq == nbk."""
    sp = inp.spec
    nb, nk = max(1, inp.ntiles(p)), max(1, inp.nbk)
    mask = np.zeros((sp.batch, sp.num_kv_heads, nb, nk), np.uint8)
    ell = np.full((sp.batch, sp.num_kv_heads, nb, nk), np.nan) if want_scores else None
    mu = np.full((sp.batch, sp.num_kv_heads, nb), np.nan) if want_scores else None
    u, nu = _units_arr(units)
    rc = _load().oracle_estimate(ctypes.byref(p), *inp._args(), _ptr(u), nu, _ptr(mask),
                                 _ptr(ell), _ptr(mu))
    assert rc == 0
    return (mask, ell, mu) if want_scores else mask


def attend(inp: Inputs, p: Params, mask, units=None):
    """fp64 output [total, Hq, d] and LSE [total, Hq] under ``mask`` (bit0 = kept).
    Rows of units not computed are NaN."""
    sp = inp.spec
    mask = np.ascontiguousarray(mask, dtype=np.uint8)
    out = np.full((sp.total_tokens, sp.num_q_heads, sp.head_dim), np.nan)
    lse = np.full((sp.total_tokens, sp.num_q_heads), np.nan)
    u, nu = _units_arr(units)
    rc = _load().oracle_attend(ctypes.byref(p), *inp._args(), _ptr(mask), _ptr(u), nu,
                               _ptr(out), _ptr(lse))
    assert rc == 0
    return out, lse


def margins(ell, mu, alpha):
    """Relative distance of each block energy from the threshold:
    E_J / (alpha * max E) - 1 = expm1(ell - ln(alpha) - mu); NaN above the diagonal."""
    return np.expm1(ell - np.log(alpha) - mu[..., None])


def kept_ratio(mask, seqlens, block_size, prefix=None):
    """Kept blocks over block-causal pairs (J <= absolute query block), over
    all (b, h)."""
    kept = 0
    tot = 0
    for b, L in enumerate(seqlens):
        n = (L + block_size - 1) // block_size
        off = 0 if prefix is None else prefix[b] // block_size
        kept += int((mask[b, :, :n, :] & 1).sum())
        tot += mask.shape[1] * sum(off + I + 1 for I in range(n))
    return kept / max(1, tot)
