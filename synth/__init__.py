"""Seeded synthetic workloads for block-sparse causal GQA prefill attention.

This module only draws inputs. It holds none of the method's arithmetic: it
draws Gaussian Q, K and V, plants salient key blocks and biased query blocks,
casts to the storage dtype (bf16, or OCP e4m3fn with per-head absmax scales)
and lays K/V out in a paged token pool. Both the GPU path (tests, bench) and
the CPU oracle consume exactly these arrays.

Every random draw comes from its own ``numpy.random.default_rng([seed, tag,
...])`` stream (PCG64 seeded through SeedSequence), so the data do not depend
on how many threads generate them or in which order:

* tag 1/2/3: Q/K/V values of sequence b, in chunks of ``_CHUNK`` tokens,
  N(0, 1) in float32;
* tag 4: one direction ``u_h`` per KV head, a normalised N(0, I) vector;
* tag 5: salient key blocks of (sequence b, KV head h): block 0 plus
  ``count`` distinct blocks drawn from ``[1, n)``;
* tag 6: sequence lengths (ragged batches), log-uniform;
* tag 7: page permutation of the shared pool (permuted page tables).

Planted structure: every key of a salient block of KV head h gets
``key_bias * u_h`` added; every query head of group h gets ``query_bias *
u_h`` in even-indexed query blocks. This reproduces the block-sparse score
pattern (vertical stripes plus locality) that the paper's needle-in-a-haystack
inputs induce, without using any of those inputs.
"""
from __future__ import annotations

import concurrent.futures as _cf
import dataclasses
import json
import math
import os
from typing import List, Optional

import numpy as np

_CHUNK = 1024
_BF16_NAN = 0x7FC0
_E4M3_NAN = 0x7F
E4M3_MAX = 448.0


def _threads() -> int:
    try:
        n = len(os.sched_getaffinity(0))
    except AttributeError:  # pragma: no cover
        n = os.cpu_count() or 1
    return max(1, min(16, n))


@dataclasses.dataclass
class Spec:
    """One synthetic workload: shapes, layout, planted structure, selection knobs."""
    name: str
    seqlens: List[int]
    num_q_heads: int
    num_kv_heads: int
    head_dim: int = 128
    block_size: int = 128
    dtype: str = "bf16"            # "bf16" | "fp8"
    page_size: int = 64            # 0: contiguous KV in the q layout
    page_order: str = "identity"   # "identity" | "permuted"
    pool_pages: int = 0            # pages in the shared pool (permuted order)
    salient_frac: float = 0.01     # fraction of key blocks planted per (b, h)
    salient_min: int = 1
    key_bias: float = 3.0
    query_bias: float = 2.0
    sink_blocks: int = 1
    window_blocks: int = 2
    recent_blocks: int = 0
    mean_correction: int = 1
    seed: int = 0
    # KV tokens before the queries of each sequence (chunked prefill, prefix
    # caching): the queries are the last seqlens[b] of prefix[b] + seqlens[b]
    # KV tokens; None = no prefix.
    prefix: Optional[List[int]] = None

    @property
    def batch(self) -> int:
        return len(self.seqlens)

    @property
    def total_tokens(self) -> int:
        return int(sum(self.seqlens))

    @property
    def max_seq_len(self) -> int:
        return int(max(self.seqlens)) if self.seqlens else 0

    @property
    def prefixes(self) -> List[int]:
        return list(self.prefix) if self.prefix is not None else [0] * self.batch

    @property
    def kvlens(self) -> List[int]:
        return [int(p + L) for p, L in zip(self.prefixes, self.seqlens)]

    @property
    def total_kv_tokens(self) -> int:
        return int(sum(self.kvlens))

    @property
    def max_kv_len(self) -> int:
        return int(max(self.kvlens)) if self.seqlens else 0

    def replace(self, **kw) -> "Spec":
        return dataclasses.replace(self, **kw)


def _normal(seed: int, tag: int, b: int, out: np.ndarray) -> None:
    """Fill ``out`` [rows, heads, d] (float32) with N(0,1), drawn in fixed-size
    token chunks (chunk c from stream [seed, tag, b, c])."""
    rows, heads, d = out.shape
    nchunks = (rows + _CHUNK - 1) // _CHUNK

    def fill(c: int) -> None:
        r0, r1 = c * _CHUNK, min(rows, (c + 1) * _CHUNK)
        g = np.random.default_rng([seed, tag, b, c])
        g.standard_normal((r1 - r0, heads, d), dtype=np.float32, out=out[r0:r1])

    if nchunks <= 1:
        for c in range(nchunks):
            fill(c)
    else:
        with _cf.ThreadPoolExecutor(_threads()) as ex:
            list(ex.map(fill, range(nchunks)))


def ragged_lengths(seed: int, batch: int, lo: int, hi: int) -> List[int]:
    """Lengths floor(exp(U(ln lo, ln hi))) drawn from stream tag 6."""
    g = np.random.default_rng([seed, 6])
    x = g.uniform(math.log(lo), math.log(hi), size=batch)
    return [int(math.floor(math.exp(v))) for v in x]


def _to_bf16_bits(x: np.ndarray) -> np.ndarray:
    import torch
    t = torch.from_numpy(np.ascontiguousarray(x)).to(torch.bfloat16)
    return t.view(torch.int16).numpy().view(np.uint16)


def _to_e4m3_bits(x: np.ndarray) -> np.ndarray:
    import torch
    t = torch.from_numpy(np.ascontiguousarray(x)).to(torch.float8_e4m3fn)
    return t.view(torch.uint8).numpy()


@dataclasses.dataclass
class Workload:
    """Host arrays of one generated workload (storage-dtype bit patterns).

    q: [total, Hq, d] (the query tokens, sequence b at rows cu[b]..cu[b+1]);
    k_tok/v_tok: [total_kv, Hkv, d] (the KV tokens, sequence b at rows
    cu_k[b]..cu_k[b+1]); scales are float32 per head (all ones for bf16).
    block_table: int32 [batch, max_pages] giving, for page j of sequence b, its
    index in a pool of ``num_pages`` pages of ``page_size`` tokens.
    """
    spec: Spec
    q: np.ndarray
    k_tok: np.ndarray
    v_tok: np.ndarray
    q_scale: np.ndarray
    k_scale: np.ndarray
    v_scale: np.ndarray
    cu_seqlens: np.ndarray
    block_table: np.ndarray
    num_pages: int
    salient: List[List[np.ndarray]]
    cu_seqlens_k: Optional[np.ndarray] = None

    def __post_init__(self):
        if self.cu_seqlens_k is None:
            self.cu_seqlens_k = self.cu_seqlens

    @property
    def max_pages(self) -> int:
        return int(self.block_table.shape[1])

    @property
    def nan_bits(self) -> int:
        return _E4M3_NAN if self.spec.dtype == "fp8" else _BF16_NAN

    def slots(self) -> np.ndarray:
        """Pool slot of every KV token (Eq. page addressing), int64 [total_kv]."""
        sp = self.spec
        cu = self.cu_seqlens_k
        out = np.empty(sp.total_kv_tokens, dtype=np.int64)
        for b, L in enumerate(sp.kvlens):
            j = np.arange(L, dtype=np.int64)
            if sp.page_size == 0:
                out[cu[b]:cu[b + 1]] = cu[b] + j
            else:
                p = sp.page_size
                out[cu[b]:cu[b + 1]] = self.block_table[b, j // p].astype(np.int64) * p + j % p
        return out

    def host_pool(self, which: str, compact: bool = True):
        """Paged K or V pool on the host; unused slots hold NaN.

        With ``compact`` the pool keeps only the pages the table references,
        renumbered in first-use order, and a matching table is returned.
        Returns (pool [slots, Hkv, d], block_table).
        """
        sp = self.spec
        tok = self.k_tok if which == "k" else self.v_tok
        if sp.page_size == 0:
            return tok, self.block_table
        bt = self.block_table
        if compact:
            used = []
            for b, L in enumerate(sp.kvlens):
                used.extend(bt[b, : (L + sp.page_size - 1) // sp.page_size].tolist())
            remap = {pg: i for i, pg in enumerate(dict.fromkeys(used))}
            bt2 = np.zeros_like(bt)
            for b, L in enumerate(sp.kvlens):
                n = (L + sp.page_size - 1) // sp.page_size
                bt2[b, :n] = [remap[x] for x in bt[b, :n]]
            npages = max(1, len(remap))
        else:
            bt2, npages = bt, self.num_pages
        pool = np.full((npages * sp.page_size,) + tok.shape[1:], self.nan_bits, dtype=tok.dtype)
        sl = np.empty(sp.total_kv_tokens, dtype=np.int64)
        cu = self.cu_seqlens_k
        for b, L in enumerate(sp.kvlens):
            j = np.arange(L, dtype=np.int64)
            sl[cu[b]:cu[b + 1]] = bt2[b, j // sp.page_size].astype(np.int64) * sp.page_size + j % sp.page_size
        pool[sl] = tok
        return pool, bt2

    def device_inputs(self, device="cuda"):
        """Torch tensors on ``device``: the full pool (NaN-poisoned), table, lengths, scales."""
        import torch
        sp = self.spec
        tdt = torch.uint8 if sp.dtype == "fp8" else torch.int16
        q = torch.from_numpy(self.q.view(np.uint8 if sp.dtype == "fp8" else np.int16)).to(device)
        ktok = torch.from_numpy(self.k_tok.view(np.uint8 if sp.dtype == "fp8" else np.int16)).to(device)
        vtok = torch.from_numpy(self.v_tok.view(np.uint8 if sp.dtype == "fp8" else np.int16)).to(device)
        if sp.page_size == 0:
            kc, vc = ktok, vtok
        else:
            nan = self.nan_bits if sp.dtype == "fp8" else np.int16(np.uint16(_BF16_NAN).view(np.int16)).item()
            shape = (self.num_pages * sp.page_size, sp.num_kv_heads, sp.head_dim)
            kc = torch.full(shape, nan, dtype=tdt, device=device)
            vc = torch.full(shape, nan, dtype=tdt, device=device)
            idx = torch.from_numpy(self.slots()).to(device)
            kc.index_copy_(0, idx, ktok)
            vc.index_copy_(0, idx, vtok)
            del ktok, vtok
        return dict(
            q=q, k_cache=kc, v_cache=vc,
            block_table=torch.from_numpy(self.block_table).to(device),
            cu_seqlens=torch.from_numpy(self.cu_seqlens).to(device),
            cu_seqlens_k=(None if self.spec.prefix is None
                          else torch.from_numpy(self.cu_seqlens_k).to(device)),
            q_scale=torch.from_numpy(self.q_scale).to(device),
            k_scale=torch.from_numpy(self.k_scale).to(device),
            v_scale=torch.from_numpy(self.v_scale).to(device),
        )


def generate(spec: Spec) -> Workload:
    """Draw the workload described by ``spec`` (deterministic in ``spec.seed``)."""
    sp = spec
    d, B, Hq, Hkv = sp.head_dim, sp.block_size, sp.num_q_heads, sp.num_kv_heads
    assert Hq % Hkv == 0
    g = Hq // Hkv
    seed = sp.seed
    pre = sp.prefixes
    assert all(x >= 0 for x in pre), "prefix lengths must be non-negative"
    kvl = sp.kvlens
    # Q, K and V are drawn for all KV positions of a sequence; Q then keeps
    # its last seqlens[b] rows, so a chunk reproduces the rows of the whole
    cu = np.zeros(sp.batch + 1, dtype=np.int32)
    cu[1:] = np.cumsum(kvl)
    total = int(cu[-1])

    ug = np.random.default_rng([seed, 4])
    u = ug.standard_normal((Hkv, d))
    u /= np.linalg.norm(u, axis=1, keepdims=True)
    u = u.astype(np.float32)

    import torch
    qf = np.empty((total, Hq, d), dtype=np.float32)
    kf = np.empty((total, Hkv, d), dtype=np.float32)
    vf = np.empty((total, Hkv, d), dtype=np.float32)
    qt, kt = torch.from_numpy(qf), torch.from_numpy(kf)
    # query bias pattern: head hq of group h gets query_bias * u_h
    qbias = torch.from_numpy(np.repeat(sp.query_bias * u, g, axis=0))          # [Hq, d]
    salient: List[List[np.ndarray]] = []
    for b, L in enumerate(kvl):
        s0 = int(cu[b])
        if L == 0:
            salient.append([np.zeros(0, dtype=np.int64) for _ in range(Hkv)])
            continue
        _normal(seed, 1, b, qf[s0:s0 + L])
        _normal(seed, 2, b, kf[s0:s0 + L])
        _normal(seed, 3, b, vf[s0:s0 + L])
        n = (L + B - 1) // B
        per_head = []
        for h in range(Hkv):
            cnt = min(n - 1, max(sp.salient_min, int(round(sp.salient_frac * n))))
            sg = np.random.default_rng([seed, 5, b, h])
            pick = (sg.choice(n - 1, size=cnt, replace=False) + 1) if cnt > 0 else np.zeros(0, dtype=np.int64)
            blocks = np.sort(np.concatenate([[0], pick])).astype(np.int64)
            per_head.append(blocks)
            kb = torch.from_numpy(sp.key_bias * u[h])
            for J in blocks:
                kt[s0 + J * B: s0 + min(L, (J + 1) * B), h, :] += kb
        # even-indexed query blocks: whole pairs of blocks, then the tail
        full = (L // (2 * B)) * 2 * B
        if full:
            qt[s0:s0 + full].view(full // (2 * B), 2, B, Hq, d)[:, 0] += qbias
        if full < L:
            qt[s0 + full:s0 + min(L, full + B)] += qbias
        salient.append(per_head)

    # query rows: the last seqlens[b] positions of every sequence
    cu_q = np.zeros(sp.batch + 1, dtype=np.int32)
    cu_q[1:] = np.cumsum(sp.seqlens)
    if sp.prefix is not None:
        rows = np.concatenate([np.arange(cu[b] + pre[b], cu[b + 1]) for b in range(sp.batch)]
                              + [np.zeros(0, np.int64)]).astype(np.int64)
    else:
        rows = None

    if sp.dtype == "bf16":
        q, k, v = _to_bf16_bits(qf), _to_bf16_bits(kf), _to_bf16_bits(vf)
        qs = np.ones(Hq, dtype=np.float32)
        ks = np.ones(Hkv, dtype=np.float32)
        vs = np.ones(Hkv, dtype=np.float32)
    elif sp.dtype == "fp8":
        def quant(x):
            t = torch.from_numpy(x)
            if x.shape[0]:
                amax = t.abs().amax(dim=(0, 2)).numpy()
            else:
                amax = np.ones(x.shape[1], np.float32)
            sc = (np.maximum(amax, 1e-30) / E4M3_MAX).astype(np.float32)
            y = (t / torch.from_numpy(sc)[None, :, None]).clamp_(-E4M3_MAX, E4M3_MAX)
            return y.to(torch.float8_e4m3fn).view(torch.uint8).numpy(), sc
        q, qs = quant(qf)
        k, ks = quant(kf)
        v, vs = quant(vf)
    else:
        raise ValueError(sp.dtype)
    del qf, kf, vf, qt, kt
    if rows is not None:
        q = np.ascontiguousarray(q[rows])

    if sp.page_size > 0:
        p = sp.page_size
        npg = [(L + p - 1) // p for L in kvl]
        max_pages = max(1, max(npg) if npg else 1)
        bt = np.zeros((sp.batch, max_pages), dtype=np.int32)
        if sp.page_order == "identity":
            off = 0
            for b, m in enumerate(npg):
                bt[b, :m] = np.arange(off, off + m)
                off += m
            num_pages = max(1, off)
        elif sp.page_order == "permuted":
            num_pages = sp.pool_pages
            assert num_pages >= sum(npg)
            perm = np.random.default_rng([seed, 7]).permutation(num_pages).astype(np.int32)
            off = 0
            for b, m in enumerate(npg):
                bt[b, :m] = perm[off:off + m]
                off += m
            # unused table entries point at a page no sequence owns (NaN-poisoned)
            spare = perm[off] if off < num_pages else 0
            for b, m in enumerate(npg):
                bt[b, m:] = spare
        else:
            raise ValueError(sp.page_order)
    else:
        bt = np.zeros((sp.batch, 1), dtype=np.int32)
        num_pages = 0
    return Workload(sp, q, k, v, qs, ks, vs, cu_q, bt, num_pages, salient,
                    cu_seqlens_k=cu if sp.prefix is not None else None)


# ---------------------------------------------------------------------------
# The five named workloads: shapes, layouts and selection knobs.
# ---------------------------------------------------------------------------

def named(name: str, seed: int = 0) -> Spec:
    """Named workload specs: the synthetic layers the tests and the benchmark run."""
    if name == "tiny2k":
        return Spec(name, [2048], 4, 1, dtype="bf16", page_size=0, salient_frac=0.0,
                    salient_min=3, sink_blocks=1, window_blocks=1, seed=seed)
    if name == "llama32k":
        return Spec(name, [32768], 32, 8, dtype="bf16", page_size=64, salient_frac=0.01,
                    salient_min=1, sink_blocks=1, window_blocks=2, seed=seed)
    if name == "llama128k_fp8":
        return Spec(name, [131072], 32, 8, dtype="fp8", page_size=64, salient_frac=0.01,
                    salient_min=1, sink_blocks=1, window_blocks=2, seed=seed)
    if name == "llama128k_bf16":
        return Spec(name, [131072], 32, 8, dtype="bf16", page_size=64, salient_frac=0.01,
                    salient_min=1, sink_blocks=1, window_blocks=2, seed=seed)
    if name == "ragged8":
        lens = ragged_lengths(seed, 8, 4096, 65536)
        return Spec(name, lens, 32, 8, dtype="bf16", page_size=64, page_order="permuted",
                    pool_pages=1 << 16, salient_frac=0.01, salient_min=1, sink_blocks=1,
                    window_blocks=2, seed=seed)
    if name == "wide128k_bf16":
        return Spec(name, [131072], 64, 8, dtype="bf16", page_size=64, salient_frac=0.005,
                    salient_min=1, sink_blocks=1, window_blocks=2, seed=seed)
    if name == "wide128k_fp8":
        return Spec(name, [131072], 64, 8, dtype="fp8", page_size=64, salient_frac=0.005,
                    salient_min=1, sink_blocks=1, window_blocks=2, seed=seed)
    raise KeyError(name)


NAMES = ["tiny2k", "llama32k", "llama128k_fp8", "llama128k_bf16", "ragged8",
         "wide128k_bf16", "wide128k_fp8"]

_ALPHA_FILE = os.path.join(os.path.dirname(__file__), "alpha.json")


def alphas() -> dict:
    """Calibrated thresholds: {workload name: {target kept ratio (str): alpha}}."""
    if not os.path.exists(_ALPHA_FILE):
        return {}
    with open(_ALPHA_FILE) as f:
        return json.load(f)


def alpha_for(name: str, target: str) -> float:
    a = alphas()
    return float(a[name]["alpha"][target])
