"""Serving-engine attention backend for the extend (prefill) phase.

The shape a continuous-batching engine needs around fp2_prefill (Sec. 4: the
sparse operator serves every extend of a request, chunked prefill included,
while decode attention stays dense):

- ``BackendConfig``: the engine-level settings, fixed at start-up (head
  counts, page size, the per-forward bounds that size the buffers, the
  selection and correction settings).
- ``PrefillBackend``: one per stream. It owns a workspace and a block-mask
  buffer sized for the largest forward the config admits, allocated once and
  reused by every layer of every forward (the library never allocates).
- ``ForwardMetadata``: built once per forward by ``init_forward_metadata``
  from the extend lengths, the cached-prefix lengths and the page table, and
  shared by all layers: the length arrays are uploaded to the device once.
- ``forward_extend``: one layer's attention over the paged cache, through the
  C ABI. The K/V of the new tokens must already be in the cache.
- Block means across forwards: ``alloc_means_cache`` gives a layer's cache of
  pooled key/value means (one slot per 128-token block of the paged pool,
  about 2/(page * bytes per element) of the KV cache). Passed to
  ``forward_extend``, a forward pools only the blocks that are new or were
  incomplete, and copies the complete blocks of the cached prefix, whose
  means an earlier forward through the same cache wrote (chunked prefill, or
  prefix pages shared between requests).

Cached prefixes may have any length (a prefix-cache hit is page-granular);
``plan_forward`` checks the lengths against the configured bounds before
anything reaches the GPU.
"""
from __future__ import annotations

import dataclasses
from typing import List, Optional, Sequence

import numpy as np

import paper_2608_19758_amd as fp2

BLOCK = fp2.BLOCK


@dataclasses.dataclass(frozen=True)
class BackendConfig:
    num_q_heads: int
    num_kv_heads: int
    page_size: int                 # tokens per KV page (> 0: paged pool)
    max_batch: int                 # sequences per forward
    max_extend_len: int            # new tokens of one sequence in one forward
    max_kv_len: int                # cached + new tokens of one sequence
    dtype: str = "bf16"            # "bf16" | "fp8"
    alpha: float = 0.1
    sink_blocks: int = 2
    window_blocks: int = 4
    recent_blocks: int = 0
    mean_correction: bool = True
    kv_splits: int = 0             # 0: cost-balanced plan on the device
    softmax_scale: float = 0.0     # <= 0: 1/sqrt(128)
    query_tile_rows: int = 0       # 0: query blocks of 128 positions; 128: 128-row tiles
    score_splits: int = 0          # 0: rows of few units split over workgroups; 1: never

    @property
    def max_pages_per_seq(self) -> int:
        return (self.max_kv_len + self.page_size - 1) // self.page_size

    def params(self, batch: int, max_extend: int, max_kv: int) -> "fp2.Params":
        return fp2.make_params(
            batch=batch, num_q_heads=self.num_q_heads, num_kv_heads=self.num_kv_heads,
            max_seq_len=max_extend, page_size=self.page_size,
            max_pages_per_seq=self.max_pages_per_seq, alpha=self.alpha,
            sink_blocks=self.sink_blocks, window_blocks=self.window_blocks,
            recent_blocks=self.recent_blocks, mean_correction=int(self.mean_correction),
            softmax_scale=self.softmax_scale, dtype=self.dtype, max_kv_len=max_kv,
            kv_splits=self.kv_splits, query_tile_rows=self.query_tile_rows,
            score_splits=self.score_splits)

    def worst_case_params(self) -> "fp2.Params":
        return self.params(self.max_batch, self.max_extend_len, self.max_kv_len)


@dataclasses.dataclass
class ForwardPlan:
    """Host part of a forward's metadata (no device memory)."""
    params: "fp2.Params"
    cu_q: np.ndarray               # int32 [batch + 1], query (new-token) rows
    cu_k: np.ndarray               # int32 [batch + 1], KV tokens (prefix + new)
    total_tokens: int


def plan_forward(cfg: BackendConfig, extend_lens: Sequence[int],
                 prefix_lens: Optional[Sequence[int]] = None) -> ForwardPlan:
    """Validate one forward against the config and build its parameters."""
    ext = [int(x) for x in extend_lens]
    pre = [0] * len(ext) if prefix_lens is None else [int(x) for x in prefix_lens]
    if len(pre) != len(ext):
        raise ValueError("extend_lens and prefix_lens differ in length")
    if len(ext) > cfg.max_batch:
        raise ValueError("batch %d > max_batch %d" % (len(ext), cfg.max_batch))
    for b, (e, p) in enumerate(zip(ext, pre)):
        if e < 0 or p < 0:
            raise ValueError("sequence %d: negative length" % b)
        if e > cfg.max_extend_len:
            raise ValueError("sequence %d: extend of %d > max_extend_len %d"
                             % (b, e, cfg.max_extend_len))
        if p + e > cfg.max_kv_len:
            raise ValueError("sequence %d: %d cached + %d new > max_kv_len %d"
                             % (b, p, e, cfg.max_kv_len))
    cu_q = np.zeros(len(ext) + 1, np.int32)
    cu_k = np.zeros(len(ext) + 1, np.int32)
    cu_q[1:] = np.cumsum(ext)
    cu_k[1:] = np.cumsum([p + e for p, e in zip(pre, ext)])
    max_e = max(ext, default=0)
    max_k = max((p + e for p, e in zip(pre, ext)), default=0)
    params = cfg.params(len(ext), max_e, max(max_k, max_e))
    return ForwardPlan(params=params, cu_q=cu_q, cu_k=cu_k, total_tokens=int(cu_q[-1]))


@dataclasses.dataclass
class ForwardMetadata:
    plan: ForwardPlan
    cu_q: object                   # device int32 [batch + 1]
    cu_k: object                   # device int32 [batch + 1]
    block_table: object            # device int32 [batch, max_pages_per_seq], dense
    pooled_blocks: object          # device int32 [batch]: cached complete prefix blocks

    @property
    def params(self):
        return self.plan.params


class PrefillBackend:
    """Extend-phase attention of one stream (see the module docstring)."""

    def __init__(self, cfg: BackendConfig, device="cuda", stream=None):
        import torch
        self.cfg = cfg
        self.device = torch.device(device)
        self.stream = stream
        worst = cfg.worst_case_params()
        need = fp2.workspace_bytes(worst)
        if need == 0 and cfg.max_batch > 0:
            raise ValueError("configuration rejected by the library: " + fp2.last_error())
        self.workspace = torch.empty(max(1, need), dtype=torch.uint8, device=self.device)
        nq, nk = fp2.num_blocks(worst), fp2.num_key_blocks(worst)
        self._mask = torch.empty(max(1, cfg.max_batch * cfg.num_kv_heads * nq * nk),
                                 dtype=torch.uint8, device=self.device)

    def init_forward_metadata(self, extend_lens: Sequence[int], prefix_lens: Optional[Sequence[int]],
                              block_table, cached_prefix_lens: Optional[Sequence[int]] = None
                              ) -> ForwardMetadata:
        """cached_prefix_lens[b]: leading tokens of sequence b whose block means an
        earlier forward wrote to the means caches used with this metadata (None:
        none); only its complete blocks are taken from the cache."""
        import torch
        plan = plan_forward(self.cfg, extend_lens, prefix_lens)
        if fp2.workspace_bytes(plan.params) > self.workspace.numel():
            raise RuntimeError("forward needs more workspace than the configured worst case")
        n = len(plan.cu_q) - 1
        cached = [0] * n if cached_prefix_lens is None else [int(x) for x in cached_prefix_lens]
        if len(cached) != n:
            raise ValueError("cached_prefix_lens and extend_lens differ in length")
        kv = np.diff(plan.cu_k)
        for b, c in enumerate(cached):
            if c < 0 or c > kv[b]:
                raise ValueError("sequence %d: %d cached tokens outside [0, %d]" % (b, c, kv[b]))
        pooled = np.array([c // BLOCK for c in cached], np.int32)
        host = np.concatenate([plan.cu_q, plan.cu_k, pooled]).astype(np.int32)
        dev = torch.from_numpy(host).to(self.device)
        w = self.cfg.max_pages_per_seq
        if not (isinstance(block_table, torch.Tensor) and block_table.is_cuda
                and block_table.dtype == torch.int32 and block_table.dim() == 2):
            raise ValueError("block_table must be a CUDA int32 tensor [batch, pages]")
        if block_table.shape[1] < w or block_table.shape[0] < n:
            raise ValueError("block_table is %s, the forward needs [>= %d, >= %d]"
                             % (tuple(block_table.shape), n, w))
        # the library reads row b at b * max_pages_per_seq: hand it a dense
        # table of exactly that width (a copy when the caller's is wider or strided)
        if block_table.shape[1] != w or not block_table.is_contiguous():
            block_table = block_table[:n, :w].contiguous()
        return ForwardMetadata(plan=plan, cu_q=dev[:n + 1], cu_k=dev[n + 1:2 * n + 2],
                               block_table=block_table, pooled_blocks=dev[2 * n + 2:])

    def alloc_means_cache(self, num_pages: int):
        """One layer's block-means cache for a pool of num_pages pages:
        (khat, vbar) bf16 [slots, num_kv_heads, 128]."""
        return fp2.alloc_means_cache(self.cfg.worst_case_params(), num_pages, self.device)

    def block_mask(self, meta: ForwardMetadata):
        """The selection mask written by the last forward_extend, as a view
        [batch, num_kv_heads, nbq, nbk] of the backend's buffer."""
        p = meta.params
        shape = (p.batch, p.num_kv_heads, max(1, fp2.num_blocks(p)), max(1, fp2.num_key_blocks(p)))
        n = int(np.prod(shape))
        return self._mask[:n].view(shape)

    def forward_extend(self, q, k_cache, v_cache, meta: ForwardMetadata, *, q_scale=None,
                       k_scale=None, v_scale=None, out=None, lse=None, want_lse=False,
                       means_cache=None):
        """One layer: q [total_new_tokens, Hq, 128] against the paged cache.
        means_cache: this layer's (khat, vbar) from alloc_means_cache, or None.
        Returns (out, lse or None)."""
        import torch
        p = meta.params
        if q.shape[0] != meta.plan.total_tokens:
            raise ValueError("q has %d rows, the forward has %d new tokens"
                             % (q.shape[0], meta.plan.total_tokens))
        if out is None:
            out = torch.empty((q.shape[0], p.num_q_heads, p.head_dim), dtype=torch.bfloat16,
                              device=q.device)
        if lse is None and want_lse:
            lse = torch.empty((q.shape[0], p.num_q_heads), dtype=torch.float32, device=q.device)
        fp2.prefill(p, q, k_cache, v_cache, meta.cu_q, meta.block_table,
                    cu_seqlens_host=meta.plan.cu_q, cu_seqlens_k=meta.cu_k,
                    cu_seqlens_k_host=meta.plan.cu_k, q_scale=q_scale, k_scale=k_scale,
                    v_scale=v_scale, out=out, lse=lse, block_mask=self.block_mask(meta),
                    workspace=self.workspace, stream=self.stream,
                    means_cache=None if means_cache is None
                    else (means_cache[0], means_cache[1], meta.pooled_blocks))
        return out, lse

    def forward_decode(self, *args, **kwargs):
        raise NotImplementedError("decode attention stays dense; this backend serves extends")
