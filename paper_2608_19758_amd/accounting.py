"""FLOP and byte accounting of the prefill operator, for measurement.

Conventions:
* dense-equivalent FLOPs of causal attention: 4 * H_q * d * L^2 / 2 per
  sequence (QK^T and PV, causal half);
* executed FLOPs of the attention kernel: every kept (b, h, I, J) costs a full
  128 x 128 tile for all g heads, 4 * d * (g * B) * B; every corrected
  (b, h, I, J) costs one pooled key for the g * B rows, 4 * d * g * B
  (Sec. 3.4 Eq. complexity counts the same terms);
* algorithmic HBM bytes: what a kernel must read and write at least once.
"""
from __future__ import annotations

import numpy as np


def dense_equiv_flops(seqlens, num_q_heads, head_dim=128):
    return float(sum(2.0 * num_q_heads * head_dim * float(L) * float(L) for L in seqlens))


def block_counts(mask, seqlens, block_size=128, correction=True):
    """Per (b, h): kept and corrected block counts over all query blocks."""
    kept = corr = 0
    for b, L in enumerate(seqlens):
        n = (L + block_size - 1) // block_size
        m = (mask[b, :, :n, :n] & 1).astype(bool)
        kept += int(m.sum())
        if correction:
            strict = np.tril(np.ones((n, n), bool), -1)
            corr += int((strict[None] & ~m).sum())
    return kept, corr


def tile_counts(mask, seqlens, positions, block_size=128, correction=True):
    """Per (b, h): kept and corrected (tile, key block) pairs for query tiles of
    ``positions`` positions (tile t lies in key block t * positions / B)."""
    kept = corr = 0
    for b, L in enumerate(seqlens):
        nt = (L + positions - 1) // positions
        nb = (L + block_size - 1) // block_size
        m = (mask[b, :, :nt, :nb] & 1).astype(bool)
        kept += int(m.sum())
        if correction:
            own = np.arange(nt) * positions // block_size
            strict = np.arange(nb)[None, :] < own[:, None]
            corr += int((strict[None] & ~m).sum())
    return kept, corr


def attention_flops(mask, seqlens, num_q_heads, num_kv_heads, head_dim=128, block_size=128,
                    correction=True, tile_rows=0):
    """(kept-block FLOPs, correction FLOPs) executed by the attention kernel.
    tile_rows > 0: the mask rows are tiles of tile_rows packed rows."""
    g = num_q_heads // num_kv_heads
    if tile_rows:
        kept, corr = tile_counts(mask, seqlens, tile_rows // g, block_size, correction)
        return (4.0 * head_dim * tile_rows * block_size * kept,
                4.0 * head_dim * tile_rows * corr)
    kept, corr = block_counts(mask, seqlens, block_size, correction)
    return (4.0 * head_dim * g * block_size * block_size * kept,
            4.0 * head_dim * g * block_size * corr)


def estimation_bytes(seqlens, num_q_heads, num_kv_heads, head_dim=128, block_size=128, elem=2):
    """Algorithmic bytes of the index stage: Q, K, V read once; pooled means
    (bf16) written and re-read once; the mask rows and the int32 kept lists
    (bounded by every causal block) written."""
    tot = 0.0
    for L in seqlens:
        n = (L + block_size - 1) // block_size
        tot += L * num_q_heads * head_dim * elem                 # Q
        tot += 2 * L * num_kv_heads * head_dim * elem            # K, V
        tot += 2 * 2 * n * num_kv_heads * head_dim * 2           # khat, vbar write + read
        tot += num_kv_heads * n * n                              # mask rows
        tot += num_kv_heads * n * (n + 1) // 2 * 4               # kept lists (upper bound)
    return tot


def pool_bytes(seqlens, num_kv_heads, head_dim=128, block_size=128, elem=2):
    """Algorithmic bytes of the block-mean kernel: K, V read; two bf16 means written."""
    tot = 0.0
    for L in seqlens:
        n = (L + block_size - 1) // block_size
        tot += 2 * L * num_kv_heads * head_dim * elem + 2 * n * num_kv_heads * head_dim * 2
    return tot


def scoring_flops(seqlens, num_q_heads, head_dim=128, block_size=128):
    """MFMA FLOPs of the fused scoring: 2 d per (query row, pooled key J <= I)."""
    tot = 0.0
    for L in seqlens:
        n = (L + block_size - 1) // block_size
        tot += 2.0 * head_dim * num_q_heads * block_size * n * (n + 1) / 2
    return tot


def csr_index_bytes(seqlen, num_q_heads, num_kv_heads, density, m_tile=128, kv_tile=64):
    """Bytes of the int32 entries of a CSR index of selected 64-token KV tiles
    per packed 128-row M-tile and KV head, as sized for the paper's design
    comparison (Tab. bsa_design)."""
    g = num_q_heads // num_kv_heads
    pos_per_tile = m_tile // g
    tiles = (g * seqlen + m_tile - 1) // m_tile
    causal = sum(-(-((i + 1) * pos_per_tile) // kv_tile) for i in range(tiles))
    entries = density * causal * num_kv_heads
    return 4.0 * entries


def dense_mask_bytes(seqlen, num_q_heads, q_tile=128, kv_tile=128):
    """One byte per (query head, 128-token Q tile, 128-token KV tile)."""
    nq = -(-seqlen // q_tile)
    nk = -(-seqlen // kv_tile)
    return float(num_q_heads * nq * nk)


def aux_flop_ratio(rho, block_size):
    """(C_idx + C_corr) / C_attn = (2 - rho) / (2 rho B), Sec. 3.4 Eq. complexity."""
    return (2.0 - rho) / (2.0 * rho * block_size)
