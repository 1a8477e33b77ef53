"""P14: the FLOP/byte accounting used by the benchmark reproduces the
closed-form numbers the paper prints (tests/golden/paper_numbers.json)."""
import json
import os

import numpy as np

from paper_2608_19758_amd import accounting as acc

GOLD = json.load(open(os.path.join(os.path.dirname(__file__), "golden", "paper_numbers.json")))


def test_index_memory_matches_paper_table():
    im = GOLD["index_memory"]
    for c in im["cases"]:
        dense = acc.dense_mask_bytes(c["seq_len"], im["num_q_heads"])
        assert dense == c["dense_mb"] * 2 ** 20
        csr = acc.csr_index_bytes(c["seq_len"], im["num_q_heads"], im["num_kv_heads"], c["density"])
        assert abs(csr / 2 ** 20 - c["csr_mb"]) < 0.5, csr / 2 ** 20


def test_aux_flop_ratio_matches_paper():
    a = GOLD["aux_flop_ratio"]
    r = acc.aux_flop_ratio(a["rho"], a["block_size"])
    assert round(100 * r) == a["percent"]


def test_flop_counts_small_mask():
    # 1 sequence of 3 blocks, g = 2: kept = diag + (2,0); corrected = (1,0), (2,1)
    m = np.zeros((1, 1, 3, 3), np.uint8)
    m[0, 0, 0, 0] = m[0, 0, 1, 1] = m[0, 0, 2, 2] = m[0, 0, 2, 0] = 1
    kept, corr = acc.block_counts(m, [384], 128)
    assert (kept, corr) == (4, 2)
    fk, fc = acc.attention_flops(m, [384], 2, 1)
    assert fk == 4 * 128 * 2 * 128 * 128 * 4 and fc == 4 * 128 * 2 * 128 * 2
    assert acc.dense_equiv_flops([384], 2) == 2 * 2 * 128 * 384 * 384


def test_tile_counts_match_block_counts_when_tile_is_block():
    """With tiles of B positions the tile accounting is the block accounting."""
    rng = np.random.default_rng(5)
    n = 9
    mask = np.zeros((1, 2, n, n), np.uint8)
    for I in range(n):
        mask[0, :, I, :I + 1] = rng.integers(0, 2, size=(2, I + 1))
        mask[0, :, I, I] = 1
    assert acc.tile_counts(mask, [n * 128 - 5], 128) == acc.block_counts(mask, [n * 128 - 5])
    f = acc.attention_flops(mask, [n * 128 - 5], 8, 2)
    assert f == acc.attention_flops(mask, [n * 128 - 5], 8, 2, tile_rows=0)


def test_tile_counts_closed_form():
    """Dense tile mask (every visible pair kept): kept = sum over tiles of
    (own block + 1), nothing corrected; empty mask: corrected = own block."""
    L, pt = 1000, 32
    nt, nb = (L + pt - 1) // pt, (L + 127) // 128
    own = np.arange(nt) * pt // 128
    full = np.zeros((1, 1, nt, nb), np.uint8)
    for t in range(nt):
        full[0, 0, t, :own[t] + 1] = 1
    assert acc.tile_counts(full, [L], pt) == (int((own + 1).sum()), 0)
    assert acc.tile_counts(np.zeros_like(full), [L], pt) == (0, int(own.sum()))
