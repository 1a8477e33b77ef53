"""Pin of the oracle's forced-block set (Sec. 3.1, the thresholding paragraph,
and Eq. select: sink blocks, the local window, the diagonal and the most recent
blocks are always kept; Sec. 4 implementation details give the sizes as
256 sink tokens and a 512-token window).

The oracle decides membership block by block. This file counts the forced
blocks of every mask row with arithmetic instead: the forced set of a row whose
query positions lie in key blocks Ja .. Jb is a prefix [0, a) (the sink) and a
suffix [t, Jb] (window counted back from Jb, the diagonal band Ja .. Jb, and the
recent blocks, all ending at Jb), so its size is a + (Jb + 1 - t) - overlap.
A window or sink off by one, a window that forgets the diagonal, or recent
blocks counted from the wrong end change at least one row count.

Also pinned by hand: the paper's defaults (256 sink tokens, 512-token window:
2 and 4 blocks of 128) force 81 of the 136 causal blocks of a 2048-token
sequence (rows 0..5 force 1, 2, 3, 4, 5, 6 blocks, rows 6..15 force 6 each),
i.e. 59.6 %.
"""
import numpy as np
import pytest

import oracle
import synth


def forced_count(nk, Ja, Jb, sink, window, recent):
    """Number of forced key blocks of a row (closed form, see the module text)."""
    a = max(0, min(sink, Jb + 1))
    t = min(Jb - window + 1, Ja, nk - recent)
    t = max(0, t)
    return a + (Jb + 1 - t) - max(0, a - t)


def test_closed_form_paper_defaults_by_hand():
    n = 16
    counts = [forced_count(n, I, I, 2, 4, 0) for I in range(n)]
    assert counts == [1, 2, 3, 4, 5, 6] + [6] * 10
    assert sum(counts) == 81
    assert round(81 / 136, 3) == 0.596


def _spec(lens, prefix=None, hq=4, hkv=2, page=64, B=128, seed=11):
    kvl = [L + (prefix[i] if prefix else 0) for i, L in enumerate(lens)]
    return synth.Spec("forced", list(lens), hq, hkv, block_size=B, page_size=page,
                      salient_frac=0.2, salient_min=1, sink_blocks=1, window_blocks=1,
                      recent_blocks=0, mean_correction=1, seed=seed, prefix=prefix,
                      pool_pages=0, page_order="identity") if kvl else None


SETS = [(0, 1, 0), (1, 1, 0), (1, 2, 0), (2, 4, 0), (3, 2, 2), (0, 0, 1), (5, 3, 4), (0, 7, 0)]


@pytest.mark.parametrize("sink,window,recent", SETS)
@pytest.mark.parametrize("alpha", [1.5, 0.0, 0.97])
def test_forced_counts_closed_form(sink, window, recent, alpha):
    """Every row's forced-bit count equals the closed form; with alpha > 1 the
    kept bits are exactly the forced ones, with alpha = 0 every causal block."""
    wl = synth.generate(_spec([1300, 129, 640], B=128))
    inp = oracle.Inputs(wl)
    mask = oracle.estimate(inp, inp.params(alpha, sink=sink, window=window, recent=recent))
    B = wl.spec.block_size
    for b, L in enumerate(wl.spec.seqlens):
        n = (L + B - 1) // B
        for h in range(wl.spec.num_kv_heads):
            for I in range(n):
                row = mask[b, h, I]
                want = forced_count(n, I, I, sink, window, recent)
                assert int(((row >> 1) & 1).sum()) == want, (b, h, I)
                kept = int((row & 1).sum())
                if alpha > 1:
                    assert kept == want
                elif alpha == 0:
                    assert kept == I + 1
                else:
                    assert want <= kept <= I + 1


@pytest.mark.parametrize("prefix", [[256], [77], [129], [1000]])
@pytest.mark.parametrize("sink,window,recent", [(1, 2, 0), (2, 1, 3), (0, 3, 1)])
def test_forced_counts_with_prefix(prefix, sink, window, recent):
    """Prefix KV: query rows at absolute positions prefix + i; a query block
    straddling two key blocks has Ja = a0 // B, Jb = a1 // B."""
    L = 700
    wl = synth.generate(_spec([L], prefix=prefix, hq=4, hkv=1, B=128))
    inp = oracle.Inputs(wl)
    mask = oracle.estimate(inp, inp.params(2.0, sink=sink, window=window, recent=recent))
    B = 128
    P0 = prefix[0]
    nk = (P0 + L + B - 1) // B
    for I in range((L + B - 1) // B):
        a0, a1 = P0 + I * B, P0 + min(L, (I + 1) * B) - 1
        Ja, Jb = a0 // B, a1 // B
        want = forced_count(nk, Ja, Jb, sink, window, recent)
        row = mask[0, 0, I]
        assert int(((row >> 1) & 1).sum()) == want, I
        assert int((row & 1).sum()) == want, I
        assert not row[Jb + 1:].any()


@pytest.mark.parametrize("tile_rows", [128, 64])
def test_forced_counts_query_tiles(tile_rows):
    """Query tiles of tile_rows packed rows (tile_rows / g positions): the tile
    lies in one key block, which is its diagonal."""
    g = 4
    wl = synth.generate(_spec([900], hq=g, hkv=1, B=128))
    inp = oracle.Inputs(wl)
    mask = oracle.estimate(inp, inp.params(2.0, sink=1, window=2, recent=1, tile_rows=tile_rows))
    Pt = tile_rows // g
    nk = (900 + 127) // 128
    for I in range((900 + Pt - 1) // Pt):
        Ja = Jb = (I * Pt) // 128
        want = forced_count(nk, Ja, Jb, 1, 2, 1)
        assert int(((mask[0, 0, I] >> 1) & 1).sum()) == want, I
