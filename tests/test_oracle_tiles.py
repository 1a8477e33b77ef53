"""Pins of the oracle's query-tile granularity (CPU only).

With tile_rows = R the selection tile is one M-tile of R packed rows of
Sec. 3.3 PackGQA (R/g positions with all g heads of a KV group; the index of
Eq. csr is per tile) instead of a block of B positions.

P17 g = 1 and R = 128: the tile is the block; bitwise equal to the default.
P18 alpha = 0 keeps every block up to the tile's key block: equals torch fp64
    SDPA with the causal mask (1e-12).
P19 the independent NumPy brute force (tests/brute.py, tile mode) agrees on
    every mask byte and to 1e-12 on outputs and LSE.
P20 block log-energies are the logsumexp of the energies of the block's tiles
    (the rows of a block are the disjoint union of its tiles' rows), 1e-12.
P21 forced bits follow the closed form with the tile's key block t*Pt/B.
P22 with a prefix, a chunk's tiles reproduce the whole sequence's tiles,
    bitwise.
"""
import numpy as np
import pytest
import torch
from scipy.special import logsumexp

import oracle
import synth
from tests import brute


def spec(lens, hq=8, hkv=2, dtype="bf16", page=16, order="identity", seed=21, prefix=None,
         sink=1, window=2, recent=0, frac=0.1):
    kvl = [L + (prefix[i] if prefix else 0) for i, L in enumerate(lens)]
    pool = sum((L + page - 1) // page for L in kvl) + 3 if order == "permuted" else 0
    return synth.Spec("tiles", list(lens), hq, hkv, dtype=dtype, page_size=page,
                      page_order=order, pool_pages=pool, salient_frac=frac, salient_min=1,
                      sink_blocks=sink, window_blocks=window, recent_blocks=recent, seed=seed,
                      prefix=prefix)


def run(wl, alpha, tile_rows=0, want_scores=False, **kw):
    inp = oracle.Inputs(wl)
    p = inp.params(alpha, tile_rows=tile_rows, **kw)
    r = oracle.estimate(inp, p, want_scores=want_scores)
    mask = r[0] if want_scores else r
    out, lse = oracle.attend(inp, p, mask)
    return (r, out, lse) if want_scores else (mask, out, lse)


@pytest.mark.parametrize("alpha", [0.0, 0.9, 2.0])
def test_p17_g1_tile_is_block(alpha):
    wl = synth.generate(spec([700, 300], hq=2, hkv=2))
    m0, o0, l0 = run(wl, alpha)
    m1, o1, l1 = run(wl, alpha, tile_rows=128)
    assert np.array_equal(m0, m1) and np.array_equal(o0, o1) and np.array_equal(l0, l1)


@pytest.mark.parametrize("case", [dict(lens=[500], hq=4, hkv=1),
                                  dict(lens=[300, 129], hq=8, hkv=2, dtype="fp8", page=64)])
def test_p18_alpha0_tiles_dense(case):
    wl = synth.generate(spec(**case))
    mask, out, _ = run(wl, 0.0, tile_rows=128)
    dense = brute.dense_sdpa(wl)
    np.testing.assert_allclose(out, dense, atol=1e-12, rtol=0)
    # every block up to the tile's key block is kept
    sp = wl.spec
    g = sp.num_q_heads // sp.num_kv_heads
    Pt = 128 // g
    for b, L in enumerate(sp.seqlens):
        for t in range((L + Pt - 1) // Pt):
            Ia = t * Pt // 128
            assert (mask[b, :, t, :Ia + 1] & 1).all() and not mask[b, :, t, Ia + 1:].any()


CASES = [dict(lens=[600, 200], hq=8, hkv=2), dict(lens=[513], hq=4, hkv=1, page=0),
         dict(lens=[400], hq=8, hkv=1, dtype="fp8", page=32, order="permuted"),
         dict(lens=[350, 90], hq=4, hkv=2, recent=1, window=1)]


@pytest.mark.parametrize("case", CASES)
@pytest.mark.parametrize("alpha", [0.0, 0.95, 2.0])
def test_p19_tiles_brute_force(case, alpha):
    wl = synth.generate(spec(**case))
    (mask, ell, mu), out, lse = run(wl, alpha, tile_rows=128, want_scores=True)
    bm, bell, bout, blse = brute.brute(wl, alpha, tile_rows=128)
    np.testing.assert_array_equal(mask, bm)
    ok = ~np.isnan(bell)
    np.testing.assert_allclose(ell[ok], bell[ok], atol=1e-12, rtol=0)
    np.testing.assert_allclose(out, bout, atol=1e-12, rtol=0)
    np.testing.assert_allclose(lse, blse, atol=1e-12, rtol=0)


@pytest.mark.parametrize("case", CASES[:3])
def test_p20_block_energy_is_logsumexp_of_tiles(case):
    wl = synth.generate(spec(**case))
    sp = wl.spec
    g = sp.num_q_heads // sp.num_kv_heads
    Pt = 128 // g
    (_, eb, _), _, _ = run(wl, 0.9, want_scores=True)
    (_, et, _), _, _ = run(wl, 0.9, tile_rows=128, want_scores=True)
    for b, L in enumerate(sp.seqlens):
        for I in range((L + 127) // 128):
            ts = range(I * 128 // Pt, min((L + Pt - 1) // Pt, (I + 1) * 128 // Pt))
            want = logsumexp(np.stack([et[b, :, t, :I + 1] for t in ts]), axis=0)
            np.testing.assert_allclose(eb[b, :, I, :I + 1], want, atol=1e-12, rtol=0)


def test_p21_forced_closed_form():
    wl = synth.generate(spec([900, 333], hq=8, hkv=2, sink=2, window=3, recent=1))
    sp = wl.spec
    mask, _, _ = run(wl, 2.0, tile_rows=128)        # alpha > 1 keeps forced blocks only
    Pt = 128 // (sp.num_q_heads // sp.num_kv_heads)
    for b, L in enumerate(sp.seqlens):
        n = (L + 127) // 128
        for t in range((L + Pt - 1) // Pt):
            Ia = t * Pt // 128
            want = np.array([J <= Ia and (J < 2 or Ia - J < 3 or J == Ia or J >= n - 1)
                             for J in range(mask.shape[-1])])
            assert ((mask[b, :, t] >> 1).astype(bool) == want[None]).all()
            assert ((mask[b, :, t] & 1).astype(bool) == want[None]).all()


@pytest.mark.parametrize("alpha", [0.0, 0.9])
def test_p22_prefix_tiles_chunk_equals_whole(alpha):
    kv, pre = [900, 650], [256, 384]
    whole = synth.generate(spec(kv, hq=4, hkv=2, page=32))
    chunk = synth.generate(spec([L - p for L, p in zip(kv, pre)], hq=4, hkv=2, page=32,
                                prefix=pre))
    mw, ow, lw = run(whole, alpha, tile_rows=128)
    mc, oc, lc = run(chunk, alpha, tile_rows=128)
    Pt = 128 // 2
    for b, (L, p) in enumerate(zip(kv, pre)):
        nt = (L - p + Pt - 1) // Pt
        np.testing.assert_array_equal(mc[b, :, :nt], mw[b, :, p // Pt:p // Pt + nt, :mc.shape[-1]])
        rw = slice(int(whole.cu_seqlens[b]) + p, int(whole.cu_seqlens[b + 1]))
        rc = slice(int(chunk.cu_seqlens[b]), int(chunk.cu_seqlens[b + 1]))
        assert np.array_equal(oc[rc], ow[rw]) and np.array_equal(lc[rc], lw[rw])
