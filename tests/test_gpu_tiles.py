"""GPU parity of the 128-packed-row query tiles (Sec. 3.3 PackGQA: the
selection tile is one M-tile of 128 packed rows, 128/g positions with all g
heads) and of the CSR index of 64-token key tiles (Eq. csr), through the C ABI.

Bars as for query blocks: mask bit-exact outside the 1e-4 margin band against
the oracle in tile mode; outputs under the GPU's mask within max-abs 2e-2
(bf16) / 6e-2 (fp8), LSE within 1e-2 / 0.0625; with g = 1 the tile is the
block and the two modes agree bit for bit. The CSR is checked entry by entry
against its definition applied to the mask on the host.
"""
import numpy as np
import pytest
import torch

import oracle
import paper_2608_19758_amd as fp2
import synth
from tests import gpu_util as gu

pytestmark = pytest.mark.gpu

R = 128   # packed rows per tile


def spec(lens, prefix=None, hq=8, hkv=2, dtype="bf16", page=64, order="identity", seed=13,
         frac=0.1, sink=1, window=2, recent=0, corr=1):
    kvl = [L + p for L, p in zip(lens, prefix)] if prefix is not None else list(lens)
    pool = sum((L + page - 1) // page for L in kvl) + 5 if (page and order == "permuted") else 0
    return synth.Spec("tiles", list(lens), hq, hkv, dtype=dtype, page_size=page,
                      page_order=order, pool_pages=pool, salient_frac=frac, salient_min=2,
                      sink_blocks=sink, window_blocks=window, recent_blocks=recent,
                      mean_correction=corr, seed=seed, prefix=prefix)


CASES = {
    "g4_paged": dict(lens=[1500, 300], hq=8, hkv=2, page=64),
    "g8_contig": dict(lens=[900], hq=16, hkv=2, page=0),
    "g2_perm_prefix": dict(lens=[700, 1], prefix=[512, 1024], hq=4, hkv=2, page=16,
                           order="permuted"),
    "g4_fp8": dict(lens=[1200], hq=8, hkv=2, dtype="fp8", page=64, recent=1),
    "g8_fp8_prefix": dict(lens=[333, 130], prefix=[256, 0], hq=8, hkv=1, dtype="fp8", page=32),
    "g4_unaligned": dict(lens=[400, 90], prefix=[50, 300], hq=8, hkv=2, page=64),
}


def _wl(name):
    c = dict(CASES[name])
    print("case", name, c, flush=True)
    return synth.generate(spec(**c))


@pytest.mark.parametrize("name,alpha", gu.alpha_cases(CASES))
def test_tiles_prefill_parity(name, alpha):
    wl = _wl(name)
    sp = wl.spec
    out, gmask, lse = gu.gpu_prefill(wl, gu.params_for(wl, alpha, query_tile_rows=R))
    inp = oracle.Inputs(wl)
    op = inp.params(alpha, tile_rows=R)
    omask, ell, mu = oracle.estimate(inp, op, want_scores=True)
    assert gmask.shape == omask.shape
    units = gu.units_of(wl, query_tile_rows=R)
    ob, ibm, ib = gu.compare_masks(gmask, omask, ell, mu, alpha, units)
    print("mask: outside-band mismatches %d, in-band mismatches %d of %d in-band" % (ob, ibm, ib))
    assert ob == 0
    oout, olse = oracle.attend(inp, op, gmask)
    gu.check_close(out, oout, lse, olse, sp.dtype)


@pytest.mark.parametrize("name", ["g4_paged", "g8_fp8_prefix"])
def test_tiles_attend_external_mask(name):
    wl = _wl(name)
    sp = wl.spec
    inp = oracle.Inputs(wl)
    op = inp.params(0.99, tile_rows=R)
    omask = oracle.estimate(inp, op)
    oout, olse = oracle.attend(inp, op, omask)
    p = gu.params_for(wl, 0.99, query_tile_rows=R)
    d = gu.device_tensors(wl)
    out, lse = fp2.attend(p, d["q"], d["k_cache"], d["v_cache"], d["cu_seqlens"],
                          torch.from_numpy(omask).cuda(), d["block_table"] if sp.page_size else None,
                          cu_seqlens_host=wl.cu_seqlens, q_scale=d["q_scale"],
                          k_scale=d["k_scale"], v_scale=d["v_scale"], want_lse=True,
                          **gu.kv_args(wl, d))
    torch.cuda.synchronize()
    gu.check_close(out.float().cpu().numpy(), oout, lse.cpu().numpy(), olse, sp.dtype,
                   label="external-mask")


@pytest.mark.parametrize("dtype", ["bf16", "fp8"])
def test_tiles_g1_equal_blocks(dtype):
    wl = synth.generate(spec([900, 200], hq=2, hkv=2, dtype=dtype))
    a = gu.gpu_prefill(wl, gu.params_for(wl, 0.98, kv_splits=1))
    b = gu.gpu_prefill(wl, gu.params_for(wl, 0.98, kv_splits=1, query_tile_rows=R))
    for x, y in zip(a, b):
        np.testing.assert_array_equal(x, y)


def csr_reference(mask, wl, Pt):
    """The definition of the CSR applied to a mask on the host."""
    sp = wl.spec
    B = sp.block_size
    offs, idx = [0], []
    for b in range(sp.batch):
        Lq, Lk = sp.seqlens[b], sp.kvlens[b]
        for h in range(sp.num_kv_heads):
            for t in range(mask.shape[2]):
                if t * Pt < Lq:
                    Jb = (Lk - Lq + min(Lq, (t + 1) * Pt) - 1) // B   # block of the last row
                    for J in range(Jb + 1):
                        if mask[b, h, t, J] & 1:
                            idx.append(2 * J)
                            if (2 * J + 1) * 64 < Lk:
                                idx.append(2 * J + 1)
                offs.append(len(idx))
    return np.array(offs, np.int32), np.array(idx, np.int32)


@pytest.mark.parametrize("name", ["g4_paged", "g2_perm_prefix", "g8_fp8_prefix", "g4_unaligned"])
@pytest.mark.parametrize("tile", [0, R])
@pytest.mark.parametrize("alpha", [0.0, 0.99])
def test_mask_to_csr(name, tile, alpha):
    wl = _wl(name)
    p = gu.params_for(wl, alpha, query_tile_rows=tile)
    d = gu.device_tensors(wl)
    out, mask, _ = fp2.prefill(p, d["q"], d["k_cache"], d["v_cache"], d["cu_seqlens"],
                               d["block_table"] if wl.spec.page_size else None,
                               q_scale=d["q_scale"], k_scale=d["k_scale"], v_scale=d["v_scale"],
                               **gu.kv_args(wl, d))
    offs, idx = fp2.mask_to_csr(p, mask, d["cu_seqlens"], cu_seqlens_host=wl.cu_seqlens,
                                **gu.kv_args(wl, d))
    torch.cuda.synchronize()
    want_o, want_i = csr_reference(mask.cpu().numpy(), wl, gu.tile_positions(wl, tile))
    got_o = offs.cpu().numpy()
    print("segments %d, entries %d (capacity %d)" % (len(want_o) - 1, want_o[-1], idx.numel()))
    np.testing.assert_array_equal(got_o, want_o)
    np.testing.assert_array_equal(idx[:got_o[-1]].cpu().numpy(), want_i)


def test_tiles_fullsize_sampled():
    """128-row tiles at the 32K bf16 shape (32 query / 8 KV heads, g = 4, so 32
    positions per tile and 8192 tiles per head), sampled units against the
    oracle."""
    sp = synth.named("llama32k")
    wl = synth.generate(sp)
    alpha = synth.alpha_for("llama32k", "0.18")
    out, gmask, lse = gu.gpu_prefill(wl, gu.params_for(wl, alpha, query_tile_rows=R))
    assert np.isfinite(out).all() and np.isfinite(lse).all()
    units = gu.units_of(wl, sample=16, seed=4, query_tile_rows=R)
    inp = oracle.Inputs(wl)
    op = inp.params(alpha, tile_rows=R)
    omask, ell, mu = oracle.estimate(inp, op, units=units, want_scores=True)
    ob, ibm, ib = gu.compare_masks(gmask, omask, ell, mu, alpha, units)
    print("mask on %d units: outside-band mismatches %d, in-band %d of %d" % (len(units), ob, ibm, ib))
    assert ob == 0
    oout, olse = oracle.attend(inp, op, gmask, units=units)
    gu.check_close(out, oout, lse, olse, "bf16", rows=gu.unit_rows(wl, units, query_tile_rows=R),
                   label="same-mask (%d sampled units)" % len(units))
