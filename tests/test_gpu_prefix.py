"""GPU parity of the prefix-KV (chunked prefill) path against the oracle,
through the C ABI.

The queries of a sequence are the last L_q of its L_kv keys (prefix
P = L_kv - L_q, a multiple of the block size): key blocks, pooled means,
mask columns and the causal mask are those of the L_kv tokens, query block I
is key block I + P/B.

Bars as for the prefill without a prefix: block means bit-exact; mask
bit-exact outside the 1e-4 margin band; outputs within max-abs 2e-2 (bf16) /
6e-2 (fp8) of the fp64 oracle under the GPU's own mask; LSE within 1e-2 /
0.0625. Without KV splits (kv_splits = 1) a chunked call reproduces, bit for
bit, the rows of the call over the whole sequence (the per-unit arithmetic
is the same in both); with the default cost-balanced plan the two calls may
split different units, so they agree up to rounding.
"""
import numpy as np
import pytest
import torch

import oracle
import paper_2608_19758_amd as fp2
import synth
from tests import brute, gpu_util as gu

pytestmark = pytest.mark.gpu


def spec(lens, prefix, hq=4, hkv=1, dtype="bf16", page=64, order="identity", seed=5, frac=0.1,
         sink=1, window=2, recent=0, corr=1):
    kvl = [L + p for L, p in zip(lens, prefix)] if prefix is not None else list(lens)
    pool = sum((L + page - 1) // page for L in kvl) + 5 if (page and order == "permuted") else 0
    return synth.Spec("prefix", list(lens), hq, hkv, dtype=dtype, page_size=page, page_order=order,
                      pool_pages=pool, salient_frac=frac, salient_min=2, sink_blocks=sink,
                      window_blocks=window, recent_blocks=recent, mean_correction=corr, seed=seed,
                      prefix=prefix)


CASES = {
    "bf16_contig": dict(lens=[700], prefix=[1024], hq=4, hkv=1, page=0),
    # an empty chunk and a one-token chunk after a prefix
    "bf16_paged_ragged": dict(lens=[300, 0, 1, 129], prefix=[512, 256, 2048, 0], hq=4, hkv=2,
                              page=64),
    "bf16_perm_p16": dict(lens=[900], prefix=[384], hq=8, hkv=1, page=16, order="permuted"),
    "g1_paged": dict(lens=[500, 260], prefix=[128, 640], hq=2, hkv=2, page=32, recent=2),
    "fp8_paged": dict(lens=[800, 200], prefix=[640, 128], hq=8, hkv=2, dtype="fp8", page=64),
    "fp8_perm": dict(lens=[333], prefix=[1152], hq=8, hkv=1, dtype="fp8", page=16,
                     order="permuted"),
    # prefixes that are not block multiples: query blocks straddle two key blocks
    "bf16_unaligned": dict(lens=[300, 129, 5, 0], prefix=[100, 1, 1000, 77], hq=4, hkv=2,
                           page=16),
    "fp8_unaligned": dict(lens=[420], prefix=[127], hq=8, hkv=2, dtype="fp8", page=64,
                          window=1, recent=1),
    "g1_unaligned_contig": dict(lens=[260, 64], prefix=[65, 129], hq=2, hkv=2, page=0),
}


def _wl(name, **kw):
    c = dict(CASES[name])
    c.update(kw)
    print("case", name, c, flush=True)
    return synth.generate(spec(**c))


@pytest.mark.parametrize("name", list(CASES))
def test_prefix_pool_bit_exact(name):
    """fp2_pool over the KV lengths equals the oracle's means of the KV tokens."""
    wl = _wl(name)
    p = gu.params_for(wl, 0.5)
    d = gu.device_tensors(wl)
    khat, vbar = fp2.pool(p, d["k_cache"], d["v_cache"], d["cu_seqlens_k"],
                          d["block_table"] if wl.spec.page_size else None,
                          cu_seqlens_host=wl.cu_seqlens_k, k_scale=d["k_scale"],
                          v_scale=d["v_scale"])
    torch.cuda.synchronize()
    inp = oracle.Inputs(wl)
    _, vb, khat_o = oracle.pool(inp, inp.params(0.5))
    np.testing.assert_array_equal(khat.view(torch.int16).cpu().numpy().view(np.uint16), khat_o)
    want_v = np.zeros(vb.shape, np.uint16)
    nz = vb != 0
    want_v[nz] = brute.bf16_round_bits(vb[nz])
    np.testing.assert_array_equal(vbar.view(torch.int16).cpu().numpy().view(np.uint16), want_v)


@pytest.mark.parametrize("name,alpha", gu.alpha_cases(CASES))
def test_prefix_prefill_parity(name, alpha):
    wl = _wl(name)
    sp = wl.spec
    p = gu.params_for(wl, alpha)
    out, gmask, lse = gu.gpu_prefill(wl, p)
    inp = oracle.Inputs(wl)
    op = gu.oracle_params(inp, alpha)
    omask, ell, mu = oracle.estimate(inp, op, want_scores=True)
    assert gmask.shape == omask.shape
    units = gu.units_of(wl)
    ob, ibm, ib = gu.compare_masks(gmask, omask, ell, mu, alpha, units)
    print("mask: outside-band mismatches %d, in-band mismatches %d of %d in-band" % (ob, ibm, ib))
    assert ob == 0
    B = sp.block_size
    for b, (L, P) in enumerate(zip(sp.seqlens, sp.prefixes)):
        nq, nk = (L + B - 1) // B, (L + P + B - 1) // B
        assert (gmask[b, :, nq:, :] == 0).all() and (gmask[b, :, :, nk:] == 0).all()
        for I in range(nq):   # nothing past the block of the last row; the band is forced
            Ja, Jb = (P + I * B) // B, (P + min(L, (I + 1) * B) - 1) // B
            assert (gmask[b, :, I, Jb + 1:] == 0).all()
            assert (gmask[b, :, I, Ja:Jb + 1] == 3).all()
    oout, olse = oracle.attend(inp, op, gmask)
    gu.check_close(out, oout, lse, olse, sp.dtype)


@pytest.mark.parametrize("name", ["bf16_paged_ragged", "fp8_perm", "bf16_unaligned"])
@pytest.mark.parametrize("corr", [0, 1])
def test_prefix_attend_external_mask(name, corr):
    """fp2_attend under the oracle's mask equals the oracle under that mask."""
    wl = _wl(name)
    sp = wl.spec
    alpha = 0.99
    inp = oracle.Inputs(wl)
    op = gu.oracle_params(inp, alpha, corr=corr)
    omask = oracle.estimate(inp, op)
    oout, olse = oracle.attend(inp, op, omask)
    p = gu.params_for(wl, alpha, corr=corr)
    d = gu.device_tensors(wl)
    out, lse = fp2.attend(p, d["q"], d["k_cache"], d["v_cache"], d["cu_seqlens"],
                          torch.from_numpy(omask).cuda(),
                          d["block_table"] if sp.page_size else None,
                          cu_seqlens_host=wl.cu_seqlens, q_scale=d["q_scale"],
                          k_scale=d["k_scale"], v_scale=d["v_scale"], want_lse=True,
                          **gu.kv_args(wl, d))
    torch.cuda.synchronize()
    gu.check_close(out.float().cpu().numpy(), oout, lse.cpu().numpy(), olse, sp.dtype,
                   label="external-mask")


CHUNKS = [
    dict(kv=[1700], pre=[512], hq=4, hkv=1, page=0),
    dict(kv=[1300, 900], pre=[768, 128], hq=8, hkv=2, page=16, order="permuted"),
    dict(kv=[2000], pre=[1024], hq=8, hkv=2, dtype="fp8", page=64),
]


@pytest.mark.parametrize("case", CHUNKS)
@pytest.mark.parametrize("alpha", [0.0, 0.99])
def test_chunk_equals_whole_on_gpu(case, alpha):
    """The chunk's mask rows, outputs and LSE equal those rows of the call over
    the whole sequence, bit for bit."""
    case = dict(case)
    kv, pre = case.pop("kv"), case.pop("pre")
    print("chunk case", kv, pre, case, alpha, flush=True)
    whole = synth.generate(spec(kv, None, **case))
    chunk = synth.generate(spec([L - P for L, P in zip(kv, pre)], pre, **case))
    ow, mw, lw = gu.gpu_prefill(whole, gu.params_for(whole, alpha, kv_splits=1, score_splits=1))
    oc, mc, lc = gu.gpu_prefill(chunk, gu.params_for(chunk, alpha, kv_splits=1, score_splits=1))
    B = whole.spec.block_size
    for b, (L, P) in enumerate(zip(kv, pre)):
        rw = slice(int(whole.cu_seqlens[b]) + P, int(whole.cu_seqlens[b + 1]))
        rc = slice(int(chunk.cu_seqlens[b]), int(chunk.cu_seqlens[b + 1]))
        nq, nk = (L - P + B - 1) // B, (L + B - 1) // B
        np.testing.assert_array_equal(mc[b, :, :nq, :nk], mw[b, :, P // B:P // B + nq, :nk])
        print("seq %d: max |chunk - whole| out %.3g" % (b, np.abs(oc[rc] - ow[rw]).max()))
        np.testing.assert_array_equal(oc[rc], ow[rw])
        np.testing.assert_array_equal(lc[rc], lw[rw])


def test_chunked_prefill_fullsize_sampled():
    """Chunked prefill at the 128K fp8 shape (32 query heads, 8 KV heads,
    paged KV): the last 32K tokens after a 96K prefix. Sampled units against
    the oracle, and the chunk's rows against the call over all 128K tokens."""
    base = synth.named("llama128k_fp8")
    alpha = synth.alpha_for("llama128k_fp8", "0.05")
    L = base.seqlens[0]
    P = L - 32768
    whole = synth.generate(base)
    chunk = synth.generate(base.replace(seqlens=[L - P], prefix=[P]))
    print("chunk of %d after prefix %d, alpha %g" % (L - P, P, alpha), flush=True)
    o1, m1, l1 = gu.gpu_prefill(chunk, gu.params_for(chunk, alpha, kv_splits=1, score_splits=1))
    ow, mw, lw = gu.gpu_prefill(whole, gu.params_for(whole, alpha, kv_splits=1, score_splits=1))
    B = base.block_size
    np.testing.assert_array_equal(m1[0], mw[0, :, P // B:, :])
    np.testing.assert_array_equal(o1, ow[P:])
    np.testing.assert_array_equal(l1, lw[P:])
    del whole, ow, mw, lw
    # the default call (cost-balanced KV splits) against the unsplit one
    oc, mc, lc = gu.gpu_prefill(chunk, gu.params_for(chunk, alpha))
    np.testing.assert_array_equal(mc, m1)
    print("planned vs unsplit: max |diff| %.3g" % np.abs(oc - o1).max())
    assert np.abs(oc - o1).max() <= gu.TOL["fp8"]
    del o1, l1
    units = gu.units_of(chunk, sample=8, seed=2)
    inp = oracle.Inputs(chunk)
    op = gu.oracle_params(inp, alpha)
    omask, ell, mu = oracle.estimate(inp, op, units=units, want_scores=True)
    ob, ibm, ib = gu.compare_masks(mc, omask, ell, mu, alpha, units)
    print("mask on %d units: outside-band mismatches %d, in-band %d of %d" % (len(units), ob, ibm, ib))
    assert ob == 0
    oout, olse = oracle.attend(inp, op, mc, units=units)
    gu.check_close(oc, oout, lc, olse, "fp8", rows=gu.unit_rows(chunk, units),
                   label="same-mask (%d sampled units)" % len(units))


@pytest.mark.parametrize("name", ["bf16_paged_ragged", "fp8_unaligned", "g1_paged"])
@pytest.mark.parametrize("ss", [1, 3, 5, 64])
def test_score_splits_parity(name, ss):
    """The scoring with its query rows split into at most `ss` parts per unit
    (uneven and empty parts included) against the oracle; the same bars as
    the prefill parity, and the kept lists agree with the mask."""
    wl = _wl(name)
    sp = wl.spec
    alpha = 0.98
    out, gmask, lse = gu.gpu_prefill(wl, gu.params_for(wl, alpha, score_splits=ss))
    inp = oracle.Inputs(wl)
    op = gu.oracle_params(inp, alpha)
    omask, ell, mu = oracle.estimate(inp, op, want_scores=True)
    ob, ibm, ib = gu.compare_masks(gmask, omask, ell, mu, alpha, gu.units_of(wl))
    print("score_splits %d: mask outside-band mismatches %d, in-band %d of %d" % (ss, ob, ibm, ib))
    assert ob == 0
    oout, olse = oracle.attend(inp, op, gmask)
    gu.check_close(out, oout, lse, olse, sp.dtype)
