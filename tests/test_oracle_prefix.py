"""Pins of the oracle's prefix-KV (chunked prefill) path (CPU only).

A sequence may hold L_kv = P + L keys of which the L queries are the last
ones.

P15 chunked == whole: the chunk's mask rows, outputs and LSE equal the rows of
    the same positions in the run over the whole sequence (the selection of a
    query block depends only on its own rows and the keys before it; Sec. 3.1
    Eq. select, Sec. 3.2 Eq. correction), bitwise.
P16 alpha = 0 with a prefix keeps every block up to the query's absolute block
    and equals dense attention with the causal mask shifted by P (torch SDPA
    with an explicit boolean mask, fp64).

Prefixes that are not block multiples (a query block straddles key blocks
Ja = a0/B and Jb = a1/B):
P23 alpha = 0 keeps exactly J <= Jb and equals the shifted-causal SDPA.
P24 the NumPy brute force (prefix-aware, both tile modes) agrees on every mask
    byte and to 1e-12 on energies, outputs and LSE.
P25 forced bits follow the closed form: sink, Jb - J < window, the band
    Ja <= J <= Jb, recent.
"""
import numpy as np
import pytest
import torch

import oracle
import synth
from tests import brute


def spec(lens, prefix=None, hq=4, hkv=1, dtype="bf16", page=0, order="identity", B=128, seed=3,
         sink=1, window=1, recent=0, corr=1, frac=0.05):
    kvl = [L + (prefix[i] if prefix else 0) for i, L in enumerate(lens)]
    pool = sum((L + page - 1) // page for L in kvl) + 5 if order == "permuted" else 0
    return synth.Spec("t", list(lens), hq, hkv, block_size=B, dtype=dtype, page_size=page,
                      page_order=order, pool_pages=pool, salient_frac=frac, salient_min=1,
                      sink_blocks=sink, window_blocks=window, recent_blocks=recent,
                      mean_correction=corr, seed=seed, prefix=prefix)


def run(wl, alpha, **kw):
    inp = oracle.Inputs(wl)
    p = inp.params(alpha, **kw)
    mask = oracle.estimate(inp, p)
    out, lse = oracle.attend(inp, p, mask)
    return mask, out, lse


CHUNKS = [
    dict(kv=[900], pre=[256]),
    dict(kv=[900], pre=[512], page=32, order="permuted"),
    dict(kv=[700, 300], pre=[384, 0], hq=4, hkv=2, page=64),
    dict(kv=[650], pre=[128], dtype="fp8", page=16),
    dict(kv=[1000], pre=[256], B=64, hq=2, hkv=2, recent=2, window=2),
]


@pytest.mark.parametrize("case", CHUNKS)
@pytest.mark.parametrize("alpha", [0.0, 0.9, 2.0])
def test_p15_chunk_equals_whole(case, alpha):
    case = dict(case)
    kv, pre = case.pop("kv"), case.pop("pre")
    whole = synth.generate(spec(kv, **case))
    chunk = synth.generate(spec([L - p for L, p in zip(kv, pre)], prefix=pre, **case))
    B = whole.spec.block_size
    # the generator reproduces the KV tokens and the query rows of the whole
    assert np.array_equal(chunk.k_tok, whole.k_tok) and np.array_equal(chunk.v_tok, whole.v_tok)
    mw, ow, lw = run(whole, alpha)
    mc, oc, lc = run(chunk, alpha)
    for b, (L, p) in enumerate(zip(kv, pre)):
        rows_w = slice(whole.cu_seqlens[b] + p, whole.cu_seqlens[b + 1])
        rows_c = slice(chunk.cu_seqlens[b], chunk.cu_seqlens[b + 1])
        assert np.array_equal(chunk.q[rows_c], whole.q[rows_w])
        nq = (L - p + B - 1) // B
        nk = (L + B - 1) // B
        assert np.array_equal(mc[b, :, :nq, :nk], mw[b, :, p // B:p // B + nq, :nk])
        assert np.array_equal(oc[rows_c], ow[rows_w])
        assert np.array_equal(lc[rows_c], lw[rows_w])


@pytest.mark.parametrize("case", [dict(lens=[300], pre=[256]),
                                  dict(lens=[200, 129], pre=[128, 384], hq=4, hkv=2, page=16),
                                  dict(lens=[150], pre=[512], dtype="fp8", page=64)])
def test_p16_alpha0_prefix_is_dense(case):
    case = dict(case)
    lens, pre = case.pop("lens"), case.pop("pre")
    wl = synth.generate(spec(lens, prefix=pre, **case))
    sp = wl.spec
    mask, out, lse = run(wl, 0.0)
    B = sp.block_size
    for b, (L, p) in enumerate(zip(lens, pre)):
        nq, nk = (L + B - 1) // B, (L + p + B - 1) // B
        want = np.zeros((nq, nk), bool)
        for I in range(nq):
            want[I, :I + p // B + 1] = True
        assert ((mask[b, :, :nq, :nk] & 1).astype(bool) == want[None]).all()
    Q, K, V = brute.decode(wl)
    g = sp.num_q_heads // sp.num_kv_heads
    cu, ck = wl.cu_seqlens, wl.cu_seqlens_k
    for b, (L, p) in enumerate(zip(lens, pre)):
        q = torch.from_numpy(Q[cu[b]:cu[b + 1]]).permute(1, 0, 2).contiguous()
        k = torch.from_numpy(K[ck[b]:ck[b + 1]]).permute(1, 0, 2).repeat_interleave(g, 0).contiguous()
        v = torch.from_numpy(V[ck[b]:ck[b + 1]]).permute(1, 0, 2).repeat_interleave(g, 0).contiguous()
        vis = torch.arange(L + p)[None, :] <= (p + torch.arange(L))[:, None]
        ref = torch.nn.functional.scaled_dot_product_attention(q, k, v, attn_mask=vis)
        np.testing.assert_allclose(out[cu[b]:cu[b + 1]], ref.permute(1, 0, 2).numpy(), atol=1e-12,
                                   rtol=0)


# Prefixes that are not multiples of the block size: a query block's rows then
# lie in two key blocks Ja = a0/B and Jb = a1/B (a0, a1 its first and last
# absolute positions).
UNALIGNED = [
    dict(lens=[300], pre=[100]),
    dict(lens=[200, 129, 5], pre=[1, 300, 1000], hq=4, hkv=2, page=16),
    dict(lens=[260], pre=[127], dtype="fp8", page=64, window=1),
    dict(lens=[150, 70], pre=[65, 129], hq=8, hkv=2, page=0, recent=1),
]


@pytest.mark.parametrize("case", UNALIGNED)
def test_p23_unaligned_alpha0_is_dense(case):
    case = dict(case)
    lens, pre = case.pop("lens"), case.pop("pre")
    wl = synth.generate(spec(lens, prefix=pre, **case))
    sp = wl.spec
    mask, out, lse = run(wl, 0.0)
    B = sp.block_size
    for b, (L, p) in enumerate(zip(lens, pre)):
        for I in range((L + B - 1) // B):
            Jb = (p + min(L, (I + 1) * B) - 1) // B
            assert (mask[b, :, I, :Jb + 1] & 1).all() and not mask[b, :, I, Jb + 1:].any()
    Q, K, V = brute.decode(wl)
    g = sp.num_q_heads // sp.num_kv_heads
    cu, ck = wl.cu_seqlens, wl.cu_seqlens_k
    for b, (L, p) in enumerate(zip(lens, pre)):
        q = torch.from_numpy(Q[cu[b]:cu[b + 1]]).permute(1, 0, 2).contiguous()
        k = torch.from_numpy(K[ck[b]:ck[b + 1]]).permute(1, 0, 2).repeat_interleave(g, 0).contiguous()
        v = torch.from_numpy(V[ck[b]:ck[b + 1]]).permute(1, 0, 2).repeat_interleave(g, 0).contiguous()
        vis = torch.arange(L + p)[None, :] <= (p + torch.arange(L))[:, None]
        ref = torch.nn.functional.scaled_dot_product_attention(q, k, v, attn_mask=vis)
        np.testing.assert_allclose(out[cu[b]:cu[b + 1]], ref.permute(1, 0, 2).numpy(), atol=1e-12,
                                   rtol=0)


@pytest.mark.parametrize("case", UNALIGNED)
@pytest.mark.parametrize("alpha", [0.9, 2.0])
@pytest.mark.parametrize("tile_rows", [0, 128])
def test_p24_unaligned_brute_force(case, alpha, tile_rows):
    case = dict(case)
    lens, pre = case.pop("lens"), case.pop("pre")
    wl = synth.generate(spec(lens, prefix=pre, **case))
    inp = oracle.Inputs(wl)
    p = inp.params(alpha, tile_rows=tile_rows)
    mask, ell, mu = oracle.estimate(inp, p, want_scores=True)
    out, lse = oracle.attend(inp, p, mask)
    bm, bell, bout, blse = brute.brute(wl, alpha, tile_rows=tile_rows)
    np.testing.assert_array_equal(mask, bm)
    ok = ~np.isnan(bell)
    np.testing.assert_allclose(ell[ok], bell[ok], atol=1e-12, rtol=0)
    np.testing.assert_allclose(out, bout, atol=1e-12, rtol=0)
    np.testing.assert_allclose(lse, blse, atol=1e-12, rtol=0)


def test_p25_unaligned_forced_closed_form():
    lens, pre = [700, 300], [100, 250]
    wl = synth.generate(spec(lens, prefix=pre, hq=4, hkv=2, sink=2, window=2, recent=1))
    mask, _, _ = run(wl, 2.0)          # alpha > 1: the forced blocks only
    B = 128
    for b, (L, p) in enumerate(zip(lens, pre)):
        n = (L + p + B - 1) // B
        for I in range((L + B - 1) // B):
            Ja, Jb = (p + I * B) // B, (p + min(L, (I + 1) * B) - 1) // B
            want = np.array([J <= Jb and (J < 2 or Jb - J < 2 or J >= Ja or J >= n - 1)
                             for J in range(mask.shape[-1])])
            assert ((mask[b, :, I] >> 1).astype(bool) == want[None]).all()
            assert ((mask[b, :, I] & 1).astype(bool) == want[None]).all()
