"""Pins of the C oracle against things other than itself (CPU only).

P1  alpha = 0 keeps every causal block -> dense causal attention (torch SDPA
    and a textbook loop).
P2  alpha > 1 leaves exactly the forced blocks; alpha = 1 adds the argmax.
P3  masks nest as alpha grows.
P4  block causality: data of later blocks changes neither mask row I nor the
    outputs of block I.
P5  the normalised form of Sec. 3.1 Eq. (1)-(2) with epsilon selects the same
    blocks as the oracle's log-energy test (Eq. select).
P6  keys constant inside each block -> the corrected output equals dense
    attention for any mask (Sec. 3.2 Eq. taylor with every delta = 0).
P7  with within-block noise independent of V, the correction lowers the error
    against dense attention (Sec. 3.2 Eq. cov / Eq. ratio).
P8  V == 1 -> every output is 1 (softmax weights incl. surrogate masses sum to 1);
    V in [0, 1] -> outputs in [0, 1].
P9  tiny inputs: an independent NumPy formulation agrees exactly on the mask
    and to 1e-12 on the output.
P10 paged (identity or permuted pages, any page size) == contiguous, bitwise.
P12 codecs against torch's casts (exhaustive for bf16 and e4m3fn decode).
"""
import math

import numpy as np
import pytest
import torch

import oracle
import synth
from tests import brute


def spec(lens, hq=4, hkv=1, dtype="bf16", page=0, order="identity", B=128, seed=1,
         sink=1, window=1, recent=0, corr=1, **kw):
    pool = 0
    if order == "permuted":
        pool = sum((L + page - 1) // page for L in lens) + 7
    return synth.Spec("t", list(lens), hq, hkv, head_dim=kw.pop("d", 128), block_size=B,
                      dtype=dtype, page_size=page, page_order=order, pool_pages=pool,
                      salient_frac=kw.pop("frac", 0.0), salient_min=kw.pop("smin", 2),
                      sink_blocks=sink, window_blocks=window, recent_blocks=recent,
                      mean_correction=corr, seed=seed, **kw)


def run(wl, alpha, **kw):
    inp = oracle.Inputs(wl)
    p = inp.params(alpha, **kw)
    mask, ell, mu = oracle.estimate(inp, p, want_scores=True)
    out, lse = oracle.attend(inp, p, mask)
    return mask, ell, mu, out, lse


CASES = [
    dict(lens=[300], hq=4, hkv=1),
    dict(lens=[128, 1, 257], hq=2, hkv=2, page=16, order="permuted"),
    dict(lens=[512], hq=8, hkv=2, B=64, page=64),
    dict(lens=[200, 64], hq=4, hkv=2, dtype="fp8", page=32),
    dict(lens=[130], hq=3, hkv=1, B=64),
]


# ---------------------------------------------------------------- P1
@pytest.mark.parametrize("case", CASES[:4])
def test_p1_alpha0_is_dense(case):
    wl = synth.generate(spec(**case))
    _, _, _, out, lse = run(wl, 0.0)
    ref = brute.dense_sdpa(wl)
    np.testing.assert_allclose(out, ref, atol=1e-12, rtol=0)
    loop = brute.dense_loop(wl)
    np.testing.assert_allclose(out, loop, atol=1e-12, rtol=0)
    mask = oracle.estimate(oracle.Inputs(wl), oracle.Inputs(wl).params(0.0))
    for b, L in enumerate(wl.spec.seqlens):
        n = (L + wl.spec.block_size - 1) // wl.spec.block_size
        tri = np.tril(np.ones((n, n), bool))
        assert ((mask[b, :, :n, :n] & 1).astype(bool) == tri[None]).all()


# ---------------------------------------------------------------- P2
@pytest.mark.parametrize("sink,window,recent", [(1, 1, 0), (2, 3, 0), (0, 1, 1), (3, 2, 2)])
def test_p2_alpha_above_one_keeps_forced_only(sink, window, recent):
    wl = synth.generate(spec([700, 333], hq=4, hkv=2, page=64, frac=0.2))
    inp = oracle.Inputs(wl)
    mask = oracle.estimate(inp, inp.params(1.5, sink=sink, window=window, recent=recent))
    B = wl.spec.block_size
    for b, L in enumerate(wl.spec.seqlens):
        n = (L + B - 1) // B
        for h in range(2):
            for I in range(n):
                f = brute.forced_set(n, I, I, sink, window, recent)
                for J in range(mask.shape[-1]):
                    want = (1 | 2) if J in f else 0
                    assert mask[b, h, I, J] == want, (b, h, I, J)


def test_p2_alpha_one_adds_argmax():
    wl = synth.generate(spec([900], hq=4, hkv=1, frac=0.3, seed=5))
    inp = oracle.Inputs(wl)
    mask = oracle.estimate(inp, inp.params(1.0, sink=0, window=1))
    bmask, bell, _, _ = brute.brute(wl, 1.0, sink=0, window=1)
    n = mask.shape[-1]
    for I in range(n):
        arg = int(np.nanargmax(bell[0, 0, I, :I + 1]))
        kept = set(np.nonzero(mask[0, 0, I] & 1)[0].tolist())
        assert kept == {arg, I}, (I, kept, arg)


# ---------------------------------------------------------------- P3
def test_p3_masks_nest_in_alpha():
    wl = synth.generate(spec([1500], hq=4, hkv=1, frac=0.1, seed=3))
    inp = oracle.Inputs(wl)
    prev = None
    ratios = []
    for a in [0.0, 0.5, 0.9, 0.97, 0.99, 0.999, 1.0, 2.0]:
        m = oracle.estimate(inp, inp.params(a)) & 1
        if prev is not None:
            assert ((m <= prev)).all(), a
        prev = m
        ratios.append(oracle.kept_ratio(m, wl.spec.seqlens, 128))
    assert all(x >= y for x, y in zip(ratios, ratios[1:]))
    assert ratios[0] == 1.0 and ratios[-1] < ratios[0]


# ---------------------------------------------------------------- P4
def test_p4_block_causality():
    sp = spec([1000], hq=4, hkv=1, frac=0.2, seed=9)
    wl = synth.generate(sp)
    wl2 = synth.generate(sp)
    B = sp.block_size
    I = 3
    rng = np.random.default_rng(0)
    # replace every Q/K/V token after block I with fresh random bf16 values
    t0 = (I + 1) * B
    for arr in (wl2.q, wl2.k_tok, wl2.v_tok):
        noise = rng.standard_normal(arr[t0:].shape).astype(np.float32) * 3
        arr[t0:] = torch.from_numpy(noise).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    m1, _, _, o1, l1 = run(wl, 0.98)
    m2, _, _, o2, l2 = run(wl2, 0.98)
    assert (m1[0, 0, :I + 1] == m2[0, 0, :I + 1]).all()
    assert (m1[0, 0, :, I + 1:][:I + 1] == 0).all()
    np.testing.assert_array_equal(o1[:t0], o2[:t0])
    np.testing.assert_array_equal(l1[:t0], l2[:t0])
    assert not np.array_equal(o1[t0:], o2[t0:])


# ---------------------------------------------------------------- P5
def _eq2_scores(wl, eps=1e-6):
    """Score_{I,J} of Sec. 3.1 Eq. (1)-(2): per-(I,J) max, rescale, normalise."""
    sp = wl.spec
    Q, K, _ = brute.decode(wl)
    B, g = sp.block_size, sp.num_q_heads // sp.num_kv_heads
    L = sp.seqlens[0]
    n = (L + B - 1) // B
    out = {}
    for h in range(sp.num_kv_heads):
        Kb = K[:L, h]
        kbar = np.stack([Kb[J * B:(J + 1) * B].mean(0) for J in range(n)])
        khat = brute.bf16_bits_to_f64(brute.bf16_round_bits(kbar))
        for I in range(n):
            qs = Q[I * B:min(L, (I + 1) * B), h * g:(h + 1) * g].reshape(-1, sp.head_dim)
            s = qs @ khat[:I + 1].T / math.sqrt(sp.head_dim)     # [rows, I+1]
            m = s.max(0)                                          # m_{I,J}
            S = np.exp(s - m).sum(0)                              # S_{I,J}
            M = m.max()
            num = S * np.exp(m - M)
            out[(h, I)] = num / (num.sum() + eps)
    return out


def test_p5_normalised_form_selects_same_blocks():
    wl = synth.generate(spec([1800], hq=4, hkv=2, frac=0.15, seed=11))
    scores = _eq2_scores(wl)
    ratios = np.concatenate([s / s.max() for s in scores.values()])
    ratios = np.unique(np.round(ratios, 15))
    inp = oracle.Inputs(wl)
    # pick alphas in the middle of gaps between attained ratios: no near-ties
    gaps = np.diff(ratios)
    picks = np.argsort(-gaps)[:5]
    for i in picks:
        a = float((ratios[i] + ratios[i + 1]) / 2)
        mask = oracle.estimate(inp, inp.params(a, sink=0, window=0))
        for (h, I), s in scores.items():
            want = (s >= a * s.max())
            want[I] = True      # diagonal is always kept
            got = (mask[0, h, I, :I + 1] & 1).astype(bool)
            assert (want == got).all(), (a, h, I)


# ---------------------------------------------------------------- P6
def _blockwise_constant_keys(wl):
    sp = wl.spec
    B = sp.block_size
    cu = wl.cu_seqlens
    for b, L in enumerate(sp.seqlens):
        for t in range(L):
            wl.k_tok[cu[b] + t] = wl.k_tok[cu[b] + (t // B) * B]
    return wl


@pytest.mark.parametrize("dtype", ["bf16", "fp8"])
def test_p6_correction_exact_for_constant_blocks(dtype):
    wl = _blockwise_constant_keys(synth.generate(spec([640, 300], hq=4, hkv=2, dtype=dtype,
                                                      page=64, frac=0.2, seed=4)))
    dense = brute.dense_sdpa(wl)
    inp = oracle.Inputs(wl)
    p = inp.params(0.5, correction=1)
    rng = np.random.default_rng(2)
    mask = oracle.estimate(inp, p)
    # any mask: randomise the non-diagonal part
    rnd = (rng.random(mask.shape) < 0.3).astype(np.uint8)
    for I in range(mask.shape[2]):
        rnd[:, :, I, I] = 1
        rnd[:, :, I, I + 1:] = 0
    for m in (mask, rnd):
        out, _ = oracle.attend(inp, p, m)
        np.testing.assert_allclose(out, dense, atol=1e-12, rtol=0)
    # and without the correction the result is not dense
    out0, _ = oracle.attend(inp, inp.params(0.5, correction=0), rnd)
    assert np.abs(out0 - dense).max() > 1e-3


# ---------------------------------------------------------------- P7
def test_p7_correction_reduces_error():
    wl = synth.generate(spec([2048], hq=4, hkv=1, frac=0.0, smin=3, seed=7))
    dense = brute.dense_sdpa(wl)
    inp = oracle.Inputs(wl)
    mask = oracle.estimate(inp, inp.params(0.99))
    on, _ = oracle.attend(inp, inp.params(0.99, correction=1), mask)
    off, _ = oracle.attend(inp, inp.params(0.99, correction=0), mask)
    e_on = np.abs(on - dense).mean()
    e_off = np.abs(off - dense).mean()
    print("P7 mean |err| with / without correction:", e_on, e_off)
    assert e_on < 0.5 * e_off


# ---------------------------------------------------------------- P8
@pytest.mark.parametrize("corr", [0, 1])
def test_p8_weights_sum_to_one(corr):
    sp = spec([700, 129], hq=4, hkv=2, page=64, frac=0.2, seed=8)
    wl = synth.generate(sp)
    one = np.uint16(0x3F80)  # bf16 1.0
    wl.v_tok[:] = one
    _, _, _, out, _ = run(wl, 0.99, correction=corr)
    np.testing.assert_allclose(out, 1.0, atol=1e-14, rtol=0)
    wl2 = synth.generate(sp)
    rng = np.random.default_rng(1)
    u = rng.random(wl2.v_tok.shape).astype(np.float32)
    wl2.v_tok[:] = torch.from_numpy(u).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    _, _, _, out2, _ = run(wl2, 0.99, correction=corr)
    assert out2.min() >= 0.0 and out2.max() <= 1.0


# ---------------------------------------------------------------- P9
@pytest.mark.parametrize("case", CASES)
@pytest.mark.parametrize("alpha", [0.0, 0.97, 0.995])
@pytest.mark.parametrize("corr", [0, 1])
def test_p9_brute_force(case, alpha, corr):
    case = dict(case)
    wl = synth.generate(spec(frac=0.2, **case))
    mask, ell, mu, out, lse = run(wl, alpha, correction=corr)
    bmask, bell, bout, blse = brute.brute(wl, alpha, correction=corr)
    np.testing.assert_allclose(ell, bell, atol=1e-12, rtol=0, equal_nan=True)
    if alpha > 0:
        marg = oracle.margins(ell, mu, alpha)
        # exact agreement is only meaningful away from exact ties
        assert np.nanmin(np.abs(marg)) > 1e-12
    np.testing.assert_array_equal(mask, bmask)
    np.testing.assert_allclose(out, bout, atol=1e-12, rtol=0)
    np.testing.assert_allclose(lse, blse, atol=1e-12, rtol=0)


# ---------------------------------------------------------------- P10
@pytest.mark.parametrize("dtype", ["bf16", "fp8"])
def test_p10_paged_equals_contiguous(dtype):
    base = spec([450, 1000, 77], hq=4, hkv=2, dtype=dtype, page=0, frac=0.1, seed=12)
    ref = run(synth.generate(base), 0.98)
    for page, order in [(64, "identity"), (16, "permuted"), (1, "permuted"), (128, "permuted")]:
        sp = spec([450, 1000, 77], hq=4, hkv=2, dtype=dtype, page=page, order=order, frac=0.1,
                  seed=12)
        got = run(synth.generate(sp), 0.98)
        for a, b in zip(ref, got):
            np.testing.assert_array_equal(a, b)


# ---------------------------------------------------------------- P12
def test_p12_bf16_decode_exhaustive():
    bits = np.arange(1 << 16, dtype=np.uint32).astype(np.uint16)
    ref = torch.from_numpy(bits.view(np.int16)).view(torch.bfloat16).to(torch.float64).numpy()
    got = np.array([oracle.bf16_decode(int(b)) for b in bits])
    same = (got == ref) | (np.isnan(got) & np.isnan(ref))
    assert same.all()


def test_p12_bf16_encode_matches_torch_on_float32():
    rng = np.random.default_rng(0)
    x = np.concatenate([
        rng.standard_normal(20000).astype(np.float32),
        (rng.standard_normal(5000) * 1e-38).astype(np.float32),      # bf16 subnormals
        np.clip(rng.standard_normal(2000) * 1e38, -3.3e38, 3.3e38).astype(np.float32),
        np.array([3.3895314e38, 3.40e38, -3.40e38, 1.0 + 2 ** -8, 1.0 + 3 * 2 ** -8,
                  2 ** -133, 2 ** -134, 1.5 * 2 ** -133, 0.0, -0.0], np.float32),
    ])
    # exact ties: 1 + k/256 with odd k
    x = np.concatenate([x, (1.0 + np.arange(1, 256, 2) / 256.0).astype(np.float32)])
    ref = torch.from_numpy(x).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    got = np.array([oracle.bf16_encode_rne(float(v)) for v in x], dtype=np.uint16)
    np.testing.assert_array_equal(got, ref)


def test_p12_bf16_encode_from_double_is_single_rounding():
    rng = np.random.default_rng(5)
    x = rng.standard_normal(20000) * np.exp(rng.uniform(-20, 20, 20000))
    ref = brute.bf16_round_bits(x)
    got = np.array([oracle.bf16_encode_rne(float(v)) for v in x], dtype=np.uint16)
    np.testing.assert_array_equal(got, ref)
    # a value just above a bf16 tie must round up even where a float32 detour ties
    v = 1.0 + 2 ** -8 + 2 ** -40
    assert oracle.bf16_encode_rne(v) == 0x3F81


def test_p12_e4m3_decode_exhaustive():
    bits = np.arange(256, dtype=np.uint8)
    ref = torch.from_numpy(bits).view(torch.float8_e4m3fn).to(torch.float64).numpy()
    got = np.array([oracle.e4m3_decode(int(b)) for b in bits])
    same = (got == ref) | (np.isnan(got) & np.isnan(ref))
    assert same.all()
    assert np.nanmax(got) == 448.0
