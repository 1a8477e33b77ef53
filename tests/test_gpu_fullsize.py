"""Full-size workloads on the GPU (the launch configuration bench.py times),
checked against the oracle on sampled (sequence, KV head, query block) units
that the oracle computes one by one, plus properties that hold at any size:
every output finite, forced-block bits exact for every block, rows past a
sequence zero, and the kept ratio equal to the oracle-calibrated one up to
blocks inside the margin band. The error against dense attention (every
block kept) on four of the sampled units is reported beside the same-mask error."""
import numpy as np
import pytest

import oracle
import synth
from paper_2608_19758_amd import accounting as acc
from tests import gpu_util as gu

pytestmark = pytest.mark.gpu

CASES = [("llama32k", "0.18"), ("llama128k_fp8", "0.05"), ("llama128k_fp8", "0.02"),
         ("llama128k_bf16", "0.05"), ("ragged8", "0.18"), ("wide128k_bf16", "0.009"),
         ("wide128k_fp8", "0.009")]


def forced_closed_form(n, sink, window, recent):
    I = np.arange(n)[:, None]
    J = np.arange(n)[None, :]
    return (J <= I) & ((J < sink) | (I - J < window) | (J == I) | (J >= n - recent))


@pytest.mark.parametrize("name,target", CASES)
def test_fullsize_sampled_parity(name, target):
    sp = synth.named(name)
    print("workload", name, "target", target, "lens", sp.seqlens, flush=True)
    wl = synth.generate(sp)
    alpha = synth.alpha_for(name, target)
    p = gu.params_for(wl, alpha)
    out, gmask, lse = gu.gpu_prefill(wl, p)
    assert np.isfinite(out).all() and np.isfinite(lse).all()
    B = sp.block_size
    for b, L in enumerate(sp.seqlens):
        n = (L + B - 1) // B
        f = forced_closed_form(n, sp.sink_blocks, sp.window_blocks, sp.recent_blocks)
        assert ((gmask[b, :, :n, :n] & 2).astype(bool) == f[None]).all()
        assert (gmask[b, :, n:, :] == 0).all() and (gmask[b, :, :, n:] == 0).all()
        assert not (gmask[b, :, :n, :n] & ~np.tril(np.ones((n, n), bool))[None]).any()

    units = gu.units_of(wl, sample=16, seed=1)
    inp = oracle.Inputs(wl)
    op = gu.oracle_params(inp, alpha)
    omask, ell, mu = oracle.estimate(inp, op, units=units, want_scores=True)
    ob, ibm, ib = gu.compare_masks(gmask, omask, ell, mu, alpha, units)
    print("mask on %d units: outside-band mismatches %d, in-band %d of %d" % (len(units), ob, ibm, ib))
    assert ob == 0
    oout, olse = oracle.attend(inp, op, gmask, units=units)
    worst = 0.0
    for rs, hs in gu.unit_rows(wl, units):
        worst = max(worst, float(np.abs(out[rs, hs] - oout[rs, hs]).max()))
        assert np.abs(lse[rs, hs] - olse[rs, hs]).max() <= gu.LSE_TOL[sp.dtype]
    print("same-mask max-abs err on sampled units %.3g (tol %g)" % (worst, gu.TOL[sp.dtype]))
    assert worst <= gu.TOL[sp.dtype]
    # reported next to it: the error of the sparse output against dense
    # attention (every block kept, the oracle at alpha = 0) on four of the units
    du = units[::4]
    op0 = gu.oracle_params(inp, 0.0)
    dmask = oracle.estimate(inp, op0, units=du)
    dout, _ = oracle.attend(inp, op0, dmask, units=du)
    dworst, num, den = 0.0, 0.0, 0.0
    for rs, hs in gu.unit_rows(wl, du):
        diff = out[rs, hs] - dout[rs, hs]
        dworst = max(dworst, float(np.abs(diff).max()))
        num += float((diff ** 2).sum())
        den += float((dout[rs, hs] ** 2).sum())
    print("vs dense attention on %d units: max-abs err %.3g, relative Frobenius %.3g "
          "(same-mask max-abs %.3g)" % (len(du), dworst, (num / max(den, 1e-300)) ** 0.5, worst))
    assert np.isfinite(dworst)
    kept = oracle.kept_ratio(gmask, sp.seqlens, B)
    want = synth.alphas()[name]["kept_ratio"][target]
    tot = sum((L + B - 1) // B * ((L + B - 1) // B + 1) // 2 for L in sp.seqlens) * sp.num_kv_heads
    print("kept ratio GPU %.5f, oracle calibration %.5f" % (kept, want))
    # a block can only flip when its energy is within the band of the threshold
    assert abs(kept - want) * tot <= max(4, 0.002 * tot)


def test_fullsize_attention_flops_accounting():
    """Executed-FLOP accounting matches a direct count on a GPU mask."""
    sp = synth.named("llama32k")
    wl = synth.generate(sp)
    out, gmask, _ = gu.gpu_prefill(wl, gu.params_for(wl, synth.alpha_for("llama32k", "0.18")))
    n = sp.max_seq_len // 128
    kept = int((gmask[0, :, :n, :n] & 1).sum())
    corr = sum(int(((gmask[0, h, I, :I] & 1) == 0).sum()) for h in range(8) for I in range(n))
    fk, fc = acc.attention_flops(gmask, sp.seqlens, 32, 8)
    assert fk == 4 * 128 * 4 * 128 * 128 * kept
    assert fc == 4 * 128 * 4 * 128 * corr


def test_maximum_sequence_length():
    """One sequence of 1,048,576 tokens, the largest the library admits (8192
    key blocks: the longest energy row, kept lists and correction lists),
    fp8, 4 query heads on 1 KV head, paged; sampled units against the oracle
    and the closed-form forced bits everywhere."""
    sp = synth.Spec("max1m", [1 << 20], 4, 1, dtype="fp8", page_size=64, salient_frac=0.005,
                    salient_min=1, sink_blocks=1, window_blocks=2, seed=17)
    print("workload 1M tokens", flush=True)
    wl = synth.generate(sp)
    alpha = 0.98
    out, gmask, lse = gu.gpu_prefill(wl, gu.params_for(wl, alpha))
    assert np.isfinite(out).all() and np.isfinite(lse).all()
    n = (1 << 20) // 128
    assert gmask.shape == (1, 1, n, n)
    f = forced_closed_form(n, 1, 2, 0)
    assert ((gmask[0, 0] & 2).astype(bool) == f).all()
    kept = oracle.kept_ratio(gmask, sp.seqlens, 128)
    print("kept ratio %.5f" % kept)
    units = [(0, 0, n - 1), (0, 0, 3)]
    inp = oracle.Inputs(wl)
    op = gu.oracle_params(inp, alpha)
    omask, ell, mu = oracle.estimate(inp, op, units=units, want_scores=True)
    ob, ibm, ib = gu.compare_masks(gmask, omask, ell, mu, alpha, units)
    print("mask on %d units: outside-band mismatches %d, in-band %d of %d" % (len(units), ob, ibm, ib))
    assert ob == 0
    oout, olse = oracle.attend(inp, op, gmask, units=units)
    worst = 0.0
    for rs, hs in gu.unit_rows(wl, units):
        worst = max(worst, float(np.abs(out[rs, hs] - oout[rs, hs]).max()))
        assert np.abs(lse[rs, hs] - olse[rs, hs]).max() <= gu.LSE_TOL["fp8"]
    print("same-mask max-abs err on sampled units %.3g" % worst)
    assert worst <= gu.TOL["fp8"]
