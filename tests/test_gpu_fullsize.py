"""Full-size workloads on the GPU, in the launch configuration bench.py times.

Every workload compares the WHOLE block mask with the oracle's (bit-exact
outside the 1e-4 band around the threshold; in-band disagreements counted),
checks the forced bits against their closed form and the oracle's kept ratio
against the stored calibration, and compares outputs and LSE with the oracle
on sampled (sequence, KV head, query block) units: all units of the 2K
workload, 768 units (every KV head at 96 query blocks, the heaviest included)
of the 128K fp8 workloads, 128 units elsewhere. The error against dense
attention (the oracle with every block kept) on a few of the units is reported
beside the same-mask error."""
import numpy as np
import pytest

import oracle
import synth
from paper_2608_19758_amd import accounting as acc
from tests import gpu_util as gu

pytestmark = pytest.mark.gpu

# (workload, kept-ratio target, mean correction override, output units compared)
CASES = [("tiny2k", "0.30", None, None),
         ("llama32k", "0.18", None, 128),
         ("llama128k_fp8", "0.10", None, 128),
         ("llama128k_fp8", "0.05", None, 768),
         ("llama128k_fp8", "0.05", 0, 768),
         ("llama128k_fp8", "0.02", None, 128),
         ("llama128k_bf16", "0.05", None, 128),
         ("ragged8", "0.18", None, 128),
         ("wide128k_bf16", "0.009", None, 128),
         ("wide128k_fp8", "0.009", None, 128)]

_cache = {}


def _workload(name):
    """One generated workload at a time (the 128K ones hold GBs on the host)."""
    if name not in _cache:
        _cache.clear()
        _cache[name] = synth.generate(synth.named(name))
    return _cache[name]


def forced_closed_form(n, sink, window, recent):
    I = np.arange(n)[:, None]
    J = np.arange(n)[None, :]
    return (J <= I) & ((J < sink) | (I - J < window) | (J == I) | (J >= n - recent))


def strided_units(wl, count):
    """count units: every KV head of each sequence at evenly strided query
    blocks, each sequence's last (heaviest) block included."""
    sp = wl.spec
    B = sp.block_size
    per_seq = max(1, count // (sp.batch * sp.num_kv_heads))
    units = set()
    for b, L in enumerate(sp.seqlens):
        n = (L + B - 1) // B
        if n == 0:
            continue
        blocks = np.unique(np.linspace(n - 1, 0, min(n, per_seq)).round().astype(int))
        for h in range(sp.num_kv_heads):
            for I in blocks:
                units.add((b, h, int(I)))
    return sorted(units)


@pytest.mark.parametrize("name,target,corr,nunits", CASES,
                         ids=["%s@%s%s" % (c[0], c[1], "" if c[2] is None else "-corr%d" % c[2])
                              for c in CASES])
def test_fullsize_parity(name, target, corr, nunits):
    sp = synth.named(name)
    print("workload", name, "target", target, "correction", corr, "lens", sp.seqlens, flush=True)
    wl = _workload(name)
    alpha = synth.alpha_for(name, target)
    p = gu.params_for(wl, alpha, corr=corr)
    out, gmask, lse = gu.gpu_prefill(wl, p)
    assert np.isfinite(out).all() and np.isfinite(lse).all()
    B = sp.block_size
    for b, L in enumerate(sp.seqlens):
        n = (L + B - 1) // B
        f = forced_closed_form(n, sp.sink_blocks, sp.window_blocks, sp.recent_blocks)
        assert ((gmask[b, :, :n, :n] & 2).astype(bool) == f[None]).all()
        assert (gmask[b, :, n:, :] == 0).all() and (gmask[b, :, :, n:] == 0).all()
        assert not (gmask[b, :, :n, :n] & ~np.tril(np.ones((n, n), bool))[None]).any()

    # the whole mask against the oracle's
    inp = oracle.Inputs(wl)
    op = gu.oracle_params(inp, alpha, corr=corr)
    omask, ell, mu = oracle.estimate(inp, op, want_scores=True)
    ob, ibm, ib = gu.compare_masks_full(gmask, omask, ell, mu, alpha)
    print("whole mask: outside-band mismatches %d, in-band mismatches %d of %d in-band"
          % (ob, ibm, ib), flush=True)
    assert ob == 0
    okept = oracle.kept_ratio(omask, sp.seqlens, B)
    gkept = oracle.kept_ratio(gmask, sp.seqlens, B)
    want = synth.alphas()[name]["kept_ratio"][target]
    print("kept ratio GPU %.6f, oracle %.6f, stored calibration %.6f" % (gkept, okept, want))
    assert okept == pytest.approx(want, rel=1e-12, abs=1e-15)
    del ell, mu

    units = gu.units_of(wl) if nunits is None else strided_units(wl, nunits)
    oout, olse = oracle.attend(inp, op, gmask, units=units)
    rows = gu.unit_rows(wl, units)
    gu.check_close(out, oout, lse, olse, sp.dtype, rows=rows,
                   label="same-mask (%d units)" % len(units))
    # reported next to it: the error of the sparse output against dense
    # attention (every block kept, the oracle at alpha = 0) on a few units
    du = units[::max(1, len(units) // 4)][:4]
    op0 = gu.oracle_params(inp, 0.0)
    dmask = oracle.estimate(inp, op0, units=du)
    dout, _ = oracle.attend(inp, op0, dmask, units=du)
    dworst, num, den = 0.0, 0.0, 0.0
    for rs, hs in gu.unit_rows(wl, du):
        diff = out[rs, hs] - dout[rs, hs]
        dworst = max(dworst, float(np.abs(diff).max()))
        num += float((diff ** 2).sum())
        den += float((dout[rs, hs] ** 2).sum())
    print("vs dense attention on %d units: max-abs err %.3g, relative Frobenius %.3g"
          % (len(du), dworst, (num / max(den, 1e-300)) ** 0.5))
    assert np.isfinite(dworst)


def test_fullsize_attention_flops_accounting():
    """Executed-FLOP accounting matches a direct count on a GPU mask."""
    sp = synth.named("llama32k")
    wl = _workload("llama32k")
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
    _cache.clear()
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
    gu.check_close(out, oout, lse, olse, "fp8", rows=gu.unit_rows(wl, units),
                   label="same-mask (%d units)" % len(units))
