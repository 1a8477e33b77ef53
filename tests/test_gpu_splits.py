"""GPU parity of the KV splits (Sec. 3.3 Eq. split and Eq. cost) with their
log-sum-exp combine, through the C ABI.

With U parts, part u of a unit walks kept-list positions [u ceil(T/U),
min((u+1) ceil(T/U), T)) and the u-th range of pruned blocks; a combine
kernel merges the partial outputs. The mask does not depend on the splits
(bitwise); the output is the unsplit one up to rounding, so both are held to
the same bars against the fp64 oracle: max-abs 2e-2 (bf16) / 6e-2 (fp8), LSE
1e-2 / 0.0625. Fixed part counts (kv_splits = n) cover more parts than kept
blocks (empty parts) and parts of a single kept block; the cost-balanced plan
(kv_splits = 0, the default) splits the heavy units of short chunks after
long prefixes, where the step budget is small.
"""
import numpy as np
import pytest
import torch

import oracle
import paper_2608_19758_amd as fp2
import synth
from tests import gpu_util as gu

pytestmark = pytest.mark.gpu


def spec(lens, prefix=None, hq=4, hkv=1, dtype="bf16", page=64, order="identity", seed=7,
         frac=0.1, sink=1, window=2, recent=0, corr=1):
    kvl = [L + p for L, p in zip(lens, prefix)] if prefix is not None else list(lens)
    pool = sum((L + page - 1) // page for L in kvl) + 5 if (page and order == "permuted") else 0
    return synth.Spec("splits", list(lens), hq, hkv, dtype=dtype, page_size=page,
                      page_order=order, pool_pages=pool, salient_frac=frac, salient_min=2,
                      sink_blocks=sink, window_blocks=window, recent_blocks=recent,
                      mean_correction=corr, seed=seed, prefix=prefix)


CASES = {
    "bf16_contig": dict(lens=[2048], hq=4, hkv=1, page=0),
    "bf16_ragged_perm": dict(lens=[1000, 129, 1], hq=8, hkv=2, page=16, order="permuted"),
    "g1_prefix": dict(lens=[600], prefix=[1280], hq=2, hkv=2, page=32),
    "fp8_paged": dict(lens=[1800, 333], hq=8, hkv=2, dtype="fp8", page=64),
    "fp8_g8_prefix": dict(lens=[300], prefix=[2048], hq=8, hkv=1, dtype="fp8", page=16,
                          order="permuted"),
    "bf16_unaligned": dict(lens=[500, 70], prefix=[1000, 31], hq=4, hkv=2, page=32),
}


def _wl(name):
    c = dict(CASES[name])
    print("case", name, c, flush=True)
    return synth.generate(spec(**c))


def _check(wl, out, gmask, lse, alpha, corr=None):
    sp = wl.spec
    inp = oracle.Inputs(wl)
    op = gu.oracle_params(inp, alpha, corr=corr)
    oout, olse = oracle.attend(inp, op, gmask)
    gu.check_close(out, oout, lse, olse, sp.dtype)
    return oout


@pytest.mark.parametrize("name", list(CASES))
@pytest.mark.parametrize("splits", [2, 3, 7, 32])
def test_splits_parity(name, splits):
    wl = _wl(name)
    alpha = 0.99
    o1, m1, l1 = gu.gpu_prefill(wl, gu.params_for(wl, alpha, kv_splits=1))
    ou, mu_, lu = gu.gpu_prefill(wl, gu.params_for(wl, alpha, kv_splits=splits))
    np.testing.assert_array_equal(mu_, m1)           # selection does not depend on the splits
    d = np.abs(ou - o1).max()
    print("splits %d: max |split - unsplit| %.3g" % (splits, d))
    _check(wl, ou, mu_, lu, alpha)


@pytest.mark.parametrize("name", ["bf16_ragged_perm", "fp8_g8_prefix"])
@pytest.mark.parametrize("corr", [0, 1])
def test_splits_attend_external_mask(name, corr):
    """fp2_attend with splits under the oracle's mask (alpha 0.5: long kept lists)."""
    wl = _wl(name)
    sp = wl.spec
    alpha = 0.5
    inp = oracle.Inputs(wl)
    op = gu.oracle_params(inp, alpha, corr=corr)
    omask = oracle.estimate(inp, op)
    oout, olse = oracle.attend(inp, op, omask)
    p = gu.params_for(wl, alpha, corr=corr, kv_splits=5)
    d = gu.device_tensors(wl)
    out, lse = fp2.attend(p, d["q"], d["k_cache"], d["v_cache"], d["cu_seqlens"],
                          torch.from_numpy(omask).cuda(), d["block_table"] if sp.page_size else None,
                          cu_seqlens_host=wl.cu_seqlens, q_scale=d["q_scale"],
                          k_scale=d["k_scale"], v_scale=d["v_scale"], want_lse=True,
                          **gu.kv_args(wl, d))
    torch.cuda.synchronize()
    gu.check_close(out.float().cpu().numpy(), oout, lse.cpu().numpy(), olse, sp.dtype,
                   label="external-mask with 5 splits")


@pytest.mark.parametrize("dtype", ["bf16", "fp8"])
def test_planned_splits_short_chunk_after_prefix(dtype):
    """A 200-token chunk after a 6K prefix: few, heavy units, so the plan's step
    budget is the 16-step minimum and most units are split; parity against the
    oracle and the unsplit call."""
    wl = synth.generate(spec([200, 70], prefix=[6144, 3072], hq=8, hkv=2, dtype=dtype, page=64))
    alpha = 0.98
    p = gu.params_for(wl, alpha)
    out, gmask, lse = gu.gpu_prefill(wl, p)
    o1, m1, _ = gu.gpu_prefill(wl, gu.params_for(wl, alpha, kv_splits=1))
    np.testing.assert_array_equal(gmask, m1)
    print("planned splits: max |split - unsplit| %.3g" % np.abs(out - o1).max())
    _check(wl, out, gmask, lse, alpha)


def test_splits_fullsize_tail_chunk_sampled():
    """The last 1K chunk of the 128K fp8 shape (127K prefix): planned splits,
    sampled units against the oracle, all rows against the unsplit call within
    the fp8 bar."""
    base = synth.named("llama128k_fp8")
    alpha = synth.alpha_for("llama128k_fp8", "0.05")
    L = base.seqlens[0]
    P = L - 1024
    wl = synth.generate(base.replace(seqlens=[L - P], prefix=[P]))
    p = gu.params_for(wl, alpha)
    out, gmask, lse = gu.gpu_prefill(wl, p)
    o1, m1, l1 = gu.gpu_prefill(wl, gu.params_for(wl, alpha, kv_splits=1))
    np.testing.assert_array_equal(gmask, m1)
    d = np.abs(out - o1).max()
    print("tail chunk: max |split - unsplit| %.3g, lse %.3g" % (d, np.abs(lse - l1).max()))
    assert d <= gu.TOL["fp8"]
    units = gu.units_of(wl, sample=6, seed=3)
    inp = oracle.Inputs(wl)
    op = gu.oracle_params(inp, alpha)
    oout, olse = oracle.attend(inp, op, gmask, units=units)
    gu.check_close(out, oout, lse, olse, "fp8", rows=gu.unit_rows(wl, units),
                   label="same-mask (%d sampled units)" % len(units))
