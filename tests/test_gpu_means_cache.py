"""GPU tests of the block-means cache (fp2_prefill_cached): a chunked prefill
that keeps the pooled means of complete blocks between its calls.

A sequence is prefilled in two calls over one paged KV pool: the first chunk
(positions [0, P)), then the rest with P tokens of prefix. The cache starts
poisoned (NaN bf16 everywhere); the first call pools every block it sees and
writes it to its slot, the second copies the P // 128 complete blocks and
pools the rest. Bars: the second call's mask, outputs and LSE equal those of
fp2_prefill without a cache bit for bit; the cache then holds, in every block's
slot, exactly the means fp2_pool computes over the whole sequence; a
pooled_blocks beyond the complete blocks is clamped (same results again).
"""
import numpy as np
import pytest
import torch

import paper_2608_19758_amd as fp2
import synth
from tests import gpu_util as gu

pytestmark = pytest.mark.gpu

B = 128
NAN_BF16 = 0x7FC0


def spec(lens, page, hq=8, hkv=2, dtype="bf16", seed=31):
    pool = sum((L + page - 1) // page for L in lens) + 9
    return synth.Spec("meanscache", list(lens), hq, hkv, dtype=dtype, page_size=page,
                      page_order="permuted", pool_pages=pool, salient_frac=0.1, salient_min=2,
                      sink_blocks=1, window_blocks=2, recent_blocks=0, mean_correction=1,
                      seed=seed)


def slot(wl, b, J):
    """The documented slot of key block J of sequence b."""
    p = wl.spec.page_size
    t = J * B
    return int(wl.block_table[b][t // p]) * ((p + B - 1) // B) + (t % p) // B


def call(wl, d, rows, kv_lens, q_lens, alpha, cache=None, pooled=None):
    """fp2_prefill(_cached) for the query rows `rows` (per sequence, a slice of
    that sequence's positions) against the first kv_lens[b] tokens of the pool."""
    sp = wl.spec
    cu_q = np.concatenate([[0], np.cumsum(q_lens)]).astype(np.int32)
    cu_k = np.concatenate([[0], np.cumsum(kv_lens)]).astype(np.int32)
    q = torch.cat([d["q"][int(wl.cu_seqlens[b]) + r.start:int(wl.cu_seqlens[b]) + r.stop]
                   for b, r in enumerate(rows)])
    p = fp2.make_params(batch=sp.batch, num_q_heads=sp.num_q_heads, num_kv_heads=sp.num_kv_heads,
                        max_seq_len=max(q_lens), page_size=sp.page_size,
                        max_pages_per_seq=wl.max_pages, alpha=alpha,
                        sink_blocks=sp.sink_blocks, window_blocks=sp.window_blocks,
                        recent_blocks=sp.recent_blocks, mean_correction=1, dtype=sp.dtype,
                        max_kv_len=max(kv_lens))
    mc = None
    if cache is not None:
        mc = (cache[0], cache[1], torch.tensor(pooled, dtype=torch.int32, device="cuda"))
    out, mask, lse = fp2.prefill(p, q, d["k_cache"], d["v_cache"], torch.from_numpy(cu_q).cuda(),
                                 d["block_table"], cu_seqlens_host=cu_q,
                                 cu_seqlens_k=torch.from_numpy(cu_k).cuda(), cu_seqlens_k_host=cu_k,
                                 q_scale=d["q_scale"], k_scale=d["k_scale"], v_scale=d["v_scale"],
                                 want_lse=True, means_cache=mc)
    torch.cuda.synchronize()
    return out.float().cpu().numpy(), mask.cpu().numpy(), lse.cpu().numpy()


CASES = [
    dict(lens=[1500, 700], cut=[640, 300], page=64, dtype="bf16"),
    dict(lens=[1300], cut=[1024], page=16, dtype="fp8"),
    dict(lens=[900, 1800], cut=[129, 1], page=200, dtype="bf16"),
    dict(lens=[2000, 333], cut=[1000, 128], page=128, dtype="fp8"),
]


@pytest.mark.parametrize("case", CASES, ids=lambda c: "p%d_%s_%s" % (c["page"], c["dtype"],
                                                                      "_".join(map(str, c["cut"]))))
def test_chunked_with_means_cache(case):
    print("means-cache case", case, flush=True)
    lens, cut = case["lens"], case["cut"]
    wl = synth.generate(spec(lens, case["page"], dtype=case["dtype"]))
    d = gu.device_tensors(wl)
    sp = wl.spec
    alpha = 0.98
    pnum = int(wl.num_pages)
    slots = fp2.means_cache_slots(gu.params_for(wl, alpha), pnum)
    assert slots == pnum * ((sp.page_size + B - 1) // B)
    kh = torch.full((slots, sp.num_kv_heads, 128), 0, dtype=torch.int16, device="cuda")
    kh.fill_(NAN_BF16)
    vb = kh.clone()
    cache = (kh.view(torch.bfloat16), vb.view(torch.bfloat16))
    # first chunk: positions [0, cut), KV = the same tokens; nothing cached yet
    r1 = [range(0, c) for c in cut]
    call(wl, d, r1, cut, cut, alpha, cache, [0] * len(lens))
    # second chunk with and without the cache
    r2 = [range(c, L) for c, L in zip(cut, lens)]
    q2 = [L - c for c, L in zip(cut, lens)]
    want = call(wl, d, r2, lens, q2, alpha)
    got = call(wl, d, r2, lens, q2, alpha, cache, [c // B for c in cut])
    for a, g in zip(want, got):
        np.testing.assert_array_equal(a, g)
    # the cache now holds the means of every block of the whole sequences
    p = gu.params_for(wl, alpha)
    khat, vbar = fp2.pool(p, d["k_cache"], d["v_cache"], d["cu_seqlens"], d["block_table"],
                          cu_seqlens_host=wl.cu_seqlens, k_scale=d["k_scale"],
                          v_scale=d["v_scale"])
    torch.cuda.synchronize()
    khat = khat.view(torch.int16).cpu().numpy()
    vbar = vbar.view(torch.int16).cpu().numpy()
    khc, vbc = kh.cpu().numpy(), vb.cpu().numpy()
    for b, L in enumerate(lens):
        for J in range((L + B - 1) // B):
            s = slot(wl, b, J)
            np.testing.assert_array_equal(khc[s], khat[b, :, J])
            np.testing.assert_array_equal(vbc[s], vbar[b, :, J])
    # pooled_blocks past the complete blocks is clamped
    again = call(wl, d, r2, lens, q2, alpha, cache, [10 ** 6] * len(lens))
    for a, g in zip(want, again):
        np.testing.assert_array_equal(a, g)
