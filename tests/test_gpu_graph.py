"""fp2_prefill captured in a HIP graph (torch.cuda.graph) and replayed.

The library only enqueues kernels on the caller's stream: it allocates,
clears and synchronises nothing (the plan kernel resets the attention's work
counter on every call, and the outputs come from torch's fill kernels), so a
serving engine can capture a call once and replay it. Bar: every replay gives
the mask, outputs and LSE of an eager call on the same inputs bit for bit,
with eager work and synchronisations between the replays and the queries
changed in place between them.
"""
import numpy as np
import pytest
import torch

import paper_2608_19758_amd as fp2
import synth
from tests import gpu_util as gu

pytestmark = pytest.mark.gpu

LENS = [1500, 700, 129]


def spec(dtype, page, seed=41):
    pool = sum((L + page - 1) // page for L in LENS) + 5
    return synth.Spec("graph", list(LENS), 8, 2, dtype=dtype, page_size=page,
                      page_order="permuted", pool_pages=pool, salient_frac=0.1, salient_min=2,
                      sink_blocks=1, window_blocks=2, recent_blocks=0, mean_correction=1,
                      seed=seed)


def bits(t):
    t = t.detach()
    if t.dtype == torch.bfloat16:
        t = t.view(torch.int16)
    elif t.dtype == torch.float32:
        t = t.view(torch.int32)
    return t.cpu().numpy()


@pytest.mark.parametrize("dtype,page,kv_splits", [("bf16", 64, 0), ("fp8", 16, 0), ("bf16", 48, 1)],
                         ids=["bf16_p64_planned", "fp8_p16_planned", "bf16_p48_nosplit"])
def test_prefill_graph_replays(dtype, page, kv_splits):
    print("graph case", dtype, page, kv_splits, flush=True)
    wl = synth.generate(spec(dtype, page))
    d = gu.device_tensors(wl)
    p = gu.params_for(wl, 0.98, kv_splits=kv_splits)

    def call():
        return fp2.prefill(p, d["q"], d["k_cache"], d["v_cache"], d["cu_seqlens"],
                           d["block_table"], cu_seqlens_host=wl.cu_seqlens, q_scale=d["q_scale"],
                           k_scale=d["k_scale"], v_scale=d["v_scale"], want_lse=True)

    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):   # warm-up off the capture
        call()
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        g_out, g_mask, g_lse = call()
    torch.cuda.synchronize()

    q0 = d["q"].clone()
    for rep in range(4):
        if rep == 2:   # new queries in place: the rows of q rotated by one token
            d["q"].copy_(torch.roll(q0, shifts=1, dims=0))
        graph.replay()
        x = torch.randn(1 << 20, device="cuda")
        float(x.sum())   # eager work and a synchronisation between replays
        got = [bits(g_mask), bits(g_out), bits(g_lse)]
        want_out, want_mask, want_lse = call()
        torch.cuda.synchronize()
        want = [bits(want_mask), bits(want_out), bits(want_lse)]
        for name, a, b in zip(["mask", "out", "lse"], want, got):
            assert np.array_equal(a, b), "replay %d: %s differs" % (rep, name)
        print("replay %d matches the eager call (kept %d)" % (rep, int((got[0] & 1).sum())),
              flush=True)
    d["q"].copy_(q0)
