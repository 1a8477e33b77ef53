"""fp2_prefill_noalloc (the prefill whose scratch is the library's static
device array) against fp2_prefill with a caller workspace, through the C ABI:
two calls in a row, the second on a smaller input, each bit for bit equal to
the workspace call (same kernels, same inputs). Also run after other GPU
work in the same process, where the array still holds an earlier call's
contents."""
import numpy as np
import pytest
import torch

import paper_2608_19758_amd as fp2
import synth
from tests import gpu_util as gu

pytestmark = pytest.mark.gpu


def _spec(lens, hq, hkv, dtype, seed):
    return synth.Spec("noalloc", list(lens), hq, hkv, dtype=dtype, page_size=64, salient_frac=0.1,
                      salient_min=2, sink_blocks=1, window_blocks=2, seed=seed)


def _both(wl, alpha):
    p = gu.params_for(wl, alpha)
    d = gu.device_tensors(wl)
    bt = d["block_table"] if wl.spec.page_size else None
    kw = dict(cu_seqlens_host=wl.cu_seqlens, q_scale=d["q_scale"], k_scale=d["k_scale"],
              v_scale=d["v_scale"])
    lse_n = torch.empty((wl.spec.total_tokens, wl.spec.num_q_heads), dtype=torch.float32,
                        device="cuda")
    on, mn, ln = fp2.prefill_noalloc(p, d["q"], d["k_cache"], d["v_cache"], d["cu_seqlens"], bt,
                                     lse=lse_n, **kw)
    torch.cuda.synchronize()
    ow, mw, lw = fp2.prefill(p, d["q"], d["k_cache"], d["v_cache"], d["cu_seqlens"], bt,
                             want_lse=True, **kw)
    torch.cuda.synchronize()
    return [t.cpu().numpy() for t in (on.view(torch.int16), mn, ln, ow.view(torch.int16), mw, lw)]


@pytest.mark.parametrize("dtype", ["bf16", "fp8"])
def test_noalloc_equals_workspace_call(dtype):
    big = synth.generate(_spec([3000, 1700], 32, 8, dtype, 5))
    small = synth.generate(_spec([900], 8, 2, dtype, 6))
    for name, wl in (("larger", big), ("smaller", small)):
        print("noalloc %s %s lens %s" % (dtype, name, wl.spec.seqlens), flush=True)
        on, mn, ln, ow, mw, lw = _both(wl, 0.98)
        np.testing.assert_array_equal(mn, mw)
        np.testing.assert_array_equal(on, ow)
        np.testing.assert_array_equal(ln, lw)


def test_noalloc_refuses_oversized_call():
    p = fp2.make_params(batch=4, num_q_heads=32, num_kv_heads=8, max_seq_len=131072,
                        page_size=64, max_pages_per_seq=2048, alpha=0.98)
    q = torch.empty((16, 32, 128), dtype=torch.bfloat16, device="cuda")
    kv = torch.empty((64, 8, 128), dtype=torch.bfloat16, device="cuda")
    cu = torch.zeros(5, dtype=torch.int32, device="cuda")
    bt = torch.zeros((4, 2048), dtype=torch.int32, device="cuda")
    with pytest.raises(fp2.Fp2Error, match="static array"):
        fp2.prefill_noalloc(p, q, kv, kv, cu, bt)
