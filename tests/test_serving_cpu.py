"""Host side of the serving backend (no GPU): per-forward validation, length
arrays, and the worst-case workspace bound every admissible forward fits."""
import numpy as np
import pytest

import paper_2608_19758_amd as fp2
from paper_2608_19758_amd import serving

CFG = serving.BackendConfig(num_q_heads=32, num_kv_heads=8, page_size=64, max_batch=4,
                            max_extend_len=8192, max_kv_len=65536, dtype="fp8")


def test_plan_forward_unaligned_prefix():
    plan = serving.plan_forward(CFG, [100, 64], [100, 4097])
    assert plan.cu_k.tolist() == [0, 200, 4361]


def test_plan_forward_arrays():
    plan = serving.plan_forward(CFG, [300, 8192, 1], [1024, 0, 4096])
    assert plan.cu_q.tolist() == [0, 300, 8492, 8493]
    assert plan.cu_k.tolist() == [0, 1324, 9516, 13613]
    assert plan.total_tokens == 8493
    p = plan.params
    assert (p.batch, p.max_seq_len, p.max_kv_len) == (3, 8192, 8192)
    assert p.max_pages_per_seq == 1024 and p.dtype == fp2.FP8_E4M3


@pytest.mark.parametrize("ext,pre,msg", [
    ([9000], [0], "max_extend_len"),
    ([8192], [65536 - 4096], "max_kv_len"),
    ([1, 1, 1, 1, 1], None, "max_batch"),
    ([1, 2], [0], "differ"),
    ([-1], None, "negative"),
])
def test_plan_forward_rejects(ext, pre, msg):
    with pytest.raises(ValueError, match=msg):
        serving.plan_forward(CFG, ext, pre)


def test_worst_case_workspace_bounds_every_forward():
    worst = fp2.workspace_bytes(CFG.worst_case_params())
    assert worst > 0
    rng = np.random.default_rng(0)
    for _ in range(200):
        b = int(rng.integers(1, CFG.max_batch + 1))
        ext = rng.integers(0, CFG.max_extend_len + 1, size=b)
        pre = rng.integers(0, CFG.max_kv_len - ext + 1)
        plan = serving.plan_forward(CFG, ext.tolist(), pre.tolist())
        assert 0 <= fp2.workspace_bytes(plan.params) <= worst
    # fixed split counts scale the partial outputs with the problem, still bounded
    cfg4 = serving.BackendConfig(**{**CFG.__dict__, "kv_splits": 4})
    worst4 = fp2.workspace_bytes(cfg4.worst_case_params())
    plan = serving.plan_forward(cfg4, [8192, 8192], [57344, 0])
    assert fp2.workspace_bytes(plan.params) <= worst4
