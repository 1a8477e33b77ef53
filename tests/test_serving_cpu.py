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


def _inputs(p, total, **over):
    import torch
    d = dict(q=torch.zeros(total, p.num_q_heads, 128, dtype=torch.uint8),
             k_cache=torch.zeros(256, p.num_kv_heads, 128, dtype=torch.uint8),
             v_cache=torch.zeros(256, p.num_kv_heads, 128, dtype=torch.uint8),
             cu_seqlens=torch.zeros(p.batch + 1, dtype=torch.int32),
             block_table=torch.zeros(p.batch, p.max_pages_per_seq, dtype=torch.int32),
             q_scale=torch.ones(p.num_q_heads), k_scale=torch.ones(p.num_kv_heads),
             v_scale=torch.ones(p.num_kv_heads))
    d.update(over)
    return d


@pytest.mark.parametrize("what,bad,msg", [
    ("block_table", "wider", "block_table must be int32"),
    ("block_table", "strided", "block_table must be contiguous"),
    ("block_table", "int64", "block_table must have dtype"),
    ("q", "bf16", "q must have 1-byte elements"),
    ("q", "strided", "q must be contiguous"),
    ("k_cache", "ragged", "k_cache: .* not a multiple"),
    ("cu_seqlens", "short", "cu_seqlens holds"),
    ("k_scale", "f64", "k_scale must have dtype"),
])
def test_binding_refuses_misshapen_tensors(what, bad, msg):
    """The C ABI takes bare pointers and reads the page table at row stride
    max_pages_per_seq: the binding refuses a table of another width, strided
    views, wrong element types and short arrays before anything is called."""
    import torch
    p = CFG.params(2, 1000, 1000)
    w = p.max_pages_per_seq
    bad_t = {
        ("block_table", "wider"): torch.zeros(2, w + 3, dtype=torch.int32),
        ("block_table", "strided"): torch.zeros(2, 2 * w, dtype=torch.int32)[:, ::2],
        ("block_table", "int64"): torch.zeros(2, w, dtype=torch.int64),
        ("q", "bf16"): torch.zeros(16, 32, 128, dtype=torch.bfloat16),
        ("q", "strided"): torch.zeros(16, 32, 256, dtype=torch.uint8)[:, :, :128],
        ("k_cache", "ragged"): torch.zeros(256 * 8 * 128 + 5, dtype=torch.uint8),
        ("cu_seqlens", "short"): torch.zeros(2, dtype=torch.int32),
        ("k_scale", "f64"): torch.ones(8, dtype=torch.float64),
    }[(what, bad)]
    d = _inputs(p, 16, **{what: bad_t})
    if what == "k_cache":
        d["v_cache"] = torch.zeros_like(bad_t)
    with pytest.raises(ValueError, match=msg):
        fp2._check_inputs(p, **d)
    # the same call with well-formed (host) tensors gets as far as the device check
    with pytest.raises(ValueError, match="must be a CUDA tensor"):
        fp2._check_inputs(p, **_inputs(p, 16))
