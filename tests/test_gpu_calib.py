"""GPU checks of the rate-calibration loops (fp2_calibrate): each kind runs,
writes nothing to its sink, and its measured rate lies between a floor that
a working loop clears and the ceiling the operation count allows -- a rate
above the vendor's dense peak (bf16 2.5 PFLOP/s, fp8 5.0 PFLOP/s) or above
every SIMD retiring one full-rate exp instruction per 4 cycles at 2.4 GHz
would mean the count is wrong."""
import pytest
import torch

import paper_2608_19758_amd as fp2

pytestmark = pytest.mark.gpu

CASES = [("mfma_bf16", 20000, 2.5e15), ("mfma_fp8", 10000, 5.0e15),
         ("exp", 10000, 256 * 4 * 64 / 4 * 2.4e9)]


@pytest.mark.parametrize("kind,iters,ceiling", CASES, ids=[c[0] for c in CASES])
def test_calibration_rate(kind, iters, ceiling):
    print("calibration case", kind, iters, flush=True)
    sink = torch.zeros(1, dtype=torch.float32, device="cuda")
    fp2.calibrate(kind, iters, sink)
    torch.cuda.synchronize()
    a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    a.record()
    ops = sum(fp2.calibrate(kind, iters, sink) for _ in range(3))
    b.record()
    torch.cuda.synchronize()
    rate = ops / (a.elapsed_time(b) * 1e-3)
    print("%s: %.4g ops/s (%.3f of the ceiling)" % (kind, rate, rate / ceiling))
    assert sink.item() == 0.0
    assert 0.2 * ceiling < rate <= 1.05 * ceiling
