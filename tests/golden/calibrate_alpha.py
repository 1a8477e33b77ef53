"""Calibrate the selection threshold alpha of each named workload (oracle only).

For every workload in ``synth.NAMES`` and each target kept-block ratio, the
oracle's block scores ell (log block energies) and row maxima mu are computed
once; the kept ratio of a threshold alpha is then the fraction of causal
blocks with ell >= ln(alpha) + mu or forced (the oracle's own rule). The ratio
does not increase with alpha, so bisection finds the alpha closest to the
target; alpha is then moved to the middle of the widest gap between attained
score ratios within +-0.2% of that value, so that as few blocks as possible sit
next to the threshold. Writes ``synth/alpha.json`` (inputs of the workloads,
not expected values).

Usage: python tests/golden/calibrate_alpha.py [name ...]
"""
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
sys.path.insert(0, ROOT)

import oracle  # noqa: E402
import synth  # noqa: E402

TARGETS = {
    "tiny2k": ["0.30"],
    "llama32k": ["0.18"],
    "llama128k_fp8": ["0.10", "0.05", "0.02"],
    "llama128k_bf16": ["0.10", "0.05", "0.02"],
    "ragged8": ["0.18"],
    "wide128k_bf16": ["0.009"],
    "wide128k_fp8": ["0.009"],
}


def forced_mask(spec, n):
    I = np.arange(n)[:, None]
    J = np.arange(n)[None, :]
    f = (J <= I) & ((J < spec.sink_blocks) | (I - J < spec.window_blocks) | (J == I)
                    | (J >= n - spec.recent_blocks))
    return f


def calibrate(name, seed=0):
    spec = synth.named(name, seed)
    t0 = time.time()
    wl = synth.generate(spec)
    inp = oracle.Inputs(wl)
    p = inp.params(0.5)
    _, ell, mu = oracle.estimate(inp, p, want_scores=True)
    t1 = time.time()
    B = spec.block_size
    # per sequence: log score ratio r = ell - mu for candidate (non-forced) causal blocks
    logr, nforced, total = [], 0, 0
    for b, L in enumerate(spec.seqlens):
        n = (L + B - 1) // B
        f = forced_mask(spec, n)
        tri = np.tril(np.ones((n, n), bool))
        for h in range(spec.num_kv_heads):
            r = ell[b, h, :n, :n] - mu[b, h, :n, None]
            logr.append(r[tri & ~f])
        nforced += int(f.sum()) * spec.num_kv_heads
        total += n * (n + 1) // 2 * spec.num_kv_heads
    logr = np.sort(np.concatenate(logr))[::-1]          # descending

    def ratio(alpha):
        kept = np.searchsorted(-logr, -np.log(alpha), side="right")  # logr >= ln alpha
        return (kept + nforced) / total

    out = {}
    for tgt in TARGETS[name]:
        target = float(tgt)
        lo, hi = 1e-6, 1.0
        for _ in range(80):
            mid = (lo + hi) / 2
            if ratio(mid) > target:
                lo = mid
            else:
                hi = mid
        a = hi if abs(ratio(hi) - target) <= abs(ratio(lo) - target) else lo
        # widest gap of attained ratios near a
        la = np.log(a)
        win = logr[(logr > la + np.log(0.998)) & (logr < la + np.log(1.002))]
        if win.size >= 2:
            gaps = -np.diff(win)
            i = int(np.argmax(gaps))
            a = float(np.exp((win[i] + win[i + 1]) / 2))
        a = float("%.9g" % a)
        out[tgt] = {"alpha": a, "kept_ratio": ratio(a)}
        print("%s target %s: alpha %.9g -> kept %.5f (oracle %.1fs)" % (name, tgt, a, ratio(a), t1 - t0),
              flush=True)
    return {"alpha": {k: v["alpha"] for k, v in out.items()},
            "kept_ratio": {k: v["kept_ratio"] for k, v in out.items()},
            "seed": seed}


def main(names):
    path = os.path.join(ROOT, "synth", "alpha.json")
    data = {}
    if os.path.exists(path):
        with open(path) as f:
            data = json.load(f)
    for n in names:
        data[n] = calibrate(n)
        with open(path, "w") as f:
            json.dump(data, f, indent=1, sort_keys=True)


if __name__ == "__main__":
    main(sys.argv[1:] or list(TARGETS))
