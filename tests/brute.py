"""Independent NumPy formulations used to pin the C oracle on tiny inputs.

These are deliberately written differently from ``oracle/oracle.c``:

* decoding goes through torch's own bf16 / float8_e4m3fn casts;
* bf16 rounding of the block mean works on the integer bit pattern of the
  double (round half to even on the 45 dropped mantissa bits);
* block scores come from the full [L, g, n] query-by-pooled-key score matrix
  and SciPy's logsumexp;
* selection sorts the row's scores;
* attention builds the full token-level weight row in which every pruned
  block's keys and values are replaced by their block means (the view in
  which the mean correction is exact, Sec. 3.2 Eq. taylor with delta = 0).
"""
from __future__ import annotations

import numpy as np
import torch
from scipy.special import logsumexp


def decode(wl):
    """float64 Q [total, Hq, d], K, V [total, Hkv, d] (token-major) via torch casts."""
    sp = wl.spec
    if sp.dtype == "bf16":
        def dec(bits):
            t = torch.from_numpy(bits.view(np.int16)).view(torch.bfloat16)
            return t.to(torch.float64).numpy()
        return dec(wl.q), dec(wl.k_tok), dec(wl.v_tok)

    def dec8(bits, sc):
        t = torch.from_numpy(bits).view(torch.float8_e4m3fn).to(torch.float64).numpy()
        return t * sc.astype(np.float64)[None, :, None]
    return dec8(wl.q, wl.q_scale), dec8(wl.k_tok, wl.k_scale), dec8(wl.v_tok, wl.v_scale)


def bf16_round_bits(x: np.ndarray) -> np.ndarray:
    """Round float64 values to bf16 (ties to even) on the double's bit pattern.

    Valid for zero and for |x| in the bf16 normal range, which is all these
    tests produce; anything else raises.
    """
    x = np.asarray(x, dtype=np.float64)
    ax = np.abs(x)
    ok = (ax == 0) | ((ax >= 2.0 ** -126) & (ax < 2.0 ** 127))
    if not ok.all():
        raise ValueError("value outside the range this helper covers")
    u = x.view(np.uint64)
    sign = (u >> np.uint64(63)).astype(np.uint32)
    mag = u & np.uint64(0x7FFFFFFFFFFFFFFF)
    keep = mag >> np.uint64(45)
    rem = mag & np.uint64((1 << 45) - 1)
    half = np.uint64(1 << 44)
    up = (rem > half) | ((rem == half) & ((keep & np.uint64(1)) == np.uint64(1)))
    keep = keep + up.astype(np.uint64)
    # keep = (biased double exponent << 7) | 7-bit mantissa
    e = (keep >> np.uint64(7)).astype(np.int64)
    m = (keep & np.uint64(0x7F)).astype(np.uint32)
    e16 = np.where(mag == 0, 0, e - 1023 + 127).astype(np.uint32)
    m = np.where(mag == 0, 0, m)
    return ((sign << 15) | (e16 << 7) | m).astype(np.uint16)


def bf16_bits_to_f64(bits: np.ndarray) -> np.ndarray:
    return (bits.astype(np.uint32) << 16).view(np.float32).astype(np.float64)


def forced_set(n, Ja, Jb, sink, window, recent):
    """Forced blocks of a query block whose rows lie in key blocks Ja .. Jb."""
    return {J for J in range(Jb + 1)
            if J < sink or Jb - J < window or J >= Ja or J >= n - recent}


def brute(wl, alpha, sink=None, window=None, recent=None, correction=None, scale=None,
          tile_rows=0):
    """mask [b, Hkv, nt, nbk], ell (same shape, NaN above the last visible
    block), out [total, Hq, d], lse.

    tile_rows > 0: a query tile is tile_rows packed rows (tile_rows / g
    positions with all g heads) instead of a block of B positions. With a
    prefix the queries sit at absolute positions prefix + i."""
    sp = wl.spec
    sink = sp.sink_blocks if sink is None else sink
    window = sp.window_blocks if window is None else window
    recent = sp.recent_blocks if recent is None else recent
    corr = sp.mean_correction if correction is None else correction
    B, d, Hq, Hkv = sp.block_size, sp.head_dim, sp.num_q_heads, sp.num_kv_heads
    g = Hq // Hkv
    scale = 1.0 / np.sqrt(d) if scale is None else scale
    Q, K, V = decode(wl)
    Pt = tile_rows // g if tile_rows else B          # positions per query tile
    nbk = max(1, (sp.max_kv_len + B - 1) // B)
    ntmax = max(1, (sp.max_seq_len + Pt - 1) // Pt)
    mask = np.zeros((sp.batch, Hkv, ntmax, nbk), np.uint8)
    ell = np.full(mask.shape, np.nan)
    out = np.full(Q.shape, np.nan)
    lse = np.full(Q.shape[:2], np.nan)
    cu, ck = wl.cu_seqlens, wl.cu_seqlens_k
    for b, Lq in enumerate(sp.seqlens):
        if Lq == 0:
            continue
        Lk = sp.kvlens[b]
        P0 = Lk - Lq
        n = (Lk + B - 1) // B
        blk = np.arange(Lk) // B
        tile = np.arange(Lq) // Pt
        for h in range(Hkv):
            Kb = K[ck[b]:ck[b] + Lk, h]
            Vb = V[ck[b]:ck[b] + Lk, h]
            kbar = np.stack([Kb[blk == J].mean(0) for J in range(n)])
            vbar = np.stack([Vb[blk == J].mean(0) for J in range(n)])
            khat = bf16_bits_to_f64(bf16_round_bits(kbar))
            Qg = Q[cu[b]:cu[b] + Lq, h * g:(h + 1) * g]         # [Lq, g, d]
            S = np.einsum("lgd,jd->lgj", Qg, khat) * scale     # [Lq, g, n]
            for t in range((Lq + Pt - 1) // Pt):
                pos = np.arange(t * Pt, min(Lq, (t + 1) * Pt))  # local positions
                Ja, Jb = (P0 + pos[0]) // B, (P0 + pos[-1]) // B
                rows = S[tile == t].reshape(-1, n)[:, :Jb + 1]
                e = logsumexp(rows, axis=0)
                ell[b, h, t, :Jb + 1] = e
                order = np.argsort(-e, kind="stable")
                top = e[order[0]]
                kept = set()
                if alpha == 0:
                    kept = set(range(Jb + 1))
                else:
                    for J in order:
                        if e[J] >= np.log(alpha) + top:
                            kept.add(int(J))
                        else:
                            break
                forced = forced_set(n, Ja, Jb, sink, window, recent)
                for J in range(Jb + 1):
                    kb = J in kept or J in forced
                    mask[b, h, t, J] = int(kb) | (int(J in forced) << 1)
                # attention rows of the tile: pruned blocks -> mean tokens
                keptb = mask[b, h, t, :n] & 1
                Km, Vm = Kb.copy(), Vb.copy()
                allowed_blk = np.zeros(n, bool)
                for J in range(Jb + 1):
                    if keptb[J]:
                        allowed_blk[J] = True
                    elif corr and J < Ja:
                        Km[blk == J] = kbar[J]
                        Vm[blk == J] = vbar[J]
                        allowed_blk[J] = True
                for j in range(g):
                    qrow = Q[cu[b] + pos, h * g + j]            # [P, d]
                    lg = qrow @ Km.T * scale                   # [P, Lk]
                    ok = allowed_blk[blk][None, :] & (np.arange(Lk)[None, :] <= P0 + pos[:, None])
                    lg = np.where(ok, lg, -np.inf)
                    m = lg.max(1, keepdims=True)
                    w = np.exp(lg - m)
                    den = w.sum(1, keepdims=True)
                    out[cu[b] + pos, h * g + j] = (w @ Vm) / den
                    lse[cu[b] + pos, h * g + j] = (m + np.log(den))[:, 0]
    return mask, ell, out, lse


def dense_sdpa(wl, scale=None):
    """Dense causal GQA attention with torch's scaled_dot_product_attention in fp64."""
    sp = wl.spec
    Q, K, V = decode(wl)
    g = sp.num_q_heads // sp.num_kv_heads
    out = np.zeros_like(Q)
    cu = wl.cu_seqlens
    for b, L in enumerate(sp.seqlens):
        if L == 0:
            continue
        q = torch.from_numpy(Q[cu[b]:cu[b] + L]).permute(1, 0, 2)               # [Hq, L, d]
        k = torch.from_numpy(K[cu[b]:cu[b] + L]).permute(1, 0, 2).repeat_interleave(g, 0)
        v = torch.from_numpy(V[cu[b]:cu[b] + L]).permute(1, 0, 2).repeat_interleave(g, 0)
        o = torch.nn.functional.scaled_dot_product_attention(
            q.contiguous(), k.contiguous(), v.contiguous(), is_causal=True, scale=scale)
        out[cu[b]:cu[b] + L] = o.permute(1, 0, 2).numpy()
    return out


def dense_loop(wl, scale=None):
    """Dense causal attention, one row at a time (textbook softmax)."""
    sp = wl.spec
    Q, K, V = decode(wl)
    g = sp.num_q_heads // sp.num_kv_heads
    scale = 1.0 / np.sqrt(sp.head_dim) if scale is None else scale
    out = np.zeros_like(Q)
    cu = wl.cu_seqlens
    for b, L in enumerate(sp.seqlens):
        for p in range(L):
            for hq in range(sp.num_q_heads):
                s = K[cu[b]:cu[b] + p + 1, hq // g] @ Q[cu[b] + p, hq] * scale
                w = np.exp(s - s.max())
                out[cu[b] + p, hq] = w @ V[cu[b]:cu[b] + p + 1, hq // g] / w.sum()
    return out
