"""CPU emulation of when the HIP kernels raise their running max.

Both the prefill attention kernel and the decode kernels form probabilities
against a running max that moves lazily: a tile's probabilities are taken
against the current (possibly stale) max, and only when some row's half-tile
sum exceeds 2^13 (or is not finite, as on the first tile where the max is
-inf) does the wave raise the max, rescale O and the running sum, and redo the
tile.  This module replays that decision, in fp64, on the same schedule as
the prefill kernel (waves of 32 query rows, 256-row workgroups, 128-key
tiles, the 32x32 accumulator's split of each 32-key block between the two
lane halves) so that a test can show which of its inputs take the rescale
path after the first tile.  It is test instrumentation for the kernel's
control flow, not a reference for its values (the oracle is that).
"""
from __future__ import annotations

import math

import numpy as np

SUM_LIMIT = 8192.0
WAVE_ROWS = 32
WG_ROWS = 256
TILE = 128


def _bf16(bits):
    a = np.asarray(bits, dtype=np.uint16).astype(np.uint32) << np.uint32(16)
    return a.view(np.float32).astype(np.float64)


def _half_of_key(offset_in_block):
    # lane half h holds keys 8*(r >> 2) + 4*h + (r & 3) of each 32-key block
    return (offset_in_block // 4) % 2


def late_raises(logits2, vis_end, wg_tiles):
    """Count tiles after the first where one wave's rescale branch runs.

    logits2 [32, K] base-2 scaled logits of one wave's rows against the
    concatenated keys; vis_end [32] one past each row's last visible key;
    wg_tiles the number of 128-key tiles the wave's workgroup visits.
    Returns the number of tiles t >= 1 whose branch fires and raises the
    finite max of some row (so a non-zero accumulator is rescaled)."""
    n_rows, K = logits2.shape
    m_run = np.full(n_rows, -np.inf)
    fired = 0
    keys = np.arange(K)
    half = _half_of_key(keys % 32)
    for t in range(wg_tiles):
        c0, c1 = t * TILE, min((t + 1) * TILE, K)
        if c0 >= K:
            x = np.full((n_rows, 0), -np.inf)
            hk = half[:0]
        else:
            x = logits2[:, c0:c1].copy()
            x[keys[None, c0:c1] >= vis_end[:, None]] = -np.inf
            hk = half[c0:c1]
        with np.errstate(invalid="ignore", over="ignore"):
            e = np.exp2(x - m_run[:, None])
            sums = np.stack([np.where(hk[None, :] == h, e, 0.0).sum(axis=1) for h in (0, 1)], 1)
        if not np.all(sums <= SUM_LIMIT) and x.shape[1]:
            m_new = np.maximum(m_run, x.max(axis=1))
            # a rescale of a non-zero accumulator: a row with a finite max
            # (it has seen keys before) whose max moves up
            if t > 0 and np.any(np.isfinite(m_run) & (m_new > m_run)):
                fired += 1
            m_run = m_new
    return fired


def prefill_late_raises(q, k, v, k_pass, anchor_len, scale=None, heads=None):
    """Late rescale count of the prefill kernel over every wave of the given
    query heads.  q [n_q, M, d], k [n_kv, M, d], k_pass [host_idx, n_kv, l_p,
    d], bf16 bits.  ``scale`` defaults to 1/sqrt(d)."""
    n_q, M, d = q.shape
    n_kv = k.shape[0]
    g = n_q // n_kv
    lp_rows = k_pass.shape[0] * k_pass.shape[2]
    if scale is None:
        scale = 1.0 / math.sqrt(d)
    s2 = scale / math.log(2.0)
    heads = range(n_q) if heads is None else heads
    total = 0
    for hq in heads:
        kv = hq // g
        kc = np.concatenate([_bf16(k[kv, :anchor_len])]
                            + [_bf16(k_pass[s, kv]) for s in range(k_pass.shape[0])]
                            + [_bf16(k[kv, anchor_len:])], axis=0)
        qh = _bf16(q[hq])
        for w0 in range(0, M, WAVE_ROWS):
            rows = np.arange(w0, w0 + WAVE_ROWS)
            valid = rows < M
            rr = np.minimum(rows, M - 1)
            vis = np.where(rr < anchor_len, rr, rr + lp_rows) + 1
            qrows = np.where(valid[:, None], qh[rr], 0.0)
            wg_last = min((w0 // WG_ROWS + 1) * WG_ROWS, M) - 1
            wg_vis = (wg_last if wg_last < anchor_len else wg_last + lp_rows) + 1
            tiles = (wg_vis + TILE - 1) // TILE
            K = min(kc.shape[0], tiles * TILE)
            logits2 = (qrows @ kc[:K].T) * s2
            total += late_raises(logits2, vis, tiles)
    return total


def decode_late_raises(q, k_cache, k_new, block, scale=None):
    """Late rescale count of a decode kernel whose split plan is one split
    (the caller checks that): every 32-row wave of a GQA group walks the
    keys [cache; new] in blocks of ``block`` keys (32: the one-wave kernel,
    128: the eight-wave kernel) from a running max of -inf.  q [n_q, n_new,
    d], k_cache [n_kv, Lc, d], k_new [n_kv, n_new, d] or None (bf16 bits).
    A block whose keys a row cannot see leaves that row's max at -inf, as in
    the kernels."""
    n_q, n_new, d = q.shape
    n_kv, lc, _ = k_cache.shape
    g = n_q // n_kv
    if scale is None:
        scale = 1.0 / math.sqrt(d)
    s2 = scale / math.log(2.0)
    total = 0
    for kv in range(n_kv):
        keys = _bf16(k_cache[kv])
        if k_new is not None:
            keys = np.concatenate([keys, _bf16(k_new[kv])], axis=0)
        K = keys.shape[0]
        R = g * n_new
        rows_q = np.stack([_bf16(q[kv * g + r // n_new, r % n_new]) for r in range(R)])
        tok = np.arange(R) % n_new
        vis_all = lc + (tok + 1 if k_new is not None else 0)
        nblk = (K + block - 1) // block
        for w0 in range(0, R, WAVE_ROWS):
            rr = np.arange(w0, min(w0 + WAVE_ROWS, R))
            logits2 = (rows_q[rr] @ keys.T) * s2
            vis = vis_all[rr]
            m_run = np.full(len(rr), -np.inf)
            idx = np.arange(K)
            half = _half_of_key(idx % 32)
            for b in range(nblk):
                c0, c1 = b * block, min((b + 1) * block, K)
                x = logits2[:, c0:c1].copy()
                x[idx[None, c0:c1] >= vis[:, None]] = -np.inf
                hk = half[c0:c1]
                with np.errstate(invalid="ignore", over="ignore"):
                    e = np.exp2(x - m_run[:, None])
                    sums = np.stack([np.where(hk[None, :] == h, e, 0.0).sum(axis=1)
                                     for h in (0, 1)], 1)
                if not np.all(sums <= SUM_LIMIT):
                    m_new = np.maximum(m_run, x.max(axis=1))
                    if b > 0 and np.any(np.isfinite(m_run) & (m_new > m_run)):
                        total += 1
                    m_run = m_new
    return total
