"""CPU model of the affine GEMM kernel's index arithmetic (test infrastructure).

The index expressions of the affine kernel (one output tile of 16 x 16 or
32 x 32 a block, k ranges of whole 16-k groups dealt to (split, wave), the
permuted k order inside a group, clamped rows, columns and k, the LDS partial
tiles of the waves, the split workspace and the fixed-order reduction)
restated in numpy for the launch shape the library reports (affine_plan, a
host-only query), and checked for every block tile (sampled for large
launches): every global read inside its operand, every k of the reduction
taken once per output tile, every output element written once, and the LDS
and workspace accesses inside their buffers.  Shares no code with the kernel
or the oracle.
"""
from __future__ import annotations

import numpy as np

from kernel_model import ModelError, cdiv, need, sample

WAVE = 64


def kpos(tsz, q, u):
    """Position inside a 16-k group of MFMA k-step u for lane quarter q."""
    if tsz == 8:
        return (u & 1) + 2 * q + 8 * (u >> 1)
    return 4 * q + u


def mfma_row(tsz, lane, r):
    """Output row of accumulator element r of a lane (16 x 16 x 4 MFMA)."""
    return (lane >> 4) + 4 * r if tsz == 8 else 4 * (lane >> 4) + r


def geometry(product, N, D, M):
    """(rows, cols, K, sAm, sAk, sBk, sBn, ldc, |A|, |B|, |C|) of a product."""
    if product == "forward":   # out = X W
        return N, M, D, D, 1, M, 1, M, N * D, D * M, N * M
    if product == "dX":        # dX = g W^T
        return N, D, M, M, 1, 1, M, D, N * M, D * M, N * D
    if product == "dW":        # dW = X^T g
        return D, M, N, 1, D, M, 1, M, N * D, N * M, D * M
    raise ModelError(f"unknown product {product}")


def check_gemm(product, N, D, M, tsz, plan, workspace_bytes):
    rows, cols, K, sAm, sAk, sBk, sBn, ldc, alen, blen, clen = geometry(product, N, D, M)
    TE, nk, splits = plan["tile"], plan["waves"], plan["splits"]
    need(TE in (16, 32) and 1 <= nk <= 8 and splits >= 1, f"{product}: plan {plan}")
    WT = TE // 16
    tm, tn = cdiv(rows, TE), cdiv(cols, TE)
    ntile = tm * tn
    need(ntile * splits < 2 ** 31 and splits <= 65535, f"{product}: grid")
    G = cdiv(K, 16)
    R = splits * nk
    # each 16-k group once per tile, over the (split, wave) ranges in order
    cover = np.zeros(G, dtype=np.int64)
    last = 0
    for r in range(R):
        lo, hi = r * G // R, (r + 1) * G // R
        need(lo == last, f"{product}: k ranges not contiguous")
        cover[lo:hi] += 1
        last = hi
    need(last == G and (cover == 1).all(), f"{product}: k groups not covered once")
    # the permuted k order covers each group
    q = np.arange(4)[:, None]
    u = np.arange(4)[None, :]
    need(sorted(kpos(tsz, q, u).ravel().tolist()) == list(range(16)),
         f"{product}: a k group's permutation")
    if splits > 1:
        need(splits * rows * cols * tsz <= workspace_bytes,
             f"{product}: partials exceed the workspace")
    lds_elems = nk * TE * TE if nk > 1 else 0
    lane = np.arange(WAVE)
    li, lq = lane & 15, lane >> 4
    tiles = sample(ntile)  # all tiles, or a fixed sample of a large launch
    written = np.zeros(rows * cols, dtype=np.int64) if len(tiles) == ntile else None
    for tile in tiles:
        i0, j0 = (tile % tm) * TE, (tile // tm) * TE
        for g in range(G):
            k = g * 16 + kpos(tsz, lq[:, None], np.arange(4)[None, :])  # (64, 4)
            part = g * 16 + 16 > K
            kc = np.minimum(k, K - 1) if part else k
            need(kc.max() < K, f"{product}: a full group reads past K")
            for x in range(WT):
                ar = np.minimum(i0 + 16 * x + li, rows - 1)
                bc = np.minimum(j0 + 16 * x + li, cols - 1)
                oa = ar[:, None] * sAm + kc * sAk
                ob = kc * sBk + bc[:, None] * sBn
                need(oa.min() >= 0 and oa.max() < alen, f"{product}: A read out of range")
                need(ob.min() >= 0 and ob.max() < blen, f"{product}: B read out of range")
        # outputs of the tile: (x, y, r, lane) -> (i, j); LDS slot of a wave's partial
        r = np.arange(4)[:, None]
        seen = set()
        for x in range(WT):
            for y in range(WT):
                ii = 16 * x + mfma_row(tsz, lane[None, :], r)
                jj = 16 * y + li[None, :] + 0 * r
                slot = ii * TE + jj
                need(slot.max() < TE * TE, f"{product}: LDS partial slot")
                seen.update((slot).ravel().tolist())
        need(len(seen) == TE * TE, f"{product}: the tile's elements not held once")
        if nk > 1:
            need((nk - 1) * TE * TE + TE * TE <= lds_elems, f"{product}: LDS partials")
        e = np.arange(TE * TE)
        gi, gj = i0 + e // TE, j0 + e % TE
        ok = (gi < rows) & (gj < cols)
        idx = gi[ok] * ldc + gj[ok]
        need(idx.size == 0 or idx.max() < clen, f"{product}: output out of range")
        if splits > 1:
            pidx = ((splits - 1) * rows + gi[ok]) * cols + gj[ok]
            need(pidx.size == 0 or pidx.max() < splits * rows * cols,
                 f"{product}: partial out of range")
        if written is not None:
            written[gi[ok] * cols + gj[ok]] += 1
    if written is not None:
        need((written == 1).all(), f"{product}: outputs not written once")
