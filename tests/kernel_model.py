"""CPU model of the conv kernels' index arithmetic (test infrastructure).

The index expressions of the conv2d kernels -- LDS layout, LDS-DMA offsets,
register staging slots, fragment reads, split reductions, epilogues and global
addresses -- restated in numpy and evaluated for every block tile, wave, lane
and loop step of a launch, with the tiling the library itself reports for the
shape (conv2d_plan / conv2d_plan_fused: host-only queries, no GPU).  For each
access the model asserts that it stays inside its buffer (an LDS region inside
the block's dynamic LDS, the accesses of a region inside it, live regions
disjoint, a global access inside its tensor), that the integer divisions the
kernels take by magic multipliers or float reciprocals are exact on the values
they meet, and that the staging slots cover what the loops read.  For the
matrix-core kernels it also checks the meaning of the indices: every fragment
an MFMA consumes holds the operand the convolution needs there (the filter
value of row m and column k, the source cell of pixel q and tap k, or a zero
on one side), every k-step is taken once and every output element written once.

A kernel change that moves an index without the matching plan change shows up
here, on the CPU, before any GPU run.  The model restates the kernels' index
expressions; it shares no code with them or with the oracle.

Launches of more than MAX_TILES tiles (or k ranges) are checked on a fixed
sample: the first and last 32 and an even spread between (a tile's index math
depends on its position only), without the whole-output coverage count.
"""
from __future__ import annotations

import numpy as np

WAVE = 64
BM = 64                 # rows of a matrix-core block tile
DMA_ZERO = 0x80000000   # out-of-range voffset: the DMA writes zeros
INT_MAX = (1 << 31) - 1


class ModelError(AssertionError):
    pass


MAX_TILES = 256


def sample(n, k=MAX_TILES):
    """All of range(n), or the fixed sample of a large launch: the first and
    last k/8 and an even spread, k in all."""
    if n <= k:
        return list(range(n))
    e = max(1, k // 8)
    return sorted(set(range(e)) | set(range(n - e, n)) |
                  set(int(v) for v in np.linspace(0, n - 1, k - 2 * e)))


def sample_pairs(m_tiles, tiles):
    """(row tile, pixel tile) pairs of a launch, sampled to about MAX_TILES."""
    if m_tiles * tiles <= MAX_TILES:
        return [(mt, t) for mt in range(m_tiles) for t in range(tiles)]
    km = min(m_tiles, 4)
    return [(mt, t) for mt in sample(m_tiles, km) for t in sample(tiles, max(MAX_TILES // km, 8))]


def need(cond, what):
    if not bool(np.all(cond)):
        raise ModelError(what)


def cdiv(a, b):
    return -(-a // b)


# ------------------------------------------------------------------ divisions
def host_magic(d):
    return ((1 << 32) + d - 1) // d


def div_magic(n, d, what="magic division"):
    """floor(n / d) as (n * ceil(2^32 / d)) >> 32 in 64-bit unsigned arithmetic,
    checked against the exact quotient."""
    n = np.asarray(n, dtype=np.int64)
    need(1 <= d < 1 << 32, f"{what}: divisor {d}")
    need(n >= 0, f"{what}: negative numerator")
    prod = (n.astype(np.uint64) & np.uint64(0xffffffff)) * np.uint64(host_magic(d))
    q = (prod >> np.uint64(32)).astype(np.int64)
    need(q == n // d, f"{what}: inexact for divisor {d}, numerators up to {n.max()}")
    return q


def div_small(n, d, what="reciprocal division"):
    """floor(n / d) through a float32 reciprocal and one correction step,
    checked against the exact quotient (and its stated range)."""
    n = np.asarray(n, dtype=np.int64)
    need((n >= 0) & (n < 1 << 22), f"{what}: numerator outside [0, 2^22)")
    need(1 <= d < 1 << 22, f"{what}: divisor {d} outside [1, 2^22)")
    rcp = np.float32(1.0) / np.float32(d)
    q = (n.astype(np.float32) * rcp).astype(np.int64)
    r = n - q * d
    q = q + (r >= d).astype(np.int64) - (r < 0).astype(np.int64)
    need(q == n // d, f"{what}: inexact for divisor {d}")
    return q


def xcd_logical_block(b, n):
    """The kernels' renumbering of block b of n (runs of consecutive logical
    blocks on one XCD); must be a permutation of the grid."""
    b = np.asarray(b, dtype=np.int64)
    m = n >> 3
    return np.where(b >= 8 * m, b, (b & 7) * m + (b >> 3))


def mfma_row(tsz, lane, r):
    """Output row held by accumulator register r of a 16x16x4 MFMA lane."""
    return (lane >> 4) + 4 * r if tsz == 8 else 4 * (lane >> 4) + r


# ------------------------------------------------------------------ buffers
class Lds:
    """A block's dynamic LDS as named byte regions."""

    def __init__(self, total, kernel):
        need(total <= 160 * 1024, f"{kernel}: {total} bytes of LDS exceed the CU's 160 KiB")
        self.total, self.kernel, self.regions = total, kernel, {}

    def region(self, name, lo, nbytes):
        need(lo >= 0 and nbytes >= 0 and lo + nbytes <= self.total,
             f"{self.kernel}: LDS region {name} [{lo}, {lo + nbytes}) outside the block's "
             f"{self.total} bytes")
        self.regions[name] = (lo, nbytes)

    def disjoint(self, *names):
        spans = sorted(self.regions[n] + (n,) for n in names)
        for (lo0, n0, a), (lo1, _, b) in zip(spans, spans[1:]):
            need(lo0 + n0 <= lo1, f"{self.kernel}: live LDS regions {a} and {b} overlap")

    def access(self, name, idx, esz, what):
        """Element indices idx (elements of esz bytes) of region name."""
        lo, nbytes = self.regions[name]
        idx = np.asarray(idx, dtype=np.int64)
        if idx.size == 0:
            return
        need(idx.min() >= 0, f"{self.kernel}: {what} below LDS region {name}")
        need((idx.max() + 1) * esz <= nbytes,
             f"{self.kernel}: {what} reaches byte {(idx.max() + 1) * esz} of LDS region "
             f"{name} ({nbytes} bytes)")


def glob(kernel, name, idx, length):
    idx = np.asarray(idx, dtype=np.int64)
    if idx.size == 0:
        return
    need((idx.min() >= 0) & (idx.max() < length),
         f"{kernel}: access to {name} at [{idx.min()}, {idx.max()}] outside its {length} elements")


class Coverage:
    """Every output element written exactly once."""

    def __init__(self, n, what):
        self.count = np.zeros(n, dtype=np.int64)
        self.what = what

    def add(self, idx):
        np.add.at(self.count, np.asarray(idx, dtype=np.int64).ravel(), 1)

    def check(self):
        need(self.count.min() >= 1, f"{self.what}: elements never written")
        need(self.count.max() <= 1, f"{self.what}: elements written more than once")


# ------------------------------------------------------------------ geometry
def gemm_view(s, pass_name):
    """The implicit GEMM of a forward / backward_data launch, as its kernel
    arguments describe it (backward_data: the flipped, transposed filter over
    the stride-up-sampled gradient, stride 1)."""
    Hout = (s.Hin + 2 * s.pad - s.Hf) // s.stride + 1
    Wout = (s.Win + 2 * s.pad - s.Wf) // s.stride + 1
    if pass_name == "forward":
        return dict(M=s.F, Cs=s.C, Sh=s.Hin, Sw=s.Win, up=1, Qh=Hout, Qw=Wout, Hf=s.Hf, Wf=s.Wf,
                    S=s.stride, Ph=s.pad, Pw=s.pad, N=s.N, bwd=False)
    return dict(M=s.C, Cs=s.F, Sh=Hout, Sw=Wout, up=s.stride, Qh=s.Hin, Qw=s.Win, Hf=s.Hf,
                Wf=s.Wf, S=1, Ph=s.Hf - 1 - s.pad, Pw=s.Wf - 1 - s.pad, N=s.N, bwd=True)


def a_element(g, mg, k):
    """Flat index into W of the GEMM operand A(m, k), k = (c, i, j)."""
    HfWf = g["Hf"] * g["Wf"]
    c, t = k // HfWf, k % HfWf
    if not g["bwd"]:
        return (mg * g["Cs"] + c) * HfWf + t
    return (c * g["M"] + mg) * HfWf + (HfWf - 1 - t)


def source_cell(g, c, yv, xv):
    """Flat source index of channel c at up-sampled position (yv, xv) of the
    padded plane, or -1 where the GEMM's B operand is zero there."""
    up = g["up"]
    inside = (yv >= 0) & (xv >= 0) & (yv % up == 0) & (xv % up == 0)
    ys, xs = np.maximum(yv, 0) // up, np.maximum(xv, 0) // up
    inside &= (ys < g["Sh"]) & (xs < g["Sw"]) & (c >= 0) & (c < g["Cs"])
    return np.where(inside, (c * g["Sh"] + ys) * g["Sw"] + xs, -1)


def tile_rows(q0, qend, Qw, S, Hf):
    return ((qend - 1) // Qw - q0 // Qw) * S + Hf


def fragment_schedule(KCK, first, step):
    """Fragment reads of the software-pipelined k loop (the next step's
    fragments are read before the current step's MFMAs): all reads, and the
    reads whose values MFMAs consume."""
    reads, used = [first], []
    kk = first
    while kk + step < KCK:
        reads += [kk + step, kk + 2 * step]
        used += [kk, kk + step]
        kk += 2 * step
    if kk < KCK:
        used.append(kk)
    return reads, used


def check_operands(g, kernel, m, kg, real_k, a_val, q, b_val):
    """An MFMA lane's operands: a_val the W element its A fragment holds for
    row m and column kg (absolute k; real_k false for a chunk's padded columns
    and for channels past the last), b_val the source cell its B fragment
    holds for pixel q (-1 = zero, -2 = never staged).  Rows past M and pixels
    past the output are not stored and may hold anything finite."""
    HfWf, K = g["Hf"] * g["Wf"], g["Cs"] * g["Hf"] * g["Wf"]
    real_k = real_k & (kg < K)
    kg = np.minimum(kg, K - 1)
    row_ok = m < g["M"]
    want_a = np.where(real_k & row_ok, a_element(g, np.minimum(m, g["M"] - 1),
                                                np.minimum(kg, K - 1)), -1)
    need(np.where(real_k & row_ok, a_val == want_a, True),
         f"{kernel}: a filter fragment holds the wrong element of W")
    t = kg % HfWf
    yv = (q // g["Qw"]) * g["S"] + t // g["Wf"] - g["Ph"]
    xv = (q % g["Qw"]) * g["S"] + t % g["Wf"] - g["Pw"]
    want_b = source_cell(g, kg // HfWf, yv, xv)
    q_ok = q < g["Qh"] * g["Qw"]
    need(np.where(real_k & q_ok, b_val == want_b, True),
         f"{kernel}: a patch fragment holds the wrong source cell")
    # columns past the last tap: one operand must be zero
    need(np.where(~real_k & row_ok & q_ok, (a_val == -1) | (b_val == -1), True),
         f"{kernel}: a padded k column meets two non-zero operands")
    need((a_val != -2) & (b_val != -2), f"{kernel}: an MFMA reads an LDS slot nothing staged")


def out_coverage(kernel, g):
    return Coverage(g["M"] * g["Qh"] * g["Qw"], f"{kernel} output")


# ====================================================== LDS-DMA implicit GEMM
def model_igemm_dma(g, p, tsz, form):
    kernel = "igemm_dma"
    M, Cs, Hf, Wf, S, Qw = g["M"], g["Cs"], g["Hf"], g["Wf"], g["S"], g["Qw"]
    Q = g["Qh"] * Qw
    HfWf, dpe = Hf * Wf, tsz // 4
    NB, TS, KC = p["tile_pixels"] // 32, p["tile_stride"], p["chunk"]
    KCK, SA = p["k_chunk"], p["slice_stride"]
    Wpad, rows_max = p["window_width"], p["window_rows"]
    src_b, a_b, stage, avec = p["window_bytes"], p["slice_bytes"], p["stage_bytes"], p["slice_vec"]
    K4 = (2 if M <= 32 else 4) if p["k_split"] == 4 else 0
    KS = p["k_split"] == 2
    pb, pool = form == "pooled_source", form == "pool_epilogue"
    bwd = g["bwd"]
    KCv = KC * HfWf
    need(NB in (1, 2, 4, 7) and 1 <= TS <= 32 * NB, f"{kernel}: tile of {TS} pixels with NB {NB}")
    need(Wpad == (Qw - 1) * S + Wf, f"{kernel}: window width")
    need(stage == src_b + a_b and src_b % 256 == 0 and a_b % 256 == 0, f"{kernel}: stage layout")
    need(not avec or (tsz == 8 and not bwd and KCv % 2 == 0), f"{kernel}: 16-byte filter DMA")
    need(KCK % 4 == 0 and 0 <= KCK - KCv < 4 and SA >= KCK, f"{kernel}: k per chunk {KCK}")
    need(not (K4 and KS) and (NB == 1 or not K4), f"{kernel}: k-split form")
    need(M > 32 or KS or K4, f"{kernel}: a 32-row filter slice needs a k-split form")
    lds = Lds(p["lds_bytes"], kernel)
    for st in (0, 1):
        lds.region(f"src{st}", st * stage, src_b)
        lds.region(f"a{st}", st * stage + src_b, a_b)
    live = ["src0", "a0", "src1", "a1"]
    if bwd and not pb:
        lds.region("mask", 2 * stage, src_b)
        live.append("mask")
    lds.disjoint(*live)

    plane = g["Sh"] * g["Sw"]
    need(Cs * plane * tsz < DMA_ZERO and M * Cs * HfWf * tsz < DMA_ZERO,
         f"{kernel}: buffer ranges reach the out-of-range marker")
    c0s = list(range(0, Cs, KC))
    need(c0s[-1] * plane * tsz <= INT_MAX, f"{kernel}: window soffset overflows")
    need(c0s[-1] * (M if bwd else 1) * HfWf * tsz <= INT_MAX, f"{kernel}: filter soffset overflows")
    tiles, m_tiles = cdiv(Q, TS), cdiv(M, BM)
    need(p["blocks"] == g["N"] * tiles * m_tiles, f"{kernel}: block count")
    nblk = p["blocks"]
    need(np.array_equal(np.sort(xcd_logical_block(np.arange(nblk), nblk)), np.arange(nblk)),
         f"{kernel}: the block renumbering is not a permutation")

    lane = np.arange(WAVE)
    lq, l16 = lane >> 4, lane & 15

    # filter slice: what each slot holds for chunk 0 (the soffset moves it by c0 channels)
    rows_a = 32 if M <= 32 else 64
    Da = rows_a * SA // 2 if avec else rows_a * SA * dpe
    NIa = cdiv(Da, WAVE)
    unit = 1024 if avec else 256
    need(cdiv(NIa, 4) <= 20, f"{kernel}: filter DMA needs {NIa} instructions, 80 offsets")
    need(NIa * unit <= a_b, f"{kernel}: filter DMA writes past the slice")
    if avec:
        need((SA * tsz) % 16 == 0, f"{kernel}: 16-byte slice rows misaligned")

    def a_slots(m0):
        d = np.arange(Da)
        e = 2 * d if avec else d // dpe
        m = div_magic(e, SA, f"{kernel} slice row")
        kk = e - m * SA
        mg = m0 + m
        ok = (mg < M) & (kk < KCv)
        if bwd:
            div_magic(np.where(ok, kk, 0), HfWf, f"{kernel} slice tap")
        el = np.where(ok, a_element(g, np.minimum(mg, M - 1), np.minimum(kk, KCv - 1)), -1)
        need(np.where(ok, el * tsz + tsz <= INT_MAX, True), f"{kernel}: filter voffset overflows")
        slots = np.full(rows_a * SA, -1, dtype=np.int64)
        if avec:  # the lane's 16 bytes: elements el and el + 1 of W
            slots[e] = el
            slots[e + 1] = np.where(ok, el + 1, -1)
        else:
            slots[e] = el
        return slots

    def a_chunk(slots, c0):
        v = np.where(slots >= 0, slots + c0 * (M if bwd else 1) * HfWf, -1)
        return np.where(v < M * Cs * HfWf, v, -1)  # past the range: 0

    # wave -> (row blocks, pixel offsets in the tile, k schedule)
    def wave_form(w):
        wm, wn = w & 1, w >> 1
        if K4:
            return [16 * x + l16 for x in range(K4)], [y * 16 + l16 for y in range(2)], \
                fragment_schedule(KCK, 4 * w, 16)
        mrow = 0 if KS else wm * 32
        sched = fragment_schedule(KCK, 4 * wm, 8) if KS else fragment_schedule(KCK, 0, 4)
        return [mrow + l16, mrow + 16 + l16], [(wn * NB + y) * 16 + l16 for y in range(NB)], sched

    taken = []
    for w in range(4):
        if K4 or (KS and w < 2) or (not KS and w == 0):
            taken += wave_form(w)[2][1]
    need(sorted(taken) == list(range(0, KCK, 4)), f"{kernel}: k-steps of a chunk not taken once")

    pairs = sample_pairs(m_tiles, tiles)
    cover = out_coverage(kernel, g) if len(pairs) == m_tiles * tiles else None
    slots_of = {}
    for mt, t in pairs:
        m0 = mt * BM
        if mt not in slots_of:
            slots_of = {mt: a_slots(m0)}
        slots = slots_of[mt]
        q0 = t * TS
        qend = min(q0 + TS, Q)
        qy0 = q0 // Qw
        rows_need = tile_rows(q0, qend, Qw, S, Hf)
        need(rows_need <= rows_max, f"{kernel}: tile {t} needs {rows_need} window rows")
        ybase = qy0 * S - g["Ph"]
        CHn = rows_need * Wpad
        Ds = KC * CHn * dpe
        NIs = cdiv(Ds, WAVE)
        need(cdiv(NIs, 4) <= 12, f"{kernel}: window DMA needs {NIs} instructions, 48 offsets")
        lds.access("src0", np.arange(NIs * WAVE * 4 // tsz), tsz, "window DMA")
        # window cell of every staged element (chunk 0), as the DMA offsets give it
        e = np.arange(Ds) // dpe
        r = div_magic(e, Wpad, f"{kernel} window row")
        x = e - r * Wpad
        c = div_small(r, rows_need, f"{kernel} window channel")
        cells = source_cell(dict(g, Cs=g["Cs"] + KC), c, ybase + r - c * rows_need, x - g["Pw"])
        need(np.where(cells >= 0, cells * tsz + tsz <= INT_MAX, True), f"{kernel}: window voffset")
        win = np.full(KC * CHn, -2, dtype=np.int64)
        win[e] = cells
        if pb:
            model_dma_pooled_source(g, p, tsz, lds, kernel, KC, CHn, rows_need, ybase, win)
        qx0 = q0 - qy0 * Qw

        def pix_off(u):
            v = qx0 + u
            dy = div_magic(v, Qw, f"{kernel} pixel row")
            return np.where(q0 + u < qend, dy * S * Wpad + (v - dy * Qw) * S, 0)

        for w in range(4):
            rows_blk, us, (reads, used) = wave_form(w)
            offs = [pix_off(u) for u in us]
            for kk in reads:
                kcol = kk + lq
                kc = np.minimum(kcol, KCv - 1)
                cc = div_magic(kc, HfWf, f"{kernel} tap channel")
                tp = kc - cc * HfWf
                ii = div_magic(tp, Wf, f"{kernel} tap row")
                ko = cc * CHn + ii * Wpad + (tp - ii * Wf)
                for rr in rows_blk:
                    lds.access("a0", rr * SA + kcol, tsz, "filter fragment read")
                for off in offs:
                    lds.access("src0", ko + off, tsz, "patch fragment read")
                if kk not in used:
                    continue
                for c0 in sorted({c0s[0], c0s[-1]}):
                    ach = a_chunk(slots, c0)
                    for rr in rows_blk:
                        ai = rr * SA + kcol
                        a_val = np.where(ai < ach.size, ach[np.minimum(ai, ach.size - 1)], -2)
                        for u, off in zip(us, offs):
                            bcell = win[ko + off]
                            b_val = np.where(bcell >= 0, bcell + c0 * plane, bcell)
                            b_val = np.where(b_val >= Cs * plane, -1, b_val)
                            check_operands(g, kernel, m0 + rr, c0 * HfWf + kcol, kcol < KCv,
                                           a_val, np.where(q0 + u < qend, q0 + u, Q), b_val)
        # epilogue buffers reuse the stages
        if K4:
            lds.region("partials", 0, p["lds_bytes"])
            lds.access("partials", (3 * 64 + 16 * K4 - 1) * 32 + 31, tsz, "k-split partials")
        if KS:
            lds.region("handover", 0, p["lds_bytes"])
            lds.access("handover", 1024 * NB - 1, tsz, "k-split hand-over")
        for w in range(4):
            wm, wn = w & 1, w >> 1
            if KS and wm == 1:
                continue
            mbase = m0 + (0 if KS else wm * 32)
            for x in range(2):
                for r4 in range(4):
                    m = mbase + x * 16 + mfma_row(tsz, lane, r4)
                    for y in range(NB):
                        q = q0 + (wn * NB + y) * 16 + l16
                        ok = (m < M) & (q < qend)
                        if cover:
                            cover.add((m * Q + q)[ok])
        if pool:
            model_pool_epilogue(g, p, tsz, lds, kernel, q0, qend, NB)
    if cover:
        cover.check()


def model_dma_pooled_source(g, p, tsz, lds, kernel, KC, CHn, rows_need, ybase, win):
    """Pooled-source staging of the LDS-DMA kernel: window owners write the
    cells of their stride regions that lie in the staged window; together the
    writes must be exactly the window's in-plane cells."""
    PS, up, Sh, Sw, Wpad = g["PS"], g["up"], g["Sh"], g["Sw"], p["window_width"]
    lds.access("src0", np.arange(KC * CHn), tsz, "window zeroing")
    last = ybase + rows_need - 1
    ys_lo = (max(ybase, 0) + up - 1) // up
    ys_hi = -1 if last < 0 else min(last // up, Sh - 1)
    written = np.zeros(KC * CHn, dtype=np.int64)
    if ys_hi >= ys_lo:
        py_lo = int(div_magic(ys_lo, PS))
        npx = int(div_magic(Sw + PS - 1, PS))
        nw = (int(div_magic(ys_hi, PS)) - py_lo + 1) * npx
        nreg = KC * nw
        need(nreg <= 256 * 4, f"{kernel}: {nreg} pool regions a chunk; the owners hold 1024")
        e = np.arange(cdiv(nreg, 256) * 256)
        c = div_small(e, nw)
        w = e - c * nw
        wy = div_small(w, npx)
        py, px = py_lo + wy, w - wy * npx
        Hp, Wp = g["Hp"], g["Wp"]
        glob(kernel, "dpool/argmax/pooled",
             (np.minimum(g["Cs"] - 1, c) * Hp + np.minimum(py, Hp - 1)) * Wp + np.minimum(px, Wp - 1),
             g["Cs"] * Hp * Wp)
        own = e < nreg
        c, py, px = c[own], py[own], px[own]
        for dy in range(PS):
            ys = py * PS + dy
            t = ys * up - ybase
            okr = (ys >= ys_lo) & (ys <= ys_hi)
            for dx in range(PS):
                xs = px * PS + dx
                x = xs * up + g["Pw"]
                ok = okr & (xs < Sw) & (x < Wpad)
                need(((t >= 0) & (t < rows_need))[ok], f"{kernel}: region cell outside the window")
                idx = (c * CHn + t * Wpad + x)[ok]
                lds.access("src0", idx, tsz, "pooled-source window write")
                np.add.at(written, idx, 1)
    in_plane = np.zeros(KC * CHn, dtype=np.int64)
    r = np.arange(KC * CHn) // Wpad
    x = np.arange(KC * CHn) % Wpad
    t = r % rows_need
    yv, xv = ybase + t, x - g["Pw"]
    ok = (yv >= 0) & (xv >= 0) & (yv % up == 0) & (xv % up == 0) & (yv // up < Sh) & (xv // up < Sw)
    in_plane[ok] = 1
    need(written == in_plane, f"{kernel}: pooled-source writes are not the window's in-plane cells")


def model_pool_epilogue(g, p, tsz, lds, kernel, q0, qend, NB):
    Qw, PS, PH, PW, Hp, Wp = g["Qw"], g["PS"], g["PH"], g["PW"], g["Hp"], g["Wp"]
    BN = 32 * NB
    need(q0 % Qw == 0 and (qend % Qw == 0), f"{kernel}: a pool tile is not whole conv rows")
    need(PS >= PH, f"{kernel}: pool windows overlap tiles")
    lds.region("pool tile", 0, p["lds_bytes"])
    lds.access("pool tile", np.arange(32 * BN), tsz, "pool tile")
    y_lo, y_hi = q0 // Qw, qend // Qw
    py = np.arange(y_lo // PS, min(Hp, cdiv(y_hi, PS)))[:, None, None, None]
    px = np.arange(Wp)[None, :, None, None]
    yy = py * PS + np.arange(PH)[None, None, :, None]
    xx = px * PS + np.arange(PW)[None, None, None, :]
    rel = (yy - y_lo) * Qw + xx
    need((rel >= 0) & (rel < qend - q0), f"{kernel}: a pool window reads outside its tile")
    lds.access("pool tile", 31 * BN + rel, tsz, "pool window read")
    glob(kernel, "pooled", ((g["M"] - 1) * Hp + py) * Wp + px, g["M"] * Hp * Wp)


def pool_coverage(kernel, g, tiles_q):
    """The pooled rows the tiles of an image produce cover every pooled row once."""
    rows = []
    for q0, qend in tiles_q:
        y_lo, y_hi = q0 // g["Qw"], qend // g["Qw"]
        rows += list(range(y_lo // g["PS"], min(g["Hp"], cdiv(y_hi, g["PS"]))))
    need(sorted(rows) == list(range(g["Hp"])), f"{kernel}: pooled rows not produced once")


# ================================================ register-staged implicit GEMM
def shifted(cells, c0, plane, limit):
    """Chunk-0 window cells moved to chunk c0 (whole channels), zero past the source."""
    v = np.where(cells >= 0, cells + c0 * plane, cells)
    return np.where(v >= limit, -1, v)


def model_igemm_reg(g, p, tsz, form):
    kernel = "igemm_reg"
    M, Cs, Hf, Wf, S, Qw = g["M"], g["Cs"], g["Hf"], g["Wf"], g["S"], g["Qw"]
    Q = g["Qh"] * Qw
    HfWf = Hf * Wf
    NB, TS, KC = p["tile_pixels"] // 32, p["tile_stride"], p["chunk"]
    KCK, SA = p["k_chunk"], p["slice_stride"]
    Wpad, rows_max, pipelined = p["window_width"], p["window_rows"], p["pipelined"]
    KCv = KC * HfWf
    CH = rows_max * Wpad
    plane = g["Sh"] * g["Sw"]
    csr = form == "csr_input"
    need(Wpad == (Qw - 1) * S + Wf and TS == 32 * NB, f"{kernel}: tiling")
    need(KCK % 4 == 0 and 0 <= KCK - KCv < 4 and SA == KCK + 1, f"{kernel}: k per chunk")
    need(p["lds_bytes"] == tsz * (KC * CH + BM * SA) + 4 * KCK, f"{kernel}: LDS size")
    need(not (csr and pipelined), f"{kernel}: CSR input takes the direct staging")
    lds = Lds(p["lds_bytes"], kernel)
    lds.region("window", 0, tsz * KC * CH)
    lds.region("slice", tsz * KC * CH, tsz * BM * SA)
    lds.region("koff", tsz * (KC * CH + BM * SA), 4 * KCK)
    lds.disjoint("window", "slice", "koff")
    tiles, m_tiles = cdiv(Q, TS), cdiv(M, BM)
    need(p["blocks"] == g["N"] * tiles * m_tiles, f"{kernel}: block count")
    lane = np.arange(WAVE)
    lq, l16 = lane >> 4, lane & 15
    ncg = cdiv(Wpad, WAVE)
    pairs = sample_pairs(m_tiles, tiles)
    cover = out_coverage(kernel, g) if len(pairs) == m_tiles * tiles else None
    c0s = sorted({0, (Cs - 1) // KC * KC})
    # filter slice: element e = (m, kk) of the 64 x KCK slice goes to slot
    # e + e / KCK (pipelined) or m * SA + kk (direct)
    e = np.arange(BM * KCK)
    if pipelined:
        need(BM * KCK <= 256 * 13, f"{kernel}: filter slice exceeds the staging registers")
        m = div_magic(e, KCK, f"{kernel} slice row")
        sidx = e + m
    else:
        m = e // KCK
        sidx = m * SA + (e - m * KCK)
    kk = e - m * KCK
    lds.access("slice", sidx, tsz, "slice store")
    slot_mt = None
    for mt, t in pairs:
        m0 = mt * BM
        if slot_mt != mt:
            slot_mt, slot = mt, {}
            for c0 in c0s:
                ok = (m0 + m < M) & (kk < KCv) & (c0 + kk // HfWf < Cs)
                sl = np.full(BM * SA, -2, dtype=np.int64)
                sl[sidx] = np.where(ok, a_element(g, np.minimum(m0 + m, M - 1),
                                                  np.minimum(c0 * HfWf + kk, Cs * HfWf - 1)), -1)
                slot[c0] = sl
        q0 = t * TS
        qend = min(q0 + TS, Q)
        qy0 = q0 // Qw
        rows_need = tile_rows(q0, qend, Qw, S, Hf)
        need(rows_need <= rows_max, f"{kernel}: tile {t} needs {rows_need} window rows")
        ybase = qy0 * S - g["Ph"]
        CHn = rows_need * Wpad
        nrows = KC * rows_need
        kv = np.arange(KCK)
        c_, t_ = kv // HfWf, kv % HfWf
        koff = np.where(kv < KCv, c_ * CHn + (t_ // Wf) * Wpad + t_ % Wf, 0)
        lds.access("koff", kv, 4, "tap offsets")
        if pipelined:
            need(nrows * ncg <= 4 * 8, f"{kernel}: {nrows * ncg} window row slots, 32 staged")
        rr = np.arange(nrows)[:, None]
        u = np.arange(Wpad)[None, :]
        lds.access("window", rr * Wpad + u, tsz, "window store")
        if csr:
            xlim = min(g["Sw"], Wpad - g["Pw"])
            need(xlim - 1 + g["Pw"] < Wpad, f"{kernel}: CSR scatter past the staged row")
        win = source_cell(dict(g, Cs=Cs + KC), rr // rows_need, ybase + rr % rows_need,
                          u - g["Pw"]).ravel()
        # all (wave, pixel block) lanes at once: q and lbase of shape (4 * NB, 64)
        wv = np.repeat(np.arange(4), NB)[:, None]
        yv = np.tile(np.arange(NB), 4)[:, None]
        q = q0 + ((wv >> 1) * NB + yv) * 16 + l16
        lb = np.where(q < qend, (q // Qw - qy0) * S * Wpad + (q % Qw) * S, 0)
        for k4 in range(0, KCK, 4):
            kcol = k4 + lq
            bi = koff[kcol] + lb
            lds.access("window", bi, tsz, "patch fragment read")
            for half in (0, 16):
                rblk = (wv & 1) * 32 + half + l16
                ai = rblk * SA + kcol
                lds.access("slice", ai, tsz, "filter fragment read")
                for c0 in c0s:
                    check_operands(g, kernel, m0 + rblk, c0 * HfWf + kcol, kcol < KCv,
                                   slot[c0][ai], np.where(q < qend, q, Q),
                                   shifted(win[bi], c0, plane, Cs * plane))
        for w in range(4):
            wm, wn = w & 1, w >> 1
            for x in range(2):
                for r4 in range(4):
                    mm = m0 + wm * 32 + x * 16 + mfma_row(tsz, lane, r4)
                    for y in range(NB):
                        qq = q0 + (wn * NB + y) * 16 + l16
                        ok = (mm < M) & (qq < qend)
                        if cover:
                            cover.add((mm * Q + qq)[ok])
    if cover:
        cover.check()


# ==================================================== small-M vector kernel
def model_small_m(g, p, tsz, form):
    kernel = "small_m"
    M, Cs, Hf, Wf, S, Qw = g["M"], g["Cs"], g["Hf"], g["Wf"], g["S"], g["Qw"]
    Q = g["Qh"] * Qw
    HfWf = Hf * Wf
    KC, MM, Wpad, rows_max = p["chunk"], p["tile_m"], p["window_width"], p["window_rows"]
    CH = rows_max * Wpad
    MW = MM * HfWf
    need(M <= 4 and MM == (1 if M == 1 else 4) and Wf <= 7, f"{kernel}: form")
    need(p["lds_bytes"] == max(tsz * (KC * CH + KC * MW), tsz * 4 * 4 * 64), f"{kernel}: LDS size")
    need(p["blocks"] == cdiv(Q, 64) * g["N"], f"{kernel}: block count")
    lds = Lds(p["lds_bytes"], kernel)
    lds.region("window", 0, tsz * KC * CH)
    lds.region("filter", tsz * KC * CH, tsz * KC * MW)
    lds.disjoint("window", "filter")
    lds.region("reduction", 0, tsz * 16 * 64)
    lane = np.arange(64)
    cover = out_coverage(kernel, g) if cdiv(Q, 64) <= MAX_TILES else None
    # every (channel, tap) of a chunk at once: arrays of shape (kc * HfWf, 64)
    for c0 in sorted({0, (Cs - 1) // KC * KC}):
        kc = min(KC, Cs - c0)
        e = np.arange(kc * MW)
        c, r = e // MW, e % MW
        m, tp = r // HfWf, r % HfWf
        filt = np.where(m < M, a_element(g, np.minimum(m, M - 1), (c0 + c) * HfWf + tp), -1)
        lds.access("filter", e, tsz, "filter store")
        glob(kernel, "W", filt[filt >= 0], M * Cs * HfWf)
        kt = np.arange(kc * HfWf)[:, None]
        cc, tt = kt // HfWf, kt % HfWf
        ii, jj = tt // Wf, tt % Wf
        for q0 in [64 * t for t in sample(cdiv(Q, 64))]:
            qend = min(q0 + 64, Q)
            qy0 = q0 // Qw
            rows = tile_rows(q0, qend, Qw, S, Hf)
            need(rows <= rows_max, f"{kernel}: tile needs {rows} window rows")
            ybase = qy0 * S - g["Ph"]
            CHn = rows * Wpad
            tot = kc * CHn
            ew = np.minimum(np.arange(cdiv(tot, 2048) * 2048), tot - 1)
            wc = div_small(ew, CHn, f"{kernel} window channel")
            rem = ew - wc * CHn
            wt = div_small(rem, Wpad, f"{kernel} window row")
            yv, xv = ybase + wt, rem - wt * Wpad - g["Pw"]
            div_small(np.maximum(yv, 0), g["up"], f"{kernel} up-sampled row")
            div_small(np.maximum(xv, 0), g["up"], f"{kernel} up-sampled column")
            cells = source_cell(g, c0 + wc, yv, xv)
            glob(kernel, "source", cells[cells >= 0], Cs * g["Sh"] * g["Sw"])
            lds.access("window", np.arange(tot), tsz, "window store")
            win = np.full(kc * CHn, -2, dtype=np.int64)
            win[ew] = cells
            q = q0 + lane
            act = q < qend
            lb = np.where(act, (q // Qw - qy0) * S * Wpad + (q % Qw) * S, 0)
            bi = cc * CHn + lb + ii * Wpad + jj
            lds.access("window", bi, tsz, "window read")
            for mm in range(MM):
                wi = cc * MW + mm * HfWf + ii * Wf + jj
                lds.access("filter", wi, tsz, "filter read")
                check_operands(g, kernel, np.full_like(bi, mm), (c0 + cc) * HfWf + tt,
                               np.ones_like(bi, dtype=bool), np.broadcast_to(filt[wi], bi.shape),
                               np.where(act, q, Q), win[bi])
            if c0 == 0:
                for m_ in range(M):
                    lds.access("reduction", (3 * 4 + m_) * 64 + lane, tsz, "partial sums")
                    if cover:
                        cover.add((m_ * Q + q)[act])
    if cover:
        cover.check()


# =================================================== filter-resident forward
def model_resident(g, p, tsz, form):
    kernel = "resident"
    M, Cs, Hf, Wf, S, Qw = g["M"], g["Cs"], g["Hf"], g["Wf"], g["S"], g["Qw"]
    Q = g["Qh"] * Qw
    HfWf, dpe = Hf * Wf, tsz // 4
    KC, KCK, SA = p["chunk"], p["k_chunk"], p["slice_stride"]
    Wpad, CH = p["window_width"], p["window_rows"] * p["window_width"]
    lds_a, stage = p["slice_bytes"], p["stage_bytes"]
    KCv = KC * HfWf
    nchunk = cdiv(Cs, KC)
    Awid, Kw = nchunk * KCK, Cs * HfWf
    need(not g["bwd"] and tsz == 8 and Q <= 256, f"{kernel}: form")
    need(CH == ((g["Qh"] - 1) * S + Hf) * Wpad and Wpad == (Qw - 1) * S + Wf, f"{kernel}: window")
    need(SA == Awid + 2 and KCK % 4 == 0 and 0 <= KCK - KCv < 4, f"{kernel}: slice layout")
    need(p["lds_bytes"] == lds_a + 2 * stage, f"{kernel}: LDS size")
    need(p["blocks"] == g["N"] * cdiv(M, 16), f"{kernel}: block count")
    lds = Lds(p["lds_bytes"], kernel)
    lds.region("slice", 0, lds_a)
    lds.region("stage0", lds_a, stage)
    lds.region("stage1", lds_a + stage, stage)
    lds.disjoint("slice", "stage0", "stage1")
    lds.region("stages", lds_a, 2 * stage)
    plane = g["Sh"] * g["Sw"]
    need(Cs * plane * tsz < DMA_ZERO, f"{kernel}: buffer range")
    need((nchunk - 1) * KC * plane * tsz <= INT_MAX, f"{kernel}: soffset overflows")
    # window DMA (whole padded image of a chunk)
    Ds = KC * CH * dpe
    NIs = cdiv(Ds, WAVE)
    need(cdiv(NIs, 16) <= 6, f"{kernel}: window DMA needs {NIs} instructions, 96 offsets")
    lds.access("stage0", np.arange(NIs * WAVE * 4 // tsz), tsz, "window DMA")
    e = np.arange(Ds) // dpe
    c = div_small(e, CH, f"{kernel} window channel")
    r = e - c * CH
    t = div_small(r, Wpad, f"{kernel} window row")
    x = r - t * Wpad
    cells = source_cell(dict(g, Cs=Cs + KC), c, t - g["Ph"], x - g["Pw"])
    win = np.full(KC * CH, -2, dtype=np.int64)
    win[e] = cells
    lane = np.arange(64)
    lq, l16 = lane >> 4, lane & 15
    cover = out_coverage(kernel, g)
    ntile = cdiv(Q, 16)
    taken = sorted(sum((fragment_schedule(KCK, 4 * kh, 16)[1] for kh in range(4)), []))
    need(taken == list(range(0, KCK, 4)), f"{kernel}: k-steps not taken once")
    for m0 in range(0, M, 16):
        # slice staging
        tot_a = 16 * Awid
        ea = np.minimum(np.arange(cdiv(tot_a, 16 * 1024) * 16 * 1024), tot_a - 1)
        rr = div_small(ea, Awid, f"{kernel} slice row")
        sl = ea - rr * Awid
        ch = div_small(sl, KCK, f"{kernel} slice chunk")
        kl = sl - ch * KCK
        k = ch * KCv + kl
        glob(kernel, "W", np.minimum(m0 + rr, M - 1) * Kw + np.minimum(k, Kw - 1), M * Kw)
        keep = (m0 + rr < M) & (kl < KCv) & (k < Kw)
        lds.access("slice", rr * SA + sl, tsz, "slice store")
        slot = np.full(16 * SA, -2, dtype=np.int64)
        slot[rr * SA + sl] = np.where(keep, (m0 + rr) * Kw + np.minimum(k, Kw - 1), -1)
        for w in range(16):
            kh, tg = w % 4, w // 4
            nt = min(4, cdiv(ntile - tg, 4)) if ntile > tg else 0
            reads, used = fragment_schedule(KCK, 4 * kh, 16)
            for chn in sorted({0, nchunk - 1}):
                c0 = chn * KC
                for kk in reads:
                    kcol = kk + lq
                    ai = l16 * SA + chn * KCK + kcol
                    lds.access("slice", ai, tsz, "filter fragment read")
                    kc = np.minimum(kcol, KCv - 1)
                    cc = div_magic(kc, HfWf, f"{kernel} tap channel")
                    tp = kc - cc * HfWf
                    ii = div_magic(tp, Wf, f"{kernel} tap row")
                    ko = cc * CH + ii * Wpad + (tp - ii * Wf)
                    for tt in range(nt):
                        q = (tg + 4 * tt) * 16 + l16
                        oy = div_magic(q, Qw, f"{kernel} pixel row")
                        pbo = np.where(q < Q, oy * S * Wpad + (q - oy * Qw) * S, 0)
                        lds.access("stage0", ko + pbo, tsz, "patch fragment read")
                        if kk in used:
                            bcell = win[ko + pbo]
                            b_val = np.where(bcell >= 0, bcell + c0 * plane, bcell)
                            b_val = np.where(b_val >= Cs * plane, -1, b_val)
                            check_operands(g, kernel, m0 + l16, c0 * HfWf + kcol, kcol < KCv,
                                           slot[ai], np.where(q < Q, q, Q), b_val)
            lds.access("stages", ((tg * 4 + 3) * 4 + 3) * 64 + lane, tsz, "k-range hand-over")
            if kh == 0:
                for r4 in range(4):
                    m = m0 + mfma_row(tsz, lane, r4)
                    for tt in range(4):
                        q = (tg + 4 * tt) * 16 + l16
                        ok = (m < M) & (q < Q)
                        cover.add((m * Q + q)[ok])
        if form == "pool_epilogue":
            lds.access("stages", 15 * Q + np.arange(Q), tsz, "pool tile")
            yy = (g["Hp"] - 1) * g["PS"] + g["PH"] - 1
            xx = (g["Wp"] - 1) * g["PS"] + g["PW"] - 1
            need(yy < g["Qh"] and xx < Qw, f"{kernel}: a pool window reads past the image")
    cover.check()


# ======================================================== backward_filter
def wgrad_geometry(s):
    Hout = (s.Hin + 2 * s.pad - s.Hf) // s.stride + 1
    Wout = (s.Win + 2 * s.pad - s.Wf) // s.stride + 1
    return dict(N=s.N, C=s.C, Hin=s.Hin, Win=s.Win, F=s.F, Hf=s.Hf, Wf=s.Wf, S=s.stride, P=s.pad,
                Hout=Hout, Wout=Wout, Q=Hout * Wout, K=s.C * s.Hf * s.Wf)


def x_cell(g, c, y, x):
    ok = (c >= 0) & (c < g["C"]) & (y >= 0) & (y < g["Hin"]) & (x >= 0) & (x < g["Win"])
    return np.where(ok, (c * g["Hin"] + y) * g["Win"] + x, -1)


def wgrad_common(g, p, tsz, kernel, threads, x_elems=None):
    """x_elems: elements of the X region when it is not nch_alloc channels of
    window_rows x window_width (the ring's slot-major DMA layout)."""
    HfWf, K = g["Hf"] * g["Wf"], g["K"]
    KR, SG, RQ = p["chunk"], p["g_stride"], p["tile_pixels"]
    Wpad, rows_max = p["window_width"], p["window_rows"]
    nch_alloc = (KR - 1) // HfWf + 2
    CH = rows_max * Wpad
    if x_elems is None:
        x_elems = nch_alloc * CH
    need(SG == RQ + 2 and RQ % 4 == 0, f"{kernel}: g tile layout")
    need(p["lds_bytes"] == tsz * (BM * SG + x_elems), f"{kernel}: LDS size")
    lds = Lds(p["lds_bytes"], kernel)
    lds.region("g", 0, tsz * BM * SG)
    lds.region("x", tsz * BM * SG, tsz * x_elems)
    lds.disjoint("g", "x")
    lds.region("all", 0, p["lds_bytes"])
    nkr, nft = cdiv(K, KR), cdiv(g["F"], BM)
    need(p["blocks"] == nkr * nft, f"{kernel}: blocks per split")
    ws_elems = p["workspace_bytes"] // tsz
    need(ws_elems == p["splits"] * (g["F"] * K + g["F"]), f"{kernel}: workspace size")
    ranges = []
    for kr in range(nkr):
        kbeg = kr * KR
        kend = min(K, kbeg + KR)
        c_lo = kbeg // HfWf
        nch = (kend - 1) // HfWf - c_lo + 1
        need(nch <= nch_alloc, f"{kernel}: k range {kr} spans {nch} channels")
        ranges.append((kbeg, kend, c_lo, nch))
    return lds, ranges, nch_alloc, CH, ws_elems


def wgrad_outputs(g, p, tsz, kernel, ranges, NBW, nwaves, ws_elems):
    """Partial dW / db stores of a split (the first and the last), and the
    split reduction's reads: every (f, k) written once per split."""
    F, K = g["F"], g["K"]
    lane = np.arange(64)
    w = np.arange(nwaves)[:, None, None, None, None]
    mb = np.arange(4)[None, :, None, None, None]
    nb = np.arange(NBW)[None, None, :, None, None]
    r4 = np.arange(4)[None, None, None, :, None]
    ln = lane[None, None, None, None, :]
    for split in sorted({0, p["splits"] - 1}):
        cover = Coverage(F * K, f"{kernel} partial dW of a split")
        for ft in range(cdiv(F, BM)):
            f = ft * BM + mb * 16 + mfma_row(tsz, ln, r4)
            for kbeg, kend, _, _ in ranges:
                k = kbeg + (w * NBW + nb) * 16 + (ln & 15)
                ok = (f < F) & (k < kend)
                idx = np.broadcast_to(f * K + k, ok.shape)[ok]
                glob(kernel, "workspace", split * F * K + idx, ws_elems)
                cover.add(idx)
        cover.check()
        glob(kernel, "workspace (db)", p["splits"] * F * K + split * F + np.arange(F), ws_elems)


def ring_contents_ok(g, kernel, T_total, splits, R):
    """Walk every split's tiles: the ring slot (oh*S + i) mod R must hold input
    row oh*S + i when tile oh reads it.  With R = Hf + 1 slots (the DMA form)
    a tile's new row lands while the previous tile still reads: it must miss
    the slots that tile reads."""
    Hf, S, Hout = g["Hf"], g["S"], g["Hout"]
    nr = min(S, Hf)
    for sp in range(splits):
        t0, t1 = sp * T_total // splits, (sp + 1) * T_total // splits
        slots = None
        prev_read = set()
        for tt in range(t0, t1):
            oh = tt % Hout
            if tt == t0 or oh == 0:
                slots = {(oh * S + t) % R: oh * S + t for t in range(Hf)}
            else:
                s0 = (oh * S + Hf - nr) % R
                for r in range(nr):
                    yr = oh * S + Hf - nr + r
                    sl = s0 + r - (R if s0 + r >= R else 0)
                    need(sl == yr % R, f"{kernel}: new row {yr} goes to slot {sl}")
                    if R > Hf:
                        need(sl not in prev_read,
                             f"{kernel}: new row {yr} lands in a slot the previous tile reads")
                    slots[sl] = yr
            prev_read = {(oh * S + i) % R for i in range(Hf)}
            for i in range(Hf):
                need(slots[(oh * S + i) % R] == oh * S + i,
                     f"{kernel}: tile of output row {oh} reads a stale ring slot")


def model_wgrad_ring(g, p, tsz, form):
    kernel = "wgrad_ring"
    HfWf, K, Wout, S, Hf = g["Hf"] * g["Wf"], g["K"], g["Wout"], g["S"], g["Hf"]
    KR, SG, RQ, Wpad = p["chunk"], p["g_stride"], p["tile_pixels"], p["window_width"]
    NBW = KR // (16 * 12)
    need(KR == 16 * NBW * 12 and NBW in (1, 2, 3), f"{kernel}: k range {KR}")
    need(RQ == cdiv(Wout, 4) * 4 and Wpad == (Wout - 1) * S + g["Wf"], f"{kernel}: tile geometry")
    nch_alloc = (KR - 1) // HfWf + 2
    nr = min(S, Hf)
    pb = form == "pooled_source"
    # X staging: bit 2 the new input row by LDS DMA into Hf + 1 slot-major slots
    # (fp32, stride 1, image under 2 GiB, LDS within 160 KB), else bit 0 a row a
    # wave through registers; bit 1 the g tile a row a wave (fp32, not the pooled
    # source)
    epi = 256 // tsz                                  # elements a DMA instruction moves
    insts = cdiv(nch_alloc * Wpad, epi)
    SLOT = insts * epi + (g["Wf"] - 1 + epi // 2) % epi  # (epi = the bank period in elements)
    xd_ok = (tsz == 4 and S == 1 and tsz * g["C"] * g["Hin"] * g["Win"] < 2 ** 31
             and tsz * (BM * SG + (Hf + 1) * SLOT) <= 160 * 1024)
    rm_ok = nr == 1 and Wpad <= 64 and RQ <= 64 and nch_alloc <= 12 * 6
    rs = p["row_staged"]
    want = (4 if xd_ok else (1 if rm_ok and not pb else 0)) | \
        (2 if (xd_ok or rm_ok) and not pb and tsz == 4 else 0)
    need(rs == want, f"{kernel}: row staging {rs}, expected {want}")
    XD = bool(rs & 4)
    R = Hf + 1 if XD else Hf
    need(p["window_rows"] == R, f"{kernel}: {p['window_rows']} ring slots")
    lds, ranges, nch_alloc, CH, ws_elems = wgrad_common(
        g, p, tsz, kernel, 768, x_elems=(R * SLOT if XD else None))
    if XD:
        CH = SLOT                                     # the slot stride

    def xo(c, sl):                                    # a channel's row in a ring slot
        return sl * SLOT + c * Wpad if XD else c * CH + sl * Wpad
    need(BM * SG >= 768, f"{kernel}: the db reduction needs 768 slots of the g tile")
    lane = np.arange(64)
    lq, l16 = lane >> 4, lane & 15
    w_it = (np.arange(12)[:, None] + 12 * np.arange(6)[None, :]).ravel()  # rows of wave w, step it
    if rs & 2:
        # wave w, step it: g row w + 12 it (< 64), lane u (< RQ); every cell once
        r = np.repeat(w_it[w_it < BM], 64)
        u = np.tile(lane, int((w_it < BM).sum()))
        ok = u < RQ
        cells = r[ok] * RQ + u[ok]
        need(np.array_equal(np.sort(cells), np.arange(BM * RQ)), f"{kernel}: g rows not staged once")
        lds.access("g", r[ok] * SG + u[ok], tsz, "g tile store")
        f = np.arange(cdiv(g["F"], BM))[:, None] * BM + r[ok][None, :]
        live = (f < g["F"]) & (u[ok][None, :] < Wout)
        for n, oh in ((0, 0), (g["N"] - 1, g["Hout"] - 1)):
            glob(kernel, "dout (row-mapped)", ((n * g["F"] + f) * g["Q"] + oh * Wout + u[ok])[live],
                 g["N"] * g["F"] * g["Q"])
    else:
        need(BM * RQ <= 768 * 5, f"{kernel}: g tile exceeds the staging registers")
        e = np.arange(BM * RQ)
        r = div_magic(e, RQ, f"{kernel} g row")
        lds.access("g", r * SG + (e - r * RQ), tsz, "g tile store")
    if pb:
        PS = g["PS"]
        npx = int(div_magic(Wout + PS - 1, PS))
        need(cdiv(BM * npx, 768) <= 5, f"{kernel}: pooled-source windows exceed the registers")
        e = np.arange(BM * npx)
        r = div_small(e, npx)
        px = e - r * npx
        for dx in range(PS):
            ox = px * PS + dx
            lds.access("g", (r * SG + ox)[ox < Wout], tsz, "pooled-source g write")
        tail = RQ - Wout
        if tail:
            e = np.arange(BM * tail)
            r = div_small(e, tail)
            lds.access("g", r * SG + Wout + e - r * tail, tsz, "g tail zeroing")
        glob(kernel, "dpool", ((g["F"] - 1) * g["Hp"] + g["Hp"] - 1) * g["Wp"] + g["Wp"] - 1,
             g["F"] * g["Hp"] * g["Wp"])
    for kbeg, kend, c_lo, nch in ranges:
        # new-row staging
        nrw = nr * Wpad
        if XD:
            # dword d = 64 i + lane of slot sl (instruction i by wave i % 12): element
            # d // (tsz / 4) = (channel c, column u); zeros (an offset past the
            # image) for padding columns, channels past the range, rows outside
            d = np.arange(insts * 64)
            e = d // (tsz // 4)
            half = d % (tsz // 4)
            c = div_magic(e, Wpad, f"{kernel} DMA channel")
            u = e - c * Wpad
            need(np.array_equal(np.unique(e[(c < nch)]), np.arange(nch * Wpad)) and
                 np.bincount(e[c < nch]).max() == tsz // 4, f"{kernel}: DMA cells not written once")
            cg, x = c_lo + c, u - g["P"]
            img = g["C"] * g["Hin"] * g["Win"]
            for oh in (1, g["Hout"] - 1):
                yr = oh + Hf - 1
                y = yr - g["P"]
                sl = yr % R
                live = (c < nch) & (cg < g["C"]) & (x >= 0) & (x < g["Win"]) & (0 <= y < g["Hin"])
                vo = ((cg * g["Hin"] + y) * g["Win"] + x) * tsz + 4 * half
                need(np.all(vo[live] >= 0) & np.all(vo[live] + 4 <= img * tsz),
                     f"{kernel}: DMA offset outside the image")
                need(img * tsz < 2 ** 31, f"{kernel}: DMA range past 2^31")
                lds.access("x", sl * SLOT + (d * 4) // tsz, tsz, "new-row DMA")
                need(np.all((d * 4) // tsz < SLOT), f"{kernel}: DMA past its slot")
        elif rs & 1:
            # wave w, step it: channel w + 12 it (< nch), lane u (< Wpad); each cell once
            c = np.repeat(w_it[w_it < nch], 64)
            rem = np.tile(lane, int((w_it < nch).sum()))
            keep = rem < Wpad
            c, rem = c[keep], rem[keep]
            need(np.array_equal(np.sort(c * Wpad + rem), np.arange(nch * Wpad)),
                 f"{kernel}: new-row cells not staged once")
            cg, x = c_lo + c, rem - g["P"]
            for n, oh in ((0, 1), (g["N"] - 1, g["Hout"] - 1)):
                y = oh * S + Hf - 1 - g["P"]
                live = (cg < g["C"]) & (x >= 0) & (x < g["Win"]) & (0 <= y < g["Hin"])
                glob(kernel, "X new row (row-mapped)",
                     (n * g["C"] * g["Hin"] * g["Win"] + (cg * g["Hin"] + y) * g["Win"] + x)[live],
                     g["N"] * g["C"] * g["Hin"] * g["Win"])
        else:
            need(nch * nrw <= 768 * 5, f"{kernel}: new rows exceed the staging registers")
            e = np.arange(nch * nrw)
            c = div_magic(e, nrw, f"{kernel} new-row channel")
            rem = e - c * nrw
            div_magic(rem, Wpad, f"{kernel} new-row row")
        for oh in range(min(g["Hout"], 2 * Hf + 2)):
            if not XD:
                s0 = (oh * S + Hf - nr) % Hf
                wrap, ring = (Hf - s0) * Wpad, Hf * Wpad
                idx = s0 * Wpad + rem - np.where(rem >= wrap, ring, 0)
                need((idx >= 0) & (idx < CH), f"{kernel}: new row outside its channel's ring")
                lds.access("x", c * CH + idx, tsz, "new-row store")
            # full staging
            e2 = np.arange(nch * Hf * Wpad)
            rw = div_magic(e2, Wpad, f"{kernel} window row")
            u = e2 - rw * Wpad
            c2 = div_small(rw, Hf, f"{kernel} window channel")
            t = rw - c2 * Hf
            rot0 = (oh * S) % R
            sl = rot0 + t - np.where(rot0 + t >= R, R, 0)
            lds.access("x", xo(c2, sl) + u, tsz, "window store")
            # fragment reads of tile oh
            rot = (oh * S) % R
            for w in range(12):
                for nb in range(NBW):
                    k = kbeg + (w * NBW + nb) * 16 + l16
                    kc = np.minimum(k, K - 1)
                    cc = div_magic(kc, HfWf, f"{kernel} column channel")
                    tp = kc - cc * HfWf
                    ii = div_magic(tp, g["Wf"], f"{kernel} column row")
                    jj = tp - ii * g["Wf"]
                    slr = rot + ii - np.where(rot + ii >= R, R, 0)
                    kof = np.where(k < kend, xo(cc - c_lo, slr) + jj, 0)
                    for qq in range(0, RQ, 4):
                        qx = qq + lq
                        qo = np.where(qx < Wout, qx * S, 0)
                        lds.access("x", kof + qo, tsz, "patch fragment read")
                        # meaning: slot sl holds input row oh*S + ((sl - rot) mod R)
                        # (the ring walk below checks that), column u holds input
                        # column u - P
                        if XD:
                            sl, cx = kof // SLOT, (kof % SLOT) // Wpad
                            ucol = (kof % SLOT) % Wpad + qo
                        else:
                            sl, cx = (kof % CH) // Wpad, kof // CH
                            ucol = (kof % CH) % Wpad + qo
                        got = x_cell(g, c_lo + cx, oh * S + (sl - rot) % R - g["P"],
                                     ucol - g["P"])
                        want = x_cell(g, cc, oh * S + ii - g["P"], qx * S + jj - g["P"])
                        live = (k < kend) & (qx < Wout)
                        need(np.where(live, (want == got) & (ucol < Wpad), True),
                             f"{kernel}: a patch fragment holds the wrong cell")
            for qq in range(0, RQ, 4):
                for mb in range(4):
                    lds.access("g", (l16 + 16 * mb) * SG + lq + qq, tsz, "g fragment read")
    tid = np.arange(768)
    lds.access("g", (tid // 12) * SG + RQ - 1, tsz, "db read")
    # the emitted masked gradient: (n, f, oh, u) for f < F, u < Wout
    f = np.arange(cdiv(g["F"], BM) * BM)[:, None]
    u = np.arange(RQ)[None, :]
    ok = (f < g["F"]) & (u < Wout)
    for n, oh in ((0, 0), (g["N"] - 1, g["Hout"] - 1)):
        glob(kernel, "g_out", ((n * g["F"] + f) * g["Q"] + oh * Wout + u)[ok], g["N"] * g["F"] * g["Q"])
    ring_contents_ok(g, kernel, g["N"] * g["Hout"], p["splits"], R)
    ring_contents_ok(g, kernel, g["N"] * g["Hout"], 1, R)
    wgrad_outputs(g, p, tsz, kernel, ranges, NBW, 12, ws_elems)


def model_wgrad_tiles(g, p, tsz, form):
    kernel = "wgrad_tiles"
    HfWf, K, Wout, S, Hf, Q = g["Hf"] * g["Wf"], g["K"], g["Wout"], g["S"], g["Hf"], g["Q"]
    KR, SG, RQ, Wpad = p["chunk"], p["g_stride"], p["tile_pixels"], p["window_width"]
    rows_max, spr, pipelined = p["window_rows"], p["row_slices"], p["pipelined"]
    NBW = KR // 64
    need(KR == 64 * NBW and NBW in (1, 2, 3), f"{kernel}: k range {KR}")
    lds, ranges, nch_alloc, CH, ws_elems = wgrad_common(g, p, tsz, kernel, 256)
    lane = np.arange(64)
    lq, l16 = lane >> 4, lane & 15
    pb = form == "pooled_source"
    tiles_per_img = g["Hout"] * spr if spr else cdiv(Q, RQ)
    if spr:
        need(Wpad == (RQ - 1) * S + g["Wf"] and rows_max == Hf, f"{kernel}: sliced tile window")
    else:
        need(Wpad == (Wout - 1) * S + g["Wf"], f"{kernel}: window width")
    if pipelined:
        need(BM * RQ <= 256 * 14 and nch_alloc * CH <= 256 * 16,
             f"{kernel}: a tile exceeds the staging registers")
    e = np.arange(BM * RQ)
    r = div_magic(e, RQ, f"{kernel} g row")
    lds.access("g", r * SG + e - r * RQ, tsz, "g tile store")
    nr_ = len(ranges)
    if tiles_per_img * nr_ <= MAX_TILES:
        t_pick, r_pick = list(range(tiles_per_img)), list(range(nr_))
    else:
        r_pick = sample(nr_, min(nr_, 4))
        t_pick = sample(tiles_per_img, max(MAX_TILES // len(r_pick), 8))
    for t in t_pick:
        if spr:
            oh = t // spr
            ow0 = (t - oh * spr) * RQ
            q0 = oh * Wout + ow0
            qend = q0 + min(RQ, Wout - ow0)
            qy0, rows_need = oh, Hf
        else:
            ow0, q0 = 0, t * RQ
            qend = min(q0 + RQ, Q)
            qy0 = q0 // Wout
            rows_need = ((qend - 1) // Wout - qy0) * S + Hf
        need(rows_need <= rows_max, f"{kernel}: tile {t} needs {rows_need} window rows")
        ybase, xbase = qy0 * S - g["P"], ow0 * S - g["P"]
        if pb:
            PS = g["PS"]
            ln = qend - q0
            rows = 1 if spr else int(div_magic(qend - 1 - qy0 * Wout, Wout)) + 1
            py_lo = int(div_magic(qy0, PS))
            py_hi = int(div_magic(qy0 + rows - 1, PS))
            px_lo = int(div_magic(ow0, PS))
            px_hi = int(div_magic(ow0 + ln - 1 if spr else Wout - 1, PS))
            npx = px_hi - px_lo + 1
            nw = (py_hi - py_lo + 1) * npx
            written = np.zeros(BM * RQ, dtype=np.int64)
            if pipelined:
                need(cdiv(BM * nw, 256) <= 8, f"{kernel}: {BM * nw} pooled windows a tile")
                e = np.arange(BM * nw)
                rr = div_small(e, nw)
                w = e - rr * nw
                wy = div_small(w, npx)
                py, px = py_lo + wy, px_lo + w - wy * npx
                for dy in range(PS):
                    oy = py * PS + dy
                    for dx in range(PS):
                        ox = px * PS + dx
                        q = oy * Wout + ox
                        ok = (oy < g["Hout"]) & (ox < Wout) & (q >= q0) & (q < qend)
                        idx = (rr * SG + q - q0)[ok]
                        lds.access("g", idx, tsz, "pooled-source g write")
                        np.add.at(written, (rr * RQ + q - q0)[ok], 1)
                tail = RQ - ln
                if tail:
                    e = np.arange(BM * tail)
                    rr = div_small(e, tail)
                    lds.access("g", rr * SG + ln + e - rr * tail, tsz, "g tail zeroing")
                want = np.zeros((BM, RQ), dtype=np.int64)
                want[:, :ln] = 1
                need(written == want.ravel(), f"{kernel}: pooled-source writes miss or repeat cells")
            else:  # direct staging: one pool_src_grad per cell
                qs = np.arange(q0, qend)
                div_magic(qs // Wout, PS, f"{kernel} pooled-source row")
                div_magic(qs % Wout, PS, f"{kernel} pooled-source column")
        for kbeg, kend, c_lo, nch in [ranges[i] for i in r_pick]:
            tot_x = nch * CH
            e = np.arange(tot_x)
            if pipelined:
                c = div_magic(e, CH, f"{kernel} window channel")
                rem = e - c * CH
                div_magic(rem, Wpad, f"{kernel} window row")
            lds.access("x", e, tsz, "window store")
            tr = (e % CH) // Wpad
            # rows past the tile's: zeros (register staging) or stale (direct staging)
            xcells = np.where(tr < rows_need,
                              x_cell(g, c_lo + e // CH, ybase + tr, xbase + (e % CH) % Wpad),
                              -1 if pipelined else -2)
            for w in range(4):
                for nb in range(NBW):
                    k = kbeg + (w * NBW + nb) * 16 + l16
                    c = k // HfWf
                    tp = k - c * HfWf
                    kof = np.where(k < kend, (c - c_lo) * CH + (tp // g["Wf"]) * Wpad + tp % g["Wf"], 0)
                    for qq in range(0, RQ + 4, 4):
                        q = q0 + qq + lq
                        rel = q - qy0 * Wout
                        dy = div_magic(np.where(q < qend, rel, 0), Wout, f"{kernel} pixel row")
                        qx = rel - dy * Wout
                        qo = np.where(q < qend, dy * S * Wpad + (qx - ow0) * S, 0)
                        lds.access("x", kof + qo, tsz, "patch fragment read")
                        if qq < RQ:
                            oh, ow = q // Wout, q % Wout
                            kc = np.minimum(k, K - 1)
                            cc, tq = kc // HfWf, kc % HfWf
                            want = x_cell(g, cc, oh * S + tq // g["Wf"] - g["P"],
                                          ow * S + tq % g["Wf"] - g["P"])
                            need(np.where((k < kend) & (q < qend), xcells[kof + qo] == want, True),
                                 f"{kernel}: a patch fragment holds the wrong cell")
        for qq in range(0, RQ + 4, 4):
            for mb in range(4):
                lds.access("all", (l16 + 16 * mb) * SG + lq + qq, tsz, "g fragment read")
    tid = np.arange(256)
    lds.access("g", (tid >> 2) * SG + RQ - 1, tsz, "db read")
    # the emitted masked gradient of the last image's last tile and filter tile
    ft = cdiv(g["F"], BM) - 1
    r = np.arange(BM)[:, None]
    u = np.arange(RQ)[None, :]
    q0 = Q - (Q - 1) % RQ - 1 if not spr else (g["Hout"] - 1) * Wout + (spr - 1) * RQ
    qend = Q
    ok = (ft * BM + r < g["F"]) & (q0 + u < qend)
    glob(kernel, "g_out", (((g["N"] - 1) * g["F"] + ft * BM) * Q + r * Q + q0 + u)[ok],
         g["N"] * g["F"] * Q)
    wgrad_outputs(g, p, tsz, kernel, ranges, NBW, 4, ws_elems)


def model_wgrad_pool_sparse(g, p, tsz, form):
    """The pool-window sum: block (image group, four filters) stages each padded
    image in LDS; a lane's windows read the K taps around their argmax cell."""
    kernel = "wgrad_pool_sparse"
    F, N, K = g["F"], g["N"], g["K"]
    groups, FW = p["splits"], p["tile_m"]
    Hx, Wx = g["Hin"] + 2 * g["P"], g["Win"] + 2 * g["P"]
    plane = Hx * Wx
    need(form == "pooled_source" and K <= 32 and FW == 4, f"{kernel}: form")
    need(p["blocks"] == cdiv(F, FW) * groups and 1 <= groups <= N, f"{kernel}: grid")
    need(p["window_width"] == Wx and p["window_rows"] == Hx, f"{kernel}: staged image")
    lds = Lds(p["lds_bytes"], kernel)
    lds.region("image", 0, tsz * g["C"] * plane)
    ws_elems = p["workspace_bytes"] // tsz
    need(groups * (F * K + F) <= ws_elems, f"{kernel}: partials exceed the workspace")
    glob(kernel, "workspace", [(groups - 1) * F * K + (F - 1) * K + K - 1,
                               groups * F * K + (groups - 1) * F + F - 1], ws_elems)
    seen = np.zeros(N, dtype=np.int64)
    for grp in range(groups):
        n0, n1 = grp * N // groups, (grp + 1) * N // groups
        need(n1 > n0, f"{kernel}: an empty image group")
        seen[n0:n1] += 1
    need(seen == 1, f"{kernel}: images not covered once by the groups")
    # staging: every padded cell once, from a valid (clamped) input element
    e = np.arange(g["C"] * plane)
    c = div_magic(e, plane, f"{kernel} image channel")
    r = e - c * plane
    yp = div_magic(r, Wx, f"{kernel} image row")
    y, x = yp - g["P"], r - yp * Wx - g["P"]
    inside = (y >= 0) & (y < g["Hin"]) & (x >= 0) & (x < g["Win"])
    lds.access("image", e, tsz, "image store")
    glob(kernel, "X", np.where(inside, (c * g["Hin"] + y) * g["Win"] + x, 0),
         g["C"] * g["Hin"] * g["Win"])
    # pool arrays of a (image, filter) plane: clamped window indices
    nwi = g["Hp"] * g["Wp"]
    w = np.arange(0, cdiv(nwi, 256) * 256)
    glob(kernel, "pool arrays", ((N - 1) * F + F - 1) * nwi + np.minimum(w, nwi - 1), N * F * nwi)
    # every cell a window routes (also the clamped cell of dead windows): its
    # K taps stay in the staged image, and tap k is input (c, oy*S+i-P, ox*S+j-P)
    div_magic(np.arange(nwi), g["Wp"], f"{kernel} window row")
    q = np.arange(g["Q"])
    oy = div_magic(q, g["Wout"], f"{kernel} cell row")
    ox = q - oy * g["Wout"]
    k = np.arange(K)
    HfWf = g["Hf"] * g["Wf"]
    kc, kt = k // HfWf, k % HfWf
    tap = kc * plane + (kt // g["Wf"]) * Wx + kt % g["Wf"]
    idx = (oy * g["S"] * Wx + ox * g["S"])[:, None] + tap[None, :]
    lds.access("image", idx, tsz, "tap read")
    yy = (oy[:, None] * g["S"] + kt // g["Wf"]) - g["P"]
    xx = (ox[:, None] * g["S"] + kt % g["Wf"]) - g["P"]
    need((idx // plane == kc) & ((idx % plane) // Wx - g["P"] == yy) & ((idx % plane) % Wx - g["P"] == xx),
         f"{kernel}: a tap reads the wrong input cell")


# ================================================================ dispatch
MODELS = {"igemm_dma": model_igemm_dma, "igemm_reg": model_igemm_reg, "small_m": model_small_m,
          "resident": model_resident, "wgrad_ring": model_wgrad_ring,
          "wgrad_tiles": model_wgrad_tiles, "wgrad_pool_sparse": model_wgrad_pool_sparse}


def check_conv(s, pass_name, dtype, plan, form="plain", pool=None):
    """Model the launch whose plan the library reports (plan: the dict of
    conv2d_plan / conv2d_plan_fused) for shape s; raises ModelError."""
    tsz = 8 if dtype == "f64" else 4
    if pass_name == "backward_filter":
        g = wgrad_geometry(s)
        plane = (g["Hout"], g["Wout"])
    else:
        g = gemm_view(s, pass_name)
        plane = (g["Qh"], g["Qw"]) if pass_name == "forward" else (g["Sh"], g["Sw"])
    if pool is not None and plan.get("fused", 1):
        ph, pw, ps, _ = pool
        g.update(PH=ph, PW=pw, PS=ps, Hp=(plane[0] - ph) // ps + 1, Wp=(plane[1] - pw) // ps + 1)
    if not plan.get("fused", 1):
        form = "plain"
    MODELS[plan["kernel"]](g, plan, tsz, form)
    if form == "pool_epilogue" and plan["kernel"] == "igemm_dma":
        TS = plan["tile_stride"]
        Q = g["Qh"] * g["Qw"]
        pool_coverage("igemm_dma", g, [(q0, min(q0 + TS, Q)) for q0 in range(0, Q, TS)])
