// conv2d backward_filter (+ fused relu mask and bias gradient) on the gfx950
// matrix cores.
//
//   g          = dout masked to out_fwd > 0 (or dout when no mask is given)
//   dW[f, k]   = sum_{n, q} g[n, f, q] * B_n[k, q],  k = (c, i, j), q = (oh, ow)
//   db[f]      = sum_{n, q} g[n, f, q]
// with B_n the (never materialised) patch matrix of image n.  This is a GEMM
// with a small output (F x C*Hf*Wf) and a very long reduction (N*Hout*Wout), so
// the reduction is split: block (f-tile, k-range, split) sums its share of the
// (image, pixel-tile) list into registers and writes one partial dW (and db)
// to the workspace; a second kernel adds the partials in split order.  The
// partition depends only on the problem sizes, so results are bitwise
// reproducible.
//
// Per pixel tile the block stages in LDS: the 64 x RQ slice of g (mask applied
// while loading) and the rows of X that the tile's windows touch for the
// channels of its k-range (zero padded).  Each of the 4 waves owns all 64 f rows
// and NBW 16-column blocks of the k-range: per 4-pixel step it reads 4 g
// fragments and NBW patch fragments and issues 4 x NBW MFMAs.
//
// Zero skip (the ZSKIP instantiations; paper, Section 3 "Sparse Operations":
// operations that are safe on sparse inputs do fewer flops): an MFMA whose g
// fragment (16 filters x 4 pixels of the masked gradient) or patch fragment
// (4 pixels x 16 columns of X) is entirely zero, by a wavefront ballot, is not
// issued.  Its product is exactly zero, so the result is bitwise that of the
// dense kernel up to the sign of zero results.
//
// Pooled source (the PB instantiations; paper, Section "Future Work": vertical
// fusion): the conv was followed by relu and a non-overlapping max-pool, and g
// is built while staging from that pool's upstream gradient, argmax and pooled
// values (pool_src_grad), so the routed gradient is never stored.
#include <algorithm>

#include "common.hpp"
#include "internal.hpp"

namespace dmlnn {
namespace {

constexpr int kThreads = 256;
constexpr int kBM = 64;
constexpr size_t kLdsBudget = 72 * 1024;
// Upper bound on resident blocks (256 CUs x 4 blocks) used to size the workspace
// without a device; the launch uses the measured occupancy, up to this bound.
constexpr int kCUs = 256;          // MI355X compute units
constexpr int kMaxThreadsPerCU = 2048;
constexpr size_t kLdsPerCU = 160 * 1024;
constexpr int kMinTiles = 2;  // fewest pixel tiles a split reduces
constexpr int kMG = 14;  // g-tile elements each thread stages per pixel tile
constexpr int kMX = 16;  // X-window elements each thread stages per pixel tile
constexpr int kMGP = 8;  // pooled source: pool windows each thread stages per pixel tile

struct WgradArgs {
    const void *X, *dout, *mask;
    void *ws;
    int N, C, Hin, Win, F, Hf, Wf, HfWf, S, P, Hout, Wout, Q, K;
    int KR, nkr, nft, RQ, tiles_per_img, T_total, splits;
    int Wpad, CH, SG;
    int pipelined;  // 1: a pixel tile fits the per-thread staging registers
    int rows_max;
    int spr;        // 0: tiles are runs of whole output rows; else slices per output row
    unsigned long long magic_rq, magic_wpad, magic_ch, magic_wout, magic_hwf, magic_wf;
    int x_dma_insts;  // ring with the X rows by LDS DMA: 64-dword instructions a slot
    PoolSrc pool;   // PB kernels: g comes from a following max-pool's backward
    void *g_out;    // or null: g (dout masked to out_fwd > 0) is also written here
                    // (by the k-range-0 blocks, each element once)
};

template <typename T, int NBW, bool ZSKIP, bool PB>
__global__ __launch_bounds__(kThreads, 2) void conv_wgrad_kernel(WgradArgs a)
{
    using MF = Mfma<T>;
    extern __shared__ __align__(16) unsigned char smem[];
    T *s_g = reinterpret_cast<T *>(smem);
    T *s_x = s_g + kBM * a.SG;

    const int tid = threadIdx.x, lane = lane_id(), wave = wave_id();
    const int L = xcd_logical_block(blockIdx.x, gridDim.x);
    const int kr = L % a.nkr;
    const int rest = L / a.nkr;
    const int ft = rest % a.nft;
    const int split = rest / a.nft;
    // 16-row blocks of the filter tile that hold filters (the others' g rows are zero)
    const int nmb = min(4, (a.F - ft * kBM + 15) / 16);

    const int kbeg = kr * a.KR;
    const int kend = min(a.K, kbeg + a.KR);
    const int c_lo = kbeg / a.HfWf;
    const int nch = (kend - 1) / a.HfWf - c_lo + 1;

    // LDS offset of column k (channel relative to c_lo, tap i, j) of this lane's blocks.
    int kof[NBW];
#pragma unroll
    for (int nb = 0; nb < NBW; ++nb) {
        int k = kbeg + (wave * NBW + nb) * 16 + (lane & 15);
        int c = k / a.HfWf, t = k - c * a.HfWf;
        int i = t / a.Wf, j = t - i * a.Wf;
        kof[nb] = (k < kend) ? (c - c_lo) * a.CH + i * a.Wpad + j : 0;
    }

    typename MF::acc_t acc[4][NBW];
#pragma unroll
    for (int mb = 0; mb < 4; ++mb)
#pragma unroll
        for (int nb = 0; nb < NBW; ++nb) acc[mb][nb] = MF::zero();
    T dbacc = T(0);

    const T *X = reinterpret_cast<const T *>(a.X);
    const T *dout = reinterpret_cast<const T *>(a.dout);
    const T *mask = reinterpret_cast<const T *>(a.mask);
    const long long t_begin = (long long)split * a.T_total / a.splits;
    const long long t_end = (long long)(split + 1) * a.T_total / a.splits;

    // Pixel tile tt covers pixels [q0, qend) of image n.  Its X window is the
    // rows_need input rows of channels c_lo .. c_lo+nch-1 that the windows touch,
    // and Wpad columns starting at input column xbase: the whole padded row when
    // tiles are runs of whole output rows, or just the columns of one slice of an
    // output row when rows are wider than a tile (spr > 0).
    struct TileGeo {
        int n, q0, qend, qy0, ow0, rows_need, ybase, xbase;
        // pooled source: the tile's cells lie in the stride regions (PS x PS
        // cells, region (py, px) holding window (py, px) in its corner) of
        // pool rows py_lo .. and columns px_lo .., npx a row, nw in all
        int py_lo, px_lo, npx, nw;
    };
    auto geo = [&](long long tt) {
        TileGeo g;
        g.n = (int)(tt / a.tiles_per_img);
        const int qt = (int)(tt - (long long)g.n * a.tiles_per_img);
        if (a.spr) {
            const int oh = qt / a.spr;
            g.ow0 = (qt - oh * a.spr) * a.RQ;
            g.q0 = oh * a.Wout + g.ow0;
            g.qend = g.q0 + min(a.RQ, a.Wout - g.ow0);
            g.qy0 = oh;
            g.rows_need = a.Hf;
        } else {
            g.ow0 = 0;
            g.q0 = qt * a.RQ;
            g.qend = min(g.q0 + a.RQ, a.Q);
            g.qy0 = g.q0 / a.Wout;
            g.rows_need = ((g.qend - 1) / a.Wout - g.qy0) * a.S + a.Hf;
        }
        g.ybase = g.qy0 * a.S - a.P;
        g.xbase = g.ow0 * a.S - a.P;
        if (PB) {
            const int len = g.qend - g.q0;
            const int rows = a.spr ? 1 : div_magic(g.qend - 1 - g.qy0 * a.Wout, a.magic_wout) + 1;
            g.py_lo = div_magic(g.qy0, a.pool.magic_ps);
            const int py_hi = div_magic(g.qy0 + rows - 1, a.pool.magic_ps);
            g.px_lo = div_magic(g.ow0, a.pool.magic_ps);
            const int px_hi = div_magic(a.spr ? g.ow0 + len - 1 : a.Wout - 1, a.pool.magic_ps);
            g.npx = px_hi - g.px_lo + 1;
            g.nw = (py_hi - g.py_lo + 1) * g.npx;
        }
        return g;
    };

    // Software pipeline: the global loads of tile tt+1 are issued into
    // registers before the MFMA loop of tile tt and written to LDS after it.
    const int tot_g = kBM * a.RQ;
    const int tot_x = nch * a.CH;  // channels x rows_max x Wpad (rows past rows_need are 0)
    constexpr int NG = PB ? 1 : kMG, NP = PB ? kMGP : 1;
    T vg[NG], vm[NG], vx[kMX];
    T pd[NP], pp[NP];  // pooled source: each owned window's gradient and pooled value
    int pa[NP];        // and argmax
    // Pooled source: element e of a tile is (filter row r, stride region w).
    auto region = [&](const TileGeo &g, int e, int &r, int &py, int &px) {
        r = div_small(e, g.nw, 1.0f / (float)g.nw);
        const int w = e - r * g.nw;
        const int wy = div_small(w, g.npx, 1.0f / (float)g.npx);
        py = g.py_lo + wy;
        px = g.px_lo + (w - wy * g.npx);
    };
    auto load = [&](const TileGeo &g) {
        const int tid = opaque(threadIdx.x);
        const size_t gbase = ((size_t)g.n * a.F + ft * kBM) * a.Q;
        if constexpr (PB) {
            // one window's three values per element (clamped: always a valid
            // address, so the loads issue together)
            const int nit = (kBM * g.nw + kThreads - 1) / kThreads;  // tile-uniform
#pragma unroll
            for (int it = 0; it < kMGP; ++it) {
                if (it >= nit) break;
                int r, py, px;
                region(g, tid + kThreads * it, r, py, px);
                const int f = min(ft * kBM + r, a.F - 1);
                const size_t o = ((size_t)g.n * a.F + f) * a.pool.Hp * a.pool.Wp +
                                 (size_t)min(py, a.pool.Hp - 1) * a.pool.Wp + min(px, a.pool.Wp - 1);
                pd[it] = reinterpret_cast<const T *>(a.pool.dpool)[o];
                pa[it] = a.pool.argmax[o];
                pp[it] = reinterpret_cast<const T *>(a.pool.pooled)[o];
            }
        } else {
#pragma unroll
        for (int it = 0; it < kMG; ++it) {
            const int e = tid + kThreads * it;
            T v = T(0), mv = T(1);
            if (e < tot_g) {
                const int r = div_magic(e, a.magic_rq), u = e - r * a.RQ;
                const int q = g.q0 + u;
                if (ft * kBM + r < a.F && q < g.qend) {
                    const size_t o = gbase + (size_t)r * a.Q + q;
                    v = dout[o];
                    if (mask) mv = mask[o];
                }
            }
            vg[it] = v;
            vm[it] = mv;
        }
        }
#pragma unroll
        for (int it = 0; it < kMX; ++it) {
            const int e = tid + kThreads * it;
            T v = T(0);
            if (e < tot_x) {
                const int c = div_magic(e, a.magic_ch), rem = e - c * a.CH;
                const int t = div_magic(rem, a.magic_wpad), u = rem - t * a.Wpad;
                const int cg = c_lo + c, y = g.ybase + t, x = g.xbase + u;
                if (t < g.rows_need && cg < a.C && y >= 0 && y < a.Hin && x >= 0 && x < a.Win)
                    v = X[(((size_t)g.n * a.C + cg) * a.Hin + y) * a.Win + x];
            }
            vx[it] = v;
        }
    };
    auto store = [&](const TileGeo &g) {
        const int tid = opaque(threadIdx.x);
        if constexpr (PB) {
            // Each element writes its region's cells that lie in the tile: the
            // window's gradient at its argmax when the pooled value is positive,
            // zeros elsewhere (every cell of the tile is in one region).
            const int len = g.qend - g.q0;
            const int nit = (kBM * g.nw + kThreads - 1) / kThreads;  // tile-uniform
#pragma unroll
            for (int it = 0; it < kMGP; ++it) {
                if (it >= nit) break;
                const int e = tid + kThreads * it;
                int r, py, px;
                region(g, e, r, py, px);
                if (e >= kBM * g.nw) continue;
                const int f = ft * kBM + r;
                const bool win = f < a.F && py < a.pool.Hp && px < a.pool.Wp && pp[it] > T(0);
                const int tgt = win ? pa[it] - f * a.Q : -1;
                T *row = s_g + r * a.SG - g.q0;
                for (int dy = 0; dy < a.pool.PS; ++dy) {
                    const int oy = py * a.pool.PS + dy;
                    for (int dx = 0; dx < a.pool.PS; ++dx) {
                        const int ox = px * a.pool.PS + dx;
                        const int q = oy * a.Wout + ox;
                        if (oy < a.Hout && ox < a.Wout && q >= g.q0 && q < g.qend)
                            row[q] = q == tgt ? pd[it] : T(0);
                    }
                }
            }
            // columns past a short tile's end stay zero
            const int tail = a.RQ - len;
            for (int e = tid; e < kBM * tail; e += kThreads) {
                const int r = div_small(e, tail, 1.0f / (float)tail);
                s_g[r * a.SG + len + (e - r * tail)] = T(0);
            }
        } else {
        T *gout = (a.g_out && kr == 0) ? reinterpret_cast<T *>(a.g_out) : nullptr;
        const size_t gbase = ((size_t)g.n * a.F + ft * kBM) * a.Q;
#pragma unroll
        for (int it = 0; it < kMG; ++it) {
            const int e = tid + kThreads * it;
            if (e < tot_g) {
                const int r = div_magic(e, a.magic_rq), u = e - r * a.RQ;
                const T v = (vm[it] > T(0)) ? vg[it] : T(0);
                s_g[r * a.SG + u] = v;
                if (gout && ft * kBM + r < a.F && g.q0 + u < g.qend)
                    gout[gbase + (size_t)r * a.Q + g.q0 + u] = v;
            }
        }
        }
#pragma unroll
        for (int it = 0; it < kMX; ++it) {
            const int e = tid + kThreads * it;
            if (e < tot_x) s_x[e] = vx[it];  // (c, t, u) at c*CH + t*Wpad + u
        }
    };
    // Fallback for tiles larger than the staging registers.
    auto stage_direct = [&](const TileGeo &g) {
        for (int r = wave; r < kBM; r += kThreads / kWave) {
            int fg = ft * kBM + r;
            size_t goff = ((size_t)g.n * a.F + fg) * a.Q;
            for (int u = lane; u < a.RQ; u += kWave) {
                int q = g.q0 + u;
                T v = T(0);
                if (fg < a.F && q < g.qend) {
                    if (PB) {
                        const int oy = q / a.Wout;
                        v = pool_src_grad<T>(a.pool, g.n, a.F, fg, a.Q, a.Wout, oy, q - oy * a.Wout);
                    } else {
                        v = dout[goff + q];
                        if (mask && !(mask[goff + q] > T(0))) v = T(0);
                        if (a.g_out && kr == 0) reinterpret_cast<T *>(a.g_out)[goff + q] = v;
                    }
                }
                s_g[r * a.SG + u] = v;
            }
        }
        const int nrows = nch * g.rows_need;
        for (int r = wave; r < nrows; r += kThreads / kWave) {
            int c = r / g.rows_need, t = r - c * g.rows_need;
            int cg = c_lo + c, y = g.ybase + t;
            bool rowok = cg < a.C && y >= 0 && y < a.Hin;
            size_t xoff = (((size_t)g.n * a.C + cg) * a.Hin + (rowok ? y : 0)) * a.Win;
            T *dst = s_x + c * a.CH + t * a.Wpad;
            for (int u = lane; u < a.Wpad; u += kWave) {
                int x = g.xbase + u;
                dst[u] = (rowok && x >= 0 && x < a.Win) ? X[xoff + x] : T(0);
            }
        }
    };

    TileGeo cur = geo(t_begin);
    if (a.pipelined && t_begin < t_end) load(cur);
    const int lq = lane >> 4;
    for (long long tt = t_begin; tt < t_end; ++tt) {
        __syncthreads();
        if (a.pipelined)
            store(cur);
        else
            stage_direct(cur);
        __syncthreads();
        const TileGeo g = cur;
        if (a.pipelined && tt + 1 < t_end) {
            cur = geo(tt + 1);
            load(cur);
        } else if (tt + 1 < t_end) {
            cur = geo(tt + 1);
        }

        if (kr == 0) {  // bias gradient: thread (f = tid/4, phase = tid%4), fixed order
            const T *gr = s_g + (tid >> 2) * a.SG;
            for (int u = tid & 3; u < a.RQ; u += 4) dbacc += gr[u];
        }

        // LDS offset of pixel q0 + qq + lane/16 inside the X window (0 past the
        // tile's end: such columns of g are zero).  The row is found relative to
        // the tile's first row, so the magic division stays exact.
        auto q_off = [&](int qq) {
            const int q = g.q0 + qq + lq;
            if (q >= g.qend) return 0;
            const int rel = q - g.qy0 * a.Wout;
            const int dy = div_magic(rel, a.magic_wout), qx = rel - dy * a.Wout;
            return dy * a.S * a.Wpad + (qx - g.ow0) * a.S;
        };
        // Fragments are software-pipelined: those of step qq+4 are read while the
        // MFMAs of step qq issue.  The reads after the last step stay inside LDS
        // (the g rows are followed by the X window) and are not used.
        const T *grow = s_g + (lane & 15) * a.SG + lq;
        T av[4], bv[NBW];
        {
            const int qo = q_off(0);
#pragma unroll
            for (int mb = 0; mb < 4; ++mb) av[mb] = grow[mb * 16 * a.SG];
#pragma unroll
            for (int nb = 0; nb < NBW; ++nb) bv[nb] = s_x[kof[nb] + qo];
        }
        for (int qq = 0; qq < a.RQ; qq += 4) {
            T nav[4], nbv[NBW];
            const int nqo = q_off(qq + 4);
#pragma unroll
            for (int mb = 0; mb < 4; ++mb) nav[mb] = grow[mb * 16 * a.SG + qq + 4];
#pragma unroll
            for (int nb = 0; nb < NBW; ++nb) nbv[nb] = s_x[kof[nb] + nqo];
            bool za[4];
#pragma unroll
            for (int mb = 0; mb < 4; ++mb) za[mb] = mb >= nmb || (ZSKIP && wave_all_zero(av[mb]));
#pragma unroll
            for (int nb = 0; nb < NBW; ++nb) {
                if (ZSKIP && wave_all_zero(bv[nb])) continue;
#pragma unroll
                for (int mb = 0; mb < 4; ++mb)
                    if (!za[mb]) acc[mb][nb] = MF::mma(av[mb], bv[nb], acc[mb][nb]);
            }
#pragma unroll
            for (int mb = 0; mb < 4; ++mb) av[mb] = nav[mb];
#pragma unroll
            for (int nb = 0; nb < NBW; ++nb) bv[nb] = nbv[nb];
        }
    }

    T *wsp = reinterpret_cast<T *>(a.ws) + (size_t)split * a.F * a.K;
#pragma unroll
    for (int mb = 0; mb < 4; ++mb)
#pragma unroll
        for (int nb = 0; nb < NBW; ++nb)
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                int f = ft * kBM + mb * 16 + MF::row(lane, r);
                int k = kbeg + (wave * NBW + nb) * 16 + (lane & 15);
                if (f < a.F && k < kend) wsp[(size_t)f * a.K + k] = acc[mb][nb][r];
            }

    if (kr == 0) {
        __syncthreads();
        T *s_red = s_g;
        s_red[tid] = dbacc;
        __syncthreads();
        if (tid < kBM) {
            int f = ft * kBM + tid;
            if (f < a.F) {
                T s = s_red[4 * tid] + s_red[4 * tid + 1] + s_red[4 * tid + 2] + s_red[4 * tid + 3];
                T *wsdb = reinterpret_cast<T *>(a.ws) + (size_t)a.splits * a.F * a.K;
                wsdb[(size_t)split * a.F + f] = s;
            }
        }
    }
}

// dW[e] (e < FK) and db[f] (e = FK + f) = sum over splits of the partials.  A
// block covers 16 outputs with 16 split phases each: thread (e, ph) sums splits
// ph, ph+16, ... in order (double accumulation), and the 16 phase sums are added
// in phase order, so the result depends only on the split count.
template <typename T>
__global__ __launch_bounds__(256) void conv_wgrad_reduce(const T *ws, T *dW, T *db, int FK, int F,
                                                         int splits)
{
    __shared__ double s_part[16][17];
    const int el = threadIdx.x & 15, ph = threadIdx.x >> 4;
    const int e = blockIdx.x * 16 + el;
    const int total = FK + (db ? F : 0);
    double sum = 0.0;
    if (e < total) {
        const T *base = e < FK ? ws + e : ws + (size_t)splits * FK + (e - FK);
        const size_t stride = e < FK ? (size_t)FK : (size_t)F;
        // eight loads in flight, then added in split order (a chain of dependent
        // loads would wait a full memory latency per split)
        int sp = ph;
        for (; sp + 7 * 16 < splits; sp += 8 * 16) {
            T v[8];
#pragma unroll
            for (int u = 0; u < 8; ++u) v[u] = base[(size_t)(sp + 16 * u) * stride];
#pragma unroll
            for (int u = 0; u < 8; ++u) sum += (double)v[u];
        }
        for (; sp < splits; sp += 16) sum += (double)base[(size_t)sp * stride];
    }
    s_part[ph][el] = sum;
    __syncthreads();
    if (ph == 0 && e < total) {
        double t = s_part[0][el];
        for (int q = 1; q < 16; ++q) t += s_part[q][el];
        if (e < FK)
            dW[e] = (T)t;
        else
            db[e - FK] = (T)t;
    }
}

// Row-ring variant for layers whose output rows fit one tile (Wout <= 60).
// A block of 12 waves covers the whole k range (up to 12 x 16 x NBW columns),
// so each g tile is staged once for all of dW's columns instead of once per
// k-range block.  A pixel tile is one output row; consecutive tiles of a block
// are consecutive rows of one image, so the X window (Hf input rows per
// channel) is a ring: input row y (counted from the top padding row, yr = y +
// P) lives in slot yr mod Hf, and the next tile only stages its min(S, Hf) new
// rows.  The first tile of a block and of each image restages all Hf rows.
constexpr int kRingThreads = 768;
constexpr int kRingWaves = kRingThreads / kWave;
constexpr int kRG = 5;  // g-tile elements each thread stages per tile
constexpr int kRX = 5;  // new X-row elements each thread stages per tile
constexpr int kRGP = 5; // pooled source: pool windows each thread stages per tile (64 x 60 / 768)
// Row-mapped staging (RM: one new input row a tile, rows of at most 64
// elements, at most 72 channels): wave w stages rows w, w + 12, ... of the g
// tile and channels w, w + 12, ... of the new input row, a lane per element,
// so each row's offsets are a wave-uniform base plus the lane: no division
// and no per-element branch, where the element mapping above pays a magic
// division per element and a branch per staged element.
constexpr int kRMG = (kBM + kRingWaves - 1) / kRingWaves;  // g rows a wave stages (6)
constexpr int kRMX = 6;                                     // channels a wave stages
// X rows by LDS DMA (XM = 2; stride 1, where the LDS holds it): the ring has
// Hf + 1 slots, slot-major ([slot][channel][Wpad], the slot stride a whole
// number of 64-dword DMA instructions plus a bank-spreading pad), so the next tile's new
// row lands in the one slot the current tile does not read, straight from
// global memory during the current tile's MFMAs: no staging registers, no LDS
// stores, and no new-row work between the barriers.

// XM: how the next tile's input row is staged: 0 an element a thread, 1 a row
// a wave through registers, 2 by LDS DMA.
template <typename T, int NBW, bool ZSKIP, bool PB, int XM>
__global__ __launch_bounds__(kRingThreads, 1) void conv_wgrad_ring_kernel(WgradArgs a)
{
    using MF = Mfma<T>;
    extern __shared__ __align__(16) unsigned char smem[];
    T *s_g = reinterpret_cast<T *>(smem);
    // XM < 2: [channel][slot][Wpad], CH = Hf * Wpad a channel; XM = 2:
    // [slot][channel][Wpad], CH the slot stride
    T *s_x = s_g + kBM * a.SG;
    constexpr bool RM = XM == 1, XD = XM == 2;
    const int R = XD ? a.rows_max : a.Hf;  // ring slots: Hf, or Hf + 1 with the DMA
    auto xoff = [&](int c, int sl) { return XD ? sl * a.CH + c * a.Wpad : c * a.CH + sl * a.Wpad; };

    const int tid = threadIdx.x, lane = lane_id(), wave = wave_id();
    const int L = xcd_logical_block(blockIdx.x, gridDim.x);
    const int kr = L % a.nkr;
    const int rest = L / a.nkr;
    const int ft = rest % a.nft;
    const int split = rest / a.nft;

    const int kbeg = kr * a.KR;
    const int kend = min(a.K, kbeg + a.KR);
    const int c_lo = kbeg / a.HfWf;
    const int nch = (kend - 1) / a.HfWf - c_lo + 1;
    const int nr = min(a.S, a.Hf);  // new input rows per consecutive tile


    typename MF::acc_t acc[4][NBW];
#pragma unroll
    for (int mb = 0; mb < 4; ++mb)
#pragma unroll
        for (int nb = 0; nb < NBW; ++nb) acc[mb][nb] = MF::zero();
    T dbacc = T(0);

    const T *X = reinterpret_cast<const T *>(a.X);
    const T *dout = reinterpret_cast<const T *>(a.dout);
    const T *mask = reinterpret_cast<const T *>(a.mask);
    const long long t_begin = (long long)split * a.T_total / a.splits;
    const long long t_end = (long long)(split + 1) * a.T_total / a.splits;

    // Input row yr (from the top padding row) of channel c_lo + c, or zeros.
    // (The offset inside an image is 32-bit: an image holds fewer than 2^31
    // elements, which the host validates.)
    auto x_at = [&](int n, int c, int yr, int u) -> T {
        const int cg = c_lo + c, y = yr - a.P, x = u - a.P;
        const T *xi = X + (size_t)n * a.C * a.Hin * a.Win;  // the image (uniform)
        if (cg < a.C && y >= 0 && y < a.Hin && x >= 0 && x < a.Win)
            return xi[(cg * a.Hin + y) * a.Win + x];
        return T(0);
    };

    static_assert(!(PB && RM), "the pooled source has its own staging");
    // fp64 keeps the element mapping for the g tile: a sixth g row a wave would spill
    constexpr bool RMG = XM != 0 && !PB && sizeof(T) == 4;
    constexpr int NG = PB ? 1 : (RMG ? kRMG : kRG), NP = PB ? kRGP : 1;
    constexpr int NX = RM ? kRMX : kRX;  // (unused with the DMA)
    T vg[NG], vm[NG], vx[NX];
    // Pooled source: element e of a row is (filter row r, pool column px): the
    // window's three values are loaded once and its PS cells of the row written
    // from them (the gradient at the argmax, zeros elsewhere).
    T pd[NP], pp[NP];
    int pa[NP];
    const int npx = PB ? div_magic(a.Wout + a.pool.PS - 1, a.pool.magic_ps) : 1;
    const float rcp_npx = 1.0f / (float)npx;
    const int nit_r = (kBM * npx + kRingThreads - 1) / kRingThreads;  // owner iterations
    auto load_g = [&](int n, int oh) {
        const int tid = opaque(threadIdx.x);
        const size_t gbase = ((size_t)n * a.F + ft * kBM) * a.Q + (size_t)oh * a.Wout;
        if constexpr (PB) {
            const int py = min(div_magic(oh, a.pool.magic_ps), a.pool.Hp - 1);
#pragma unroll
            for (int it = 0; it < kRGP; ++it) {
                if (it >= nit_r) break;
                const int e = tid + kRingThreads * it;
                const int r = div_small(e, npx, rcp_npx), px = e - r * npx;
                const int f = min(ft * kBM + r, a.F - 1);
                const size_t o = (((size_t)n * a.F + f) * a.pool.Hp + py) * a.pool.Wp +
                                 min(px, a.pool.Wp - 1);
                pd[it] = reinterpret_cast<const T *>(a.pool.dpool)[o];
                pa[it] = a.pool.argmax[o];
                pp[it] = reinterpret_cast<const T *>(a.pool.pooled)[o];
            }
            return;
        }
        if constexpr (RMG) {
            const int ln = tid & (kWave - 1);
            const T *gb = dout + gbase, *mbp = mask ? mask + gbase : nullptr;
#pragma unroll
            for (int it = 0; it < NG; ++it) {
                const int r = wave + kRingWaves * it;  // wave-uniform
                T v = T(0), mv = T(1);
                if (r < kBM && ft * kBM + r < a.F && ln < a.Wout) {
                    const unsigned o = (unsigned)(r * a.Q) + ln;  // < F*Q < 2^31
                    v = gb[o];
                    if (mask) mv = mbp[o];
                }
                vg[it] = v;
                vm[it] = mv;
            }
            return;
        }
#pragma unroll
        for (int it = 0; it < NG; ++it) {
            const int e = tid + kRingThreads * it;
            T v = T(0), mv = T(1);
            if (e < kBM * a.RQ) {
                const int r = div_magic(e, a.magic_rq), u = e - r * a.RQ;
                if (ft * kBM + r < a.F && u < a.Wout) {
                    const size_t o = gbase + (unsigned)(r * a.Q + u);  // < F*Q < 2^31
                    v = dout[o];
                    if (mask) mv = mask[o];
                }
            }
            vg[it] = v;
            vm[it] = mv;
        }
    };
    auto store_g = [&](int n, int oh) {
        const int tid = opaque(threadIdx.x);
        if constexpr (PB) {
            (void)n;
            const int py = div_magic(oh, a.pool.magic_ps);
#pragma unroll
            for (int it = 0; it < kRGP; ++it) {
                if (it >= nit_r) break;
                const int e = tid + kRingThreads * it;
                const int r = div_small(e, npx, rcp_npx), px = e - r * npx;
                if (e >= kBM * npx) continue;
                const int f = ft * kBM + r;
                const bool win = f < a.F && py < a.pool.Hp && px < a.pool.Wp && pp[it] > T(0);
                const int tgt = win ? pa[it] - f * a.Q - oh * a.Wout : -1;
                for (int dx = 0; dx < a.pool.PS; ++dx) {
                    const int ox = px * a.pool.PS + dx;
                    if (ox < a.Wout) s_g[r * a.SG + ox] = ox == tgt ? pd[it] : T(0);
                }
            }
            return;
        }
        (void)n;
        if constexpr (RMG) {
            const int ln = tid & (kWave - 1);
#pragma unroll
            for (int it = 0; it < NG; ++it) {
                const int r = wave + kRingWaves * it;
                if (r < kBM && ln < a.RQ) s_g[r * a.SG + ln] = (vm[it] > T(0)) ? vg[it] : T(0);
            }
            return;
        }
#pragma unroll
        for (int it = 0; it < NG; ++it) {
            const int e = tid + kRingThreads * it;
            if (e < kBM * a.RQ) {
                const int r = div_magic(e, a.magic_rq), u = e - r * a.RQ;
                s_g[r * a.SG + u] = (vm[it] > T(0)) ? vg[it] : T(0);
            }
        }
    };
    // The staged tile's masked gradient to g_out (k-range 0 only): issued after
    // the barrier that ends the staging phase, from the registers the tile was
    // loaded into (before the next tile's loads reuse them), so the stores
    // leave the phase in which the matrix pipe idles.
    T *const gout = (!PB && a.g_out && kr == 0) ? reinterpret_cast<T *>(a.g_out) : nullptr;
    constexpr bool kLoadInLoop = sizeof(T) == 8;  // where the next tile's loads issue (below)
    auto emit_g = [&](int n, int oh) {
        if (PB || !gout) return;
        const int tid = opaque(threadIdx.x);
        if constexpr (RMG) {
            const int ln = tid & (kWave - 1);
            T *gb = gout + ((size_t)n * a.F + ft * kBM) * a.Q + (size_t)oh * a.Wout;
#pragma unroll
            for (int it = 0; it < NG; ++it) {
                const int r = wave + kRingWaves * it;
                if (r < kBM && ft * kBM + r < a.F && ln < a.Wout)
                    gb[(unsigned)(r * a.Q) + ln] = (vm[it] > T(0)) ? vg[it] : T(0);
            }
            return;
        }
#pragma unroll
        for (int it = 0; it < NG; ++it) {
            const int e = tid + kRingThreads * it;
            if (e < kBM * a.RQ) {
                const int r = div_magic(e, a.magic_rq), u = e - r * a.RQ;
                if (u < a.Wout && ft * kBM + r < a.F)
                    gout[((size_t)n * a.F + ft * kBM + r) * a.Q + (size_t)oh * a.Wout + u] =
                        (vm[it] > T(0)) ? vg[it] : T(0);
            }
        }
    };
    // The nr new rows of tile oh (rows yr = oh*S + Hf - nr + r).
    const int nrw = nr * a.Wpad;
    auto load_x = [&](int n, int oh) {
        const int tid = opaque(threadIdx.x);
        if constexpr (RM) {  // the one new row yr = oh*S + Hf - 1, channel c_lo + c a wave-row
            const int ln = tid & (kWave - 1);
            const int y = oh * a.S + a.Hf - 1 - a.P, x = ln - a.P;
            const bool ok = ln < a.Wpad && x >= 0 && x < a.Win && y >= 0 && y < a.Hin;
            const T *xi = X + (size_t)n * a.C * a.Hin * a.Win;  // the image
#pragma unroll
            for (int it = 0; it < NX; ++it) {
                const int c = wave + kRingWaves * it, cg = c_lo + c;
                T v = T(0);
                if (c < nch && cg < a.C && ok) v = xi[(unsigned)((cg * a.Hin + y) * a.Win) + x];
                vx[it] = v;
            }
            return;
        }
#pragma unroll
        for (int it = 0; it < kRX; ++it) {
            const int e = tid + kRingThreads * it;
            T v = T(0);
            if (e < nch * nrw) {
                const int c = div_magic(e, a.magic_ch), rem = e - c * nrw;
                const int r = div_magic(rem, a.magic_wpad), u = rem - r * a.Wpad;
                v = x_at(n, c, oh * a.S + a.Hf - nr + r, u);
            }
            vx[it] = v;
        }
    };
    // New row r goes to slot (s0 + r) mod Hf, s0 = (oh*S + Hf - nr) mod Hf (the
    // same for the whole block); r < nr <= Hf, so the wrap is one subtraction of
    // Hf rows, taken from the offset rem = r*Wpad + u within the channel's rows.
    // This phase sits between the two barriers with the matrix pipe idle, so it
    // avoids per-element division and modulo.
    auto store_x = [&](int oh) {
        const int tid = opaque(threadIdx.x);
        const int s0 = (oh * a.S + a.Hf - nr) % a.Hf;
        if constexpr (RM) {
            const int ln = tid & (kWave - 1);
#pragma unroll
            for (int it = 0; it < NX; ++it) {
                const int c = wave + kRingWaves * it;
                if (c < nch && ln < a.Wpad) s_x[c * a.CH + s0 * a.Wpad + ln] = vx[it];
            }
            return;
        }
        const int base = s0 * a.Wpad, wrap = (a.Hf - s0) * a.Wpad, ring = a.Hf * a.Wpad;
#pragma unroll
        for (int it = 0; it < kRX; ++it) {
            const int e = tid + kRingThreads * it;
            if (e < nch * nrw) {
                const int c = div_magic(e, a.magic_ch), rem = e - c * nrw;
                s_x[c * a.CH + base + rem - (rem >= wrap ? ring : 0)] = vx[it];
            }
        }
    };
    // All Hf rows of tile oh, straight from global memory (first tile of an image).
    // Element e is row rw = e / Wpad of the window (channel c = rw / Hf, filter
    // row t), column u; row t goes to slot (oh*S + t) mod Hf = rot0 + t, less Hf
    // once it reaches Hf.  Magic and reciprocal divisions (e < 2^16, rw < 2^22):
    // this runs between the barriers with the matrix pipe idle.
    auto stage_x_full = [&](int n, int oh) {
        const int tot = XD ? nch * a.Hf * a.Wpad : nch * a.CH;  // (CH = Hf * Wpad without the DMA)
        const int rot0 = (oh * a.S) % R;
        const float rcp_hf = 1.0f / (float)a.Hf;
        for (int e = tid; e < tot; e += kRingThreads) {
            const int rw = div_magic(e, a.magic_wpad), u = e - rw * a.Wpad;
            const int c = div_small(rw, a.Hf, rcp_hf), t = rw - c * a.Hf;
            const int sl = rot0 + t - (rot0 + t >= R ? R : 0);
            s_x[xoff(c, sl) + u] = x_at(n, c, oh * a.S + t, u);
        }
    };
    // XD: the new row yr = oh + Hf - 1 of tile oh (stride 1) into slot yr mod R,
    // every channel of the k range: dword d of the slot (instruction d / 64,
    // taken by wave (d / 64) mod 12) is element d / (sizeof(T) / 4) = (channel c,
    // column u); the padding columns, the channels past the range and the
    // rows outside the image load zeros (an offset past the buffer).
    auto dma_x = [&](int n, int oh) {
        const int yr = oh + a.Hf - 1, y = yr - a.P, sl = yr % R;
        const size_t img = (size_t)a.C * a.Hin * a.Win;
        const i32x4 rs = buffer_rsrc(X + (size_t)n * img, (unsigned)(img * sizeof(T)));
        const int ln = opaque(threadIdx.x) & (kWave - 1);
        constexpr int EPI = kWave * 4 / (int)sizeof(T);  // elements an instruction moves
        for (int i = wave; i < a.x_dma_insts; i += kRingWaves) {
            const int d = i * kWave + ln;
            const int e = sizeof(T) == 8 ? d >> 1 : d;
            const int half = sizeof(T) == 8 ? (d & 1) : 0;
            const int c = div_magic(e, a.magic_wpad), u = e - c * a.Wpad;
            const int cg = c_lo + c, x = u - a.P;
            const bool ok = c < nch && cg < a.C && x >= 0 && x < a.Win && y >= 0 && y < a.Hin;
            const int vo = ok ? (int)(((cg * a.Hin + y) * a.Win + x) * (int)sizeof(T)) + 4 * half
                              : kDmaZero;  // < the image's bytes < 2^31
            dma_dword(rs, s_x + sl * a.CH + i * EPI, vo, 0);
        }
    };

    if (t_begin < t_end) {
        const int n0 = (int)(t_begin / a.Hout), oh0 = (int)(t_begin - (long long)n0 * a.Hout);
        load_g(n0, oh0);
        if (PB) {
            // the g-tile columns past the row are never written by the windows
            const int tail = a.RQ - a.Wout;
            for (int e = tid; e < kBM * tail; e += kRingThreads) {
                const int r = div_small(e, tail, 1.0f / (float)tail);
                s_g[r * a.SG + a.Wout + (e - r * tail)] = T(0);
            }
        }
        store_g(n0, oh0);
        stage_x_full(n0, oh0);
        __syncthreads();
        emit_g(n0, oh0);
        if (!kLoadInLoop && t_begin + 1 < t_end) {
            const long long t1 = t_begin + 1;
            const int n1 = (int)(t1 / a.Hout), oh1 = (int)(t1 - (long long)n1 * a.Hout);
            load_g(n1, oh1);
            if (oh1 != 0) {
                if constexpr (XD)
                    dma_x(n1, oh1);
                else
                    load_x(n1, oh1);
            }
        }
    }
    const int lq = lane >> 4;
    // (image, output row) of the current tile, advanced by one row per tile
    // (no 64-bit division per tile)
    int cn = (int)(t_begin / a.Hout), coh = (int)(t_begin - (long long)cn * a.Hout);
    for (long long tt = t_begin; tt < t_end; ++tt) {
        const int n = cn, oh = coh;
        const int n1 = oh + 1 < a.Hout ? n : n + 1, oh1 = oh + 1 < a.Hout ? oh + 1 : 0;
        // LDS offset of column k = (c, i, j) of this lane's blocks: filter row i
        // of this tile sits in slot (oh*S + i) mod R.
        const int rot = (oh * a.S) % R;
        int kof[NBW];
#pragma unroll
        for (int nb = 0; nb < NBW; ++nb) {
            const int k = kbeg + (wave * NBW + nb) * 16 + (lane & 15);
            const int c = div_magic(k, a.magic_hwf), t = k - c * a.HfWf;
            const int i = div_magic(t, a.magic_wf), j = t - i * a.Wf;
            int sl = rot + i;
            sl -= sl >= R ? R : 0;
            kof[nb] = k < kend ? xoff(c - c_lo, sl) + j : 0;
        }

        if (kr == 0) {  // bias gradient: thread (f = tid/12, phase = tid%12), fixed order
            const T *gr = s_g + (tid / 12) * a.SG;
            for (int u = tid % 12; u < a.RQ; u += 12) dbacc += gr[u];
        }

        const T *grow = s_g + (lane & 15) * a.SG + lq;
        // fp64: the next tile's loads are issued inside this tile's MFMA loop,
        // at a k-step that differs per wave (the g tile and the X row at steps
        // six waves apart): the three waves of a SIMD then do their address
        // work at different times and the other two keep the matrix pipe fed
        // (all at once after the barrier, it idled: 1-2% of the pass).  fp32
        // (half the matrix time per tile) issues them after the barrier,
        // which measured faster there.
        const bool pf = kLoadInLoop && tt + 1 < t_end;
        const int pfg = min(4 * wave, a.RQ - 4);
        const int pfx = min(4 * ((wave + kRingWaves / 2) % kRingWaves), a.RQ - 4);
        for (int qq = 0; qq < a.RQ; qq += 4) {
            if (qq == pfg && pf) load_g(n1, oh1);
            if (qq == pfx && pf && oh1 != 0) {
                if constexpr (XD)
                    dma_x(n1, oh1);
                else
                    load_x(n1, oh1);
            }
            const int qx = qq + lq;
            const int qo = qx < a.Wout ? qx * a.S : 0;
            T av[4];
#pragma unroll
            for (int mb = 0; mb < 4; ++mb) av[mb] = grow[mb * 16 * a.SG + qq];
            bool za[4];
#pragma unroll
            for (int mb = 0; mb < 4; ++mb) za[mb] = ZSKIP && wave_all_zero(av[mb]);
#pragma unroll
            for (int nb = 0; nb < NBW; ++nb) {
                const T bv = s_x[kof[nb] + qo];
                if (ZSKIP && wave_all_zero(bv)) continue;
#pragma unroll
                for (int mb = 0; mb < 4; ++mb)
                    if (!za[mb]) acc[mb][nb] = MF::mma(av[mb], bv, acc[mb][nb]);
            }
        }

        if (tt + 1 < t_end) {
            __syncthreads();
            store_g(n1, oh1);
            if (oh1 == 0)
                stage_x_full(n1, oh1);
            else if constexpr (!XD)
                store_x(oh1);
            if constexpr (XD) wait_dma();  // this wave's DMA of the new row has landed
            __syncthreads();
            emit_g(n1, oh1);
            if (!kLoadInLoop && tt + 2 < t_end) {
                const int n2 = oh1 + 1 < a.Hout ? n1 : n1 + 1, oh2 = oh1 + 1 < a.Hout ? oh1 + 1 : 0;
                load_g(n2, oh2);
                if (oh2 != 0) {
                    if constexpr (XD)
                        dma_x(n2, oh2);
                    else
                        load_x(n2, oh2);
                }
            }
        }
        cn = n1;
        coh = oh1;
    }

    T *wsp = reinterpret_cast<T *>(a.ws) + (size_t)split * a.F * a.K;
#pragma unroll
    for (int mb = 0; mb < 4; ++mb)
#pragma unroll
        for (int nb = 0; nb < NBW; ++nb)
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                int f = ft * kBM + mb * 16 + MF::row(lane, r);
                int k = kbeg + (wave * NBW + nb) * 16 + (lane & 15);
                if (f < a.F && k < kend) wsp[(size_t)f * a.K + k] = acc[mb][nb][r];
            }

    if (kr == 0) {
        __syncthreads();
        T *s_red = s_g;
        s_red[tid] = dbacc;
        __syncthreads();
        if (tid < kBM) {
            int f = ft * kBM + tid;
            if (f < a.F) {
                T sum = T(0);
                for (int p = 0; p < 12; ++p) sum += s_red[12 * tid + p];
                T *wsdb = reinterpret_cast<T *>(a.ws) + (size_t)a.splits * a.F * a.K;
                wsdb[(size_t)split * a.F + f] = sum;
            }
        }
    }
}

// The most splits a launch may use, and the workspace holds: one resident
// round of blocks on a 256-CU device at one CU's LDS and thread limits (the
// launch takes the occupancy HIP reports, which is never above these), with at
// least kMinTiles pixel tiles per split.
long long split_bound(size_t lds, int threads, int per_split, long long T_total)
{
    long long per_cu = (long long)(kLdsPerCU / std::max<size_t>(lds, 1));
    per_cu = std::min<long long>(per_cu, kMaxThreadsPerCU / threads);
    per_cu = std::max<long long>(per_cu, 1);
    long long sp = kCUs * per_cu / per_split;
    sp = std::min(sp, T_total / kMinTiles);
    return std::max<long long>(sp, 1);
}

struct WPlan {
    int NBW, KR, nkr, nft, RQ, tiles_per_img, splits, Wpad, CH, SG, rows_max, pipelined, spr;
    int rowmap = 0;  // ring: row-mapped staging (one new row a tile, rows <= 64, <= 72 channels)
    int xdma = 0;    // ring: X rows by LDS DMA into Hf + 1 slot-major slots (stride 1)
    int x_dma_insts = 0;
    long long T_total;
    size_t lds;
};

size_t wlds(size_t tsz, int SG, int nch, int CH, int RQ)
{
    (void)RQ;
    return tsz * ((size_t)kBM * SG + (size_t)nch * CH);
}

bool make_wplan(size_t tsz, const ConvDims &d, WPlan &p)
{
    const int K = d.C * d.Hf * d.Wf;
    const int HfWf = d.Hf * d.Wf;
    const int Q = d.Hout * d.Wout;
    p.NBW = K > 128 ? 3 : (K > 64 ? 2 : 1);
    p.KR = 64 * p.NBW;
    p.nkr = (K + p.KR - 1) / p.KR;
    p.nft = (d.F + kBM - 1) / kBM;
    p.Wpad = (d.Wout - 1) * d.stride + d.Wf;
    const int nch_alloc = (p.KR - 1) / HfWf + 2;
    p.spr = 0;
    if (d.Wout > 56) {
        // Rows wider than a tile: each tile is one slice of an output row (at
        // most 56 pixels, a multiple of 4) and its X window spans only the
        // slice's input columns.
        int spr = (d.Wout + 55) / 56;
        int rq = ((d.Wout + spr - 1) / spr + 3) / 4 * 4;
        spr = (d.Wout + rq - 1) / rq;
        p.spr = spr;
        p.RQ = rq;
        p.rows_max = d.Hf;
        p.Wpad = (rq - 1) * d.stride + d.Wf;
        p.CH = p.rows_max * p.Wpad;
        p.SG = rq + 2;
        p.lds = wlds(tsz, p.SG, nch_alloc, p.CH, rq);
        if (p.lds > 160 * 1024) return false;
        p.pipelined = kBM * p.RQ <= kThreads * kMG && (long long)nch_alloc * p.CH <= kThreads * kMX;
        p.tiles_per_img = d.Hout * spr;
        p.T_total = (long long)d.N * p.tiles_per_img;
        p.splits = (int)split_bound(p.lds, kThreads, p.nkr * p.nft, p.T_total);
        return true;
    }
    // Pixel tile: whole output rows (at most 56 pixels so the g tile fits the
    // staging registers), a multiple of 4.
    int rq = d.Wout * (56 / d.Wout);
    if (rq > Q) rq = Q;
    rq = ((rq + 3) / 4) * 4;
    for (;;) {
        const bool aligned = rq % d.Wout == 0;
        int rows_max = aligned ? (rq / d.Wout - 1) * d.stride + d.Hf
                               : ((d.Wout + rq - 2) / d.Wout) * d.stride + d.Hf;
        int CH = rows_max * p.Wpad;
        int SG = rq + 2;  // 2 mod 4: the g-tile fragment reads are free of bank conflicts
        size_t lds = wlds(tsz, SG, nch_alloc, CH, rq);
        if (lds <= kLdsBudget || rq <= 4) {
            p.RQ = rq;
            p.CH = CH;
            p.SG = SG;
            p.rows_max = rows_max;
            p.lds = lds;
            break;
        }
        rq = ((rq / 2 + 3) / 4) * 4;
    }
    if (p.lds > 160 * 1024) return false;
    p.pipelined = kBM * p.RQ <= kThreads * kMG && (long long)nch_alloc * p.CH <= kThreads * kMX;
    p.tiles_per_img = (Q + p.RQ - 1) / p.RQ;
    p.T_total = (long long)d.N * p.tiles_per_img;
    p.splits = (int)split_bound(p.lds, kThreads, p.nkr * p.nft, p.T_total);
    return true;
}

// Plan for the row-ring kernel, or false when the layer does not suit it: rows
// wider than 60 outputs, a k range that 12 waves cover poorly, or an LDS window
// over the per-CU budget.
bool make_rplan(size_t tsz, const ConvDims &d, WPlan &p)
{
    const int K = d.C * d.Hf * d.Wf;
    const int HfWf = d.Hf * d.Wf;
    if (d.Wout > 60) return false;
    double best = 0.0;
    int nbw = 0;
    for (int cand = 3; cand >= 1; --cand) {
        const int kr = 16 * cand * kRingWaves;
        const int nkr = (K + kr - 1) / kr;
        const double eff = (double)K / ((double)nkr * kr);
        if (eff > best + 1e-9) {
            best = eff;
            nbw = cand;
        }
    }
    if (best < 0.85) return false;
    p.NBW = nbw;
    p.KR = 16 * nbw * kRingWaves;
    p.nkr = (K + p.KR - 1) / p.KR;
    p.nft = (d.F + kBM - 1) / kBM;
    p.RQ = (d.Wout + 3) / 4 * 4;
    p.SG = p.RQ + 2;
    p.spr = 0;
    p.rows_max = d.Hf;
    p.Wpad = (d.Wout - 1) * d.stride + d.Wf;
    p.CH = d.Hf * p.Wpad;
    const int nch_alloc = (p.KR - 1) / HfWf + 2;
    const int nr = d.stride < d.Hf ? d.stride : d.Hf;
    if (kBM * p.SG < kRingThreads) return false;  // the db reduction reuses the g tile
    if (kBM * p.RQ > kRingThreads * kRG) return false;
    if ((long long)nch_alloc * nr * p.Wpad > (long long)kRingThreads * kRX) return false;
    p.lds = tsz * ((size_t)kBM * p.SG + (size_t)nch_alloc * p.CH);
    if (p.lds > 160 * 1024) return false;
    p.rowmap = nr == 1 && p.Wpad <= kWave && p.RQ <= kWave && nch_alloc <= kRingWaves * kRMX;
    // X rows by LDS DMA, fp32 only: stride 1 (the new row misses the current
    // tile's slots), an image under 2 GiB (32-bit buffer offsets), and the Hf +
    // 1 slots in LDS.  (In fp64 the DMA measured slower than the row-mapped
    // registers it replaces: the ResNet layer's backward_filter 1.084-1.088
    // against 1.069-1.072 ms; fp32 0.684 against 0.691-0.694.)
    {
        const int epi = kWave * 4 / (int)tsz;  // elements a 64-dword instruction moves
        const int insts = (nch_alloc * p.Wpad + epi - 1) / epi;
        // The slot stride past the DMA'd extent: two taps a filter row apart
        // (j = Wf - 1, then j = 0 of the next row) are slot - (Wf - 1) elements
        // apart; half the 256-byte bank period puts their 16-lane pieces of a
        // fragment read in disjoint banks.
        const int period = 256 / (int)tsz;
        const int slot = insts * epi + (d.Wf - 1 + period / 2) % period;
        const size_t ldsx = tsz * ((size_t)kBM * p.SG + (size_t)(d.Hf + 1) * slot);
        const size_t img = tsz * (size_t)d.C * d.Hin * d.Win;
        if (tsz == 4 && d.stride == 1 && img < 0x80000000ull && ldsx <= 160 * 1024) {
            p.xdma = 1;
            p.x_dma_insts = insts;
            p.rows_max = d.Hf + 1;
            p.CH = slot;
            p.lds = ldsx;
        }
    }
    p.pipelined = 1;
    p.tiles_per_img = d.Hout;
    p.T_total = (long long)d.N * d.Hout;
    p.splits = (int)split_bound(p.lds, kRingThreads, p.nkr * p.nft, p.T_total);
    return true;
}

template <typename T, bool ZSKIP, bool PB, int XM>
void (*ring_kernel(int nbw))(WgradArgs)
{
    return nbw == 3 ? conv_wgrad_ring_kernel<T, 3, ZSKIP, PB, XM>
                    : (nbw == 2 ? conv_wgrad_ring_kernel<T, 2, ZSKIP, PB, XM>
                                : conv_wgrad_ring_kernel<T, 1, ZSKIP, PB, XM>);
}

// The ring kernel of a plan's X staging (the pooled source has no row-mapped form).
template <typename T, bool ZSKIP, bool PB>
void (*ring_kernel_for(const WPlan &p))(WgradArgs)
{
    if (p.xdma) return ring_kernel<T, ZSKIP, PB, 2>(p.NBW);
    if constexpr (!PB)
        if (p.rowmap) return ring_kernel<T, ZSKIP, PB, 1>(p.NBW);
    return ring_kernel<T, ZSKIP, PB, 0>(p.NBW);
}

// Blocks resident at once for a launch of kernel k, taken as the smaller of k's
// and its other zero-skip instantiation's (kz, or null): the two can differ in
// registers and so in occupancy, and the split count -- with it the summation
// order -- then stays the same under either zero-skip mode.
int common_slots(void (*k)(WgradArgs), void (*kz)(WgradArgs), int threads, size_t lds)
{
    int slots = resident_slots(k, threads, lds);
    if (kz && allow_dynamic_lds(kz, lds) == hipSuccess)
        slots = std::min(slots, resident_slots(kz, threads, lds));
    return slots;
}

template <typename T, bool ZSKIP, bool PB>
hipError_t launch_ring(WgradArgs a, const WPlan &p, void *dW, void *db, hipStream_t s)
{
    void (*k)(WgradArgs) = ring_kernel_for<T, ZSKIP, PB>(p);
    void (*kz)(WgradArgs) = nullptr;  // the other zero-skip form (the pooled source has none)
    if constexpr (!PB) kz = ring_kernel_for<T, !ZSKIP, PB>(p);
    hipError_t e = allow_dynamic_lds(k, p.lds);
    if (e != hipSuccess) return e;
    const int per_split = p.nkr * p.nft;
    int splits = common_slots(k, kz, kRingThreads, p.lds) / per_split;
    if (splits > p.splits) splits = p.splits;
    if (splits < 1) splits = 1;
    a.splits = splits;
    hipLaunchKernelGGL(k, dim3(splits * per_split), dim3(kRingThreads), p.lds, s, a);
    e = hipGetLastError();
    if (e != hipSuccess) return e;
    const int FK = a.F * a.K;
    const int total = FK + (db ? a.F : 0);
    hipLaunchKernelGGL((conv_wgrad_reduce<T>), dim3((total + 15) / 16), dim3(256), 0, s,
                       reinterpret_cast<const T *>(a.ws), reinterpret_cast<T *>(dW),
                       reinterpret_cast<T *>(db), FK, a.F, a.splits);
    return hipGetLastError();
}

template <typename T, bool ZSKIP, bool PB>
hipError_t launch_w(WgradArgs a, const WPlan &p, void *dW, void *db, hipStream_t s)
{
    auto k = p.NBW == 3 ? conv_wgrad_kernel<T, 3, ZSKIP, PB>
                        : (p.NBW == 2 ? conv_wgrad_kernel<T, 2, ZSKIP, PB>
                                      : conv_wgrad_kernel<T, 1, ZSKIP, PB>);
    void (*kz)(WgradArgs) = nullptr;  // the other zero-skip form (the pooled source has none)
    if constexpr (!PB)
        kz = p.NBW == 3 ? conv_wgrad_kernel<T, 3, !ZSKIP, PB>
                        : (p.NBW == 2 ? conv_wgrad_kernel<T, 2, !ZSKIP, PB>
                                      : conv_wgrad_kernel<T, 1, !ZSKIP, PB>);
    hipError_t e = allow_dynamic_lds(k, p.lds);
    if (e != hipSuccess) return e;
    // One resident round: as many splits as the device holds blocks at once (a
    // second, partial round would nearly double the time), within the workspace.
    const int per_split = p.nkr * p.nft;
    int slots = common_slots(k, kz, kThreads, p.lds);
    int splits = slots / per_split;
    // at most p.splits: at least kMinTiles tiles per split (tiny layers would
    // otherwise spend their time in block start-up and in the split reduction)
    // and within the workspace
    if (splits > p.splits) splits = p.splits;
    if (splits < 1) splits = 1;
    a.splits = splits;
    dim3 grid(splits * per_split), block(kThreads);
    hipLaunchKernelGGL(k, grid, block, p.lds, s, a);
    e = hipGetLastError();
    if (e != hipSuccess) return e;
    const int FK = a.F * a.K;
    const int total = FK + (db ? a.F : 0);
    hipLaunchKernelGGL((conv_wgrad_reduce<T>), dim3((total + 15) / 16), dim3(256), 0, s,
                       reinterpret_cast<const T *>(a.ws), reinterpret_cast<T *>(dW),
                       reinterpret_cast<T *>(db), FK, a.F, a.splits);
    return hipGetLastError();
}

// Most stride regions of a pool (PS x PS cells holding one window each) that
// one pixel tile of the plan meets: the tiled kernel's pooled-source staging
// holds kMGP of them per thread.
int max_regions(const WPlan &p, const ConvDims &d, int PS)
{
    int best = 0;
    for (int qt = 0; qt < p.tiles_per_img; ++qt) {
        int qy0, rows, ox0, ox1;
        if (p.spr) {
            const int oh = qt / p.spr, ow0 = (qt - oh * p.spr) * p.RQ;
            const int len = p.RQ < d.Wout - ow0 ? p.RQ : d.Wout - ow0;
            qy0 = oh;
            rows = 1;
            ox0 = ow0;
            ox1 = ow0 + len - 1;
        } else {
            const int Q = d.Hout * d.Wout, q0 = qt * p.RQ;
            const int qend = q0 + p.RQ < Q ? q0 + p.RQ : Q;
            qy0 = q0 / d.Wout;
            rows = (qend - 1) / d.Wout - qy0 + 1;
            ox0 = 0;
            ox1 = d.Wout - 1;
        }
        const int nw = ((qy0 + rows - 1) / PS - qy0 / PS + 1) * (ox1 / PS - ox0 / PS + 1);
        best = nw > best ? nw : best;
    }
    return best;
}

// The plan a backward_filter call takes: the row ring when the layer suits it,
// else the 4-wave split kernel.
bool choose_wplan(size_t tsz, const ConvDims &d, WPlan &p, bool &ring)
{
    WPlan r;
    ring = make_rplan(tsz, d, r);
    if (ring) {
        p = r;
        return true;
    }
    return make_wplan(tsz, d, p);
}

// Pooled source with a short filter row (K = C*Hf*Wf <= kSpK; LeNet conv1: K =
// 25).  The routed gradient g holds at most one non-zero cell per pool window:
// the window's argmax, when its pooled value is positive (every other cell of
// the conv output is zero).  So dW and db are sums over the windows rather
// than over all pixels (paper, Section 3 "Sparse Operations": an operator that
// is safe on sparse input does work in proportion to the non-zeros; here the
// zeros are known from the pool's argmax without looking at them).
//
// Block (image group, group of four filters), one wave per filter.  For each
// image of the group the block stages the zero-padded input image in LDS;
// each lane then takes windows w, w + 64, ... of its filter's plane (their
// three pool values loaded kSpB windows at a time) and for a non-zero window
// adds d * X[n, c, oy*S + i - P, ox*S + j - P] (an LDS read) to its K
// accumulators and d to the bias one.  The wave's sums are added in a fixed
// butterfly and written as split `group` of the split workspace, which the
// same fixed-order reduction as the split kernels completes.
constexpr int kSpK = 32;
constexpr int kSpFilters = 4;                 // filters (waves) per block
constexpr int kSpThreads = kSpFilters * kWave;
constexpr int kSpB = 2;                       // windows whose pool values load together
constexpr int kSpStage = 8;                   // image elements a thread loads together
constexpr size_t kSpLds = 64 * 1024;          // the padded image, at most

// Divisors of the window sum as host magic numbers (every numerator is below
// 2^16: the staged image holds at most 8192 elements).
struct SparseMagic {
    unsigned long long plane, wx, wp;
};

template <typename T>
__global__ __launch_bounds__(kSpThreads) void conv_wgrad_pool_sparse_kernel(WgradArgs a,
                                                                            int groups,
                                                                            SparseMagic mg)
{
    extern __shared__ __align__(16) unsigned char smem[];
    T *s_x = reinterpret_cast<T *>(smem);  // [C][Hin + 2P][Win + 2P], zero borders
    __shared__ int s_tap[kSpK];
    const int tid = threadIdx.x, lane = lane_id(), wave = wave_id();
    const int nfg = (a.F + kSpFilters - 1) / kSpFilters;
    const int grp = blockIdx.x / nfg, f = (blockIdx.x - grp * nfg) * kSpFilters + wave;
    const int n0 = (int)((long long)grp * a.N / groups);
    const int n1 = (int)((long long)(grp + 1) * a.N / groups);
    const int Hx = a.Hin + 2 * a.P, Wx = a.Win + 2 * a.P, plane = Hx * Wx;
    if (tid < kSpK) {  // column k = (c, i, j): its offset from the window origin
        const int k = min(tid, a.K - 1);
        const int c = k / a.HfWf, t = k - c * a.HfWf, i = t / a.Wf;
        s_tap[tid] = c * plane + i * Wx + (t - i * a.Wf);
    }
    const PoolSrc &p = a.pool;
    const T *X = reinterpret_cast<const T *>(a.X);
    const T *dpool = reinterpret_cast<const T *>(p.dpool);
    const T *pooled = reinterpret_cast<const T *>(p.pooled);
    const int nwi = p.Hp * p.Wp;  // windows of one (image, filter) plane
    const int fc = min(f, a.F - 1);  // waves past the last filter compute and drop
    T acc[kSpK + 1];
#pragma unroll
    for (int k = 0; k <= kSpK; ++k) acc[k] = T(0);
    for (int n = n0; n < n1; ++n) {
        __syncthreads();  // the previous image's readers are done
        const T *xn = X + (size_t)n * a.C * a.Hin * a.Win;
        // kSpStage loads a thread before any store, so they are in flight together
        const int tot = a.C * plane;
        for (int base = 0; base < tot; base += kSpStage * kSpThreads) {
            T v[kSpStage];
            bool in[kSpStage];
#pragma unroll
            for (int u = 0; u < kSpStage; ++u) {
                const int e = min(base + u * kSpThreads + tid, tot - 1);
                const int c = div_magic(e, mg.plane), r = e - c * plane;
                const int yp = div_magic(r, mg.wx), xp = r - yp * Wx;
                const int y = yp - a.P, x = xp - a.P;
                in[u] = y >= 0 && y < a.Hin && x >= 0 && x < a.Win;
                v[u] = xn[in[u] ? (c * a.Hin + y) * a.Win + x : 0];
            }
#pragma unroll
            for (int u = 0; u < kSpStage; ++u) {
                const int e = base + u * kSpThreads + tid;
                if (e < tot) s_x[e] = in[u] ? v[u] : T(0);
            }
        }
        __syncthreads();
        const size_t pbase = ((size_t)n * a.F + fc) * nwi;
        for (int w0 = lane; w0 < nwi; w0 += kSpB * kWave) {
            T pv[kSpB], d[kSpB];
            int am[kSpB];
#pragma unroll
            for (int b = 0; b < kSpB; ++b) {  // clamped: every load issues before any use
                const size_t o = pbase + min(w0 + b * kWave, nwi - 1);
                pv[b] = pooled[o];
                d[b] = dpool[o];
                am[b] = p.argmax[o];
            }
#pragma unroll
            for (int b = 0; b < kSpB; ++b) {
                const int w = w0 + b * kWave;
                const int qa = am[b] - fc * a.Q;  // the argmax cell in the conv output plane
                const int q = min(max(qa, 0), a.Q - 1);
                const int oy = div_magic(q, a.magic_wout), ox = q - oy * a.Wout;
                const int py = div_magic(min(w, nwi - 1), mg.wp), px = w - py * p.Wp;
                // the cell must lie in its window, as the routing defines it
                const int ry = oy - py * p.PS, rx = ox - px * p.PS;
                const bool live = w < nwi && pv[b] > T(0) && qa == q && ry >= 0 && ry < p.PH &&
                                  rx >= 0 && rx < p.PW;
                const T de = live ? d[b] : T(0);
                const T *xw = s_x + oy * a.S * Wx + ox * a.S;  // the window origin
                // all kSpK columns, no branch: columns past K repeat tap K-1
                // into accumulators that are never stored
#pragma unroll
                for (int k = 0; k < kSpK; ++k) acc[k] += de * xw[s_tap[k]];
                acc[kSpK] += de;
            }
        }
    }
    // butterfly over the wave's lanes (fixed order)
#pragma unroll
    for (int k = 0; k <= kSpK; ++k) {
        T v = acc[k];
#pragma unroll
        for (int off = kWave / 2; off > 0; off >>= 1) v += __shfl_xor(v, off, kWave);
        acc[k] = v;
    }
    if (f < a.F && lane == 0) {
        T *ws = reinterpret_cast<T *>(a.ws);
#pragma unroll
        for (int k = 0; k < kSpK; ++k)
            if (k < a.K) ws[(size_t)grp * a.F * a.K + (size_t)f * a.K + k] = acc[k];
        ws[(size_t)groups * a.F * a.K + (size_t)grp * a.F + f] = acc[kSpK];
    }
}

// Whether a pooled-source backward_filter takes the window sum: short filter
// rows and a padded input image that fits the block's LDS.
bool sparse_fits(size_t tsz, const ConvDims &d)
{
    return d.C * d.Hf * d.Wf <= kSpK &&
           tsz * d.C * (size_t)(d.Hin + 2 * d.pad) * (d.Win + 2 * d.pad) <= kSpLds;
}

size_t sparse_lds(size_t tsz, const ConvDims &d)
{
    return tsz * d.C * (size_t)(d.Hin + 2 * d.pad) * (d.Win + 2 * d.pad);
}

// Image groups of the window sum: one per image up to the workspace's split
// count (each group is a split of the reduction).
int sparse_groups(int N, int ws_splits) { return std::max(1, std::min(N, ws_splits)); }

template <typename T>
hipError_t launch_pool_sparse(WgradArgs a, int groups, size_t lds, void *dW, void *db,
                              hipStream_t s)
{
    a.splits = groups;
    auto k = conv_wgrad_pool_sparse_kernel<T>;
    hipError_t e = allow_dynamic_lds(k, lds);
    if (e != hipSuccess) return e;
    const int nfg = (a.F + kSpFilters - 1) / kSpFilters;
    const int Wx = a.Win + 2 * a.P;
    const SparseMagic mg = {host_magic((a.Hin + 2 * a.P) * Wx), host_magic(Wx),
                            host_magic(a.pool.Wp)};
    hipLaunchKernelGGL(k, dim3(nfg * groups), dim3(kSpThreads), lds, s, a, groups, mg);
    e = hipGetLastError();
    if (e != hipSuccess) return e;
    const int FK = a.F * a.K;
    const int total = FK + (db ? a.F : 0);
    hipLaunchKernelGGL((conv_wgrad_reduce<T>), dim3((total + 15) / 16), dim3(256), 0, s,
                       reinterpret_cast<const T *>(a.ws), reinterpret_cast<T *>(dW),
                       reinterpret_cast<T *>(db), FK, a.F, groups);
    return hipGetLastError();
}

}  // namespace

size_t conv_wgrad_workspace_bytes(int dtype, const ConvDims &d)
{
    const size_t tsz = dtype == 0 ? sizeof(double) : sizeof(float);
    WPlan p;
    bool ring;
    if (!choose_wplan(tsz, d, p, ring)) return 0;
    const size_t K = (size_t)d.C * d.Hf * d.Wf;
    return tsz * (size_t)p.splits * ((size_t)d.F * K + (size_t)d.F);
}

hipError_t wgrad_plan_info(int dtype, const ConvDims &d, int pool_ps, ConvPlanInfo &info)
{
    const size_t tsz = dtype == 0 ? sizeof(double) : sizeof(float);
    WPlan p;
    bool ring;
    if (!choose_wplan(tsz, d, p, ring)) return hipErrorInvalidValue;
    if (pool_ps && sparse_fits(tsz, d)) {
        const int groups = sparse_groups(d.N, p.splits);
        info.kernel = kWgradPoolSparse;
        info.tile_m = kSpFilters;
        info.blocks = (d.F + kSpFilters - 1) / kSpFilters * groups;
        info.chunk = d.C * d.Hf * d.Wf;
        info.k_split = 1;
        info.splits = groups;
        info.window_width = d.Win + 2 * d.pad;
        info.window_rows = d.Hin + 2 * d.pad;
        info.lds = sparse_lds(tsz, d);
        info.tile_stride = kSpB * kWave;
        info.fused = 1;
        return hipSuccess;
    }
    info.kernel = ring ? kWgradRing : kWgradTiles;
    info.tile_m = kBM;
    info.tile_pixels = p.RQ;
    info.blocks = p.nkr * p.nft;
    info.chunk = p.KR;
    info.k_split = 1;
    info.splits = p.splits;
    info.window_width = p.Wpad;
    info.window_rows = p.rows_max;
    info.lds = p.lds;
    info.g_stride = p.SG;
    info.row_slices = p.spr;
    info.tile_stride = p.RQ;
    info.pipelined = p.pipelined;
    if (pool_ps && !ring && kBM * max_regions(p, d, pool_ps) > kThreads * kMGP) info.pipelined = 0;
    info.fused = pool_ps ? 1 : 0;
    info.row_staged = 0;
    if (ring) {
        if (p.xdma)
            info.row_staged |= 4;
        else if (p.rowmap && !pool_ps)
            info.row_staged |= 1;
        if ((p.xdma || p.rowmap) && !pool_ps && tsz == 4) info.row_staged |= 2;
    }
    return hipSuccess;
}

hipError_t launch_conv_backward_filter(int dtype, const void *X, const void *dout,
                                       const void *out_fwd, void *dW, void *db,
                                       const ConvDims &d, void *ws, int zero_skip,
                                       hipStream_t s, const PoolSrc *pool, void *g_out)
{
    const size_t tsz = dtype == 0 ? sizeof(double) : sizeof(float);
    WPlan p;
    bool ring;
    if (!choose_wplan(tsz, d, p, ring)) return hipErrorInvalidValue;
    WgradArgs a = {};
    a.X = X;
    a.dout = dout;
    a.mask = out_fwd;
    a.ws = ws;
    a.N = d.N;
    a.C = d.C;
    a.Hin = d.Hin;
    a.Win = d.Win;
    a.F = d.F;
    a.Hf = d.Hf;
    a.Wf = d.Wf;
    a.HfWf = d.Hf * d.Wf;
    a.S = d.stride;
    a.P = d.pad;
    a.Hout = d.Hout;
    a.Wout = d.Wout;
    a.Q = d.Hout * d.Wout;
    a.K = d.C * d.Hf * d.Wf;
    a.KR = p.KR;
    a.nkr = p.nkr;
    a.nft = p.nft;
    a.RQ = p.RQ;
    a.tiles_per_img = p.tiles_per_img;
    a.T_total = (int)p.T_total;
    a.splits = p.splits;
    a.Wpad = p.Wpad;
    a.CH = p.CH;
    a.SG = p.SG;
    a.rows_max = p.rows_max;
    a.x_dma_insts = p.x_dma_insts;
    a.pipelined = p.pipelined;
    a.spr = p.spr;
    a.magic_rq = host_magic(p.RQ);
    a.magic_wpad = host_magic(p.Wpad);
    a.magic_wout = host_magic(d.Wout);
    a.magic_hwf = host_magic(a.HfWf);
    a.magic_wf = host_magic(d.Wf);
    a.g_out = pool ? nullptr : g_out;
    if (pool) {
        // the pooled source has no zero-skip form (its routed gradient has no
        // all-zero fragments: one cell per window holds a value)
        a.pool = *pool;
        a.mask = nullptr;
        if (sparse_fits(tsz, d)) {  // short filter rows: the sum over the pool windows
            const int groups = sparse_groups(d.N, p.splits);
            const size_t lds = sparse_lds(tsz, d);
            return dtype == 0 ? launch_pool_sparse<double>(a, groups, lds, dW, db, s)
                              : launch_pool_sparse<float>(a, groups, lds, dW, db, s);
        }
        // the tiled kernel's register staging holds kMGP windows a thread; more
        // take the direct staging path (one cell at a time)
        if (!ring && kBM * max_regions(p, d, pool->PS) > kThreads * kMGP) a.pipelined = 0;
        a.magic_ch = ring ? host_magic((d.stride < d.Hf ? d.stride : d.Hf) * p.Wpad)
                          : host_magic(p.CH);
        if (ring)
            return dtype == 0 ? launch_ring<double, false, true>(a, p, dW, db, s)
                              : launch_ring<float, false, true>(a, p, dW, db, s);
        return dtype == 0 ? launch_w<double, false, true>(a, p, dW, db, s)
                          : launch_w<float, false, true>(a, p, dW, db, s);
    }
    if (ring) {
        // the ring's new-row staging divides by the new rows' span per channel
        a.magic_ch = host_magic((d.stride < d.Hf ? d.stride : d.Hf) * p.Wpad);
        if (dtype == 0)
            return zero_skip ? launch_ring<double, true, false>(a, p, dW, db, s)
                             : launch_ring<double, false, false>(a, p, dW, db, s);
        return zero_skip ? launch_ring<float, true, false>(a, p, dW, db, s)
                         : launch_ring<float, false, false>(a, p, dW, db, s);
    }
    a.magic_ch = host_magic(p.CH);
    if (dtype == 0)
        return zero_skip ? launch_w<double, true, false>(a, p, dW, db, s)
                         : launch_w<double, false, false>(a, p, dW, db, s);
    return zero_skip ? launch_w<float, true, false>(a, p, dW, db, s)
                     : launch_w<float, false, false>(a, p, dW, db, s);
}

}  // namespace dmlnn
