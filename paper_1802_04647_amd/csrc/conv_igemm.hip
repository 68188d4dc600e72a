// conv2d forward (+ fused bias_add and relu) and conv2d backward_data (+ fused
// relu mask) as one implicit-im2col GEMM on the gfx950 matrix cores.
//
// Both passes compute, per image n,
//   out[n, m, qy, qx] = sum_{c, i, j} A(m, c, i, j) * src_v(n, c, qy*S + i - P, qx*S + j - P)
// i.e. a GEMM  out_n[M x Q] = A[M x K] * B_n[K x Q]  with K = Cs*Hf*Wf and the
// patch matrix B_n never materialised:
//   forward:   A = W (M = F filters), src = X, (S, P) = (stride, pad).
//   backward:  A(m=c, f, i, j) = W[f, c, Hf-1-i, Wf-1-j] (flipped and transposed),
//              src = relu-masked dout, virtually up-sampled by the stride (a
//              gradient value sits at every stride-th position, zeros between),
//              (S, P) = (1, Hf-1-pad) for rows and (1, Wf-1-pad) for columns,
//              output Hin x Win.
// This is the lowering of the paper's Section 3 ("Sparse Operations") done
// implicitly: the patch tile is built in LDS from the row-major N x (C*H*W)
// matrix and consumed straight from there.
//
// Tiling: a block (4 waves) owns 64 output rows (m) by 32*NB output pixels of
// one image.  Waves are arranged 2 (m) x 2 (pixels); each wave issues
// 2 x NB independent 16x16x4 MFMAs per k-step.  K is walked in chunks of KC
// source channels; per chunk the block stages (a) the KC x rows x Wpad window of
// source rows its pixels touch, zero-padded, and (b) the 64 x KC*Hf*Wf slice of
// A, both in LDS.  A per-chunk table maps k -> LDS offset of tap (c,i,j); each
// lane adds the offset of its own pixel.
#include <algorithm>
#include <type_traits>

#include "common.hpp"
#include "internal.hpp"

namespace dmlnn {
namespace {

constexpr int kThreads = 256;
constexpr int kMaxBanks = 8;  // filter banks one horizontally fused launch may carry
constexpr int kBM = 64;
constexpr size_t kLdsBudget = 72 * 1024;  // two blocks per CU
constexpr int kMS = 8;    // source-row slots each wave stages per chunk
constexpr int kMA = 13;   // filter elements each thread stages per chunk

struct IgemmArgs {
    const void *src;   // [N][Cs][Sh][Sw]
    const void *mask;  // same shape as src (backward only) or null
    const void *wgt;   // W [F][C][Hf][Wf]
    const void *bias;  // [M] or null (forward only)
    void *out;         // [N][M][Q]
    int M, Cs, Sh, Sw, up;
    int Qw, Q;
    int Hf, Wf, HfWf;
    int S, Ph, Pw;
    int relu;
    int tiles_per_img;
    int TS;         // pixels between consecutive tile origins (<= 32 NB; less when a
                    // fused pool needs tiles of whole row groups)
    int KC, KCK;
    int Wpad, CH, SA;
    int pipelined;  // 1: chunk fits the per-thread staging registers
    int ksplit;     // LDS-DMA kernel, M <= 32: the two m-halves of waves split the
                    // k-steps of the same 32 rows instead of taking 32 rows each
    // Fused max-pool epilogue (forward, LDS-DMA kernel): PH x PW windows at
    // stride PS, no padding, giving Hp x Wp per filter; pooled [N][M][Hp*Wp]
    // and the in-row argmax of each window within the conv output row.
    void *pool_out;
    int32_t *pool_idx;
    int PH, PW, PS, Hp, Wp;
    // Horizontal fusion (forward): rows [bank_off[b], bank_off[b+1]) of M belong
    // to filter bank b, whose output is bank_out[b] ([N][F_b][Q]).  nbanks <= 1:
    // a single output at out.
    int nbanks;
    int bank_off[kMaxBanks + 1];
    void *bank_out[kMaxBanks];
    int require_dma;  // 1: return hipErrorNotSupported instead of using the register path
    int k4;           // LDS-DMA kernel with NB = 1: 0, or the row blocks (2 or 4) of the
                      // four-way k split
    // Sparse input (forward, register-staged kernel): X given in CSR; csr_row
    // holds, for every image row (n, c, y), the position of its first non-zero
    // (N*Cs*Sh + 1 entries, the last = nnz), csr_col / csr_val the CSR columns
    // (c*Sh*Sw + y*Sw + x) and values.
    int csr;  // 1: the input is the CSR arrays below (csr_col / csr_val may be
              // null when there are no non-zeros)
    const int32_t *csr_row;
    const int32_t *csr_col;
    const void *csr_val;
    unsigned long long magic_kck, magic_hw, magic_wf;
    unsigned long long magic_wpad, magic_sa, magic_qw;  // LDS-DMA kernel set-up
    // Pooled source (backward, the PB instantiations): the conv was followed by
    // relu and a non-overlapping max-pool, and the masked dout is built while
    // staging from that pool's gradient, argmax and pooled values (src and
    // mask are unused).
    int pb;
    PoolSrc pool;
};

template <typename T, int NB, bool BWD, bool ZSKIP, bool CSR = false, bool PB = false>
__global__ __launch_bounds__(kThreads, 2) void conv_igemm_kernel(IgemmArgs a)
{
    using MF = Mfma<T>;
    extern __shared__ __align__(16) unsigned char smem[];
    T *s_src = reinterpret_cast<T *>(smem);
    T *s_a = s_src + a.KC * a.CH;
    int *s_koff = reinterpret_cast<int *>(s_a + kBM * a.SA);

    const int tid = threadIdx.x, lane = lane_id(), wave = wave_id();
    const int wm = wave & 1, wn = wave >> 1;
    const int n = blockIdx.x / a.tiles_per_img;
    const int tile = blockIdx.x - n * a.tiles_per_img;
    const int m0 = blockIdx.y * kBM;
    const int q0 = tile * a.TS;
    const int qend = min(q0 + a.TS, a.Q);
    const int qy0 = q0 / a.Qw;
    const int rows_need = ((qend - 1) / a.Qw - qy0) * a.S + a.Hf;
    const int ybase = qy0 * a.S - a.Ph;
    const int CHn = rows_need * a.Wpad;  // channel stride of this tile's staged window
    const int KCv = a.KC * a.HfWf;       // real (unpadded) k per chunk

    for (int kk = tid; kk < a.KCK; kk += kThreads) {
        int off = 0;
        if (kk < KCv) {
            int c = kk / a.HfWf, t = kk - c * a.HfWf;
            int i = t / a.Wf, j = t - i * a.Wf;
            off = c * CHn + i * a.Wpad + j;
        }
        s_koff[kk] = off;
    }

    int lbase[NB];
#pragma unroll
    for (int y = 0; y < NB; ++y) {
        int q = q0 + (wn * NB + y) * 16 + (lane & 15);
        int qy = q / a.Qw, qx = q - qy * a.Qw;
        lbase[y] = (q < qend) ? (qy - qy0) * a.S * a.Wpad + qx * a.S : 0;
    }

    typename MF::acc_t acc[2][NB];
#pragma unroll
    for (int x = 0; x < 2; ++x)
#pragma unroll
        for (int y = 0; y < NB; ++y) acc[x][y] = MF::zero();

    const size_t img = (size_t)n * a.Cs * a.Sh * a.Sw;
    const T *src = PB ? nullptr : reinterpret_cast<const T *>(a.src) + img;
    const T *msk = (BWD && !PB && a.mask) ? reinterpret_cast<const T *>(a.mask) + img : nullptr;
    const T *wgt = reinterpret_cast<const T *>(a.wgt);

    // Staging is software-pipelined: the global loads of chunk c0+KC are issued
    // into registers before the MFMA loop of chunk c0 and written to LDS after
    // it.  Source rows: wave w owns row slots w, w+4, ... of the chunk's
    // KC*rows_need staged rows (times 64-wide column groups).  Filter slice:
    // thread t owns elements t, t+256, ... of the 64 x KCK slice.
    const int nrows = a.KC * rows_need;
    const int ncg = (a.Wpad + kWave - 1) / kWave;
    const int tot_a = kBM * a.KCK;
    T vs[kMS], vm[kMS], va[kMA];

    auto load = [&](int c0) {
        const int tid = opaque(threadIdx.x);
#pragma unroll
        for (int it = 0; it < kMS; ++it) {
            const int slot = wave + 4 * it;
            const int r = slot / ncg, cgi = slot - r * ncg;
            T v = T(0), mv = T(1);
            if (PB) {
                // branch-free: a clamped cell, dropped when outside the window
                // (r is wave-uniform, so the row terms are too)
                const int c = r / rows_need, t = r - c * rows_need;
                const int cg = c0 + c, yv = ybase + t;
                const int ys = max(yv, 0) / a.up;
                const int u = lane + kWave * cgi;
                const int xv = u - a.Pw;
                const int xs = max(xv, 0) / a.up;
                const bool ok = r < nrows && cg < a.Cs && yv >= 0 && ys * a.up == yv &&
                                ys < a.Sh && u < a.Wpad && xv >= 0 && xs * a.up == xv && xs < a.Sw;
                const T pg = pool_src_grad<T>(a.pool, n, a.Cs, min(cg, a.Cs - 1), a.Sh * a.Sw,
                                              a.Sw, min(ys, a.Sh - 1), min(xs, a.Sw - 1));
                v = ok ? pg : T(0);
            } else if (r < nrows) {
                const int c = r / rows_need, t = r - c * rows_need;
                const int cg = c0 + c, yv = ybase + t;
                const int ys = yv / a.up;
                const int u = lane + kWave * cgi;
                const int xv = u - a.Pw;
                const int xs = xv / a.up;
                if (cg < a.Cs && yv >= 0 && ys * a.up == yv && ys < a.Sh && u < a.Wpad &&
                    xv >= 0 && xs * a.up == xv && xs < a.Sw) {
                    const size_t o = ((size_t)cg * a.Sh + ys) * a.Sw + xs;
                    v = src[o];
                    if (BWD && msk) mv = msk[o];
                }
            }
            vs[it] = v;
            vm[it] = mv;
        }
#pragma unroll
        for (int it = 0; it < kMA; ++it) {
            const int e = tid + kThreads * it;
            T v = T(0);
            if (e < tot_a) {
                const int m = div_magic(e, a.magic_kck);
                const int kk = e - m * a.KCK;
                const int c = div_magic(kk, a.magic_hw);
                const int t = kk - c * a.HfWf;
                const int mg = m0 + m;
                if (mg < a.M && kk < KCv && c0 + c < a.Cs) {
                    if (!BWD)
                        v = wgt[((size_t)mg * a.Cs + c0) * a.HfWf + kk];
                    else
                        v = wgt[((size_t)(c0 + c) * a.M + mg) * a.HfWf + (a.HfWf - 1 - t)];
                }
            }
            va[it] = v;
        }
    };

    auto store = [&]() {
        const int tid = opaque(threadIdx.x);
#pragma unroll
        for (int it = 0; it < kMS; ++it) {
            const int slot = wave + 4 * it;
            const int r = slot / ncg, cgi = slot - r * ncg;
            const int u = lane + kWave * cgi;
            if (r < nrows && u < a.Wpad) {
                T v = vs[it];
                if (BWD && !(vm[it] > T(0))) v = T(0);
                s_src[r * a.Wpad + u] = v;  // row r = (channel, staged row), dense
            }
        }
#pragma unroll
        for (int it = 0; it < kMA; ++it) {
            const int e = tid + kThreads * it;
            if (e < tot_a) s_a[e + div_magic(e, a.magic_kck)] = va[it];  // row stride KCK + 1
        }
    };

    // Fallback for chunks larger than the staging registers: load and store
    // directly (one memory round trip per row slot; correct for any size).
    auto stage_direct = [&](int c0) {
        if (CSR) {
            // Each wave zeroes its window rows, then scatters the row's non-zeros
            // (LDS writes of one wave land in issue order).  A staged row holds
            // window columns [0, Wpad), i.e. input columns [-Pw, Wpad - Pw): with a
            // stride above 1 the last input columns can lie past the last window
            // (they feed no output) and are skipped, as are columns outside the
            // image row, so no input, well-formed or not, writes outside the row.
            const T *val = reinterpret_cast<const T *>(a.csr_val);
            for (int r = wave; r < nrows; r += kThreads / kWave) {
                const int c = r / rows_need, t = r - c * rows_need;
                const int cg = c0 + c, yv = ybase + t;
                T *dst = s_src + r * a.Wpad;
                for (int u = lane; u < a.Wpad; u += kWave) dst[u] = T(0);
                if (cg < a.Cs && yv >= 0 && yv < a.Sh) {
                    const size_t ri = ((size_t)n * a.Cs + cg) * a.Sh + yv;
                    const int kb = a.csr_row[ri], ke = a.csr_row[ri + 1];
                    const int base = (cg * a.Sh + yv) * a.Sw;
                    const int xlim = min(a.Sw, a.Wpad - a.Pw);
                    for (int k = kb + lane; k < ke; k += kWave) {
                        const int x = a.csr_col[k] - base;
                        if (x >= 0 && x < xlim) dst[x + a.Pw] = val[k];
                    }
                }
            }
        }
        for (int r = wave; !CSR && r < nrows; r += kThreads / kWave) {
            const int c = r / rows_need, t = r - c * rows_need;
            const int cg = c0 + c, yv = ybase + t;
            const int ys = yv / a.up;
            const bool rowok = cg < a.Cs && yv >= 0 && ys * a.up == yv && ys < a.Sh;
            const size_t roff = ((size_t)cg * a.Sh + (rowok ? ys : 0)) * a.Sw;
            for (int u = lane; u < a.Wpad; u += kWave) {
                T v = T(0);
                const int xv = u - a.Pw;
                const int xs = xv / a.up;
                if (rowok && xv >= 0 && xs * a.up == xv && xs < a.Sw) {
                    if (PB) {
                        v = pool_src_grad<T>(a.pool, n, a.Cs, cg, a.Sh * a.Sw, a.Sw, ys, xs);
                    } else {
                        v = src[roff + xs];
                        if (BWD && msk && !(msk[roff + xs] > T(0))) v = T(0);
                    }
                }
                s_src[r * a.Wpad + u] = v;
            }
        }
        for (int e = tid; e < tot_a; e += kThreads) {
            const int m = e / a.KCK, kk = e - m * a.KCK;
            const int c = kk / a.HfWf, t = kk - c * a.HfWf;
            const int mg = m0 + m;
            T v = T(0);
            if (mg < a.M && kk < KCv && c0 + c < a.Cs) {
                if (!BWD)
                    v = wgt[((size_t)mg * a.Cs + c0) * a.HfWf + kk];
                else
                    v = wgt[((size_t)(c0 + c) * a.M + mg) * a.HfWf + (a.HfWf - 1 - t)];
            }
            s_a[m * a.SA + kk] = v;
        }
    };

    if (a.pipelined) load(0);
    for (int c0 = 0; c0 < a.Cs; c0 += a.KC) {
        __syncthreads();
        if (a.pipelined)
            store();
        else
            stage_direct(c0);
        __syncthreads();
        if (a.pipelined && c0 + a.KC < a.Cs) load(c0 + a.KC);

        const T *arow0 = s_a + (wm * 32 + (lane & 15)) * a.SA + (lane >> 4);
        const T *arow1 = arow0 + 16 * a.SA;
        const int *kof = s_koff + (lane >> 4);
        for (int kk = 0; kk < a.KCK; kk += 4) {
            T av0 = arow0[kk], av1 = arow1[kk];
            int ko = kof[kk];
#pragma unroll
            for (int y = 0; y < NB; ++y) {
                T bv = s_src[ko + lbase[y]];
                if (ZSKIP && wave_all_zero(bv)) continue;
                acc[0][y] = MF::mma(av0, bv, acc[0][y]);
                acc[1][y] = MF::mma(av1, bv, acc[1][y]);
            }
        }
    }

    T *out = reinterpret_cast<T *>(a.out) + (size_t)n * a.M * a.Q;
    const T *bias = reinterpret_cast<const T *>(a.bias);
#pragma unroll
    for (int x = 0; x < 2; ++x)
#pragma unroll
        for (int y = 0; y < NB; ++y)
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                int m = m0 + wm * 32 + x * 16 + MF::row(lane, r);
                int q = q0 + (wn * NB + y) * 16 + (lane & 15);
                if (m < a.M && q < qend) {
                    T v = acc[x][y][r];
                    if (!BWD) {
                        if (bias) v += bias[m];
                        v = relu_if(v, a.relu);
                    }
                    out[(size_t)m * a.Q + q] = v;
                }
            }
}

// ---------------------------------------------------------------------------
// LDS-DMA variant (the default path).  Same tiling and MFMA loop as above, but
// each chunk's source window and filter slice are copied global -> LDS by the
// buffer unit (buffer_load ... lds), double-buffered: the copies of chunk c+1
// are issued right before the MFMA loop of chunk c, with no register staging
// and no LDS store phase.  Zero padding, image borders, the k padding and a
// ragged last channel chunk all come from the buffer range check: lanes whose
// element lies outside the image (or beyond the tensor) get an out-of-range
// offset and write 0.  Each lane's byte offset within a chunk is the same for
// every chunk and stays in a register; the chunk's channel offset is the scalar
// soffset.  In the backward pass the relu mask source is copied into one LDS
// window and folded into the chunk's source window before its MFMAs.
// The fp64 forward pass moves the filter slice 16 bytes per lane when a chunk
// holds an even number of taps: a slice row is a contiguous run of the filter
// row, each lane's element pair lies inside it, and the four-times-larger
// instructions let a chunk take more channels (LeNet conv2: 2 instead of 1).
// The backward pass reads the filter flipped and channel-major, so its pairs
// are not contiguous and it keeps the 4-byte form.
constexpr int kMaxDmaS = 12;  // source-window DMA instructions per wave per chunk
// Filter-slice DMA instructions per wave per chunk.  (Twice as many offset
// registers for the one- and two-column-block tiles, which would allow larger
// chunks, measured slower on the LeNet layers: the longer unrolled set-up and
// issue code cost more than the saved barriers.)
constexpr int dma_a_max(int) { return 20; }
// Rows of the staged filter slice: layers with M <= 32 take the k-split (or
// four-way) forms, whose waves only read rows 0..31.
__host__ __device__ constexpr int dma_a_rows(int M) { return M <= 32 ? 32 : kBM; }
constexpr size_t kLdsPerBlock = 80 * 1024;  // two blocks per CU (160 KiB)
constexpr size_t kLdsPerBlock32 = 53 * 1024;  // three blocks per CU (fp32)

struct DmaLayout {
    int src_bytes, a_bytes, stage_bytes;  // per-stage regions, 256-byte multiples; a_bytes
                                          // has 256 bytes of slack
    int a_vec;  // 1: the filter slice moves 16 bytes per lane (fp64 forward, chunks of
                // an even number of taps: every pair of elements is contiguous in the
                // filter, and no pair mixes a tap with a zero column)
};

template <typename T, int NB, bool BWD, bool ZSKIP, bool KS, bool POOL, int K4 = 0,
          bool PB = false>
__global__ __launch_bounds__(kThreads, 2) __attribute__((amdgpu_waves_per_eu(2, sizeof(T) == 4 ? 3 : 2))) void conv_igemm_dma_kernel(IgemmArgs a, DmaLayout L,
                                                                     unsigned w_bytes)
{
    using MF = Mfma<T>;
    constexpr int dpe = sizeof(T) / 4;  // dwords per element
    extern __shared__ __align__(16) unsigned char smem[];
    unsigned char *stages = smem;

    const int tid = threadIdx.x, lane = lane_id(), wave = wave_id();
    const int wm = wave & 1, wn = wave >> 1;
    // Consecutive tiles of an image share the halo rows of their source
    // windows: the blocks are renumbered so that runs of consecutive tiles go
    // to one XCD, whose L2 then serves the second read of each halo row (dealt
    // round-robin, neighbours sat on different XCDs and fetched the halo from
    // HBM again: backward_data read 1.29 GB of HBM for 0.82 GB of operands).
    const int Lb = xcd_logical_block(blockIdx.x + gridDim.x * blockIdx.y, gridDim.x * gridDim.y);
    const int bx = Lb % gridDim.x, by = Lb / gridDim.x;
    const int n = bx / a.tiles_per_img;
    const int tile = bx - n * a.tiles_per_img;
    const int m0 = by * kBM;
    const int q0 = tile * a.TS;
    const int qend = min(q0 + a.TS, a.Q);
    const int qy0 = q0 / a.Qw;
    const int rows_need = ((qend - 1) / a.Qw - qy0) * a.S + a.Hf;
    const int ybase = qy0 * a.S - a.Ph;
    const int CHn = rows_need * a.Wpad;
    const int KCv = a.KC * a.HfWf;

    // Set-up index math avoids runtime integer division (a long VALU sequence
    // each; the offsets below take dozens): the divisors are launch constants
    // with host magic numbers, or the block's row count through a float
    // reciprocal.  A pixel u < 32 NB past the tile's first column splits as
    // (qx0 + u) / Qw with both operands below 2^16 (the plan bounds Qw).
    const int qx0 = q0 - qy0 * a.Qw;
    auto pix_off = [&](int u) {
        const int v = qx0 + u, dy = div_magic(v, a.magic_qw);
        return dy * a.S * a.Wpad + (v - dy * a.Qw) * a.S;
    };
    int lbase[NB];
#pragma unroll
    for (int y = 0; y < NB; ++y) {
        const int u = (wn * NB + y) * 16 + (lane & 15);
        lbase[y] = (q0 + u < qend) ? pix_off(u) : 0;
    }

    typename MF::acc_t acc[2][NB];
#pragma unroll
    for (int x = 0; x < 2; ++x)
#pragma unroll
        for (int y = 0; y < NB; ++y) acc[x][y] = MF::zero();
    // K4 (NB = 1 tiles of small layers): every wave covers the whole 16*K4 x 32
    // tile and the four waves split the k-steps (wave w takes steps 4w, 4w+16,
    // ...); the partial tiles are added in wave order after the last chunk.
    constexpr int R4 = K4 ? K4 : 1;
    typename MF::acc_t acc4[R4][2];
    int lb4[2];
    if (K4) {
#pragma unroll
        for (int x = 0; x < R4; ++x)
#pragma unroll
            for (int y = 0; y < 2; ++y) acc4[x][y] = MF::zero();
#pragma unroll
        for (int y = 0; y < 2; ++y) {
            const int u = y * 16 + (lane & 15);
            lb4[y] = (q0 + u < qend) ? pix_off(u) : 0;
        }
    }

    const size_t img = (size_t)a.Cs * a.Sh * a.Sw;
    const unsigned img_bytes = (unsigned)(img * sizeof(T));
    const bool has_mask = BWD && !PB && a.mask != nullptr;
    const i32x4 rs_src = buffer_rsrc(reinterpret_cast<const T *>(a.src) + (size_t)n * img, img_bytes);
    const i32x4 rs_msk = has_mask ? buffer_rsrc(reinterpret_cast<const T *>(a.mask) + (size_t)n * img,
                                                img_bytes)
                                  : rs_src;
    const i32x4 rs_w = buffer_rsrc(a.wgt, w_bytes);

    // Per-lane byte offsets inside a chunk (channel c0 excluded), or kDmaZero.
    const int Ds = a.KC * CHn * dpe;
    const int NIs = (Ds + kWave - 1) / kWave;
    constexpr int kMaxDmaA = dma_a_max(NB);
    const bool avec = sizeof(T) == 8 && !BWD && L.a_vec;
    // filter-slice DMA units (dwords, or pairs of elements) and instructions
    const int Da = avec ? dma_a_rows(a.M) * a.SA / 2 : dma_a_rows(a.M) * a.SA * dpe;
    const int NIa = (Da + kWave - 1) / kWave;
    int vs_off[kMaxDmaS], va_off[kMaxDmaA];
    // Window element e (< 12 * 4 * 64) -> (row r, column x) by the magic of
    // Wpad, r -> (channel c, row t) through the reciprocal of rows_need.
    const float rcp_rows = 1.0f / (float)rows_need;
#pragma unroll
    for (int j = 0; j < kMaxDmaS; ++j) {
        const int ii = wave + 4 * j, d = ii * kWave + lane;
        int off = kDmaZero;
        if (ii < NIs && d < Ds) {
            const int e = d / dpe, h = d - e * dpe;
            const int r = div_magic(e, a.magic_wpad), x = e - r * a.Wpad;
            const int c = div_small(r, rows_need, rcp_rows), t = r - c * rows_need;
            const int yv = ybase + t, xv = x - a.Pw;
            bool in = yv >= 0 && xv >= 0;
            int ys = yv, xs = xv;
            if (a.up != 1) {  // backward_data of a strided layer: up-sampled source
                ys = max(yv, 0) / a.up;
                xs = max(xv, 0) / a.up;
                in = in && ys * a.up == yv && xs * a.up == xv;
            }
            if (in && ys < a.Sh && xs < a.Sw)
                off = (int)((((size_t)c * a.Sh + ys) * a.Sw + xs) * sizeof(T)) + 4 * h;
        }
        vs_off[j] = off;
    }
#pragma unroll
    for (int j = 0; j < kMaxDmaA; ++j) {
        const int ii = wave + 4 * j, d = ii * kWave + lane;
        int off = kDmaZero;
        if (ii < NIa && d < Da) {
            const int e = avec ? 2 * d : d / dpe, h = avec ? 0 : d - e * dpe;
            const int m = div_magic(e, a.magic_sa), kk = e - m * a.SA;
            const int mg = m0 + m;
            if (mg < a.M && kk < KCv) {
                size_t el;
                if (!BWD) {
                    el = (size_t)mg * a.Cs * a.HfWf + kk;
                } else {
                    const int c = div_magic(kk, a.magic_hw), t = kk - c * a.HfWf;
                    el = ((size_t)c * a.M + mg) * a.HfWf + (a.HfWf - 1 - t);
                }
                off = (int)(el * sizeof(T)) + 4 * h;
            }
        }
        va_off[j] = off;
    }

    // LDS: two stages of [source window][A slice], then one mask window (the
    // backward pass's relu mask lands there and is folded into the source
    // window of its stage before that stage's MFMAs read it).
    auto stage_src = [&](int st) { return reinterpret_cast<T *>(stages + st * L.stage_bytes); };
    auto stage_a = [&](int st) {
        return reinterpret_cast<T *>(stages + st * L.stage_bytes + L.src_bytes);
    };
    T *const s_msk = reinterpret_cast<T *>(stages + 2 * L.stage_bytes);
    auto issue = [&](int st, int c0) {
        unsigned char *ps = reinterpret_cast<unsigned char *>(stage_src(st));
        unsigned char *pm = reinterpret_cast<unsigned char *>(s_msk);
        unsigned char *pa = reinterpret_cast<unsigned char *>(stage_a(st));
        const int so_src = (int)((size_t)c0 * a.Sh * a.Sw * sizeof(T));
        const int so_w = (int)((size_t)c0 * (BWD ? a.M : 1) * a.HfWf * sizeof(T));
#pragma unroll
        for (int j = 0; j < kMaxDmaS; ++j) {
            const int ii = wave + 4 * j;
            if (!PB && ii < NIs) {
                dma_dword(rs_src, ps + ii * 256, vs_off[j], so_src);
                if (has_mask) dma_dword(rs_msk, pm + ii * 256, vs_off[j], so_src);
            }
        }
        if (avec) {
#pragma unroll
            for (int j = 0; j < kMaxDmaA; ++j) {
                const int ii = wave + 4 * j;
                if (ii < NIa) dma_x4(rs_w, pa + ii * 1024, va_off[j], so_w);
            }
        } else {
#pragma unroll
            for (int j = 0; j < kMaxDmaA; ++j) {
                const int ii = wave + 4 * j;
                if (ii < NIa) dma_dword(rs_w, pa + ii * 256, va_off[j], so_w);
            }
        }
    };

    // PB: the gradient window of a chunk is written from registers by window
    // owners.  Element e of a chunk is (channel c, stride region (py, px)) of
    // the pool: the PS x PS cells whose window is (py, px).  Its owner loads
    // the window's gradient, argmax and pooled value once and writes the
    // region's cells that lie in the staged window: the gradient at the argmax
    // when the pooled value is positive, zeros elsewhere.  The loads of chunk
    // c+1 are issued before the MFMAs of chunk c and written to the other stage
    // after them.  Window cells outside the gradient plane (padding, the
    // up-sampling gaps) are zeroed once and never written again.
    constexpr int kRP = 4;  // regions a thread owns per chunk (the plan keeps KC to that)
    constexpr int NRP = PB ? kRP : 1;
    T rd[NRP], rpv[NRP];
    int ra[NRP];
    int ys_lo = 0, ys_hi = -1, py_lo = 0, npx = 1, nw = 0;
    if (PB) {
        // gradient rows the window holds: ys*up - ybase in [0, rows_need)
        const int last = ybase + rows_need - 1;
        ys_lo = (max(ybase, 0) + a.up - 1) / a.up;
        ys_hi = last < 0 ? -1 : min(last / a.up, a.Sh - 1);
        if (ys_hi >= ys_lo) {
            py_lo = div_magic(ys_lo, a.pool.magic_ps);
            npx = div_magic(a.Sw + a.pool.PS - 1, a.pool.magic_ps);
            nw = (div_magic(ys_hi, a.pool.magic_ps) - py_lo + 1) * npx;
        }
    }
    const int nreg = a.KC * nw;
    const int nreg_it = (nreg + kThreads - 1) / kThreads;  // iterations with owners (block-uniform)
    const float rcp_nw = 1.0f / (float)max(nw, 1), rcp_npx = 1.0f / (float)npx;
    auto region = [&](int e, int &c, int &py, int &px) {
        c = div_small(e, max(nw, 1), rcp_nw);
        const int w = e - c * nw;
        const int wy = div_small(w, npx, rcp_npx);
        py = py_lo + wy;
        px = w - wy * npx;
    };
    auto rload = [&](int cn) {
#pragma unroll
        for (int i = 0; i < NRP; ++i) {
            if (i >= nreg_it) break;
            int c, py, px;
            region(tid + kThreads * i, c, py, px);
            const size_t o = (((size_t)n * a.Cs + min(cn + c, a.Cs - 1)) * a.pool.Hp +
                              min(py, a.pool.Hp - 1)) * a.pool.Wp + min(px, a.pool.Wp - 1);
            rd[i] = reinterpret_cast<const T *>(a.pool.dpool)[o];
            ra[i] = a.pool.argmax[o];
            rpv[i] = reinterpret_cast<const T *>(a.pool.pooled)[o];
        }
    };
    auto rstore = [&](int cn, T *win) {
        const int Qs = a.Sh * a.Sw;
#pragma unroll
        for (int i = 0; i < NRP; ++i) {
            if (i >= nreg_it) break;
            const int e = tid + kThreads * i;
            int c, py, px;
            region(e, c, py, px);
            if (e >= nreg) continue;
            const int cg = cn + c;
            const bool ok = cg < a.Cs && py < a.pool.Hp && px < a.pool.Wp && rpv[i] > T(0);
            const int tgt = ok ? ra[i] - cg * Qs : -1;
            T *wc = win + c * CHn;
            for (int dy = 0; dy < a.pool.PS; ++dy) {
                const int ys = py * a.pool.PS + dy;
                if (ys < ys_lo || ys > ys_hi) continue;
                const int t = ys * a.up - ybase;
                for (int dx = 0; dx < a.pool.PS; ++dx) {
                    const int xs = px * a.pool.PS + dx, x = xs * a.up + a.Pw;
                    if (xs < a.Sw && x < a.Wpad) wc[t * a.Wpad + x] = ys * a.Sw + xs == tgt ? rd[i] : T(0);
                }
            }
        }
    };
    if (PB) {
        for (int e = tid; e < a.KC * CHn; e += kThreads) {
            stage_src(0)[e] = T(0);
            stage_src(1)[e] = T(0);
        }
        __syncthreads();
        rload(0);
    }
    issue(0, 0);
    if (PB) rstore(0, stage_src(0));
    wait_dma();
    __syncthreads();
    int st = 0;
    for (int c0 = 0; c0 < a.Cs; c0 += a.KC) {
        if (has_mask) {
            // dout * (out_fwd > 0) in place; the mask window is free again after
            // the barrier, so the next chunk's mask may land in it.
            T *w = stage_src(st);
            const int nel = a.KC * CHn;
            for (int e = tid; e < nel; e += kThreads)
                if (!(s_msk[e] > T(0))) w[e] = T(0);
            __syncthreads();
        }
        if (c0 + a.KC < a.Cs) {
            issue(st ^ 1, c0 + a.KC);
            if (PB) rload(c0 + a.KC);
        }

        const T *s_src = stage_src(st);
        const int mrow = KS ? 0 : wm * 32;
        const T *arow0 = stage_a(st) + (mrow + (lane & 15)) * a.SA + (lane >> 4);
        const T *arow1 = arow0 + 16 * a.SA;
        // Fragments are software-pipelined in two register sets: the A/B
        // fragments of step kk+4 are read while the MFMAs of step kk issue, so
        // LDS latency overlaps the matrix pipe.  sched_group_barrier pins that
        // issue order (the scheduler would otherwise sink a set's reads down to
        // its MFMAs).  Reads past the last step land in the A slice's slack (in
        // bounds, unused).  The tap offset of a step is computed
        // arithmetically, so the B reads need no dependent LDS read.
        // Steps past the chunk's last tap read tap KCv-1 instead: a finite value
        // that meets a zero column of A, and no branch splits the loop body.
        auto tap_off = [&](int k) {
            const int kc = min(k, KCv - 1);
            const int c = div_magic(kc, a.magic_hw), t = kc - c * a.HfWf;
            const int i = div_magic(t, a.magic_wf), j = t - i * a.Wf;
            return c * CHn + i * a.Wpad + j;
        };
        T a0[2], a1[2], b0[NB], b1[NB];
        auto frag = [&](int kk, T &fa0, T &fa1, T (&fb)[NB]) {
            fa0 = arow0[kk];
            fa1 = arow1[kk];
            const int ko = tap_off(kk + (lane >> 4));
#pragma unroll
            for (int y = 0; y < NB; ++y) fb[y] = s_src[ko + lbase[y]];
        };
        auto mma_step = [&](T fa0, T fa1, const T (&fb)[NB]) {
#pragma unroll
            for (int y = 0; y < NB; ++y) {
                const T bv = fb[y];
                if (ZSKIP && wave_all_zero(bv)) continue;
                acc[0][y] = MF::mma(fa0, bv, acc[0][y]);
                acc[1][y] = MF::mma(fa1, bv, acc[1][y]);
            }
        };
        if (!K4) {
            // With ksplit, wave half wm takes the steps kk = 4*wm, 4*wm + 8, ...
            const int kstep = KS ? 8 : 4;
            int kk = KS ? 4 * wm : 0;
            frag(kk, a0[0], a1[0], b0);
            for (; kk + kstep < a.KCK; kk += 2 * kstep) {
                frag(kk + kstep, a0[1], a1[1], b1);
                mma_step(a0[0], a1[0], b0);
                frag(kk + 2 * kstep, a0[0], a1[0], b0);
                mma_step(a0[1], a1[1], b1);
                if (!ZSKIP) {
                    // Issue order: a set's reads, then the other set's MFMAs.
                    __builtin_amdgcn_sched_group_barrier(0x100, NB + 2, 0);
                    __builtin_amdgcn_sched_group_barrier(0x008, 2 * NB, 0);
                    __builtin_amdgcn_sched_group_barrier(0x100, NB + 2, 0);
                    __builtin_amdgcn_sched_group_barrier(0x008, 2 * NB, 0);
                }
            }
            if (kk < a.KCK) mma_step(a0[0], a1[0], b0);
        } else {
            const T *ar = stage_a(st) + (lane & 15) * a.SA + (lane >> 4);
            T fa[2][R4], fb[2][2];
            auto frag4 = [&](int k, T (&A)[R4], T (&B)[2]) {
#pragma unroll
                for (int x = 0; x < R4; ++x) A[x] = ar[16 * x * a.SA + k];
                const int ko = tap_off(k + (lane >> 4));
#pragma unroll
                for (int y = 0; y < 2; ++y) B[y] = s_src[ko + lb4[y]];
            };
            auto mma4 = [&](const T (&A)[R4], const T (&B)[2]) {
#pragma unroll
                for (int y = 0; y < 2; ++y) {
                    if (ZSKIP && wave_all_zero(B[y])) continue;
#pragma unroll
                    for (int x = 0; x < R4; ++x) acc4[x][y] = MF::mma(A[x], B[y], acc4[x][y]);
                }
            };
            int kk = 4 * wave;
            frag4(kk, fa[0], fb[0]);
            for (; kk + 16 < a.KCK; kk += 32) {
                frag4(kk + 16, fa[1], fb[1]);
                mma4(fa[0], fb[0]);
                frag4(kk + 32, fa[0], fb[0]);
                mma4(fa[1], fb[1]);
                if (!ZSKIP) {
                    __builtin_amdgcn_sched_group_barrier(0x100, R4 + 2, 0);
                    __builtin_amdgcn_sched_group_barrier(0x008, 2 * R4, 0);
                    __builtin_amdgcn_sched_group_barrier(0x100, R4 + 2, 0);
                    __builtin_amdgcn_sched_group_barrier(0x008, 2 * R4, 0);
                }
            }
            if (kk < a.KCK) mma4(fa[0], fb[0]);
        }
        // the next chunk's gradient window, into the stage no wave reads now
        if (PB && c0 + a.KC < a.Cs) rstore(c0 + a.KC, stage_src(st ^ 1));
        wait_dma();
        __syncthreads();
        st ^= 1;
    }

    if (K4) {
        // Partial tiles to LDS, then each wave sums (in wave order) the part of
        // the tile the standard epilogue expects it to hold.
        T *s_p = reinterpret_cast<T *>(smem);
#pragma unroll
        for (int x = 0; x < R4; ++x)
#pragma unroll
            for (int y = 0; y < 2; ++y)
#pragma unroll
                for (int r = 0; r < 4; ++r)
                    s_p[(wave * 64 + 16 * x + MF::row(lane, r)) * 32 + 16 * y + (lane & 15)] =
                        acc4[x][y][r];
        __syncthreads();
#pragma unroll
        for (int x = 0; x < 2; ++x)
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                const int ml = wm * 32 + 16 * x + MF::row(lane, r), col = wn * 16 + (lane & 15);
                T v = T(0);
                if (ml < 16 * R4)
#pragma unroll
                    for (int w = 0; w < 4; ++w) v += s_p[(w * 64 + ml) * 32 + col];
                acc[x][0][r] = v;
            }
        __syncthreads();
    }
    bool active = true;  // this wave holds final values of its rows
    if (KS) {
        // Waves wm = 1 hand their partial tiles to the waves wm = 0 of the same
        // columns, which add them (fixed order) and store.  The stages are free:
        // every wave has passed the last chunk's barrier.
        T *s_red = reinterpret_cast<T *>(smem);
        if (wm == 1)
#pragma unroll
            for (int x = 0; x < 2; ++x)
#pragma unroll
                for (int y = 0; y < NB; ++y)
#pragma unroll
                    for (int r = 0; r < 4; ++r)
                        s_red[(((wn * 2 + x) * NB + y) * 4 + r) * kWave + lane] = acc[x][y][r];
        __syncthreads();
        if (wm == 1) {
            if (!POOL) return;
            active = false;
        } else {
#pragma unroll
            for (int x = 0; x < 2; ++x)
#pragma unroll
                for (int y = 0; y < NB; ++y)
#pragma unroll
                    for (int r = 0; r < 4; ++r)
                        acc[x][y][r] += s_red[(((wn * 2 + x) * NB + y) * 4 + r) * kWave + lane];
        }
    }
    const int mbase = m0 + (KS ? 0 : wm * 32);
    if (!BWD && active) {  // bias and relu, in place
        const T *bias = reinterpret_cast<const T *>(a.bias);
#pragma unroll
        for (int x = 0; x < 2; ++x)
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                const int m = mbase + x * 16 + MF::row(lane, r);
                const T bm = (bias && m < a.M) ? bias[m] : T(0);
#pragma unroll
                for (int y = 0; y < NB; ++y) acc[x][y][r] = relu_if(acc[x][y][r] + bm, a.relu);
            }
    }
    if (active && a.out) {
        T *out = reinterpret_cast<T *>(a.out) + (size_t)n * a.M * a.Q;
#pragma unroll
        for (int x = 0; x < 2; ++x)
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                const int m = mbase + x * 16 + MF::row(lane, r);
                if (m >= a.M) continue;
                T *orow = out + (size_t)m * a.Q;
                if (!BWD && a.nbanks > 1) {  // the row's filter bank and its output
                    int b = 0;
                    while (b + 1 < a.nbanks && m >= a.bank_off[b + 1]) ++b;
                    const int Fb = a.bank_off[b + 1] - a.bank_off[b];
                    orow = reinterpret_cast<T *>(a.bank_out[b]) +
                           ((size_t)n * Fb + (m - a.bank_off[b])) * a.Q;
                }
#pragma unroll
                for (int y = 0; y < NB; ++y) {
                    const int q = q0 + (wn * NB + y) * 16 + (lane & 15);
                    if (q < qend) orow[q] = acc[x][y][r];
                }
            }
    }
    if (POOL) {
        // The tile is whole rows of conv output [y_lo, y_hi); the pooled rows
        // whose windows start in it lie wholly inside it (PS >= PH, tiles a
        // multiple of PS rows).  Per 32-row half: the half's values go to LDS
        // ([32][32 NB]), then every thread scans windows (first maximum wins,
        // strict >, as the standalone pooling kernel does).
        constexpr int BN = 32 * NB;
        T *s_t = reinterpret_cast<T *>(smem);
        const int y_lo = q0 / a.Qw, y_hi = qend / a.Qw;  // q0, qend: multiples of Qw
        const int py_lo = y_lo / a.PS;
        const int py_hi = min(a.Hp, (y_hi + a.PS - 1) / a.PS);
        const int npool = (py_hi - py_lo) * a.Wp;
        T *pout = reinterpret_cast<T *>(a.pool_out) + (size_t)n * a.M * a.Hp * a.Wp;
        int32_t *pidx = a.pool_idx + (size_t)n * a.M * a.Hp * a.Wp;
        for (int half = 0; half < (KS ? 1 : 2); ++half) {
            __syncthreads();
            if (active && (KS || wm == half))
#pragma unroll
                for (int x = 0; x < 2; ++x)
#pragma unroll
                    for (int y = 0; y < NB; ++y)
#pragma unroll
                        for (int r = 0; r < 4; ++r) {
                            const int u = (wn * NB + y) * 16 + (lane & 15);
                            if (q0 + u < qend)
                                s_t[(x * 16 + MF::row(lane, r)) * BN + u] = acc[x][y][r];
                        }
            __syncthreads();
            for (int e = tid; e < 32 * npool; e += kThreads) {
                const int rr = e / npool, pe = e - rr * npool;
                const int m = m0 + half * 32 + rr;
                if (m >= a.M) continue;
                const int py = py_lo + pe / a.Wp, px = pe - (pe / a.Wp) * a.Wp;
                T best = T(0);
                int bidx = -1;
                for (int i = 0; i < a.PH; ++i) {
                    const int yy = py * a.PS + i;
                    for (int j = 0; j < a.PW; ++j) {
                        const int xx = px * a.PS + j;
                        const T v = s_t[rr * BN + (yy - y_lo) * a.Qw + xx];
                        if (bidx < 0 || v > best) {
                            best = v;
                            bidx = yy * a.Qw + xx;
                        }
                    }
                }
                const size_t o = (size_t)m * a.Hp * a.Wp + (size_t)py * a.Wp + px;
                pout[o] = best;
                pidx[o] = m * a.Q + bidx;
            }
        }
    }
}

// Layers with at most four output rows (forward with F <= 4, backward_data
// with C <= 4): a matrix-core tile is at least 16 rows, so nearly all of its
// work would be padding.  Here the products run on the vector ALU.  A block
// covers 64 consecutive pixels of one image (a lane per pixel) with four waves
// that split the source channels (wave w takes channels w, w+4, ... of each
// chunk); their partial sums are added in wave order at the end.  Per chunk
// of KC channels the block stages the window rows its pixels read (the masked
// dout in the backward pass) and the chunk's filter values in LDS; a lane then
// walks its channels' taps, the Wf taps of a window row unrolled so their LDS
// reads overlap.  Filter values are read by all lanes at one address (an LDS
// broadcast).
constexpr int kSmallM = 4;
constexpr int kSmallPix = 64;
constexpr int kSmallWaves = 4;
constexpr int kSmallMaxWf = 7;
constexpr int kSmallStage = 8;  // window elements each thread loads before storing
constexpr size_t kSmallLds = 32 * 1024;

// WF: the filter width when it is 3 or 5 (taps fully unrolled), else 0 (any
// width up to kSmallMaxWf).  MM: 1 when M = 1, else 4 (filter rows past M are
// staged as zeros, so no row test is needed).
template <typename T, bool BWD, int WF, int MM, bool PB = false>
__global__ __launch_bounds__(kSmallPix * kSmallWaves) void conv_small_m_kernel(IgemmArgs a)
{
    extern __shared__ __align__(16) unsigned char smem[];
    const int tid = threadIdx.x, lane = lane_id(), wave = wave_id();
    const int n = blockIdx.y;
    const int q0 = blockIdx.x * kSmallPix, qend = min(q0 + kSmallPix, a.Q);
    const int qy0 = q0 / a.Qw;
    const int rows = ((qend - 1) / a.Qw - qy0) * a.S + a.Hf;
    const int ybase = qy0 * a.S - a.Ph;
    const int CHn = rows * a.Wpad;
    T *s_win = reinterpret_cast<T *>(smem);  // [KC][rows][Wpad]
    T *s_w = s_win + (size_t)a.KC * a.CH;    // [KC][MM][Hf*Wf]; CH = the largest rows * Wpad
    const int q = q0 + lane;
    const bool act = q < qend;
    int lb = 0;
    if (act) {
        const int qy = q / a.Qw, qx = q - qy * a.Qw;
        lb = (qy - qy0) * a.S * a.Wpad + qx * a.S;
    }
    const size_t img = (size_t)a.Cs * a.Sh * a.Sw;
    const T *src = PB ? nullptr : reinterpret_cast<const T *>(a.src) + (size_t)n * img;
    const T *msk = (BWD && !PB && a.mask) ? reinterpret_cast<const T *>(a.mask) + (size_t)n * img
                                          : nullptr;
    const T *W = reinterpret_cast<const T *>(a.wgt);
    const int MW = MM * a.HfWf;
    const float rcp_ch = 1.0f / (float)CHn, rcp_wpad = 1.0f / (float)a.Wpad;
    const float rcp_up = 1.0f / (float)a.up;
    const T *mskp = msk ? msk : src;  // loaded either way; used only with a mask
    T acc[MM];
#pragma unroll
    for (int m = 0; m < MM; ++m) acc[m] = T(0);

    for (int c0 = 0; c0 < a.Cs; c0 += a.KC) {
        const int kc = min(a.KC, a.Cs - c0);
        __syncthreads();  // the previous chunk's readers are done
        // Window element e = (c, t, x) of the chunk.  Each thread issues eight
        // loads before using any: cells outside the source read element 0 of
        // the image (a valid address) and are zeroed afterwards, so no branch
        // splits the loads (a load under a divergent branch is waited for at
        // the branch's end).
        const int tot = kc * CHn;
        for (int base = 0; base < tot; base += kSmallStage * kSmallPix * kSmallWaves) {
            T v[kSmallStage], mv[kSmallStage];
            bool ok[kSmallStage];
#pragma unroll
            for (int u = 0; u < kSmallStage; ++u) {
                const int e = min(base + u * kSmallPix * kSmallWaves + tid, tot - 1);
                const int c = div_small(e, CHn, rcp_ch), rem = e - c * CHn;
                const int t = div_small(rem, a.Wpad, rcp_wpad), x = rem - t * a.Wpad;
                const int yv = ybase + t, xv = x - a.Pw;
                const int ys = div_small(max(yv, 0), a.up, rcp_up);
                const int xs = div_small(max(xv, 0), a.up, rcp_up);
                const bool in = yv >= 0 && xv >= 0 && ys * a.up == yv && xs * a.up == xv &&
                                ys < a.Sh && xs < a.Sw;
                ok[u] = in;
                if (PB) {
                    // branch-free: a clamped cell, dropped by ok[u] when outside
                    v[u] = pool_src_grad<T>(a.pool, n, a.Cs, c0 + c, a.Sh * a.Sw, a.Sw,
                                            min(ys, a.Sh - 1), min(xs, a.Sw - 1));
                    mv[u] = T(1);
                } else {
                    const size_t o = in ? ((size_t)(c0 + c) * a.Sh + ys) * a.Sw + xs : 0;
                    v[u] = src[o];
                    mv[u] = mskp[o];
                }
            }
#pragma unroll
            for (int u = 0; u < kSmallStage; ++u) {
                const int e = base + u * kSmallPix * kSmallWaves + tid;
                if (e < tot) s_win[e] = (ok[u] && (!msk || mv[u] > T(0))) ? v[u] : T(0);
            }
        }
        for (int e = tid; e < kc * MW; e += kSmallPix * kSmallWaves) {
            const int c = e / MW, r = e - c * MW;
            const int m = r / a.HfWf, tp = r - m * a.HfWf;
            const size_t el = BWD ? ((size_t)(c0 + c) * a.M + m) * a.HfWf + (a.HfWf - 1 - tp)
                                  : ((size_t)m * a.Cs + (c0 + c)) * a.HfWf + tp;
            s_w[e] = m < a.M ? W[el] : T(0);
        }
        __syncthreads();
        if (act) {
            for (int c = wave; c < kc; c += kSmallWaves) {
                const T *wrow = s_win + c * CHn + lb;
                const T *wc = s_w + c * MW;
                for (int i = 0; i < a.Hf; ++i) {
                    if constexpr (WF > 0) {
                        // a window row's taps: all LDS reads first, then the FMAs
                        T v[WF], w[MM][WF];
#pragma unroll
                        for (int j = 0; j < WF; ++j) v[j] = wrow[i * a.Wpad + j];
#pragma unroll
                        for (int m = 0; m < MM; ++m)
#pragma unroll
                            for (int j = 0; j < WF; ++j) w[m][j] = wc[m * a.HfWf + i * WF + j];
#pragma unroll
                        for (int j = 0; j < WF; ++j)
#pragma unroll
                            for (int m = 0; m < MM; ++m) acc[m] += w[m][j] * v[j];
                    } else {
                        for (int j = 0; j < a.Wf; ++j) {
                            const T v = wrow[i * a.Wpad + j];
#pragma unroll
                            for (int m = 0; m < MM; ++m) acc[m] += wc[m * a.HfWf + i * a.Wf + j] * v;
                        }
                    }
                }
            }
        }
    }
    // partial sums of the four channel groups, added in wave order
    __syncthreads();
    T *s_red = reinterpret_cast<T *>(smem);  // [wave][M][64]
#pragma unroll
    for (int m = 0; m < MM; ++m)
        if (m < a.M) s_red[(wave * kSmallM + m) * kSmallPix + lane] = acc[m];
    __syncthreads();
    T *out = reinterpret_cast<T *>(a.out) + (size_t)n * a.M * a.Q;
    const T *bias = reinterpret_cast<const T *>(a.bias);
    for (int e = tid; e < a.M * kSmallPix; e += kSmallPix * kSmallWaves) {
        const int m = e / kSmallPix, u = e - m * kSmallPix;
        if (q0 + u >= qend) continue;
        T v = s_red[m * kSmallPix + u];
#pragma unroll
        for (int w = 1; w < kSmallWaves; ++w) v += s_red[(w * kSmallM + m) * kSmallPix + u];
        if (!BWD) v = relu_if(v + (bias ? bias[m] : T(0)), a.relu);
        out[(size_t)m * a.Q + q0 + u] = v;
    }
}

// Channel chunk of the small-M kernel: the largest whose window and filter
// values fit kSmallLds; 0 when not even one channel fits.
int small_m_plan(size_t tsz, int M, int Cs, int Qw, int Q, int Hf, int Wf, int S, int &CH,
                 int &Wpad)
{
    Wpad = (Qw - 1) * S + Wf;
    int rows_max = 0;
    for (int q0 = 0; q0 < Q; q0 += kSmallPix) {
        const int qe = (q0 + kSmallPix < Q ? q0 + kSmallPix : Q) - 1;
        const int r = (qe / Qw - q0 / Qw) * S + Hf;
        rows_max = r > rows_max ? r : rows_max;
    }
    CH = rows_max * Wpad;
    if (Wf > kSmallMaxWf) return 0;
    const int MM = M == 1 ? 1 : kSmallM;
    const size_t per_c = tsz * ((size_t)CH + (size_t)MM * Hf * Wf);
    size_t kc = kSmallLds / per_c;
    if (kc > (size_t)Cs) kc = Cs;
    return (int)kc;
}

// ---------------------------------------------------------------------------
// Filter-resident forward for small images with a moderate K (LeNet conv2: 64
// images of 14x14, K = 800).  There the 64-row tiles above re-stage the whole
// filter from L2 for every 32 pixels; here a block owns 16 filters of one
// image and keeps their whole 16 x K slice in LDS, loaded once, while the
// image's padded source window streams through in channel chunks (LDS DMA,
// double-buffered, exactly as above).  The waves form four tile groups (group
// g takes every fourth 16-pixel tile of the image from tile g, at most four:
// Q <= 256), so a wave issues up to four independent MFMAs per k-step from one
// filter fragment, times kResKs k ranges (alternate k-steps; the partial tiles
// are added in range order at the end): with one block per CU (the slice and
// the two chunks take most of its LDS) that keeps four waves per SIMD.  The
// slice is stored chunk by chunk, each chunk's taps padded to a multiple of 4
// (zeros), so a chunk's k-steps read it at a fixed offset.  The epilogue adds
// the bias, applies relu and stores, or pools (the whole image is in the block:
// every pooled window lies inside it).
constexpr int kResRows = 16;
constexpr int kResNT = 4;       // 16-pixel tiles per wave at most
constexpr int kResKs = 4;                      // k ranges (alternate k-steps)
constexpr int kResWaves = 4 * kResKs;          // four tile groups x kResKs
constexpr int kResThreads = kResWaves * kWave;
constexpr int kResMaxDma = 6;  // source-window DMA instructions per wave per chunk

template <typename T, bool POOL>
__global__ __launch_bounds__(kResThreads) __attribute__((amdgpu_waves_per_eu(2))) void conv_resident_kernel(IgemmArgs a, int lds_a_bytes, int stage_bytes)
{
    using MF = Mfma<T>;
    constexpr int dpe = sizeof(T) / 4;
    extern __shared__ __align__(16) unsigned char smem[];
    T *s_a = reinterpret_cast<T *>(smem);  // [16][SA]
    unsigned char *stages = smem + lds_a_bytes;
    auto stage_src = [&](int st) { return reinterpret_cast<T *>(stages + st * stage_bytes); };

    const int tid = threadIdx.x, lane = lane_id(), wave = wave_id();
    // tile group and k range: the waves of one SIMD (wave mod 4) hold the four
    // tile groups, so a group with one tile more than the others does not load
    // one SIMD alone
    const int kh = wave % kResKs, tg = wave / kResKs;
    const int n = blockIdx.x, m0 = blockIdx.y * kResRows;
    const int KCv = a.KC * a.HfWf;
    const int nchunk = (a.Cs + a.KC - 1) / a.KC;
    const int Kw = a.Cs * a.HfWf;  // filter row length
    const int Awid = nchunk * a.KCK;

    // Source window of a chunk: [KC][Hpad][Wpad], row t / column x of the
    // padded image (input row t - Ph, column x - Pw), zeros outside.  Per-lane
    // DMA offsets are chunk-invariant; the chunk's channel offset is soffset.
    const size_t img = (size_t)a.Cs * a.Sh * a.Sw;
    const i32x4 rs_src = buffer_rsrc(reinterpret_cast<const T *>(a.src) + (size_t)n * img,
                                     (unsigned)(img * sizeof(T)));
    const int Ds = a.KC * a.CH * dpe;
    const int NIs = (Ds + kWave - 1) / kWave;
    const float rcp_ch = 1.0f / (float)a.CH, rcp_wpad = 1.0f / (float)a.Wpad;
    int vs_off[kResMaxDma];
#pragma unroll
    for (int j = 0; j < kResMaxDma; ++j) {
        const int ii = wave + kResWaves * j, d = ii * kWave + lane;
        int off = kDmaZero;
        if (ii < NIs && d < Ds) {
            const int e = d / dpe, h = d - e * dpe;
            const int c = div_small(e, a.CH, rcp_ch), r = e - c * a.CH;
            const int t = div_small(r, a.Wpad, rcp_wpad), x = r - t * a.Wpad;
            const int y = t - a.Ph, xs = x - a.Pw;
            if (y >= 0 && y < a.Sh && xs >= 0 && xs < a.Sw)
                off = (int)((((size_t)c * a.Sh + y) * a.Sw + xs) * sizeof(T)) + 4 * h;
        }
        vs_off[j] = off;
    }
    auto issue = [&](int st, int c0) {
        unsigned char *ps = reinterpret_cast<unsigned char *>(stage_src(st));
        const int so = (int)((size_t)c0 * a.Sh * a.Sw * sizeof(T));
#pragma unroll
        for (int j = 0; j < kResMaxDma; ++j) {
            const int ii = wave + kResWaves * j;
            if (ii < NIs) dma_dword(rs_src, ps + ii * 256, vs_off[j], so);
        }
    };
    issue(0, 0);

    // The filter slice, once: slot ch * KCK + kl of row r holds
    // W[m0 + r][ch * KC * HfWf + kl] for kl < KC * HfWf inside the filter row,
    // else 0.  Sixteen branch-free loads per thread in flight before the
    // stores (one round trip for the LeNet slice, 16 x 800, over 1024 threads).
    const T *W = reinterpret_cast<const T *>(a.wgt);
    const int tot_a = kResRows * Awid;
    const float rcp_aw = 1.0f / (float)Awid, rcp_kck = 1.0f / (float)a.KCK;
    constexpr int kAB = 16;
    for (int base = 0; base < tot_a; base += kAB * kResThreads) {
        T v[kAB];
#pragma unroll
        for (int u = 0; u < kAB; ++u) {
            const int e = min(base + u * kResThreads + tid, tot_a - 1);
            const int r = div_small(e, Awid, rcp_aw), sl = e - r * Awid;
            const int ch = div_small(sl, a.KCK, rcp_kck), kl = sl - ch * a.KCK;
            const int k = ch * KCv + kl;
            v[u] = W[(size_t)min(m0 + r, a.M - 1) * Kw + min(k, Kw - 1)];
        }
#pragma unroll
        for (int u = 0; u < kAB; ++u) {
            const int e = base + u * kResThreads + tid;
            if (e < tot_a) {
                const int r = div_small(e, Awid, rcp_aw), sl = e - r * Awid;
                const int ch = div_small(sl, a.KCK, rcp_kck), kl = sl - ch * a.KCK;
                const int k = ch * KCv + kl;
                s_a[r * a.SA + sl] = (m0 + r < a.M && kl < KCv && k < Kw) ? v[u] : T(0);
            }
        }
    }

    // Window offset of this lane's pixel in each of the wave's tiles (0 past Q:
    // a valid address whose results are not stored).
    int pb[kResNT];
#pragma unroll
    for (int tt = 0; tt < kResNT; ++tt) {
        const int q = (tg + 4 * tt) * 16 + (lane & 15);
        const int oy = div_magic(q, a.magic_qw), ox = q - oy * a.Qw;
        pb[tt] = q < a.Q ? oy * a.S * a.Wpad + ox * a.S : 0;
    }
    // tiles of this group that hold pixels (wave-uniform): the others skip
    // their fragment reads and MFMAs
    const int ntile = (a.Q + 15) / 16;
    const int nt = ntile > tg ? min(kResNT, (ntile - tg + 3) / 4) : 0;
    typename MF::acc_t acc[kResNT];
#pragma unroll
    for (int tt = 0; tt < kResNT; ++tt) acc[tt] = MF::zero();
    wait_dma();
    __syncthreads();

    // Steps past the chunk's last tap read tap KCv - 1 (finite) against a zero
    // filter column.  The prefetch after a chunk's last step reads past its
    // slots, inside LDS (the slice is followed by the stages), unused.
    auto tap_off = [&](int k) {
        const int kc = min(k, KCv - 1);
        const int c = div_magic(kc, a.magic_hw), t = kc - c * a.HfWf;
        const int i = div_magic(t, a.magic_wf), j = t - i * a.Wf;
        return c * a.CH + i * a.Wpad + j;
    };
    for (int ch = 0; ch < nchunk; ++ch) {
        const int st = ch & 1;
        if (ch + 1 < nchunk) issue(st ^ 1, (ch + 1) * a.KC);
        const T *s_src = stage_src(st);
        const T *arow = s_a + (lane & 15) * a.SA + ch * a.KCK + (lane >> 4);
        T fa0, fa1, fb0[kResNT], fb1[kResNT];
        auto frag = [&](int kk, T &fa, T (&fb)[kResNT]) {
            fa = arow[kk];
            const int ko = tap_off(kk + (lane >> 4));
#pragma unroll
            for (int tt = 0; tt < kResNT; ++tt)
                if (tt < nt) fb[tt] = s_src[ko + pb[tt]];
        };
        auto mma_step = [&](T fa, const T (&fb)[kResNT]) {
#pragma unroll
            for (int tt = 0; tt < kResNT; ++tt)
                if (tt < nt) acc[tt] = MF::mma(fa, fb[tt], acc[tt]);
        };
        // k range kh takes the steps 4 kh, 4 kh + KST, ...
        constexpr int KST = 4 * kResKs;
        int kk = 4 * kh;
        frag(kk, fa0, fb0);
        for (; kk + KST < a.KCK; kk += 2 * KST) {
            frag(kk + KST, fa1, fb1);
            mma_step(fa0, fb0);
            frag(kk + 2 * KST, fa0, fb0);
            mma_step(fa1, fb1);
            __builtin_amdgcn_sched_group_barrier(0x100, kResNT + 1, 0);
            __builtin_amdgcn_sched_group_barrier(0x008, kResNT, 0);
            __builtin_amdgcn_sched_group_barrier(0x100, kResNT + 1, 0);
            __builtin_amdgcn_sched_group_barrier(0x008, kResNT, 0);
        }
        if (kk < a.KCK) mma_step(fa0, fb0);
        wait_dma();
        __syncthreads();
    }

    // The other k ranges hand their partial tiles to the first, one range at a
    // time through the stages (free after the last barrier); the first adds
    // them in range order.
    {
        T *s_red = reinterpret_cast<T *>(stages);  // [4 tile groups][kResNT][4][64]
        for (int h = 1; h < kResKs; ++h) {  // the other ranges, in order
            if (kh == h)
#pragma unroll
                for (int tt = 0; tt < kResNT; ++tt)
#pragma unroll
                    for (int r = 0; r < 4; ++r)
                        s_red[((tg * kResNT + tt) * 4 + r) * kWave + lane] = acc[tt][r];
            __syncthreads();
            if (kh == 0)
#pragma unroll
                for (int tt = 0; tt < kResNT; ++tt)
#pragma unroll
                    for (int r = 0; r < 4; ++r)
                        acc[tt][r] += s_red[((tg * kResNT + tt) * 4 + r) * kWave + lane];
            __syncthreads();
        }
    }
    // Epilogue (first k range): bias and relu, then the conv output and/or the pool.
    const T *bias = reinterpret_cast<const T *>(a.bias);
#pragma unroll
    for (int r = 0; r < 4; ++r) {
        const int m = m0 + MF::row(lane, r);
        const T bm = (bias && m < a.M) ? bias[m] : T(0);
#pragma unroll
        for (int tt = 0; tt < kResNT; ++tt) acc[tt][r] = relu_if(acc[tt][r] + bm, a.relu);
    }
    if (a.out && kh == 0) {
        T *out = reinterpret_cast<T *>(a.out) + (size_t)n * a.M * a.Q;
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            const int m = m0 + MF::row(lane, r);
#pragma unroll
            for (int tt = 0; tt < kResNT; ++tt) {
                const int q = (tg + 4 * tt) * 16 + (lane & 15);
                if (m < a.M && q < a.Q) out[(size_t)m * a.Q + q] = acc[tt][r];
            }
        }
    }
    if (POOL) {
        // the 16 x Q tile to LDS (the stages are free after the last barrier),
        // then every thread scans windows: first maximum wins (strict >)
        T *s_t = reinterpret_cast<T *>(stages);
        if (kh == 0)
#pragma unroll
            for (int r = 0; r < 4; ++r)
#pragma unroll
                for (int tt = 0; tt < kResNT; ++tt) {
                    const int q = (tg + 4 * tt) * 16 + (lane & 15);
                    if (q < a.Q) s_t[MF::row(lane, r) * a.Q + q] = acc[tt][r];
                }
        __syncthreads();
        const int npool = a.Hp * a.Wp;
        T *pout = reinterpret_cast<T *>(a.pool_out) + (size_t)n * a.M * npool;
        int32_t *pidx = a.pool_idx + (size_t)n * a.M * npool;
        for (int e = tid; e < kResRows * npool; e += kResThreads) {
            const int rr = e / npool, pe = e - rr * npool;
            const int m = m0 + rr;
            if (m >= a.M) continue;
            const int py = pe / a.Wp, px = pe - py * a.Wp;
            T best = T(0);
            int bidx = -1;
            for (int i = 0; i < a.PH; ++i) {
                const int yy = py * a.PS + i;
                for (int j = 0; j < a.PW; ++j) {
                    const int xx = px * a.PS + j;
                    const T v = s_t[rr * a.Q + yy * a.Qw + xx];
                    if (bidx < 0 || v > best) {
                        best = v;
                        bidx = yy * a.Qw + xx;
                    }
                }
            }
            const size_t o = (size_t)m * npool + pe;
            pout[o] = best;
            pidx[o] = m * a.Q + bidx;
        }
    }
}

// Host-side tile selection ----------------------------------------------------

struct Plan {
    int NB, KC, KCK, Wpad, CH, SA, tiles_per_img, TS, m_tiles, pipelined;
    size_t lds;
};

size_t lds_bytes(size_t tsz, int KC, int CH, int SA, int KCK)
{
    return tsz * ((size_t)KC * CH + (size_t)kBM * SA) + sizeof(int) * (size_t)KCK;
}

bool make_plan(size_t tsz, int M, int Cs, int Qw, int Q, int Hf, int Wf, int S, int nimg,
               Plan &p, int align = 0)
{
    static const int kNB64[] = {7, 4, 2, 1}, kNB32[] = {7, 4, 2, 1};
    const int HfWf = Hf * Wf;
    p.m_tiles = (M + kBM - 1) / kBM;
    double best = -1.0;
    const int *cand = tsz == 8 ? kNB64 : kNB32;
    const int ncand = 4;
    for (int ci = 0; ci < ncand; ++ci) {
        const int NB = cand[ci];
        int BN = 32 * NB;
        // a fused epilogue needs tiles of whole row groups (or one tile per
        // image): the tile origins step by the largest multiple of the group
        // that fits, and the rest of the 32 NB pixels is masked
        const int TS = (!align || BN >= Q) ? BN : (BN / align) * align;
        if (TS == 0) continue;
        int tiles = (Q + TS - 1) / TS;
        double fill = (double)Q / ((double)tiles * BN);
        double blocks = (double)nimg * tiles * p.m_tiles;
        double occ = blocks >= 512.0 ? 1.0 : blocks / 512.0;
        double score = fill * occ;
        if (score > best + 1e-9) {
            best = score;
            p.NB = NB;
            p.tiles_per_img = tiles;
            p.TS = TS;
        }
    }
    if (best < 0.0) return false;
    // Input rows a tile of TS consecutive outputs reads: the exact maximum over
    // the tiles of an image (a tile that starts a row spans one row fewer than
    // the general bound when TS is a multiple of the output width).
    int rows_max = 0;
    for (int t = 0; t < p.tiles_per_img; ++t) {
        const int qa = t * p.TS, qb = (qa + p.TS < Q ? qa + p.TS : Q) - 1;
        const int r = (qb / Qw - qa / Qw) * S + Hf;
        rows_max = r > rows_max ? r : rows_max;
    }
    p.Wpad = (Qw - 1) * S + Wf;
    p.CH = rows_max * p.Wpad;
    // Largest channel chunk whose staging fits the per-thread register slots
    // (pipelined path) and the LDS budget; otherwise the largest that fits the
    // LDS budget alone (direct-staging path).
    const int ncg = (p.Wpad + 63) / 64;
    auto kck_of = [&](int kc) { return ((kc * HfWf + 3) / 4) * 4; };
    auto fits_lds = [&](int kc) {
        return lds_bytes(tsz, kc, p.CH, kck_of(kc) + 1, kck_of(kc)) <= kLdsBudget;
    };
    auto fits_regs = [&](int kc) {
        return (kc * rows_max * ncg + 3) / 4 <= kMS && kBM * kck_of(kc) <= kThreads * kMA;
    };
    int kc = Cs;
    while (kc > 1 && !(fits_regs(kc) && fits_lds(kc))) --kc;
    p.pipelined = fits_regs(kc) && fits_lds(kc);
    if (!p.pipelined) {
        kc = Cs;
        while (kc > 1 && !fits_lds(kc)) --kc;
    }
    p.KC = kc;
    p.KCK = kck_of(kc);
    p.SA = p.KCK + 1;
    p.lds = lds_bytes(tsz, p.KC, p.CH, p.SA, p.KCK);
    return p.lds <= 160 * 1024;
}

// LDS-DMA plan: the largest channel chunk (up to 16) whose per-wave DMA
// instruction counts fit the offset registers and whose two stages fit the
// per-block LDS share.  False when the problem needs the register-staged path
// (very wide rows, very large filters, or tensors of 2 GiB and more, whose byte
// offsets would reach the out-of-range marker).
// pb_rpc (pooled source): the most pool regions one channel of a staged window
// meets; a chunk's regions must fit the owners' registers (kRP a thread).
bool make_dma_plan(size_t tsz, bool bwd, int pb_rpc, int M, int Cs, int HfWf, int rows_max,
                   int Wpad, size_t img_bytes, size_t w_bytes, Plan &p, DmaLayout &L)
{
    const int max_a = dma_a_max(p.NB), rows_a = dma_a_rows(M);
    if (img_bytes >= 0x80000000ull || w_bytes >= 0x80000000ull) return false;
    const long long dpe = (long long)tsz / 4;
    // The largest chunk that fits, unless a chunk at least half as large has no
    // padded k-steps (KC*Hf*Wf a multiple of 4): then the largest such chunk.
    int first = 0, exact = 0;
    Plan pf = p, pe = p;
    DmaLayout lf = {}, le = {};
    for (int kc = Cs < 16 ? Cs : 16; kc >= 1; --kc) {
        // row stride of the A slice: 2 mod 4 elements, so the 32 lanes of a half-wave
        // (16 rows x 2 k) hit distinct banks (an odd stride conflicts)
        const int kck = ((kc * HfWf + 3) / 4) * 4, sa = kck + 2;
        // fp64 rows of sa = 2 mod 4 elements start 16-byte aligned in LDS
        const bool vec = tsz == 8 && !bwd && (kc * HfWf) % 2 == 0;
        const long long nis = ((long long)kc * rows_max * Wpad * dpe + kWave - 1) / kWave;
        const long long nia = vec ? ((long long)rows_a * sa / 2 + kWave - 1) / kWave
                                  : ((long long)rows_a * sa * dpe + kWave - 1) / kWave;
        if ((nis + 3) / 4 > kMaxDmaS || (nia + 3) / 4 > max_a) continue;
        if (pb_rpc && kc * pb_rpc > kThreads * 4) continue;
        DmaLayout l;
        l.src_bytes = (int)nis * 256;
        l.a_bytes = (int)nia * (vec ? 1024 : 256) + 256;  // + slack read by the last step's prefetch
        l.a_vec = vec;
        l.stage_bytes = l.src_bytes + l.a_bytes;
        // + the mask window of the backward pass (not with a pooled source)
        const size_t total = 2 * (size_t)l.stage_bytes + (bwd && !pb_rpc ? (size_t)l.src_bytes : 0);
        // fp32 kernels fit three blocks per CU in registers; keep LDS to a third
        if (total > (tsz == 4 ? kLdsPerBlock32 : kLdsPerBlock)) continue;
        Plan q = p;
        q.KC = kc;
        q.KCK = kck;
        q.SA = sa;
        q.lds = total;
        if (!first) {
            first = kc;
            pf = q;
            lf = l;
        }
        if (kck == kc * HfWf && 2 * kc >= first) {
            exact = kc;
            pe = q;
            le = l;
            break;
        }
    }
    if (!first) return false;
    p = exact ? pe : pf;
    L = exact ? le : lf;
    return true;
}

template <typename T, int NB, bool BWD, bool KS, bool POOL, int K4 = 0, bool PB = false>
hipError_t launch_dma_ks(const IgemmArgs &a, const Plan &p, const DmaLayout &L, unsigned w_bytes,
                         int nimg, int zero_skip, hipStream_t s)
{
    dim3 grid(nimg * p.tiles_per_img, p.m_tiles), block(kThreads);
    hipError_t e;
    if (PB) {  // the pooled source has no zero-skip form
        auto k = conv_igemm_dma_kernel<T, NB, BWD, false, KS, POOL, K4, true>;
        if ((e = allow_dynamic_lds(k, p.lds)) != hipSuccess) return e;
        hipLaunchKernelGGL(k, grid, block, p.lds, s, a, L, w_bytes);
    } else if (zero_skip) {
        auto k = conv_igemm_dma_kernel<T, NB, BWD, true, KS, POOL, K4>;
        if ((e = allow_dynamic_lds(k, p.lds)) != hipSuccess) return e;
        hipLaunchKernelGGL(k, grid, block, p.lds, s, a, L, w_bytes);
    } else {
        auto k = conv_igemm_dma_kernel<T, NB, BWD, false, KS, POOL, K4>;
        if ((e = allow_dynamic_lds(k, p.lds)) != hipSuccess) return e;
        hipLaunchKernelGGL(k, grid, block, p.lds, s, a, L, w_bytes);
    }
    return hipGetLastError();
}

template <typename T, int NB, bool BWD, bool POOL, bool PB = false>
hipError_t launch_dma_k4(const IgemmArgs &a, const Plan &p, const DmaLayout &L, unsigned w_bytes,
                         int nimg, int zero_skip, hipStream_t s)
{
    if constexpr (NB == 1) {
        if (a.k4 == 4)
            return launch_dma_ks<T, NB, BWD, false, POOL, 4, PB>(a, p, L, w_bytes, nimg, zero_skip,
                                                                 s);
        if (a.k4 == 2)
            return launch_dma_ks<T, NB, BWD, false, POOL, 2, PB>(a, p, L, w_bytes, nimg, zero_skip,
                                                                 s);
    }
    if (a.ksplit)
        return launch_dma_ks<T, NB, BWD, true, POOL, 0, PB>(a, p, L, w_bytes, nimg, zero_skip, s);
    return launch_dma_ks<T, NB, BWD, false, POOL, 0, PB>(a, p, L, w_bytes, nimg, zero_skip, s);
}

template <typename T, int NB, bool BWD>
hipError_t launch_dma(const IgemmArgs &a, const Plan &p, const DmaLayout &L, unsigned w_bytes,
                      int nimg, int zero_skip, hipStream_t s)
{
    if (!BWD && a.pool_out)
        return launch_dma_k4<T, NB, false, true>(a, p, L, w_bytes, nimg, zero_skip, s);
    if (BWD && a.pb) return launch_dma_k4<T, NB, true, false, true>(a, p, L, w_bytes, nimg, 0, s);
    return launch_dma_k4<T, NB, BWD, false>(a, p, L, w_bytes, nimg, zero_skip, s);
}

template <typename T, int NB, bool BWD>
hipError_t launch_nb(const IgemmArgs &a, const Plan &p, int nimg, int zero_skip, hipStream_t s)
{
    dim3 grid(nimg * p.tiles_per_img, p.m_tiles), block(kThreads);
    hipError_t e;
    if (!BWD && a.csr) {
        auto k = zero_skip ? conv_igemm_kernel<T, NB, false, true, true>
                           : conv_igemm_kernel<T, NB, false, false, true>;
        if ((e = allow_dynamic_lds(k, p.lds)) != hipSuccess) return e;
        hipLaunchKernelGGL(k, grid, block, p.lds, s, a);
        return hipGetLastError();
    }
    if (BWD && a.pb) {
        auto k = conv_igemm_kernel<T, NB, true, false, false, true>;
        if ((e = allow_dynamic_lds(k, p.lds)) != hipSuccess) return e;
        hipLaunchKernelGGL(k, grid, block, p.lds, s, a);
        return hipGetLastError();
    }
    if (zero_skip) {
        auto k = conv_igemm_kernel<T, NB, BWD, true>;
        if ((e = allow_dynamic_lds(k, p.lds)) != hipSuccess) return e;
        hipLaunchKernelGGL(k, grid, block, p.lds, s, a);
    } else {
        auto k = conv_igemm_kernel<T, NB, BWD, false>;
        if ((e = allow_dynamic_lds(k, p.lds)) != hipSuccess) return e;
        hipLaunchKernelGGL(k, grid, block, p.lds, s, a);
    }
    return hipGetLastError();
}

// Plan of the filter-resident forward, or false when it does not apply: at
// most 256 output pixels, enough blocks (images x 16-filter groups) to fill
// the CUs, and a 16-row filter slice that leaves room in LDS for two source
// chunks.  The chunk is the largest whose DMA fits the offset registers,
// preferring one without padded k-steps.
struct ResPlan {
    int KC, KCK, SA, Wpad, CH, lds_a, stage;
    size_t lds;
};

bool res_plan(size_t tsz, int M, int Cs, int Sh, int Sw, int Qh, int Qw, int Hf, int Wf, int S,
              int nimg, bool pool, ResPlan &r)
{
    const int Q = Qh * Qw, HfWf = Hf * Wf;
    if (Q > kResNT * 4 * 16) return false;
    // the per-image buffer range and the chunk's soffset are 32-bit byte offsets
    // that must stay below the out-of-range marker
    if ((size_t)Cs * Sh * Sw * tsz >= 0x80000000ull) return false;
    if ((long long)nimg * ((M + kResRows - 1) / kResRows) < 128) return false;
    r.Wpad = (Qw - 1) * S + Wf;
    r.CH = ((Qh - 1) * S + Hf) * r.Wpad;
    const long long dpe = (long long)tsz / 4;
    int first = 0;
    for (int kc = Cs < 16 ? Cs : 16; kc >= 1; --kc) {
        const int kcv = kc * HfWf, kck = (kcv + 3) / 4 * 4;
        const int nchunk = (Cs + kc - 1) / kc;
        const long long nis = ((long long)kc * r.CH * dpe + kWave - 1) / kWave;
        if ((nis + kResWaves - 1) / kResWaves > kResMaxDma) continue;
        const long long sa = (long long)nchunk * kck + 2;  // 2 mod 4
        // + slack for the prefetch after a chunk's last step
        const long long lds_a = (kResRows * sa * (long long)tsz + 64 * (long long)tsz + 255) / 256 * 256;
        long long stage = nis * 256;
        // the stages also hold the k-half reduction and the pooling tile
        const long long need = std::max((long long)4 * kResNT * 4 * kWave,
                                        pool ? (long long)kResRows * Q : 0LL) * (long long)tsz;
        if (2 * stage < need) stage = (need / 2 + 255) / 256 * 256;
        const long long total = lds_a + 2 * stage;
        if (total > 160 * 1024) continue;
        // the largest chunk that fits, unless one at least half as large has no
        // padded k-steps: then the largest such
        const bool exact = kck == kcv;
        if (first && !(exact && 2 * kc >= first)) continue;
        r.KC = kc;
        r.KCK = kck;
        r.SA = (int)sa;
        r.lds_a = (int)lds_a;
        r.stage = (int)stage;
        r.lds = (size_t)total;
        if (!first) first = kc;
        if (exact) break;
    }
    return first > 0;
}

// Geometry of one forward / backward_data launch (the GEMM view: M output rows,
// Cs source channels of Sh x Sw, Qh x Qw output pixels) and the fused forms it
// carries, as the kernel choice sees them.
struct ConvGeo {
    int M, Cs, Sh, Sw, Qh, Qw, Hf, Wf, S, nimg;
    bool pool;
    int PS;
    int csr, nbanks, require_dma, zero_skip;
    int pb;            // backward from a pooled source
    int pb_ps, pb_up;  // its pool stride; the stride up-sampling the gradient
};

// The kernel family a launch takes and its tiling.
struct ConvChoice {
    int kernel;   // ConvKernel
    Plan p, pd;   // tiling (register-staged kernel; pd: the LDS-DMA kernel's)
    DmaLayout L;  // LDS-DMA staging layout
    ResPlan rp;   // filter-resident forward
    int small_kc, small_CH, small_Wpad, small_MM;  // small-M kernel
    int k4, ksplit;                               // LDS-DMA in-block k split
    size_t lds;   // dynamic LDS per block
};

// Kernel selection for a forward or backward_data pass, host only (no device
// access): the small-M vector kernel for at most four output rows, the
// filter-resident forward for small fp64 images, else the LDS-DMA implicit
// GEMM, else the register-staged one.  hipErrorNotSupported when a fused form
// (pool epilogue, filter banks) needs the LDS-DMA kernel and the shape does
// not fit it; hipErrorInvalidValue when no tiling fits.
hipError_t choose_conv(size_t tsz, bool bwd, const ConvGeo &g, ConvChoice &c)
{
    c = ConvChoice{};
    const int HfWf = g.Hf * g.Wf, Q = g.Qh * g.Qw;
    if (g.M <= kSmallM && !g.pool && !g.csr && g.nbanks <= 1 && !g.require_dma) {
        const int kc = small_m_plan(tsz, g.M, g.Cs, g.Qw, Q, g.Hf, g.Wf, g.S, c.small_CH,
                                    c.small_Wpad);
        if (kc >= 1) {
            c.kernel = kConvSmallM;
            c.small_kc = kc;
            c.small_MM = g.M == 1 ? 1 : kSmallM;
            // the chunk buffers, or the final reduction ([4 waves][4 rows][64 pixels])
            c.lds = tsz * ((size_t)kc * c.small_CH + (size_t)kc * c.small_MM * HfWf);
            const size_t red = tsz * kSmallWaves * kSmallM * kSmallPix;
            if (c.lds < red) c.lds = red;
            return hipSuccess;
        }
    }
    // The filter-resident forward, fp64 only (in fp32 the 64-row tiles measured
    // faster on LeNet conv2: 40 against 43 us); it has no zero-skip form.
    if (!bwd && tsz == 8 && !g.csr && g.nbanks <= 1 && !g.zero_skip && g.M >= kResRows &&
        res_plan(tsz, g.M, g.Cs, g.Sh, g.Sw, g.Qh, g.Qw, g.Hf, g.Wf, g.S, g.nimg, g.pool, c.rp)) {
        c.kernel = kConvResident;
        c.lds = c.rp.lds;
        return hipSuccess;
    }
    if (!make_plan(tsz, g.M, g.Cs, g.Qw, Q, g.Hf, g.Wf, g.S, g.nimg, c.p,
                   g.pool ? g.Qw * g.PS : 0))
        return g.pool ? hipErrorNotSupported : hipErrorInvalidValue;
    const size_t img_bytes = (size_t)g.Cs * g.Sh * g.Sw * tsz;
    const size_t w_bytes = (size_t)g.M * g.Cs * HfWf * tsz;
    if (g.csr) c.p.pipelined = 0;  // sparse staging is the direct path only
    c.pd = c.p;
    // pooled source: the pool regions one channel of a staged window can meet
    // (its rows hold at most dr gradient rows)
    int pb_rpc = 0;
    if (bwd && g.pb) {
        const int dr = (c.p.CH / c.p.Wpad - 1) / g.pb_up + 1;
        pb_rpc = ((dr - 1) / g.pb_ps + 2) * ((g.Sw + g.pb_ps - 1) / g.pb_ps);
    }
    if (!g.csr && make_dma_plan(tsz, bwd, pb_rpc, g.M, g.Cs, HfWf, c.p.CH / c.p.Wpad,
                                c.p.Wpad, img_bytes, w_bytes, c.pd, c.L)) {
        c.kernel = kConvDma;
        // The smallest tiles (NB = 1: small layers with few blocks) split the
        // k-steps four ways so every wave has 4 or 8 independent MFMAs per step,
        // when a chunk has enough steps to share (12+) and enough rows (M > 16).
        // (LeNet conv2 forward, 13 steps a chunk: 64 -> 60 us against the 2 x 2
        // wave form.)
        c.k4 = (c.pd.NB == 1 && c.pd.KCK >= 48 && g.M > 16) ? (g.M <= 32 ? 2 : 4) : 0;
        c.ksplit = !c.k4 && g.M <= 32;
        if (c.ksplit) {  // the partial-tile hand-over reuses the stages
            const size_t red = tsz * (size_t)2 * 2 * c.pd.NB * 4 * kWave;
            if (c.pd.lds < red) c.pd.lds = red;
        }
        if (c.k4) {  // so do the four partial tiles
            const size_t red = tsz * (size_t)4 * 64 * 32;
            if (c.pd.lds < red) c.pd.lds = red;
        }
        if (g.pool) {  // so does the pooling tile (32 rows x 32 NB)
            const size_t pt = tsz * (size_t)32 * 32 * c.pd.NB;
            if (c.pd.lds < pt) c.pd.lds = pt;
            if (c.pd.lds > (tsz == 4 ? kLdsPerBlock32 : kLdsPerBlock)) return hipErrorNotSupported;
        }
        c.lds = c.pd.lds;
        return hipSuccess;
    }
    if (g.pool || g.require_dma) return hipErrorNotSupported;  // fused epilogues: LDS-DMA only
    c.kernel = kConvReg;
    c.lds = c.p.lds;
    return hipSuccess;
}

template <typename T, bool BWD>
hipError_t launch_typed(IgemmArgs a, int M, int Cs, int Qh, int Qw, int nimg, int zero_skip,
                        hipStream_t s)
{
    a.M = M;
    a.Cs = Cs;
    a.Qw = Qw;
    a.Q = Qh * Qw;
    a.HfWf = a.Hf * a.Wf;
    const bool pool = !BWD && a.pool_out;
    ConvGeo g = {M, Cs, a.Sh, a.Sw, Qh, Qw, a.Hf, a.Wf, a.S, nimg, pool, a.PS, a.csr,
                 a.nbanks, a.require_dma, zero_skip, a.pb, a.pool.PS, a.up};
    ConvChoice c;
    const hipError_t ce = choose_conv(sizeof(T), BWD, g, c);
    if (ce != hipSuccess) return ce;
    if (c.kernel == kConvSmallM) {
        a.KC = c.small_kc;
        a.CH = c.small_CH;
        a.Wpad = c.small_Wpad;
        auto pick = [&](auto mm, auto pbc) {
            constexpr int MM = decltype(mm)::value;
            constexpr bool PBV = decltype(pbc)::value;
            return a.Wf == 3 ? conv_small_m_kernel<T, BWD, 3, MM, PBV>
                             : (a.Wf == 5 ? conv_small_m_kernel<T, BWD, 5, MM, PBV>
                                          : conv_small_m_kernel<T, BWD, 0, MM, PBV>);
        };
        auto pick_pb = [&](auto mm) {
            if constexpr (BWD)
                if (a.pb) return pick(mm, std::true_type());
            return pick(mm, std::false_type());
        };
        auto k = M == 1 ? pick_pb(std::integral_constant<int, 1>())
                        : pick_pb(std::integral_constant<int, kSmallM>());
        hipError_t e = allow_dynamic_lds(k, c.lds);
        if (e != hipSuccess) return e;
        dim3 grid((a.Q + kSmallPix - 1) / kSmallPix, nimg);
        hipLaunchKernelGGL(k, grid, dim3(kSmallPix * kSmallWaves), c.lds, s, a);
        return hipGetLastError();
    }
    if constexpr (!BWD && sizeof(T) == 8) {
        if (c.kernel == kConvResident) {
            const ResPlan &rp = c.rp;
            a.KC = rp.KC;
            a.KCK = rp.KCK;
            a.SA = rp.SA;
            a.Wpad = rp.Wpad;
            a.CH = rp.CH;
            a.magic_hw = host_magic(a.HfWf);
            a.magic_wf = host_magic(a.Wf);
            a.magic_qw = host_magic(Qw);
            auto k = pool ? conv_resident_kernel<T, true> : conv_resident_kernel<T, false>;
            hipError_t e = allow_dynamic_lds(k, rp.lds);
            if (e != hipSuccess) return e;
            dim3 grid(nimg, (M + kResRows - 1) / kResRows);
            hipLaunchKernelGGL(k, grid, dim3(kResThreads), rp.lds, s, a, rp.lds_a, rp.stage);
            return hipGetLastError();
        }
    }
    if (c.kernel == kConvResident) return hipErrorInvalidValue;  // not reached
    const Plan &p = c.p;
    a.tiles_per_img = p.tiles_per_img;
    a.TS = p.TS;
    a.KC = p.KC;
    a.KCK = p.KCK;
    a.Wpad = p.Wpad;
    a.CH = p.CH;
    a.SA = p.SA;
    a.pipelined = p.pipelined;
    a.magic_kck = host_magic(p.KCK);
    a.magic_hw = host_magic(a.HfWf);
    a.magic_wf = host_magic(a.Wf);
    if (c.kernel == kConvDma) {
        const Plan &pd = c.pd;
        const unsigned w_bytes = (unsigned)((size_t)M * Cs * a.HfWf * sizeof(T));
        IgemmArgs ad = a;
        ad.KC = pd.KC;
        ad.KCK = pd.KCK;
        ad.SA = pd.SA;
        ad.magic_wpad = host_magic(pd.Wpad);
        ad.magic_sa = host_magic(pd.SA);
        ad.magic_qw = host_magic(Qw);
        ad.k4 = c.k4;
        ad.ksplit = c.ksplit;
        switch (pd.NB) {
        case 7: return launch_dma<T, 7, BWD>(ad, pd, c.L, w_bytes, nimg, zero_skip, s);
        case 4: return launch_dma<T, 4, BWD>(ad, pd, c.L, w_bytes, nimg, zero_skip, s);
        case 2: return launch_dma<T, 2, BWD>(ad, pd, c.L, w_bytes, nimg, zero_skip, s);
        default: return launch_dma<T, 1, BWD>(ad, pd, c.L, w_bytes, nimg, zero_skip, s);
        }
    }
    switch (p.NB) {
    case 7: return launch_nb<T, 7, BWD>(a, p, nimg, zero_skip, s);
    case 4: return launch_nb<T, 4, BWD>(a, p, nimg, zero_skip, s);
    case 2: return launch_nb<T, 2, BWD>(a, p, nimg, zero_skip, s);
    default: return launch_nb<T, 1, BWD>(a, p, nimg, zero_skip, s);
    }
}

}  // namespace

hipError_t conv_plan_info(int dtype, int pass, const ConvDims &d, int zero_skip, int form,
                          int ph, int pw, int ps, int pp, ConvPlanInfo &info)
{
    info = ConvPlanInfo{};
    if (pass == 1) return wgrad_plan_info(dtype, d, form == kFormPooledSource ? ps : 0, info);
    const size_t tsz = dtype == 0 ? sizeof(double) : sizeof(float);
    const bool bwd = pass == 2;
    // backward_data is the same GEMM over the up-sampled gradient: M = C rows,
    // F source channels of Hout x Wout, Hin x Win output pixels, stride 1
    ConvGeo g = bwd ? ConvGeo{d.C, d.F, d.Hout, d.Wout, d.Hin, d.Win, d.Hf, d.Wf, 1, d.N,
                              false, 0, 0, 0, 0, zero_skip, 0, 0, 1}
                    : ConvGeo{d.F, d.C, d.Hin, d.Win, d.Hout, d.Wout, d.Hf, d.Wf, d.stride,
                              d.N, false, 0, 0, 0, 0, zero_skip, 0, 0, 1};
    // the fused forms as their calls set them up (the pool form fuses only
    // unpadded pools whose stride is at least the window height; the calls fall
    // back to the plain kernels when the fused kernel does not fit)
    bool applied = true;
    if (!bwd && form == kFormPoolEpilogue && pp == 0 && ps >= ph) {
        g.pool = true;
        g.PS = ps;
    } else if (!bwd && form == kFormBanks) {
        g.nbanks = 2;
        g.require_dma = 1;
    } else if (!bwd && form == kFormCsr) {
        g.csr = 1;
    } else if (bwd && form == kFormPooledSource) {
        g.pb = 1;
        g.pb_ps = ps;
        g.pb_up = d.stride;
        g.zero_skip = 0;
    } else {
        applied = false;
    }
    (void)pw;
    ConvChoice c;
    hipError_t e = choose_conv(tsz, bwd, g, c);
    info.fused = applied && e == hipSuccess;
    if (e == hipErrorNotSupported && (g.pool || g.nbanks > 1)) {
        g.pool = false;
        g.nbanks = 0;
        g.require_dma = 0;
        e = choose_conv(tsz, bwd, g, c);
    }
    if (e != hipSuccess) return e;
    const int Q = g.Qh * g.Qw;
    info.kernel = c.kernel;
    info.lds = c.lds;
    info.k_split = 1;
    switch (c.kernel) {
    case kConvSmallM:
        info.tile_m = c.small_MM;
        info.tile_pixels = kSmallPix;
        info.tile_stride = kSmallPix;
        info.blocks = (Q + kSmallPix - 1) / kSmallPix * d.N;
        info.chunk = c.small_kc;
        info.window_width = c.small_Wpad;
        info.window_rows = c.small_CH / c.small_Wpad;
        break;
    case kConvResident:
        info.tile_m = kResRows;
        info.tile_pixels = Q;
        info.blocks = d.N * ((g.M + kResRows - 1) / kResRows);
        info.chunk = c.rp.KC;
        info.k_split = kResKs;
        info.window_width = c.rp.Wpad;
        info.window_rows = c.rp.CH / c.rp.Wpad;
        info.tile_stride = Q;
        info.k_chunk = c.rp.KCK;
        info.slice_stride = c.rp.SA;
        info.stage_bytes = c.rp.stage;
        info.slice_bytes = c.rp.lds_a;
        break;
    default: {
        const Plan &p = c.kernel == kConvDma ? c.pd : c.p;
        info.tile_m = kBM;
        info.tile_pixels = 32 * p.NB;
        info.blocks = d.N * p.tiles_per_img * p.m_tiles;
        info.chunk = p.KC;
        info.k_split = c.k4 ? 4 : (c.ksplit ? 2 : 1);
        info.window_width = p.Wpad;
        info.window_rows = p.CH / p.Wpad;
        info.tile_stride = p.TS;
        info.k_chunk = p.KCK;
        info.slice_stride = p.SA;
        info.pipelined = c.kernel == kConvReg ? p.pipelined : 0;
        if (c.kernel == kConvDma) {
            info.stage_bytes = c.L.stage_bytes;
            info.window_bytes = c.L.src_bytes;
            info.slice_bytes = c.L.a_bytes;
            info.slice_vec = c.L.a_vec;
        }
    }
    }
    return hipSuccess;
}

hipError_t launch_conv_forward(int dtype, const void *X, const void *W, const void *b, void *out,
                               const ConvDims &d, int relu, int zero_skip, hipStream_t s)
{
    IgemmArgs a = {};
    a.src = X;
    a.mask = nullptr;
    a.wgt = W;
    a.bias = b;
    a.out = out;
    a.Sh = d.Hin;
    a.Sw = d.Win;
    a.up = 1;
    a.Hf = d.Hf;
    a.Wf = d.Wf;
    a.S = d.stride;
    a.Ph = d.pad;
    a.Pw = d.pad;
    a.relu = relu;
    if (dtype == 0)
        return launch_typed<double, false>(a, d.F, d.C, d.Hout, d.Wout, d.N, zero_skip, s);
    return launch_typed<float, false>(a, d.F, d.C, d.Hout, d.Wout, d.N, zero_skip, s);
}

hipError_t launch_conv_forward_pool(int dtype, const void *X, const void *W, const void *b,
                                    void *out, void *pooled, int32_t *argmax, const ConvDims &d,
                                    int relu, int ph, int pw, int ps, int Hp, int Wp,
                                    int zero_skip, hipStream_t s)
{
    // Fused only when every pooled window lies inside one tile of whole rows:
    // no pool padding and a stride no smaller than the window height.
    if (ps < ph) return hipErrorNotSupported;
    IgemmArgs a = {};
    a.src = X;
    a.mask = nullptr;
    a.wgt = W;
    a.bias = b;
    a.out = out;
    a.Sh = d.Hin;
    a.Sw = d.Win;
    a.up = 1;
    a.Hf = d.Hf;
    a.Wf = d.Wf;
    a.S = d.stride;
    a.Ph = d.pad;
    a.Pw = d.pad;
    a.relu = relu;
    a.pool_out = pooled;
    a.pool_idx = argmax;
    a.PH = ph;
    a.PW = pw;
    a.PS = ps;
    a.Hp = Hp;
    a.Wp = Wp;
    if (dtype == 0)
        return launch_typed<double, false>(a, d.F, d.C, d.Hout, d.Wout, d.N, zero_skip, s);
    return launch_typed<float, false>(a, d.F, d.C, d.Hout, d.Wout, d.N, zero_skip, s);
}

hipError_t launch_conv_forward_multi(int dtype, const void *X, const void *Wcat,
                                     const void *bcat, void *const *outs, const int *Fs,
                                     int nbanks, const ConvDims &d, int relu, int zero_skip,
                                     hipStream_t s)
{
    if (nbanks < 1 || nbanks > kMaxBanks) return hipErrorInvalidValue;
    IgemmArgs a = {};
    a.src = X;
    a.mask = nullptr;
    a.wgt = Wcat;
    a.bias = bcat;
    a.out = outs[0];
    a.Sh = d.Hin;
    a.Sw = d.Win;
    a.up = 1;
    a.Hf = d.Hf;
    a.Wf = d.Wf;
    a.S = d.stride;
    a.Ph = d.pad;
    a.Pw = d.pad;
    a.relu = relu;
    a.nbanks = nbanks;
    a.bank_off[0] = 0;
    for (int b = 0; b < nbanks; ++b) {
        a.bank_off[b + 1] = a.bank_off[b] + Fs[b];
        a.bank_out[b] = outs[b];
    }
    a.require_dma = 1;
    const int M = a.bank_off[nbanks];
    if (dtype == 0) return launch_typed<double, false>(a, M, d.C, d.Hout, d.Wout, d.N, zero_skip, s);
    return launch_typed<float, false>(a, M, d.C, d.Hout, d.Wout, d.N, zero_skip, s);
}

namespace {
// row_index[i] for image row i = (n, c, y): the first position of CSR row n whose
// column is >= c*Hin*Win + y*Win (binary search within the row's range, which is
// clamped to [0, nnz], so any rowptr keeps every read in bounds).
__global__ __launch_bounds__(256) void csr_row_index_kernel(const int32_t *rowptr,
                                                            const int32_t *colidx, int nnz,
                                                            int32_t *row_index, int N, int C,
                                                            int Hin, int Win)
{
    const long long total = (long long)N * C * Hin;
    for (long long i = (long long)blockIdx.x * 256 + threadIdx.x; i <= total;
         i += (long long)gridDim.x * 256) {
        if (i == total) {
            row_index[i] = min(max(rowptr[N], 0), nnz);
            continue;
        }
        const int n = (int)(i / ((long long)C * Hin));
        const int cy = (int)(i - (long long)n * C * Hin);  // c*Hin + y
        int lo = min(max(rowptr[n], 0), nnz);
        int hi = min(max(rowptr[n + 1], lo), nnz);
        const int key = cy * Win;
        while (lo < hi) {
            const int mid = lo + (hi - lo) / 2;
            if (colidx[mid] < key)
                lo = mid + 1;
            else
                hi = mid;
        }
        row_index[i] = lo;
    }
}
}  // namespace

hipError_t launch_conv_forward_csr(int dtype, const int32_t *rowptr, const int32_t *colidx,
                                   const void *vals, int nnz, int32_t *row_index, const void *W,
                                   const void *b, void *out, const ConvDims &d, int relu,
                                   int zero_skip, hipStream_t s)
{
    const long long rows = (long long)d.N * d.C * d.Hin + 1;
    long long g = (rows + 255) / 256;
    if (g > 4096) g = 4096;
    hipLaunchKernelGGL(csr_row_index_kernel, dim3((int)g), dim3(256), 0, s, rowptr, colidx, nnz,
                       row_index, d.N, d.C, d.Hin, d.Win);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    IgemmArgs a = {};
    a.src = nullptr;  // not read: the staging takes the CSR arrays
    a.wgt = W;
    a.bias = b;
    a.out = out;
    a.Sh = d.Hin;
    a.Sw = d.Win;
    a.up = 1;
    a.Hf = d.Hf;
    a.Wf = d.Wf;
    a.S = d.stride;
    a.Ph = d.pad;
    a.Pw = d.pad;
    a.relu = relu;
    a.csr = 1;
    a.csr_row = row_index;
    a.csr_col = colidx;
    a.csr_val = vals;
    if (dtype == 0)
        return launch_typed<double, false>(a, d.F, d.C, d.Hout, d.Wout, d.N, zero_skip, s);
    return launch_typed<float, false>(a, d.F, d.C, d.Hout, d.Wout, d.N, zero_skip, s);
}

hipError_t launch_conv_backward_data(int dtype, const void *W, const void *dout,
                                     const void *out_fwd, void *dX, const ConvDims &d,
                                     int zero_skip, hipStream_t s, const PoolSrc *pool)
{
    IgemmArgs a = {};
    a.src = dout;
    a.mask = out_fwd;
    if (pool) {
        a.pb = 1;
        a.pool = *pool;
        a.src = pool->dpool;
        a.mask = nullptr;
        zero_skip = 0;
    }
    a.wgt = W;
    a.bias = nullptr;
    a.out = dX;
    a.Sh = d.Hout;
    a.Sw = d.Wout;
    a.up = d.stride;
    a.Hf = d.Hf;
    a.Wf = d.Wf;
    a.S = 1;
    a.Ph = d.Hf - 1 - d.pad;  // full correlation: the flipped filter's pad per axis
    a.Pw = d.Wf - 1 - d.pad;
    a.relu = 0;
    if (dtype == 0)
        return launch_typed<double, true>(a, d.C, d.F, d.Hin, d.Win, d.N, zero_skip, s);
    return launch_typed<float, true>(a, d.C, d.F, d.Hin, d.Win, d.N, zero_skip, s);
}

}  // namespace dmlnn
