// affine forward/backward (paper, Section 2: the affine layer is the matrix
// product of the inputs with the weights plus a broadcast bias row, and its
// backward returns the input, weight and bias gradients in that order) on the
// gfx950 matrix cores.
//
// One strided GEMM kernel serves all three products:
//   forward  out = X W + b        (A = X,        B = W)
//   dX = g W^T                    (A = g,        B = W viewed transposed)
//   dW = X^T g                    (A = X viewed transposed, B = g)
// where g = dout masked to out_fwd > 0 when a relu mask is given.  A block
// owns a 16 x 16 output tile and up to 16 waves that split K (one MFMA per
// 4-deep k-step); their partial tiles are added in wave order
// (deterministic).  Column sums of g (db) use a separate fixed-order kernel.
#include "common.hpp"
#include "internal.hpp"

namespace dmlnn {
namespace {

constexpr int kTJ = 16;      // output tile columns
constexpr int kMaxKW = 16;   // waves splitting K inside a block

struct GemmArgs {
    const void *A, *Amask;  // A(i,k) = A[i*sAm + k*sAk]; mask has the same strides
    const void *B, *Bmask;  // B(k,j) = B[k*sBk + j*sBn]
    const void *bias;       // per column j, or null
    void *C;                // C[i*ldc + j]
    long long sAm, sAk, sBk, sBn, ldc;
    int M, N, K, relu;
    int kw_len;             // k per wave (a multiple of 16)
};

// A block owns a 16 x 16 output tile; its waves split K into contiguous
// ranges of kw_len (a multiple of 16) and read their MFMA fragments straight
// from global memory (the products here have at most a few MB of operands,
// which stay in L2).
//
// k is walked in groups of 16 (four MFMA k-steps).  Inside a group the k
// order is permuted so that an operand stored with k contiguous (X for the
// forward product, g and W for dX) is read with 16-byte vector loads: lane
// quarter q holds k = 2q, 2q+1, 8+2q, 9+2q of the group in its four steps
// (fp64; for fp32 k = 4q..4q+3).  Each step still covers four distinct k, the
// four steps cover the group, and both operands use the same order, so the
// products are unchanged.  A 16-row fragment then reads 64 contiguous bytes
// per row per load instead of 32, which halves the L1 cache accesses that
// bound these loads.  Operands with rows contiguous keep per-step loads.
//
// These products are small, so a wave's time is load latency: groups are
// loaded two at a time, one batch ahead (two register sets), so one batch's
// loads are in flight while the previous batch's MFMAs issue.  Rows and
// columns past the matrix edge read a clamped (valid) row or column; they only
// feed outputs that are not stored.  A partial last group (K not a multiple
// of 16) reads clamped k and zeroes B past the range.  A relu mask is loaded
// beside its operand and applied just before the MFMA.  The per-wave partial
// tiles are added in wave order (deterministic).
template <typename T>
struct GemmFrag {
    // position in the group of k-step u for lane quarter q
    static __device__ __forceinline__ int kpos(int q, int u)
    {
        if (sizeof(T) == 8) return (u & 1) + 2 * q + 8 * (u >> 1);
        return 4 * q + u;
    }
    // the four values of a k-contiguous row at group start p (16-byte aligned)
    static __device__ __forceinline__ void vload(const T *p, int q, T (&v)[4])
    {
        if constexpr (sizeof(T) == 8) {
            const double2 lo = *reinterpret_cast<const double2 *>(p + 2 * q);
            const double2 hi = *reinterpret_cast<const double2 *>(p + 8 + 2 * q);
            v[0] = lo.x;
            v[1] = lo.y;
            v[2] = hi.x;
            v[3] = hi.y;
        } else {
            const float4 x = *reinterpret_cast<const float4 *>(p + 4 * q);
            v[0] = x.x;
            v[1] = x.y;
            v[2] = x.z;
            v[3] = x.w;
        }
    }
};

// Waves per block at most: the masked fp64 forms hold two register sets of
// operands and masks, more than the 128 registers a 16-wave block leaves.
template <typename T, bool MA, bool MB>
constexpr int gemm_max_waves() { return (sizeof(T) == 8 && (MA || MB)) ? 8 : kMaxKW; }

template <typename T, bool MA, bool MB, bool VA, bool VB>
__global__ __launch_bounds__((gemm_max_waves<T, MA, MB>() * kWave)) void gemm_kernel(GemmArgs g)
{
    using MF = Mfma<T>;
    using FR = GemmFrag<T>;
    extern __shared__ __align__(16) unsigned char smem[];
    T *s_red = reinterpret_cast<T *>(smem);  // [wave][16 * kTJ]

    const int tid = threadIdx.x, lane = lane_id(), wave = wave_id();
    const int nw = blockDim.x / kWave;
    // Blocks are dealt to the 8 XCDs round-robin (block b to XCD b mod 8), and
    // each XCD has its own L2.  Tile t = (ti, tj), ti fastest, is renumbered so
    // that every XCD owns a contiguous run of tiles: the row tiles of a column
    // strip then share one L2 copy of that strip of B (for the LeNet products
    // B is a 12.8 MB weight matrix, larger than one L2).
    const int ntile = gridDim.x * gridDim.y, bl = blockIdx.x + gridDim.x * blockIdx.y;
    const int per = ntile / 8, rem = ntile % 8, xcd = bl % 8;
    const int t = xcd * per + min(xcd, rem) + bl / 8;
    const int i0 = (t % gridDim.x) * 16, j0 = (t / gridDim.x) * kTJ;
    const int kbeg = wave * g.kw_len, kend = min(g.K, kbeg + g.kw_len);
    const int ngrp = kend > kbeg ? (kend - kbeg + 15) / 16 : 0;
    const bool ragged = ((kend - kbeg) & 15) != 0;  // the last group is partial
    const T *A = reinterpret_cast<const T *>(g.A);
    const T *Am = reinterpret_cast<const T *>(g.Amask);
    const T *B = reinterpret_cast<const T *>(g.B);
    const T *Bm = reinterpret_cast<const T *>(g.Bmask);
    const int li = lane & 15, q = lane >> 4;
    const long long arow = (long long)min(i0 + li, g.M - 1) * g.sAm;
    const long long bcol = (long long)min(j0 + li, g.N - 1) * g.sBn;

    struct Grp {
        T a[4], b[4];
        T am[4], bm[4];  // used only with a mask (MA / MB)
    };
    // one group of 16 k from k0; `part`: the wave's partial last group
    auto load_grp = [&](int k0, bool part, Grp &f) {
        if (part) {
#pragma unroll
            for (int u = 0; u < 4; ++u) {
                const int k = k0 + FR::kpos(q, u), kc = min(k, kend - 1);
                const long long oa = arow + (long long)kc * g.sAk;
                const long long ob = (long long)kc * g.sBk + bcol;
                f.a[u] = A[oa];
                if (MA) f.am[u] = Am[oa];
                const T bv = B[ob];
                f.b[u] = k < kend ? bv : T(0);
                if (MB) f.bm[u] = Bm[ob];
            }
            return;
        }
        if constexpr (VA) {
            FR::vload(A + arow + k0, q, f.a);
            if constexpr (MA) FR::vload(Am + arow + k0, q, f.am);
        } else {
#pragma unroll
            for (int u = 0; u < 4; ++u) {
                const long long oa = arow + (long long)(k0 + FR::kpos(q, u)) * g.sAk;
                f.a[u] = A[oa];
                if (MA) f.am[u] = Am[oa];
            }
        }
        if constexpr (VB) {
            FR::vload(B + bcol + k0, q, f.b);
            if constexpr (MB) FR::vload(Bm + bcol + k0, q, f.bm);
        } else {
#pragma unroll
            for (int u = 0; u < 4; ++u) {
                const long long ob = (long long)(k0 + FR::kpos(q, u)) * g.sBk + bcol;
                f.b[u] = B[ob];
                if (MB) f.bm[u] = Bm[ob];
            }
        }
    };
    typename MF::acc_t acc = MF::zero();
    auto mma_grp = [&](const Grp &f) {
#pragma unroll
        for (int u = 0; u < 4; ++u) {
            const T av = MA ? (f.am[u] > T(0) ? f.a[u] : T(0)) : f.a[u];
            const T bv = MB ? (f.bm[u] > T(0) ? f.b[u] : T(0)) : f.b[u];
            acc = MF::mma(av, bv, acc);
        }
    };
    // batch b = groups 2b and 2b + 1 (the second may not exist)
    auto load_batch = [&](int b, Grp (&f)[2]) {
        const int g0 = 2 * b;
        load_grp(kbeg + 16 * g0, ragged && g0 == ngrp - 1, f[0]);
        if (g0 + 1 < ngrp) load_grp(kbeg + 16 * g0 + 16, ragged && g0 + 1 == ngrp - 1, f[1]);
    };
    auto mma_batch = [&](int b, const Grp (&f)[2]) {
        mma_grp(f[0]);
        if (2 * b + 1 < ngrp) mma_grp(f[1]);
    };
    const int nbatch = (ngrp + 1) / 2;
    Grp f0[2], f1[2];
    if (nbatch > 0) load_batch(0, f0);
    int i = 0;
    for (; i + 1 < nbatch; i += 2) {
        load_batch(i + 1, f1);
        mma_batch(i, f0);
        if (i + 2 < nbatch) load_batch(i + 2, f0);
        mma_batch(i + 1, f1);
    }
    if (i < nbatch) mma_batch(i, f0);

    T *C = reinterpret_cast<T *>(g.C);
    const T *bias = reinterpret_cast<const T *>(g.bias);
    if (nw == 1) {  // one wave: no partial tiles to add
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            const int ii = i0 + MF::row(lane, r), j = j0 + li;
            if (ii < g.M && j < g.N) {
                T v = acc[r];
                if (bias) v += bias[j];
                C[(long long)ii * g.ldc + j] = relu_if(v, g.relu);
            }
        }
        return;
    }
#pragma unroll
    for (int r = 0; r < 4; ++r) s_red[wave * 16 * kTJ + MF::row(lane, r) * kTJ + li] = acc[r];
    __syncthreads();
    for (int e = tid; e < 16 * kTJ; e += blockDim.x) {
        const int ii = i0 + e / kTJ, j = j0 + e % kTJ;
        if (ii < g.M && j < g.N) {
            T v = s_red[e];
            for (int w = 1; w < nw; ++w) v += s_red[w * 16 * kTJ + e];
            if (bias) v += bias[j];
            C[(long long)ii * g.ldc + j] = relu_if(v, g.relu);
        }
    }
}

// Products with a moderate K and many columns (the LeNet dX = g W^T: 64 x 3136
// from K = 512): the 16 x K strip of A (masked) is staged in LDS once per
// block, and the block's four waves each stream their own 16 columns of B
// over the whole K.  Splitting K across waves instead (above) makes every
// 16-column tile re-read A and its mask from L2: for dX that is 100 MB of
// 32-byte row pieces, and the L1 throughput on those pieces bounds the time.
// k is walked in the same permuted 16-groups as above (A from LDS at the
// permuted positions, B with 16-byte loads when k-contiguous), four groups
// per batch, loaded one batch ahead.  Each column block has two waves, one
// per half of the k groups, so twice as many B loads are in flight per CU
// (the product has too few tiles for more than one block per CU); the second
// half's partial tile is added to the first's through LDS (fixed order).
constexpr int kLdsACols = 4;                 // 16-column blocks per block
constexpr int kLdsAWaves = 2 * kLdsACols;    // two k halves each
constexpr int kLdsAMaxK = 1024;

template <typename T, bool MA, bool VB>
__global__ __launch_bounds__(kLdsAWaves * kWave) void gemm_lds_a_kernel(GemmArgs g)
{
    using MF = Mfma<T>;
    using FR = GemmFrag<T>;
    extern __shared__ __align__(16) unsigned char smem[];
    T *s_a = reinterpret_cast<T *>(smem);  // [16][SK], k past K zero

    const int tid = threadIdx.x, lane = lane_id(), wave = wave_id();
    const int ntile = gridDim.x * gridDim.y, bl = blockIdx.x + gridDim.x * blockIdx.y;
    const int per = ntile / 8, rem = ntile % 8, xcd = bl % 8;
    const int t = xcd * per + min(xcd, rem) + bl / 8;
    const int i0 = (t % gridDim.x) * 16;
    const int cb = wave % kLdsACols, kh = wave / kLdsACols;  // column block, k half
    const int j0 = (t / gridDim.x) * (16 * kLdsACols) + 16 * cb;
    const int K16 = (g.K + 15) / 16 * 16;
    const int SK = K16 + 2;  // 2 mod 4
    const T *A = reinterpret_cast<const T *>(g.A);
    const T *Am = reinterpret_cast<const T *>(g.Amask);
    const T *B = reinterpret_cast<const T *>(g.B);

    // Stage A: element (r, k) at s_a[r * SK + k].  With k contiguous in memory
    // consecutive threads take consecutive k, else consecutive rows.  Eight
    // branch-free loads per thread before any store (clamped rows and k).
    const bool kfast = g.sAk == 1;
    const int tot = 16 * K16;
    for (int base = 0; base < tot; base += 8 * kLdsAWaves * kWave) {
        T v[8], mv[8];
#pragma unroll
        for (int u = 0; u < 8; ++u) {
            const int e = min(base + u * kLdsAWaves * kWave + tid, tot - 1);
            const int r = kfast ? e / K16 : e % 16, k = kfast ? e % K16 : e / 16;
            const long long o = (long long)min(i0 + r, g.M - 1) * g.sAm +
                                (long long)min(k, g.K - 1) * g.sAk;
            v[u] = A[o];
            mv[u] = MA ? Am[o] : T(1);
        }
#pragma unroll
        for (int u = 0; u < 8; ++u) {
            const int e = base + u * kLdsAWaves * kWave + tid;
            if (e < tot) {
                const int r = kfast ? e / K16 : e % 16, k = kfast ? e % K16 : e / 16;
                s_a[r * SK + k] = (k < g.K && mv[u] > T(0)) ? v[u] : T(0);
            }
        }
    }
    __syncthreads();

    const int li = lane & 15, q = lane >> 4;
    const long long bcol = (long long)min(j0 + li, g.N - 1) * g.sBn;
    const T *arow = s_a + li * SK;
    constexpr int kG = 4;  // groups per batch
    // this wave's groups: [g_lo, g_hi) of the K16 / 16
    const int ngrp_all = K16 / 16, nh = (ngrp_all + 1) / 2;
    const int g_lo = kh ? nh : 0, g_hi = kh ? ngrp_all : nh;
    const int ngrp = g_hi - g_lo, nbatch = (ngrp + kG - 1) / kG;
    auto load_b = [&](int b, T (&f)[kG][4]) {
#pragma unroll
        for (int gg = 0; gg < kG; ++gg) {
            const int k0 = (g_lo + min(b * kG + gg, max(ngrp - 1, 0))) * 16;
            if (VB && k0 + 16 <= g.K) {
                FR::vload(B + bcol + k0, q, f[gg]);
            } else {
#pragma unroll
                for (int u = 0; u < 4; ++u) {
                    const int k = k0 + FR::kpos(q, u);
                    const T bv = B[(long long)min(k, g.K - 1) * g.sBk + bcol];
                    f[gg][u] = k < g.K ? bv : T(0);
                }
            }
        }
    };
    typename MF::acc_t acc = MF::zero();
    auto mma_b = [&](int b, const T (&f)[kG][4]) {
#pragma unroll
        for (int gg = 0; gg < kG; ++gg) {
            if (b * kG + gg >= ngrp) break;
            const int k0 = (g_lo + b * kG + gg) * 16;
#pragma unroll
            for (int u = 0; u < 4; ++u) acc = MF::mma(arow[k0 + FR::kpos(q, u)], f[gg][u], acc);
        }
    };
    T f0[kG][4], f1[kG][4];
    if (nbatch > 0) load_b(0, f0);
    int b = 0;
    for (; b + 1 < nbatch; b += 2) {
        load_b(b + 1, f1);
        mma_b(b, f0);
        if (b + 2 < nbatch) load_b(b + 2, f0);
        mma_b(b + 1, f1);
    }
    if (b < nbatch) mma_b(b, f0);

    // the second k half hands its partial tile to the first (past the A strip)
    T *s_red = s_a + 16 * SK;  // [kLdsACols][4][64]
    if (kh == 1)
#pragma unroll
        for (int r = 0; r < 4; ++r) s_red[(cb * 4 + r) * kWave + lane] = acc[r];
    __syncthreads();
    if (kh == 1) return;
#pragma unroll
    for (int r = 0; r < 4; ++r) acc[r] += s_red[(cb * 4 + r) * kWave + lane];

    T *C = reinterpret_cast<T *>(g.C);
    const T *bias = reinterpret_cast<const T *>(g.bias);
#pragma unroll
    for (int r = 0; r < 4; ++r) {
        const int ii = i0 + MF::row(lane, r), j = j0 + li;
        if (ii < g.M && j < g.N) {
            T v = acc[r];
            if (bias) v += bias[j];
            C[(long long)ii * g.ldc + j] = relu_if(v, g.relu);
        }
    }
}

// db[j] = sum_i g[i, j], g masked by out_fwd > 0 if given.  A block covers 16
// columns with 16 row phases each: thread (j, ph) sums rows ph, ph+16, ... in
// order, and the 16 phase sums are added in phase order (deterministic).
template <typename T>
__global__ __launch_bounds__(256) void colsum_kernel(const T *G, const T *mask, T *db, int N,
                                                     int M)
{
    __shared__ T s_part[16][17];
    const int jl = threadIdx.x & 15, ph = threadIdx.x >> 4;
    const int j = blockIdx.x * 16 + jl;
    T s = T(0);
    if (j < M)
        for (int i = ph; i < N; i += 16) {
            T v = G[(size_t)i * M + j];
            if (mask && !(mask[(size_t)i * M + j] > T(0))) v = T(0);
            s += v;
        }
    s_part[ph][jl] = s;
    __syncthreads();
    if (ph == 0 && j < M) {
        T t = s_part[0][jl];
        for (int q = 1; q < 16; ++q) t += s_part[q][jl];
        db[j] = t;
    }
}

// An operand takes the vector loads when k is contiguous and every row start
// is 16-byte aligned.
template <typename T>
bool vec_ok(const void *p, long long s_row, long long s_k)
{
    constexpr long long e = 16 / sizeof(T);  // elements per 16 bytes
    return s_k == 1 && s_row % e == 0 && reinterpret_cast<uintptr_t>(p) % 16 == 0;
}

template <typename T, bool MA, bool MB>
auto pick_gemm(bool va, bool vb)
{
    return va ? (vb ? gemm_kernel<T, MA, MB, true, true> : gemm_kernel<T, MA, MB, true, false>)
              : (vb ? gemm_kernel<T, MA, MB, false, true> : gemm_kernel<T, MA, MB, false, false>);
}

// Waves per block: enough that each walks about 16 k-steps (two batches), at
// most 16; the per-wave k range is a multiple of 16.
template <typename T>
hipError_t gemm(GemmArgs g, hipStream_t s)
{
    if (g.Amask && g.Bmask) return hipErrorInvalidValue;  // one masked operand at most
    // A strip in LDS: K up to 1024, no mask on B, and enough 16 x 64 tiles
    const long long tiles64 = (long long)((g.M + 15) / 16) * ((g.N + 63) / 64);
    if (!g.Bmask && g.K <= kLdsAMaxK && g.K >= 64 && tiles64 >= 128) {
        const bool vb = vec_ok<T>(g.B, g.sBn, g.sBk);
        auto k = g.Amask ? (vb ? gemm_lds_a_kernel<T, true, true> : gemm_lds_a_kernel<T, true, false>)
                         : (vb ? gemm_lds_a_kernel<T, false, true> : gemm_lds_a_kernel<T, false, false>);
        const size_t lds = sizeof(T) * (16 * ((size_t)(g.K + 15) / 16 * 16 + 2) +
                                         (size_t)kLdsACols * 4 * kWave);
        hipError_t e = allow_dynamic_lds(k, lds);
        if (e != hipSuccess) return e;
        dim3 grid((g.M + 15) / 16, (g.N + 16 * kLdsACols - 1) / (16 * kLdsACols));
        hipLaunchKernelGGL(k, grid, dim3(kLdsAWaves * kWave), lds, s, g);
        return hipGetLastError();
    }
    const int grps = (g.K + 15) / 16;
    const int max_w = g.Amask ? gemm_max_waves<T, true, false>()
                              : (g.Bmask ? gemm_max_waves<T, false, true>() : kMaxKW);
    int nw = (grps + 3) / 4;
    nw = nw < 1 ? 1 : (nw > max_w ? max_w : nw);
    g.kw_len = ((grps + nw - 1) / nw) * 16;
    const bool va = vec_ok<T>(g.A, g.sAm, g.sAk) && (!g.Amask || vec_ok<T>(g.Amask, g.sAm, g.sAk));
    const bool vb = vec_ok<T>(g.B, g.sBn, g.sBk) && (!g.Bmask || vec_ok<T>(g.Bmask, g.sBn, g.sBk));
    const size_t lds = nw > 1 ? (size_t)nw * 16 * kTJ * sizeof(T) : 0;
    auto k = g.Amask ? pick_gemm<T, true, false>(va, vb)
                     : (g.Bmask ? pick_gemm<T, false, true>(va, vb) : pick_gemm<T, false, false>(va, vb));
    hipError_t e = allow_dynamic_lds(k, lds);
    if (e != hipSuccess) return e;
    dim3 grid((g.M + 15) / 16, (g.N + kTJ - 1) / kTJ);
    hipLaunchKernelGGL(k, grid, dim3(nw * kWave), lds, s, g);
    return hipGetLastError();
}

}  // namespace

hipError_t launch_affine_fwd(int dtype, const void *X, const void *W, const void *b, void *out,
                             int N, int D, int M, int relu, hipStream_t s)
{
    GemmArgs g = {};
    g.A = X;
    g.sAm = D;
    g.sAk = 1;
    g.B = W;
    g.sBk = M;
    g.sBn = 1;
    g.bias = b;
    g.C = out;
    g.ldc = M;
    g.M = N;
    g.N = M;
    g.K = D;
    g.relu = relu;
    return dtype == 0 ? gemm<double>(g, s) : gemm<float>(g, s);
}

hipError_t launch_affine_bwd(int dtype, const void *dout, const void *X, const void *W,
                             const void *out_fwd, void *dX, void *dW, void *db, int N, int D,
                             int M, hipStream_t s)
{
    hipError_t e;
    if (dX) {  // dX[n, d] = sum_m g[n, m] W[d, m]
        GemmArgs g = {};
        g.A = dout;
        g.Amask = out_fwd;
        g.sAm = M;
        g.sAk = 1;
        g.B = W;
        g.sBk = 1;
        g.sBn = M;
        g.C = dX;
        g.ldc = D;
        g.M = N;
        g.N = D;
        g.K = M;
        e = dtype == 0 ? gemm<double>(g, s) : gemm<float>(g, s);
        if (e != hipSuccess) return e;
    }
    if (dW) {  // dW[d, m] = sum_n X[n, d] g[n, m]
        GemmArgs g = {};
        g.A = X;
        g.sAm = 1;
        g.sAk = D;
        g.B = dout;
        g.Bmask = out_fwd;
        g.sBk = M;
        g.sBn = 1;
        g.C = dW;
        g.ldc = M;
        g.M = D;
        g.N = M;
        g.K = N;
        e = dtype == 0 ? gemm<double>(g, s) : gemm<float>(g, s);
        if (e != hipSuccess) return e;
    }
    if (db) {
        dim3 grid((M + 15) / 16);
        if (dtype == 0)
            hipLaunchKernelGGL(colsum_kernel<double>, grid, dim3(256), 0, s, (const double *)dout,
                               (const double *)out_fwd, (double *)db, N, M);
        else
            hipLaunchKernelGGL(colsum_kernel<float>, grid, dim3(256), 0, s, (const float *)dout,
                               (const float *)out_fwd, (float *)db, N, M);
        return hipGetLastError();
    }
    return hipSuccess;
}

}  // namespace dmlnn
