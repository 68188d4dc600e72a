// affine forward/backward (paper, Section 2 listing: scores = X %*% W + b and
// [dX, dW, db] = affine::backward(...)) on the gfx950 matrix cores.
//
// One strided GEMM kernel serves all three products:
//   forward  out = X W + b        (A = X,        B = W)
//   dX = g W^T                    (A = g,        B = W viewed transposed)
//   dW = X^T g                    (A = X viewed transposed, B = g)
// where g = dout masked to out_fwd > 0 when a relu mask is given; the mask is
// applied as the operand is loaded.  A block owns a 16 x 16 output tile and up
// to 16 waves that split K (one MFMA per 4-deep k-step); their partial tiles
// are added in wave order (deterministic).  Column sums of g (db) use a
// separate fixed-order kernel.
#include <type_traits>

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
    int kw_len;             // k per wave (a multiple of 4)
};

// A block owns a (16 TM) x 16 output tile (each B fragment feeds TM MFMAs, so B
// is read once per 16 TM rows); its waves split K into contiguous ranges
// of kw_len and read their MFMA fragments straight from global memory (the
// products here have at most a few MB of operands, which stay in L2).  The
// per-wave partial tiles are added in wave order (deterministic).  Rows and
// columns past the matrix edge read a clamped (valid) row or column: they only
// feed outputs that are not stored.  The main loop takes whole batches of kU
// steps with no k test, so its loads issue back to back; the tail zeroes k
// past the wave's range.  MA / MB: A / B carries a relu mask.
template <typename T, bool MA, bool MB, int kTM>
__global__ __launch_bounds__(kMaxKW * kWave) void gemm_kernel(GemmArgs g)
{
    using MF = Mfma<T>;
    constexpr int kTI = 16 * kTM;
    constexpr int kU = kTM == 1 ? 8 : 4;  // 4-deep k-steps loaded before their MFMAs
    extern __shared__ __align__(16) unsigned char smem[];
    T *s_red = reinterpret_cast<T *>(smem);  // [wave][kTI * kTJ]

    const int tid = threadIdx.x, lane = lane_id(), wave = wave_id();
    const int nw = blockDim.x / kWave;
    const int i0 = blockIdx.x * kTI, j0 = blockIdx.y * kTJ;
    const int kbeg = wave * g.kw_len, kend = min(g.K, kbeg + g.kw_len);
    const T *A = reinterpret_cast<const T *>(g.A);
    const T *Am = reinterpret_cast<const T *>(g.Amask);
    const T *B = reinterpret_cast<const T *>(g.B);
    const T *Bm = reinterpret_cast<const T *>(g.Bmask);
    const int li = lane & 15, lk = lane >> 4;
    long long arow[kTM];
#pragma unroll
    for (int x = 0; x < kTM; ++x) arow[x] = (long long)min(i0 + 16 * x + li, g.M - 1) * g.sAm;
    const long long bcol = (long long)min(j0 + li, g.N - 1) * g.sBn;

    auto ldA = [&](int x, int k) -> T {
        const long long o = arow[x] + (long long)k * g.sAk;
        const T v = A[o];
        if (MA) return Am[o] > T(0) ? v : T(0);
        return v;
    };
    auto ldB = [&](int k) -> T {
        const long long o = (long long)k * g.sBk + bcol;
        const T v = B[o];
        if (MB) return Bm[o] > T(0) ? v : T(0);
        return v;
    };

    typename MF::acc_t acc[kTM];
#pragma unroll
    for (int x = 0; x < kTM; ++x) acc[x] = MF::zero();
    int kk = kbeg;
    for (; kk + 4 * kU <= kend; kk += 4 * kU) {
        T a[kU][kTM], b[kU];
#pragma unroll
        for (int u = 0; u < kU; ++u) {
#pragma unroll
            for (int x = 0; x < kTM; ++x) a[u][x] = ldA(x, kk + 4 * u + lk);
            b[u] = ldB(kk + 4 * u + lk);
        }
#pragma unroll
        for (int u = 0; u < kU; ++u)
#pragma unroll
            for (int x = 0; x < kTM; ++x) acc[x] = MF::mma(a[u][x], b[u], acc[x]);
    }
    for (; kk < kend; kk += 4) {
        const int k = kk + lk;
        const int kc = min(k, kend - 1);
        T b = ldB(kc);
        b = k < kend ? b : T(0);
#pragma unroll
        for (int x = 0; x < kTM; ++x) acc[x] = MF::mma(ldA(x, kc), b, acc[x]);
    }

#pragma unroll
    for (int x = 0; x < kTM; ++x)
#pragma unroll
        for (int r = 0; r < 4; ++r)
            s_red[wave * kTI * kTJ + (16 * x + MF::row(lane, r)) * kTJ + li] = acc[x][r];
    __syncthreads();
    T *C = reinterpret_cast<T *>(g.C);
    const T *bias = reinterpret_cast<const T *>(g.bias);
    for (int e = tid; e < kTI * kTJ; e += blockDim.x) {
        const int i = i0 + e / kTJ, j = j0 + e % kTJ;
        if (i < g.M && j < g.N) {
            T v = s_red[e];
            for (int w = 1; w < nw; ++w) v += s_red[w * kTI * kTJ + e];
            if (bias) v += bias[j];
            C[(long long)i * g.ldc + j] = relu_if(v, g.relu);
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

// Waves per block: about 128 k each, at most 16 (a power of two).
template <typename T>
hipError_t gemm(GemmArgs g, hipStream_t s)
{
    int nw = 1;
    while (nw < kMaxKW && 2 * nw * 128 <= g.K) nw <<= 1;
    g.kw_len = ((g.K + nw - 1) / nw + 3) / 4 * 4;
    // 64-row tiles when that still leaves at least 128 blocks, else 16-row tiles
    const bool tall = (long long)((g.M + 63) / 64) * ((g.N + kTJ - 1) / kTJ) >= 128;
    const int kTI = tall ? 64 : 16;
    const size_t lds = (size_t)nw * kTI * kTJ * sizeof(T);
    auto pick = [&](auto tm) {
        constexpr int TM = decltype(tm)::value;
        return g.Amask ? (g.Bmask ? gemm_kernel<T, true, true, TM> : gemm_kernel<T, true, false, TM>)
                       : (g.Bmask ? gemm_kernel<T, false, true, TM>
                                  : gemm_kernel<T, false, false, TM>);
    };
    auto k = tall ? pick(std::integral_constant<int, 4>()) : pick(std::integral_constant<int, 1>());
    hipError_t e = allow_dynamic_lds(k, lds);
    if (e != hipSuccess) return e;
    dim3 grid((g.M + kTI - 1) / kTI, (g.N + kTJ - 1) / kTJ);
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
    {  // dW[d, m] = sum_n X[n, d] g[n, m]
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
