// affine forward/backward (paper, Section 2 listing: scores = X %*% W + b and
// [dX, dW, db] = affine::backward(...)) on the gfx950 matrix cores.
//
// One strided GEMM kernel serves all three products:
//   forward  out = X W + b        (A = X,        B = W)
//   dX = g W^T                    (A = g,        B = W viewed transposed)
//   dW = X^T g                    (A = X viewed transposed, B = g)
// where g = dout masked to out_fwd > 0 when a relu mask is given; the mask is
// applied while the operand tile is staged.  A block owns a 32 x 32 output tile;
// its 4 waves each take every 4th 4-deep k-step of a staged K-chunk (2 x 2
// MFMAs per step), and the four partial tiles are added in wave order at the
// end (deterministic).  Column sums of g (db) use a separate fixed-order kernel.
#include "common.hpp"
#include "internal.hpp"

namespace dmlnn {
namespace {

constexpr int kThreads = 256;
constexpr int kT = 32;    // output tile edge
constexpr int kKC = 64;   // k per staged chunk

struct GemmArgs {
    const void *A, *Amask;  // A(i,k) = A[i*sAm + k*sAk]; mask has the same strides
    const void *B, *Bmask;  // B(k,j) = B[k*sBk + j*sBn]
    const void *bias;       // per column j, or null
    void *C;                // C[i*ldc + j]
    long long sAm, sAk, sBk, sBn, ldc;
    int M, N, K, relu;
};

template <typename T>
__global__ __launch_bounds__(kThreads) void gemm_kernel(GemmArgs g)
{
    using MF = Mfma<T>;
    // operand tiles during the K loop; the four per-wave partial tiles afterwards
    constexpr int kStage = kT * (kKC + 1) + kKC * (kT + 1);
    constexpr int kWords = kStage > 4 * kT * kT ? kStage : 4 * kT * kT;
    __shared__ T smem[kWords];
    T(*s_a)[kKC + 1] = reinterpret_cast<T(*)[kKC + 1]>(smem);
    T(*s_b)[kT + 1] = reinterpret_cast<T(*)[kT + 1]>(smem + kT * (kKC + 1));
    T(*s_red)[kT * kT] = reinterpret_cast<T(*)[kT * kT]>(smem);

    const int tid = threadIdx.x, lane = lane_id(), wave = wave_id();
    const int i0 = blockIdx.x * kT, j0 = blockIdx.y * kT;
    const T *A = reinterpret_cast<const T *>(g.A);
    const T *Am = reinterpret_cast<const T *>(g.Amask);
    const T *B = reinterpret_cast<const T *>(g.B);
    const T *Bm = reinterpret_cast<const T *>(g.Bmask);

    typename MF::acc_t acc[2][2];
#pragma unroll
    for (int x = 0; x < 2; ++x)
#pragma unroll
        for (int y = 0; y < 2; ++y) acc[x][y] = MF::zero();

    for (int k0 = 0; k0 < g.K; k0 += kKC) {
        __syncthreads();
        for (int e = tid; e < kT * kKC; e += kThreads) {
            // A tile: rows i, columns k (k fastest when A is k-contiguous)
            int r, c;
            if (g.sAk == 1) { r = e / kKC; c = e % kKC; } else { c = e / kT; r = e % kT; }
            int i = i0 + r, k = k0 + c;
            T v = T(0);
            if (i < g.M && k < g.K) {
                long long o = (long long)i * g.sAm + (long long)k * g.sAk;
                v = A[o];
                if (Am && !(Am[o] > T(0))) v = T(0);
            }
            s_a[r][c] = v;
        }
        for (int e = tid; e < kT * kKC; e += kThreads) {
            int r, c;  // r = k row, c = j column
            if (g.sBn == 1) { r = e / kT; c = e % kT; } else { c = e / kKC; r = e % kKC; }
            int k = k0 + r, j = j0 + c;
            T v = T(0);
            if (k < g.K && j < g.N) {
                long long o = (long long)k * g.sBk + (long long)j * g.sBn;
                v = B[o];
                if (Bm && !(Bm[o] > T(0))) v = T(0);
            }
            s_b[r][c] = v;
        }
        __syncthreads();
#pragma unroll
        for (int st = 0; st < kKC / 4 / 4; ++st) {
            const int kk = (st * 4 + wave) * 4 + (lane >> 4);
            T a0 = s_a[lane & 15][kk], a1 = s_a[16 + (lane & 15)][kk];
            T b0 = s_b[kk][lane & 15], b1 = s_b[kk][16 + (lane & 15)];
            acc[0][0] = MF::mma(a0, b0, acc[0][0]);
            acc[0][1] = MF::mma(a0, b1, acc[0][1]);
            acc[1][0] = MF::mma(a1, b0, acc[1][0]);
            acc[1][1] = MF::mma(a1, b1, acc[1][1]);
        }
    }

    __syncthreads();
#pragma unroll
    for (int x = 0; x < 2; ++x)
#pragma unroll
        for (int y = 0; y < 2; ++y)
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                int i = x * 16 + MF::row(lane, r), j = y * 16 + (lane & 15);
                s_red[wave][i * kT + j] = acc[x][y][r];
            }
    __syncthreads();
    T *C = reinterpret_cast<T *>(g.C);
    const T *bias = reinterpret_cast<const T *>(g.bias);
    for (int e = tid; e < kT * kT; e += kThreads) {
        int i = i0 + e / kT, j = j0 + e % kT;
        if (i < g.M && j < g.N) {
            T v = ((s_red[0][e] + s_red[1][e]) + s_red[2][e]) + s_red[3][e];
            if (bias) v += bias[j];
            C[(long long)i * g.ldc + j] = relu_if(v, g.relu);
        }
    }
}

// db[j] = sum_i g[i, j] (rows in order), g masked by out_fwd > 0 if given.
template <typename T>
__global__ __launch_bounds__(256) void colsum_kernel(const T *G, const T *mask, T *db, int N,
                                                     int M)
{
    const int j = blockIdx.x * 256 + threadIdx.x;
    if (j >= M) return;
    T s = T(0);
    for (int i = 0; i < N; ++i) {
        T v = G[(size_t)i * M + j];
        if (mask && !(mask[(size_t)i * M + j] > T(0))) v = T(0);
        s += v;
    }
    db[j] = s;
}

template <typename T>
hipError_t gemm(const GemmArgs &g, hipStream_t s)
{
    dim3 grid((g.M + kT - 1) / kT, (g.N + kT - 1) / kT);
    hipLaunchKernelGGL(gemm_kernel<T>, grid, dim3(kThreads), 0, s, g);
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
        dim3 grid((M + 255) / 256);
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
