// Fused softmax + cross-entropy forward and backward (paper, Section 2: the
// softmax classifier's training loop chains the softmax forward, the
// cross-entropy backward and the softmax backward; here the three are one pass
// whose result equals that chain).  Per row, with m = max_k s:
//   p = exp(s - m) / sum exp(s - m)
//   row loss = -sum_k y (s - m - log sum exp(s - m))
//   ds = (p * sum_k y - y) / N
// and loss = (1/N) * sum of row losses.  Blocks of 16 waves; lanes run across
// the K columns of a row with butterfly-shuffle reductions.  One block does the
// whole call, or (with a workspace) up to kSmMaxBlocks blocks each write their
// share of the loss to the workspace and a one-wave pass adds the shares.
#include "common.hpp"
#include "internal.hpp"

namespace dmlnn {
namespace {

// Rows are processed by lane segments of width sw (a power of two >= K, at most
// 64): a wave holds 64/sw rows at once and the waves of the grid (16 a block)
// take consecutive row groups.  Per-row losses are summed per segment in row
// order, then over (wave, segment) in order within a block, then over blocks in
// block order: the loss is deterministic for a given block count.
template <typename T>
__device__ __forceinline__ T seg_sum(T v, int sw)
{
    for (int off = sw >> 1; off > 0; off >>= 1) v += __shfl_xor(v, off, kWave);
    return v;
}

template <typename T>
__device__ __forceinline__ T seg_max(T v, int sw)
{
    for (int off = sw >> 1; off > 0; off >>= 1) {
        T o = __shfl_xor(v, off, kWave);
        v = o > v ? o : v;
    }
    return v;
}

constexpr int kSmThreads = 1024;
constexpr int kSmWaves = kSmThreads / kWave;
constexpr int kSmMaxBlocks = 2048;  // blocks of a call with a workspace (one loss share each)

// part: null (one block: the loss goes to *loss) or one element a block (the
// block's share of the sum of row losses, before the 1/N).
template <typename T>
__global__ __launch_bounds__(kSmThreads) void softmax_xent_kernel(const T *S, const T *Y, T *P,
                                                                  T *dS, T *loss, T *part, int N,
                                                                  int K, int sw)
{
    __shared__ T s_part[kSmThreads];
    const int lane = lane_id(), wave = wave_id();
    const int rpw = kWave / sw, seg = lane / sw, sl = lane - seg * sw;
    const int wave_g = blockIdx.x * kSmWaves + wave, nwaves = gridDim.x * kSmWaves;
    const T invN = T(1) / T(N);
    T total = T(0);
    if (K <= sw) {
        // At most one column per lane: s and y are loaded once, into registers,
        // and each exponential is taken once (the same values and reduction
        // order as the general loop below).
        for (int r0 = wave_g * rpw; r0 < N; r0 += nwaves * rpw) {
            const int n = r0 + seg;
            const bool ok = n < N && sl < K;
            const size_t o = ok ? (size_t)n * K + sl : 0;
            const T s0 = S[o], y0 = Y[o];
            const T sk = ok ? s0 : T(-INFINITY), yk = ok ? y0 : T(0);
            const T m = seg_max(sk, sw);
            const T e = ok ? exp(sk - m) : T(0);
            const T se = seg_sum(e, sw), ys = seg_sum(yk, sw);
            const T lse = m + log(se);
            const T rl = seg_sum(ok ? -(yk * (sk - lse)) : T(0), sw);
            if (ok) {
                const T p = e / se;
                if (P) P[o] = p;
                dS[o] = (p * ys - yk) * invN;
            }
            if (n < N) total += rl;
        }
    } else {
        for (int r0 = wave_g * rpw; r0 < N; r0 += nwaves * rpw) {
            const int n = r0 + seg;
            const bool ok = n < N;
            const T *s = S + (size_t)n * K;
            const T *y = Y + (size_t)n * K;
            T m = -INFINITY;
            if (ok)
                for (int k = sl; k < K; k += sw) m = s[k] > m ? s[k] : m;
            m = seg_max(m, sw);
            T se = T(0), ys = T(0);
            if (ok)
                for (int k = sl; k < K; k += sw) {
                    se += exp(s[k] - m);
                    ys += y[k];
                }
            se = seg_sum(se, sw);
            ys = seg_sum(ys, sw);
            const T lse = m + log(se);
            T rl = T(0);
            if (ok)
                for (int k = sl; k < K; k += sw) {
                    const T sk = s[k], yk = y[k];
                    const T p = exp(sk - m) / se;
                    if (P) P[(size_t)n * K + k] = p;
                    dS[(size_t)n * K + k] = (p * ys - yk) * invN;
                    rl -= yk * (sk - lse);
                }
            rl = seg_sum(rl, sw);
            if (ok) total += rl;
        }
    }
    s_part[threadIdx.x] = total;
    __syncthreads();
    if (threadIdx.x == 0) {
        // segment i (wave i / rpw, segment i % rpw) keeps its sum at s_part[i * sw];
        // the sums are added in segment order, read sixteen at a time so the
        // LDS reads overlap instead of each waiting for the previous add
        const int nseg = kSmWaves * rpw;
        T t = T(0);
        for (int i0 = 0; i0 < nseg; i0 += 16) {
            T v[16];
#pragma unroll
            for (int u = 0; u < 16; ++u) v[u] = s_part[min(i0 + u, nseg - 1) * sw];
#pragma unroll
            for (int u = 0; u < 16; ++u)
                if (i0 + u < nseg) t += v[u];
        }
        if (part)
            part[blockIdx.x] = t;
        else
            *loss = t * invN;
    }
}

// The loss from the blocks' shares: lane l adds shares l, l + 64, ... in order,
// then a fixed butterfly adds the 64 lane sums (lane 0 ends with the total).
template <typename T>
__global__ __launch_bounds__(kWave) void softmax_loss_reduce(const T *part, int G, T *loss, int N)
{
    const int lane = threadIdx.x;
    T t = T(0);
    for (int b = lane; b < G; b += kWave) t += part[b];
    for (int off = kWave / 2; off > 0; off >>= 1) t += __shfl_xor(t, off, kWave);
    if (lane == 0) *loss = t * (T(1) / T(N));
}

// Row-wise softmax alone (forward-only scoring): same segment layout, no loss.
template <typename T>
__global__ __launch_bounds__(kSmThreads) void softmax_kernel(const T *S, T *P, int N, int K, int sw)
{
    const int lane = lane_id(), wave = wave_id();
    const int rpw = kWave / sw, seg = lane / sw, sl = lane - seg * sw;
    const int wave_g = blockIdx.x * kSmWaves + wave, nwaves = gridDim.x * kSmWaves;
    if (K <= sw) {  // one column per lane at most, as in softmax_xent_kernel
        for (int r0 = wave_g * rpw; r0 < N; r0 += nwaves * rpw) {
            const int n = r0 + seg;
            const bool ok = n < N && sl < K;
            const size_t o = ok ? (size_t)n * K + sl : 0;
            const T s0 = S[o];
            const T sk = ok ? s0 : T(-INFINITY);
            const T m = seg_max(sk, sw);
            const T e = ok ? exp(sk - m) : T(0);
            const T se = seg_sum(e, sw);
            if (ok) P[o] = e / se;
        }
        return;
    }
    for (int r0 = wave_g * rpw; r0 < N; r0 += nwaves * rpw) {
        const int n = r0 + seg;
        const bool ok = n < N;
        const T *s = S + (size_t)n * K;
        T m = -INFINITY;
        if (ok)
            for (int k = sl; k < K; k += sw) m = s[k] > m ? s[k] : m;
        m = seg_max(m, sw);
        T se = T(0);
        if (ok)
            for (int k = sl; k < K; k += sw) se += exp(s[k] - m);
        se = seg_sum(se, sw);
        if (ok)
            for (int k = sl; k < K; k += sw) P[(size_t)n * K + k] = exp(s[k] - m) / se;
    }
}

}  // namespace

hipError_t launch_softmax(int dtype, const void *S, void *P, int N, int K, hipStream_t s)
{
    int sw = 1;
    while (sw < K && sw < kWave) sw <<= 1;
    const long long rows_per_block = (long long)kSmWaves * (kWave / sw);
    long long g = (N + rows_per_block - 1) / rows_per_block;
    if (g > 1024) g = 1024;
    if (dtype == 0)
        hipLaunchKernelGGL(softmax_kernel<double>, dim3((int)g), dim3(kSmThreads), 0, s,
                           (const double *)S, (double *)P, N, K, sw);
    else
        hipLaunchKernelGGL(softmax_kernel<float>, dim3((int)g), dim3(kSmThreads), 0, s,
                           (const float *)S, (float *)P, N, K, sw);
    return hipGetLastError();
}

namespace {

int softmax_segment(int K)
{
    int sw = 1;
    while (sw < K && sw < kWave) sw <<= 1;
    return sw;
}

// Blocks a call would use with an unbounded workspace: one per 16 waves' rows,
// at most kSmMaxBlocks.
long long softmax_blocks(int N, int K)
{
    const long long rows_per_block = (long long)kSmWaves * (kWave / softmax_segment(K));
    return std::min<long long>((N + rows_per_block - 1) / rows_per_block, kSmMaxBlocks);
}

template <typename T>
hipError_t launch_xent(const void *S, const void *Y, void *P, void *dS, void *loss, int N, int K,
                       void *ws, size_t ws_bytes, hipStream_t s)
{
    const int sw = softmax_segment(K);
    long long G = ws ? std::min<long long>(softmax_blocks(N, K), (long long)(ws_bytes / sizeof(T)))
                     : 1;
    if (G <= 1) {
        hipLaunchKernelGGL(softmax_xent_kernel<T>, dim3(1), dim3(kSmThreads), 0, s,
                           (const T *)S, (const T *)Y, (T *)P, (T *)dS, (T *)loss, (T *)nullptr,
                           N, K, sw);
        return hipGetLastError();
    }
    hipLaunchKernelGGL(softmax_xent_kernel<T>, dim3((int)G), dim3(kSmThreads), 0, s, (const T *)S,
                       (const T *)Y, (T *)P, (T *)dS, (T *)loss, (T *)ws, N, K, sw);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(softmax_loss_reduce<T>, dim3(1), dim3(kWave), 0, s, (const T *)ws, (int)G,
                       (T *)loss, N);
    return hipGetLastError();
}

}  // namespace

size_t softmax_xent_workspace_bytes(int dtype, int N, int K)
{
    const long long G = softmax_blocks(N, K);
    return G > 1 ? (size_t)G * (dtype == 0 ? sizeof(double) : sizeof(float)) : 0;
}

hipError_t launch_softmax_xent(int dtype, const void *S, const void *Y, void *P, void *dS,
                               void *loss, int N, int K, void *ws, size_t ws_bytes, hipStream_t s)
{
    return dtype == 0 ? launch_xent<double>(S, Y, P, dS, loss, N, K, ws, ws_bytes, s)
                      : launch_xent<float>(S, Y, P, dS, loss, N, K, ws, ws_bytes, s);
}

}  // namespace dmlnn
