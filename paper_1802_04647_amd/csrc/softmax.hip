// Fused softmax + cross-entropy forward and backward (paper, Section 2 listing:
// probs = softmax::forward(scores); dprobs = cross_entropy_loss::backward(probs, y);
// dscores = softmax::backward(dprobs, scores)).  Per row, with m = max_k s:
//   p = exp(s - m) / sum exp(s - m)
//   row loss = -sum_k y (s - m - log sum exp(s - m))
//   ds = (p * sum_k y - y) / N
// and loss = (1/N) * sum of row losses.  One block; wave w takes rows w, w+4, ...
// with lanes across the K columns and butterfly-shuffle reductions; the four wave
// totals are added in wave order, so the loss is deterministic.
#include "common.hpp"
#include "internal.hpp"

namespace dmlnn {
namespace {

template <typename T>
__device__ __forceinline__ T wave_sum(T v)
{
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) v += __shfl_xor(v, off, kWave);
    return v;
}

template <typename T>
__device__ __forceinline__ T wave_max(T v)
{
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) {
        T o = __shfl_xor(v, off, kWave);
        v = o > v ? o : v;
    }
    return v;
}

template <typename T>
__global__ __launch_bounds__(256) void softmax_xent_kernel(const T *S, const T *Y, T *P, T *dS,
                                                           T *loss, int N, int K)
{
    __shared__ T s_tot[4];
    const int lane = lane_id(), wave = wave_id();
    const T invN = T(1) / T(N);
    T total = T(0);
    for (int n = wave; n < N; n += 4) {
        const T *s = S + (size_t)n * K;
        const T *y = Y + (size_t)n * K;
        T m = -INFINITY;
        for (int k = lane; k < K; k += kWave) m = s[k] > m ? s[k] : m;
        m = wave_max(m);
        T se = T(0), ys = T(0);
        for (int k = lane; k < K; k += kWave) {
            se += exp(s[k] - m);
            ys += y[k];
        }
        se = wave_sum(se);
        ys = wave_sum(ys);
        const T lse = m + log(se);
        T rl = T(0);
        for (int k = lane; k < K; k += kWave) {
            const T p = exp(s[k] - m) / se;
            if (P) P[(size_t)n * K + k] = p;
            dS[(size_t)n * K + k] = (p * ys - y[k]) * invN;
            rl -= y[k] * (s[k] - lse);
        }
        total += wave_sum(rl);
    }
    if (lane == 0) s_tot[wave] = total;
    __syncthreads();
    if (threadIdx.x == 0) *loss = (((s_tot[0] + s_tot[1]) + s_tot[2]) + s_tot[3]) * invN;
}

}  // namespace

hipError_t launch_softmax_xent(int dtype, const void *S, const void *Y, void *P, void *dS,
                               void *loss, int N, int K, hipStream_t s)
{
    if (dtype == 0)
        hipLaunchKernelGGL(softmax_xent_kernel<double>, dim3(1), dim3(256), 0, s,
                           (const double *)S, (const double *)Y, (double *)P, (double *)dS,
                           (double *)loss, N, K);
    else
        hipLaunchKernelGGL(softmax_xent_kernel<float>, dim3(1), dim3(256), 0, s, (const float *)S,
                           (const float *)Y, (float *)P, (float *)dS, (float *)loss, N, K);
    return hipGetLastError();
}

}  // namespace dmlnn
