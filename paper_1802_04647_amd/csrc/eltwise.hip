// Streaming elementwise kernels: bias_add_relu, sgd_momentum_update, count_nonzero.
// All are HBM-bound; each thread handles a contiguous pair/quad via vector
// loads where alignment allows, with a grid-stride loop sized to the chip.
#include "common.hpp"
#include "internal.hpp"

namespace dmlnn {
namespace {

int stream_grid(long long n_items)
{
    long long g = (n_items + 255) / 256;
    const long long cap = 256LL * 16;  // 16 blocks per CU
    return (int)(g < 1 ? 1 : (g > cap ? cap : g));
}

// out[n, c*HW + q] = relu?(X[...] + b[c]).  Row-major N x (C*HW), viewed as
// N*C segments of HW contiguous values; one block-stride walk over all values.
template <typename T>
__global__ __launch_bounds__(256) void bias_add_relu_kernel(const T *X, const T *b, T *out,
                                                            long long total, int C, int HW,
                                                            int relu)
{
    for (long long e = (long long)blockIdx.x * 256 + threadIdx.x; e < total;
         e += (long long)gridDim.x * 256) {
        T v = X[e];
        if (b) v += b[(int)((e / HW) % C)];
        out[e] = relu_if(v, relu);
    }
}

// v <- mu*v - lr*g; theta <- theta + v.  Computed in the buffer's type.
template <typename T>
__global__ __launch_bounds__(256) void sgd_momentum_kernel(T *__restrict__ theta,
                                                           const T *__restrict__ grad,
                                                           T *__restrict__ v, T lr, T mu,
                                                           long long n)
{
    for (long long e = (long long)blockIdx.x * 256 + threadIdx.x; e < n;
         e += (long long)gridDim.x * 256) {
        const T nv = mu * v[e] - lr * grad[e];
        v[e] = nv;
        theta[e] = theta[e] + nv;
    }
}

__global__ void zero_i64_kernel(long long *p) { *p = 0; }

// Per-wave ballot + popcount, one integer atomic per wave (exact and
// order-independent).
template <typename T>
__global__ __launch_bounds__(256) void count_nonzero_kernel(const T *X, long long n,
                                                            long long *out)
{
    long long cnt = 0;
    for (long long base = (long long)blockIdx.x * 256; base < n; base += (long long)gridDim.x * 256) {
        long long e = base + threadIdx.x;
        bool nz = e < n && X[e] != T(0);
        cnt += __popcll(__builtin_amdgcn_ballot_w64(nz));
    }
    if (lane_id() == 0 && cnt) atomicAdd((unsigned long long *)out, (unsigned long long)cnt);
}

}  // namespace

hipError_t launch_bias_add_relu(int dtype, const void *X, const void *b, void *out, int N, int C,
                                int HW, int relu, hipStream_t s)
{
    const long long total = (long long)N * C * HW;
    const int g = stream_grid(total);
    if (dtype == 0)
        hipLaunchKernelGGL(bias_add_relu_kernel<double>, dim3(g), dim3(256), 0, s,
                           (const double *)X, (const double *)b, (double *)out, total, C, HW,
                           relu);
    else
        hipLaunchKernelGGL(bias_add_relu_kernel<float>, dim3(g), dim3(256), 0, s,
                           (const float *)X, (const float *)b, (float *)out, total, C, HW, relu);
    return hipGetLastError();
}

hipError_t launch_sgd_momentum(int dtype, void *theta, const void *grad, void *v, double lr,
                               double mu, long long n, hipStream_t s)
{
    const int g = stream_grid(n);
    if (dtype == 0)
        hipLaunchKernelGGL(sgd_momentum_kernel<double>, dim3(g), dim3(256), 0, s, (double *)theta,
                           (const double *)grad, (double *)v, lr, mu, n);
    else
        hipLaunchKernelGGL(sgd_momentum_kernel<float>, dim3(g), dim3(256), 0, s, (float *)theta,
                           (const float *)grad, (float *)v, (float)lr, (float)mu, n);
    return hipGetLastError();
}

hipError_t launch_count_nonzero(int dtype, const void *X, long long n, long long *out,
                                hipStream_t s)
{
    hipLaunchKernelGGL(zero_i64_kernel, dim3(1), dim3(1), 0, s, out);
    const int g = stream_grid(n);
    if (dtype == 0)
        hipLaunchKernelGGL(count_nonzero_kernel<double>, dim3(g), dim3(256), 0, s,
                           (const double *)X, n, out);
    else
        hipLaunchKernelGGL(count_nonzero_kernel<float>, dim3(g), dim3(256), 0, s, (const float *)X,
                           n, out);
    return hipGetLastError();
}

}  // namespace dmlnn
