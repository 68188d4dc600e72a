// The NN library's other optimizers (paper, Section 2, "NN Library": Adagrad,
// Adam, RMSprop, SGD, SGD with momentum and SGD with Nesterov momentum) as
// fused elementwise updates: one pass reads theta, grad and the optimizer state
// and writes theta and the state.  All are HBM-bound streams; the arithmetic is
// done in the buffer's type.  SGD with momentum lives in eltwise.hip.
#include "common.hpp"
#include "internal.hpp"

namespace dmlnn {
namespace {

int optim_grid(long long n)
{
    long long g = (n + 255) / 256;
    const long long cap = 256LL * 16;
    return (int)(g < 1 ? 1 : (g > cap ? cap : g));
}

#define DMLNN_FOR_EACH(e, n)                                                                      \
    for (long long e = (long long)blockIdx.x * 256 + threadIdx.x; e < (n);                        \
         e += (long long)gridDim.x * 256)

// theta <- theta - lr * g
template <typename T>
__global__ __launch_bounds__(256) void sgd_kernel(T *__restrict__ theta, const T *__restrict__ g,
                                                  T lr, long long n)
{
    DMLNN_FOR_EACH(e, n) theta[e] = theta[e] - lr * g[e];
}

// v' = mu v - lr g;  theta <- theta - mu v + (1 + mu) v'
template <typename T>
__global__ __launch_bounds__(256) void sgd_nesterov_kernel(T *__restrict__ theta,
                                                           const T *__restrict__ g,
                                                           T *__restrict__ v, T lr, T mu,
                                                           long long n)
{
    DMLNN_FOR_EACH(e, n)
    {
        const T vp = v[e];
        const T vn = mu * vp - lr * g[e];
        v[e] = vn;
        theta[e] = theta[e] - mu * vp + (T(1) + mu) * vn;
    }
}

// c <- c + g^2;  theta <- theta - lr g / (sqrt(c) + eps)
template <typename T>
__global__ __launch_bounds__(256) void adagrad_kernel(T *__restrict__ theta,
                                                      const T *__restrict__ g,
                                                      T *__restrict__ c, T lr, T eps, long long n)
{
    DMLNN_FOR_EACH(e, n)
    {
        const T ge = g[e];
        const T cn = c[e] + ge * ge;
        c[e] = cn;
        theta[e] = theta[e] - lr * ge / (sqrt(cn) + eps);
    }
}

// c <- rho c + (1 - rho) g^2;  theta <- theta - lr g / (sqrt(c) + eps)
template <typename T>
__global__ __launch_bounds__(256) void rmsprop_kernel(T *__restrict__ theta,
                                                      const T *__restrict__ g,
                                                      T *__restrict__ c, T lr, T rho, T eps,
                                                      long long n)
{
    DMLNN_FOR_EACH(e, n)
    {
        const T ge = g[e];
        const T cn = rho * c[e] + (T(1) - rho) * ge * ge;
        c[e] = cn;
        theta[e] = theta[e] - lr * ge / (sqrt(cn) + eps);
    }
}

// m <- b1 m + (1 - b1) g;  v <- b2 v + (1 - b2) g^2;
// theta <- theta - lr_t m / (sqrt(v) + eps), lr_t = lr sqrt(1 - b2^t) / (1 - b1^t)
template <typename T>
__global__ __launch_bounds__(256) void adam_kernel(T *__restrict__ theta, const T *__restrict__ g,
                                                   T *__restrict__ m, T *__restrict__ v, T lr_t,
                                                   T b1, T b2, T eps, long long n)
{
    DMLNN_FOR_EACH(e, n)
    {
        const T ge = g[e];
        const T mn = b1 * m[e] + (T(1) - b1) * ge;
        const T vn = b2 * v[e] + (T(1) - b2) * ge * ge;
        m[e] = mn;
        v[e] = vn;
        theta[e] = theta[e] - lr_t * mn / (sqrt(vn) + eps);
    }
}

#undef DMLNN_FOR_EACH

}  // namespace

hipError_t launch_sgd(int dtype, void *theta, const void *grad, double lr, long long n,
                      hipStream_t s)
{
    const int gr = optim_grid(n);
    if (dtype == 0)
        hipLaunchKernelGGL(sgd_kernel<double>, dim3(gr), dim3(256), 0, s, (double *)theta,
                           (const double *)grad, lr, n);
    else
        hipLaunchKernelGGL(sgd_kernel<float>, dim3(gr), dim3(256), 0, s, (float *)theta,
                           (const float *)grad, (float)lr, n);
    return hipGetLastError();
}

hipError_t launch_sgd_nesterov(int dtype, void *theta, const void *grad, void *v, double lr,
                               double mu, long long n, hipStream_t s)
{
    const int gr = optim_grid(n);
    if (dtype == 0)
        hipLaunchKernelGGL(sgd_nesterov_kernel<double>, dim3(gr), dim3(256), 0, s,
                           (double *)theta, (const double *)grad, (double *)v, lr, mu, n);
    else
        hipLaunchKernelGGL(sgd_nesterov_kernel<float>, dim3(gr), dim3(256), 0, s,
                           (float *)theta, (const float *)grad, (float *)v, (float)lr, (float)mu,
                           n);
    return hipGetLastError();
}

hipError_t launch_adagrad(int dtype, void *theta, const void *grad, void *cache, double lr,
                          double eps, long long n, hipStream_t s)
{
    const int gr = optim_grid(n);
    if (dtype == 0)
        hipLaunchKernelGGL(adagrad_kernel<double>, dim3(gr), dim3(256), 0, s, (double *)theta,
                           (const double *)grad, (double *)cache, lr, eps, n);
    else
        hipLaunchKernelGGL(adagrad_kernel<float>, dim3(gr), dim3(256), 0, s, (float *)theta,
                           (const float *)grad, (float *)cache, (float)lr, (float)eps, n);
    return hipGetLastError();
}

hipError_t launch_rmsprop(int dtype, void *theta, const void *grad, void *cache, double lr,
                          double decay, double eps, long long n, hipStream_t s)
{
    const int gr = optim_grid(n);
    if (dtype == 0)
        hipLaunchKernelGGL(rmsprop_kernel<double>, dim3(gr), dim3(256), 0, s, (double *)theta,
                           (const double *)grad, (double *)cache, lr, decay, eps, n);
    else
        hipLaunchKernelGGL(rmsprop_kernel<float>, dim3(gr), dim3(256), 0, s, (float *)theta,
                           (const float *)grad, (float *)cache, (float)lr, (float)decay,
                           (float)eps, n);
    return hipGetLastError();
}

hipError_t launch_adam(int dtype, void *theta, const void *grad, void *m, void *v, double lr,
                       double beta1, double beta2, double eps, long long t, long long n,
                       hipStream_t s)
{
    // The step's effective rate, formed once on the host in fp64.
    const double lr_t = lr * sqrt(1.0 - pow(beta2, (double)t)) / (1.0 - pow(beta1, (double)t));
    const int gr = optim_grid(n);
    if (dtype == 0)
        hipLaunchKernelGGL(adam_kernel<double>, dim3(gr), dim3(256), 0, s, (double *)theta,
                           (const double *)grad, (double *)m, (double *)v, lr_t, beta1, beta2,
                           eps, n);
    else
        hipLaunchKernelGGL(adam_kernel<float>, dim3(gr), dim3(256), 0, s, (float *)theta,
                           (const float *)grad, (float *)m, (float *)v, (float)lr_t,
                           (float)beta1, (float)beta2, (float)eps, n);
    return hipGetLastError();
}

}  // namespace dmlnn
