// max_pool2d forward (value + in-row argmax) and backward (gradient routing).
// Paper, Section 3 "Builtin NN Functions": pooling and its backward are builtins.
//
// Both are memory-bound streaming kernels over the row-major N x (C*H*W)
// matrices.  Forward: one thread per output, window scanned row by row,
// replacing the running maximum only on a strictly larger value (first maximum
// wins ties; +0 and -0 compare equal).  Backward: windows that do not overlap
// (stride >= window, no padding) are routed by one thread per stride region
// (the stride x stride input cells holding one window in their corner): it
// reads the window's gradient and argmax once and writes all of the region's
// cells (the gradient at the argmax, zeros elsewhere).  Other windows: one
// thread per INPUT cell gathers the outputs whose window covers it and whose
// argmax is that cell.  Either way every dX element is written exactly once,
// without atomics and in a fixed order.
#include "common.hpp"
#include "internal.hpp"

namespace dmlnn {
namespace {

template <typename T>
__global__ __launch_bounds__(256) void max_pool_fwd_kernel(const T *__restrict__ X,
                                                           T *__restrict__ out,
                                                           int32_t *__restrict__ argmax,
                                                           long long total, int C, int Hin,
                                                           int Win, int Hf, int Wf, int S, int P,
                                                           int Hout, int Wout)
{
    for (long long e = (long long)blockIdx.x * 256 + threadIdx.x; e < total;
         e += (long long)gridDim.x * 256) {
        const int ow = (int)(e % Wout);
        long long r = e / Wout;
        const int oh = (int)(r % Hout);
        r /= Hout;
        const int c = (int)(r % C);
        const long long n = r / C;
        const T *plane = X + (size_t)n * C * Hin * Win + (size_t)c * Hin * Win;
        const int h0 = oh * S - P, w0 = ow * S - P;
        T best = T(0);
        int bidx = -1;
        for (int i = 0; i < Hf; ++i) {
            const int h = h0 + i;
            if (h < 0 || h >= Hin) continue;
            for (int j = 0; j < Wf; ++j) {
                const int w = w0 + j;
                if (w < 0 || w >= Win) continue;
                const T v = plane[h * Win + w];
                if (bidx < 0 || v > best) {
                    best = v;
                    bidx = h * Win + w;
                }
            }
        }
        out[e] = best;
        argmax[e] = c * Hin * Win + bidx;
    }
}

// One thread per input cell of a (n, c) plane: blockIdx.y walks the planes,
// blockIdx.x * 256 + threadIdx.x the cells (32-bit index math per plane).
template <typename T>
__global__ __launch_bounds__(256) void max_pool_bwd_kernel(const T *__restrict__ dout,
                                                           const int32_t *__restrict__ argmax,
                                                           const T *__restrict__ pooled,
                                                           T *__restrict__ dX, long long planes,
                                                           int C, int Hin, int Win, int Hf,
                                                           int Wf, int S, int P, int Hout,
                                                           int Wout)
{
    const int HW = Hin * Win;
    const bool disjoint = S >= Hf && S >= Wf && P == 0;
    for (long long pl = blockIdx.y; pl < planes; pl += gridDim.y) {
        const int c = (int)(pl % C);
        const size_t obase = (size_t)pl * Hout * Wout;
        T *dXp = dX + (size_t)pl * HW;
        for (int idx = blockIdx.x * 256 + threadIdx.x; idx < HW; idx += gridDim.x * 256) {
            const int h = idx / Win, w = idx - (idx / Win) * Win;
            const int32_t me = c * HW + idx;
            if (disjoint) {
                // Windows do not overlap: at most one window covers the cell.
                const int oh = h / S, ow = w / S;
                // (the three reads are independent, so they are issued together)
                const bool in = oh < Hout && ow < Wout && h - oh * S < Hf && w - ow * S < Wf;
                const size_t o = in ? obase + (size_t)oh * Wout + ow : obase;
                const int32_t am = argmax[o];
                const T d = dout[o];
                const T pv = pooled ? pooled[o] : T(1);
                dXp[idx] = (in && am == me && pv > T(0)) ? d : T(0);
                continue;
            }
            // outputs (oh, ow) whose window [oh*S-P, oh*S-P+Hf) contains h
            int oh_lo = h + P - Hf + 1;
            oh_lo = oh_lo <= 0 ? 0 : (oh_lo + S - 1) / S;
            int oh_hi = (h + P) / S;
            if (oh_hi > Hout - 1) oh_hi = Hout - 1;
            int ow_lo = w + P - Wf + 1;
            ow_lo = ow_lo <= 0 ? 0 : (ow_lo + S - 1) / S;
            int ow_hi = (w + P) / S;
            if (ow_hi > Wout - 1) ow_hi = Wout - 1;
            T acc = T(0);
            for (int oh = oh_lo; oh <= oh_hi; ++oh)
                for (int ow = ow_lo; ow <= ow_hi; ++ow) {
                    const size_t o = obase + (size_t)oh * Wout + ow;
                    // with pooled given, the relu before the pool gates the route:
                    // the routed cell holds the pooled value, so its relu mask is
                    // pooled > 0
                    if (argmax[o] == me && (!pooled || pooled[o] > T(0))) acc += dout[o];
                }
            dXp[idx] = acc;
        }
    }
}

// Disjoint windows: thread (plane, region ry, rx) of the Ry x Rx stride regions
// (Ry = ceil(Hin / S)) writes the region's cells of dX.  VEC2 (S == 2 and an
// even Win, so every plane and region row is 2-element aligned): a region row
// is one 2-element vector store.
template <typename T, bool VEC2>
__global__ __launch_bounds__(256) void max_pool_bwd_regions_kernel(
    const T *__restrict__ dout, const int32_t *__restrict__ argmax, const T *__restrict__ pooled,
    T *__restrict__ dX, long long planes, int C, int Hin, int Win, int S, int Hout, int Wout,
    int Ry, int Rx)
{
    typedef T T2 __attribute__((ext_vector_type(2)));
    const int HW = Hin * Win, R = Ry * Rx;
    for (long long pl = blockIdx.y; pl < planes; pl += gridDim.y) {
        const int c = (int)(pl % C);
        const T *dp = dout + (size_t)pl * Hout * Wout;
        const int32_t *ap = argmax + (size_t)pl * Hout * Wout;
        const T *pp = pooled ? pooled + (size_t)pl * Hout * Wout : nullptr;
        T *dXp = dX + (size_t)pl * HW;
        for (int idx = blockIdx.x * 256 + threadIdx.x; idx < R; idx += gridDim.x * 256) {
            const int ry = idx / Rx, rx = idx - ry * Rx;
            const bool win = ry < Hout && rx < Wout;
            const int o = win ? ry * Wout + rx : 0;  // a valid address either way
            const int32_t am = ap[o];
            const T d = dp[o];
            const T pv = pp ? pp[o] : T(1);
            // in-plane index of the routed cell, or -1
            const int tgt = (win && pv > T(0)) ? am - c * HW : -1;
            for (int dy = 0; dy < S; ++dy) {
                const int y = ry * S + dy;
                if (y >= Hin) break;
                const int q = y * Win + rx * S;
                if (VEC2) {
                    T2 v;
                    v.x = q == tgt ? d : T(0);
                    v.y = q + 1 == tgt ? d : T(0);
                    *reinterpret_cast<T2 *>(dXp + q) = v;
                } else {
                    for (int dx = 0; dx < S && rx * S + dx < Win; ++dx)
                        dXp[q + dx] = q + dx == tgt ? d : T(0);
                }
            }
        }
    }
}

int grid_for(long long total)
{
    long long g = (total + 255) / 256;
    const long long cap = 256LL * 64;
    return (int)(g < 1 ? 1 : (g > cap ? cap : g));
}

}  // namespace

hipError_t launch_max_pool_fwd(int dtype, const void *X, void *out, int32_t *argmax, int N, int C,
                               int Hin, int Win, int Hf, int Wf, int stride, int pad, int Hout,
                               int Wout, hipStream_t s)
{
    const long long total = (long long)N * C * Hout * Wout;
    const int g = grid_for(total);
    if (dtype == 0)
        hipLaunchKernelGGL(max_pool_fwd_kernel<double>, dim3(g), dim3(256), 0, s,
                           (const double *)X, (double *)out, argmax, total, C, Hin, Win, Hf, Wf,
                           stride, pad, Hout, Wout);
    else
        hipLaunchKernelGGL(max_pool_fwd_kernel<float>, dim3(g), dim3(256), 0, s, (const float *)X,
                           (float *)out, argmax, total, C, Hin, Win, Hf, Wf, stride, pad, Hout,
                           Wout);
    return hipGetLastError();
}

hipError_t launch_max_pool_bwd(int dtype, const void *dout, const int32_t *argmax,
                               const void *pooled, void *dX, int N, int C, int Hin, int Win,
                               int Hf, int Wf, int stride, int pad, int Hout, int Wout,
                               hipStream_t s)
{
    const long long planes = (long long)N * C;
    const int HW = Hin * Win;
    if (stride >= Hf && stride >= Wf && pad == 0) {
        // disjoint windows: one thread per stride region
        const int Ry = (Hin + stride - 1) / stride, Rx = (Win + stride - 1) / stride;
        const int R = Ry * Rx;
        int gx = (R + 255) / 256;
        if (gx > 8) gx = 8;
        long long gy = planes;
        const long long cap = 32768 / gx;
        if (gy > cap) gy = cap;
        const dim3 grid(gx, (unsigned)gy);
        const size_t tsz = dtype == 0 ? sizeof(double) : sizeof(float);
        const bool vec2 = stride == 2 && Win % 2 == 0 && (uintptr_t)dX % (2 * tsz) == 0;
        if (dtype == 0) {
            auto k = vec2 ? max_pool_bwd_regions_kernel<double, true>
                          : max_pool_bwd_regions_kernel<double, false>;
            hipLaunchKernelGGL(k, grid, dim3(256), 0, s, (const double *)dout, argmax,
                               (const double *)pooled, (double *)dX, planes, C, Hin, Win, stride,
                               Hout, Wout, Ry, Rx);
        } else {
            auto k = vec2 ? max_pool_bwd_regions_kernel<float, true>
                          : max_pool_bwd_regions_kernel<float, false>;
            hipLaunchKernelGGL(k, grid, dim3(256), 0, s, (const float *)dout, argmax,
                               (const float *)pooled, (float *)dX, planes, C, Hin, Win, stride,
                               Hout, Wout, Ry, Rx);
        }
        return hipGetLastError();
    }
    // About 16k blocks in all, each thread walking several cells and planes:
    // tiny one-element blocks would leave the dispatcher as the bottleneck.
    int gx = (HW + 1023) / 1024;
    if (gx > 8) gx = 8;
    long long gy = planes;
    const long long cap = 16384 / gx;
    if (gy > cap) gy = cap;
    const dim3 grid(gx, (unsigned)gy);
    if (dtype == 0)
        hipLaunchKernelGGL(max_pool_bwd_kernel<double>, grid, dim3(256), 0, s,
                           (const double *)dout, argmax, (const double *)pooled, (double *)dX,
                           planes, C, Hin, Win, Hf, Wf, stride, pad, Hout, Wout);
    else
        hipLaunchKernelGGL(max_pool_bwd_kernel<float>, grid, dim3(256), 0, s,
                           (const float *)dout, argmax, (const float *)pooled, (float *)dX,
                           planes, C, Hin, Win, Hf, Wf, stride, pad, Hout, Wout);
    return hipGetLastError();
}

}  // namespace dmlnn
