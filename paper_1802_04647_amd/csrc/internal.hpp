// Host-side launch interface between the C ABI (api.hip) and the kernel files.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace dmlnn {

struct PoolSrc;  // common.hpp

// ---------------------------------------------------------------- conv2d ----
// Geometry of one conv2d call (already validated).
struct ConvDims {
    int N, C, Hin, Win, F, Hf, Wf, stride, pad, Hout, Wout;
};

// Kernel families of the conv2d passes (reported by the plan query).
enum ConvKernel {
    kConvDma = 1,       // implicit GEMM, LDS-DMA staging (forward / backward_data)
    kConvReg = 2,       // implicit GEMM, register-staged (forward / backward_data)
    kConvSmallM = 3,    // vector-ALU kernel for at most four output rows
    kConvResident = 4,  // filter-resident forward for small images (fp64)
    kWgradRing = 5,     // backward_filter, row ring over the whole k range
    kWgradTiles = 6,    // backward_filter, 4-wave (f-tile, k-range, split) blocks
    kWgradPoolSparse = 7  // backward_filter from a pooled source, small k: the pool windows
};

// What the plan query reports about one pass (host only, no device access).
struct ConvPlanInfo {
    int kernel;        // ConvKernel
    int tile_m;        // GEMM rows of a block tile
    int tile_pixels;   // output pixels of a block tile (backward_filter: a pixel tile)
    int blocks;        // blocks of the main launch (backward_filter: per split)
    int chunk;         // source channels staged per chunk (backward_filter: k columns a block covers)
    int k_split;       // in-block split of the k-steps: 1, 2 or 4
    int splits;        // backward_filter: the most reduction splits a launch uses
    int window_width;  // staged window row length (elements)
    int window_rows;   // staged window rows per channel
    size_t lds;        // dynamic LDS bytes per block
    int tile_stride, k_chunk, slice_stride, stage_bytes, window_bytes, slice_bytes, slice_vec;
    int g_stride, row_slices;
    int pipelined;  // register-staged kernels: loads held in registers across the MFMAs
    int fused;      // fused forms: 1 when the fused kernel runs, 0 for the unfused fallback
    int row_staged; // row ring: bit 0 new input row a row per wave, bit 1 the g tile so,
                    // bit 2 the new input row by LDS DMA
};

// Fused forms a plan query may ask about (the values of dmlnn_conv_form).
enum ConvForm { kFormPlain = 0, kFormPoolEpilogue = 1, kFormPooledSource = 2, kFormCsr = 3,
                kFormBanks = 4 };
// form: ConvForm; ph, pw, ps, pp: the pool of the pool forms (else unused).
hipError_t conv_plan_info(int dtype, int pass, const ConvDims &d, int zero_skip, int form,
                          int ph, int pw, int ps, int pp, ConvPlanInfo &info);

// Forward (relu(conv + b)) and input-gradient passes share one implicit-GEMM
// kernel family; see conv_igemm.hip.
hipError_t launch_conv_forward(int dtype, const void *X, const void *W, const void *b, void *out,
                               const ConvDims &d, int relu, int zero_skip, hipStream_t s);
// relu(conv + b) followed by max-pooling in the same kernel's epilogue (out may be
// null).  hipErrorNotSupported when the shape does not allow the fused epilogue.
hipError_t launch_conv_forward_pool(int dtype, const void *X, const void *W, const void *b,
                                    void *out, void *pooled, int32_t *argmax, const ConvDims &d,
                                    int relu, int ph, int pw, int ps, int Hp, int Wp,
                                    int zero_skip, hipStream_t s);
// Several filter banks over one input in one launch (horizontal fusion): Wcat is
// the banks' filters stacked ([sum F][C*Hf*Wf]), bcat their biases (or null);
// bank b writes outs[b] ([N][Fs[b]*Hout*Wout]).  At most 8 banks.
// hipErrorNotSupported when the shape needs the register-staged path.
hipError_t launch_conv_forward_multi(int dtype, const void *X, const void *Wcat,
                                     const void *bcat, void *const *outs, const int *Fs,
                                     int nbanks, const ConvDims &d, int relu, int zero_skip,
                                     hipStream_t s);
// Sparse-input forward: X as CSR (rowptr N+1, colidx/vals nnz); row_index is a
// caller workspace of N*C*Hin + 1 int32.
hipError_t launch_conv_forward_csr(int dtype, const int32_t *rowptr, const int32_t *colidx,
                                   const void *vals, int nnz, int32_t *row_index, const void *W,
                                   const void *b, void *out, const ConvDims &d, int relu,
                                   int zero_skip, hipStream_t s);
hipError_t launch_conv_backward_data(int dtype, const void *W, const void *dout,
                                     const void *out_fwd, void *dX, const ConvDims &d,
                                     int zero_skip, hipStream_t s, const PoolSrc *pool = nullptr);

// Filter/bias gradient: split reduction into a workspace, then a fixed-order sum.
size_t conv_wgrad_workspace_bytes(int dtype, const ConvDims &d);
// The backward_filter part of conv_plan_info.
// pool_ps: the pool stride of a pooled source, or 0.
hipError_t wgrad_plan_info(int dtype, const ConvDims &d, int pool_ps, ConvPlanInfo &info);
// pool (optional): dout is not given; g is built from a following max-pool's
// backward (see PoolSrc in common.hpp).
hipError_t launch_conv_backward_filter(int dtype, const void *X, const void *dout,
                                       const void *out_fwd, void *dW, void *db,
                                       const ConvDims &d, void *ws, int zero_skip,
                                       hipStream_t s, const PoolSrc *pool = nullptr,
                                       void *g_out = nullptr);

// ----------------------------------------------------------------- others ----
hipError_t launch_bias_add_relu(int dtype, const void *X, const void *b, void *out, int N, int C,
                                int HW, int relu, hipStream_t s);
hipError_t launch_max_pool_fwd(int dtype, const void *X, void *out, int32_t *argmax, int N, int C,
                               int Hin, int Win, int Hf, int Wf, int stride, int pad, int Hout,
                               int Wout, hipStream_t s);
// pooled (the forward's pooled values) may be null; when given, a route only
// counts where pooled > 0 (the relu mask of the pooled layer).
hipError_t launch_max_pool_bwd(int dtype, const void *dout, const int32_t *argmax,
                               const void *pooled, void *dX, int N, int C, int Hin, int Win,
                               int Hf, int Wf, int stride, int pad, int Hout, int Wout,
                               hipStream_t s);
// Launch shape of one affine product C (M x N) = A (M x K) B (K x N): the
// output tile of a block (wt x wt tiles of 16 x 16), the waves splitting its
// k range, and the block k splits, whose partial products take
// splits x M x N elements of workspace when splits > 1.
struct GemmPlan {
    int wt = 1, nk = 1, splits = 1;
    size_t workspace_bytes = 0;
};
GemmPlan gemm_plan(int M, int N, int K, size_t elem, size_t workspace_bytes);
// The largest workspace any of the affine layer's three products splits into.
size_t affine_workspace_bytes(int dtype, int N, int D, int M);
hipError_t launch_affine_fwd(int dtype, const void *X, const void *W, const void *b, void *out,
                             int N, int D, int M, int relu, void *workspace,
                             size_t workspace_bytes, hipStream_t s);
hipError_t launch_affine_bwd(int dtype, const void *dout, const void *X, const void *W,
                             const void *out_fwd, void *dX, void *dW, void *db, int N, int D,
                             int M, int relu_input, void *workspace, size_t workspace_bytes,
                             hipStream_t s);
// ws: null, or ws_bytes of scratch for the blocks' loss shares (see softmax.hip)
hipError_t launch_softmax_xent(int dtype, const void *S, const void *Y, void *P, void *dS,
                               void *loss, int N, int K, void *ws, size_t ws_bytes,
                               hipStream_t s);
size_t softmax_xent_workspace_bytes(int dtype, int N, int K);
hipError_t launch_softmax(int dtype, const void *S, void *P, int N, int K, hipStream_t s);
hipError_t launch_sgd_momentum(int dtype, void *theta, const void *grad, void *v, double lr,
                               double mu, long long n, hipStream_t s);
hipError_t launch_count_nonzero(int dtype, const void *X, long long n, long long *out,
                                hipStream_t s);

// ------------------------------------------------------------ optimizers ----
hipError_t launch_sgd(int dtype, void *theta, const void *grad, double lr, long long n,
                      hipStream_t s);
hipError_t launch_sgd_nesterov(int dtype, void *theta, const void *grad, void *v, double lr,
                               double mu, long long n, hipStream_t s);
hipError_t launch_adagrad(int dtype, void *theta, const void *grad, void *cache, double lr,
                          double eps, long long n, hipStream_t s);
hipError_t launch_rmsprop(int dtype, void *theta, const void *grad, void *cache, double lr,
                          double decay, double eps, long long n, hipStream_t s);
hipError_t launch_adam(int dtype, void *theta, const void *grad, void *m, void *v, double lr,
                       double beta1, double beta2, double eps, long long t, long long n,
                       hipStream_t s);

}  // namespace dmlnn
