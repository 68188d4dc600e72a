/*
 * dmlnn.h — C ABI of libdmlnn.so, the MI355X (gfx950) implementation of the
 * conv2d layer of a DML-style neural-network library and the ops around it.
 *
 * Source of the semantics: "Deep Learning with Apache SystemML" (Pansare et
 * al., arXiv 1802.04647).
 *   - Section 3, "Tensor Representation": a tensor [N, C, H, W] is stored as an
 *     N x (C*H*W) matrix, the dimensions after the first folded into the
 *     column index.  Reading used throughout: row-major, column index
 *     c*H*W + h*W + w.  Filters are F x (C*Hf*Wf) with column c*Hf*Wf + i*Wf + j.
 *   - Section 3, "Builtin NN Functions": conv2d and pooling, and their backward
 *     functions, are builtins.
 *   - Section 2 (NN library and its softmax-classifier listing): layers with
 *     init/forward/backward; affine (X W plus a bias row); softmax;
 *     cross-entropy; SGD (and SGD with momentum among the optimizers).
 *
 * Conventions shared by every entry point
 *   - Tensor pointers are DEVICE pointers to contiguous row-major buffers that
 *     the caller allocates and owns.  The library never allocates device memory
 *     and keeps no pointer after a call returns.
 *   - `dtype` selects the element type of every floating-point buffer of the
 *     call: DMLNN_F64 (double) or DMLNN_F32 (float).  Index buffers are int32.
 *   - `stream` is a hipStream_t (NULL = the default stream).  Calls are
 *     asynchronous on that stream; outputs are valid once the stream reaches
 *     the call.
 *   - Outputs are overwritten (never accumulated into).  Inputs are never
 *     written.  Buffers must not alias, except where a call says so.
 *   - Every call validates its arguments on the host before launching anything.
 *     On failure it returns a nonzero dmlnn_status, launches nothing, and
 *     dmlnn_last_error() describes the problem.  Faults inside a kernel surface
 *     at the next synchronisation of the stream.
 *   - Element counts of every buffer must be below 2^31.
 *   - Entry points keep no state between calls (except the zero-skip mode) and
 *     may be called from several host threads.
 */
#ifndef DMLNN_H
#define DMLNN_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#if defined(__GNUC__) || defined(__clang__)
#define DMLNN_API __attribute__((visibility("default")))
#else
#define DMLNN_API
#endif

typedef enum {
    DMLNN_F64 = 0,
    DMLNN_F32 = 1,
    /* The two bounds widen the type to the whole int range, so any int a caller
     * passes is a value of the type and an invalid one is reported
     * (DMLNN_ERR_DTYPE) rather than undefined.  They are not dtypes. */
    DMLNN_DTYPE_RANGE_MIN_ = -0x7fffffff - 1,
    DMLNN_DTYPE_RANGE_MAX_ = 0x7fffffff
} dmlnn_dtype;

typedef enum {
    DMLNN_OK = 0,
    DMLNN_ERR_ARG = 1,       /* a size, stride, pad or flag is out of range       */
    DMLNN_ERR_NULL = 2,      /* a required pointer is NULL                         */
    DMLNN_ERR_DTYPE = 3,     /* dtype is not DMLNN_F64 / DMLNN_F32                 */
    DMLNN_ERR_WORKSPACE = 4, /* workspace missing or smaller than required         */
    DMLNN_ERR_DEVICE = 5,    /* no usable gfx950 device / HIP runtime error        */
    DMLNN_ERR_LAUNCH = 6     /* a kernel launch was rejected                       */
} dmlnn_status;

/* Output size of a convolution or pooling window along one axis:
 * floor((Hin + 2*pad - Hf) / stride) + 1 (symmetric zero padding).
 * Host-only.  Returns <= 0 when the arguments are invalid or no window fits. */
DMLNN_API int conv2d_out_dim(int Hin, int Hf, int stride, int pad);

/* ---------------------------------------------------------------- conv2d ----
 * Paper: Section 3, "Builtin NN Functions" (conv2d is a builtin) and "Sparse
 * Operations" (conv2d is computed by lowering: the stored filter matrix times
 * the patch matrix, i.e. cross-correlation without a filter flip).
 *
 * Shapes: X is N x (C*Hin*Win); W is F x (C*Hf*Wf); b has F entries;
 * out is N x (F*Hout*Wout) with Hout = conv2d_out_dim(Hin,Hf,stride,pad) and
 * Wout = conv2d_out_dim(Win,Wf,stride,pad), both required to be >= 1.
 * Requires N, C, Hin, Win, F, Hf, Wf >= 1, stride >= 1, pad >= 0.
 */

/* Forward with bias_add and relu fused into the epilogue:
 *   pre[n,f,oh,ow] = b[f] + sum_{c,i,j} W[f,c,i,j] * x[n,c,oh*stride+i-pad,ow*stride+j-pad]
 *   (x is 0 outside the image);  out = relu ? max(pre, 0) : pre.
 * b may be NULL (no bias).  relu is 0 or 1. */
DMLNN_API int conv2d_forward(dmlnn_dtype dtype, const void *X, const void *W, const void *b, void *out,
                   int N, int C, int Hin, int Win, int F, int Hf, int Wf,
                   int stride, int pad, int relu, void *stream);

/* Bytes of device workspace that conv2d_backward_filter needs for these sizes
 * (a deterministic split of the reduction over images and pixels).  Depends
 * only on the arguments.  Returns 0 when the arguments are invalid. */
DMLNN_API size_t conv2d_backward_filter_workspace_size(dmlnn_dtype dtype, int N, int C, int Hin, int Win,
                                             int F, int Hf, int Wf, int stride, int pad);

/* Filter and bias gradients, with the relu mask fused into the prologue:
 *   g = dout where out_fwd > 0, else 0   (out_fwd == NULL: g = dout, no relu)
 *   dW[f,c,i,j] = sum_{n,oh,ow} g[n,f,oh,ow] * x[n,c,oh*stride+i-pad,ow*stride+j-pad]
 *   db[f]       = sum_{n,oh,ow} g[n,f,oh,ow]              (db may be NULL)
 * dout and out_fwd are N x (F*Hout*Wout); dW is F x (C*Hf*Wf).
 * `workspace` is a device buffer of at least
 * conv2d_backward_filter_workspace_size(...) bytes, owned by the caller; its
 * contents on entry are ignored and on return are undefined.  The reduction
 * order is fixed, so results are bitwise reproducible run to run. */
DMLNN_API int conv2d_backward_filter(dmlnn_dtype dtype, const void *X, const void *dout, const void *out_fwd,
                           void *dW, void *db, int N, int C, int Hin, int Win,
                           int F, int Hf, int Wf, int stride, int pad,
                           void *workspace, size_t workspace_bytes, void *stream);

/* conv2d_backward_filter that also writes the masked gradient it stages,
 *   g_out[n,f,oh,ow] = g[n,f,oh,ow]   (g as in conv2d_backward_filter),
 * so that conv2d_backward_data can take g_out as its dout with out_fwd = NULL
 * and skip the mask (paper, Section "Future Work": vertical fusion across the
 * layer's two backward functions; the relu mask is applied once).  g_out is a
 * caller-owned N x (F*Hout*Wout) device buffer; it may be dout itself (masked
 * in place: each element is read and written by the one thread that stages
 * it), but must not overlap X, dW, db, the workspace or a distinct out_fwd
 * (DMLNN_ERR_ARG).  Otherwise as conv2d_backward_filter: same workspace, same
 * results bit for bit. */
DMLNN_API int conv2d_backward_filter_emit(dmlnn_dtype dtype, const void *X, const void *dout,
                                          const void *out_fwd, void *dW, void *db, void *g_out,
                                          int N, int C, int Hin, int Win, int F, int Hf, int Wf,
                                          int stride, int pad, void *workspace,
                                          size_t workspace_bytes, void *stream);

/* conv2d_backward_filter for callers that cannot allocate device memory (code
 * under HIP graph capture, tight serving loops, harnesses that forbid
 * hipMalloc): the same computation, plan and result — bitwise equal to
 * conv2d_backward_filter for the same arguments — with the split reduction's
 * partials kept in a scratch array the library holds in device memory
 * (DMLNN_NOALLOC_SCRATCH_BYTES per GPU, reserved when the library's code is
 * loaded on that GPU and held until the process ends) instead of a caller
 * workspace.  The call allocates nothing.  Sizes whose workspace
 * (conv2d_backward_filter_workspace_size) exceeds DMLNN_NOALLOC_SCRATCH_BYTES
 * are rejected with DMLNN_ERR_WORKSPACE before anything is launched.  Every
 * call on one GPU uses that GPU's one scratch array: calls that overlap in time
 * on one GPU (on different streams, or from different host threads without
 * ordering) race and give undefined results; calls in one stream order are
 * safe.  Each call writes every scratch entry it later reads, so nothing left
 * by an earlier call is ever read. */
#define DMLNN_NOALLOC_SCRATCH_BYTES (80u * 1024u * 1024u)
DMLNN_API int conv2d_backward_filter_noalloc(dmlnn_dtype dtype, const void *X, const void *dout,
                                             const void *out_fwd, void *dW, void *db, int N,
                                             int C, int Hin, int Win, int F, int Hf, int Wf,
                                             int stride, int pad, void *stream);

/* Input gradient, with the relu mask fused into the prologue:
 *   dX[n,c,h,w] = sum_{f,i,j} W[f,c,i,j] * g[n,f,(h+pad-i)/stride,(w+pad-j)/stride]
 * over the (i,j) whose quotients are exact and inside the output; input cells
 * that no window covers get 0.  g as in conv2d_backward_filter.
 * dX is N x (C*Hin*Win). */
DMLNN_API int conv2d_backward_data(dmlnn_dtype dtype, const void *W, const void *dout, const void *out_fwd,
                         void *dX, int N, int C, int Hin, int Win, int F, int Hf, int Wf,
                         int stride, int pad, void *stream);

/* Zero-skip mode for the conv2d kernels (paper, Section 3 "Sparse Operations":
 * a sparse-input / dense-filter operator does fewer floating-point operations).
 * mode 0 = dense (default), 1 = skip every MFMA step whose staged input
 * fragment is entirely zero (a wavefront ballot).  Where both modes run the
 * same kernel, results are bitwise equal up to the sign of zero results.  The
 * filter-resident forward has no skip form: with the skip on, that pass runs
 * the LDS-DMA kernel, whose summation order differs (equal within rounding);
 * conv2d_plan reports which kernel runs.  Process-wide setting; returns the
 * previous mode, or -1 for an invalid mode. */
DMLNN_API int dmlnn_set_zero_skip(int mode);

/* ------------------------------------------------------------ conv2d_plan ----
 * Which kernel a conv2d pass would run for these sizes, and its tiling: a
 * host-only query (no device access, launches nothing) for profiling and tests.
 * The choice depends only on the arguments, as in the call itself (for
 * backward_filter, `splits` is the most reduction splits a launch may use;
 * the launch takes fewer when the device holds fewer blocks at once).
 * pass: DMLNN_PASS_FORWARD (conv2d_forward), DMLNN_PASS_BACKWARD_FILTER,
 * DMLNN_PASS_BACKWARD_DATA.  zero_skip: the zero-skip mode the call would run
 * under (0 or 1).  Returns DMLNN_OK and fills *plan, or an error status
 * (DMLNN_ERR_ARG also when no tiling fits). */
typedef enum {
    DMLNN_PASS_FORWARD = 0,
    DMLNN_PASS_BACKWARD_FILTER = 1,
    DMLNN_PASS_BACKWARD_DATA = 2
} dmlnn_conv_pass;

typedef enum {
    DMLNN_KERNEL_IGEMM_DMA = 1,      /* implicit GEMM, matrix cores, LDS-DMA staging     */
    DMLNN_KERNEL_IGEMM_REG = 2,      /* implicit GEMM, matrix cores, register staging    */
    DMLNN_KERNEL_SMALL_M = 3,        /* vector-ALU kernel for at most four output rows    */
    DMLNN_KERNEL_RESIDENT = 4,       /* filter-resident forward for small images (fp64)   */
    DMLNN_KERNEL_WGRAD_RING = 5,     /* backward_filter: row ring over the whole k range  */
    DMLNN_KERNEL_WGRAD_TILES = 6,    /* backward_filter: (filter tile, k range) blocks    */
    DMLNN_KERNEL_WGRAD_POOL_SPARSE = 7 /* backward_filter from a pooled source with at most
                                          32 filter columns: a sum over the pool windows  */
} dmlnn_conv_kernel;

typedef struct {
    int kernel;        /* dmlnn_conv_kernel */
    int zero_skip;     /* 1: the kernel's zero-skip instantiation runs (the small-M and
                          resident kernels have none: 0 there under either mode) */
    int tile_m;        /* GEMM rows of a block tile (filters; channels for backward_data) */
    int tile_pixels;   /* output pixels of a block tile (backward_filter: of a pixel tile) */
    int blocks;        /* blocks of the main launch (backward_filter: per split) */
    int chunk;         /* source channels staged per chunk (backward_filter: the k
                          columns one block covers) */
    int k_split;       /* wave groups of a block that split the k-steps (1, 2 or 4) */
    int splits;        /* backward_filter: the most reduction splits; else 0 */
    int window_width;  /* staged input-window row length, elements */
    int window_rows;   /* staged input-window rows per channel */
    size_t lds_bytes;  /* dynamic LDS per block */
    size_t workspace_bytes; /* backward_filter: conv2d_backward_filter_workspace_size; else 0 */
    /* Layout of the staged tiles (for tools that model the kernels' LDS use):
     * implicit-GEMM kernels: pixels between tile origins, k per chunk (padded to
     * whole k-steps), row stride of the staged filter slice, bytes of a stage,
     * of its input window and of its filter slice, 1 when the slice moves 16
     * bytes a lane; backward_filter: row stride of the staged gradient tile and
     * the slices a wide output row is cut into (0: tiles are whole rows). */
    int tile_stride, k_chunk, slice_stride, stage_bytes, window_bytes, slice_bytes, slice_vec;
    int g_stride, row_slices;
    int pipelined;     /* register-staged kernels: 1 when a tile's global loads are held in
                          registers across the previous tile's MFMAs, 0 when staged directly */
    int fused;         /* conv2d_plan_fused: 1 when the fused kernel runs, 0 when the call
                          falls back to the plain kernels (then described here) */
    int row_staged;    /* backward_filter row ring, how a tile is staged: bit 0 the new
                          input row a row per wave through registers (each row a
                          wave-uniform base plus the lane), bit 1 the gradient tile the
                          same way, bit 2 the new input row by LDS DMA into the one free
                          slot of an Hf + 1 slot ring (then window_rows = Hf + 1); 0
                          where elements are dealt out to threads */
} dmlnn_conv_plan;

DMLNN_API int conv2d_plan(dmlnn_dtype dtype, int pass, int N, int C, int Hin, int Win, int F,
                          int Hf, int Wf, int stride, int pad, int zero_skip,
                          dmlnn_conv_plan *plan);

/* The same query for the fused calls (paper, Section "Future Work": vertical
 * and horizontal fusion; Section 3 "Sparse Operations" for the CSR input).
 * form:
 *   DMLNN_FORM_PLAIN            as conv2d_plan;
 *   DMLNN_FORM_POOL_EPILOGUE    conv2d_forward_pool (pass FORWARD);
 *   DMLNN_FORM_POOLED_SOURCE    conv2d_backward_filter_pooled / conv2d_backward_data_pooled
 *                               (pass BACKWARD_FILTER / BACKWARD_DATA);
 *   DMLNN_FORM_CSR_INPUT        conv2d_forward_csr (pass FORWARD);
 *   DMLNN_FORM_BANKS            conv2d_forward_multi (pass FORWARD, F = the banks' total;
 *                               when not fused each bank runs as a plain forward, whose plans
 *                               conv2d_plan gives).
 * pool_h, pool_w, pool_stride, pool_pad: the pool of the two pool forms (validated as the
 * calls validate them), else ignored.  Returns DMLNN_ERR_ARG for a form that does not apply
 * to the pass. */
typedef enum {
    DMLNN_FORM_PLAIN = 0,
    DMLNN_FORM_POOL_EPILOGUE = 1,
    DMLNN_FORM_POOLED_SOURCE = 2,
    DMLNN_FORM_CSR_INPUT = 3,
    DMLNN_FORM_BANKS = 4
} dmlnn_conv_form;

DMLNN_API int conv2d_plan_fused(dmlnn_dtype dtype, int pass, int form, int pool_h, int pool_w,
                                int pool_stride, int pool_pad, int N, int C, int Hin, int Win,
                                int F, int Hf, int Wf, int stride, int pad, int zero_skip,
                                dmlnn_conv_plan *plan);

/* nnz-driven operator choice for a dense operand (paper, Section 3 "Sparse
 * Operations": the number of non-zeros kept for every intermediate selects
 * among the physical conv2d operators).  Given the number of non-zeros of the
 * operand a pass stages — X for DMLNN_PASS_FORWARD and
 * DMLNN_PASS_BACKWARD_FILTER, the gradient dout for DMLNN_PASS_BACKWARD_DATA —
 * for instance read back from count_nonzero, returns the zero-skip mode worth
 * setting with dmlnn_set_zero_skip: 1 when the kernel the pass takes in the
 * dense mode has a skip form and, with the zeros spread independently at that
 * density, at least 5% of its
 * 64-value input fragments are expected to be all zero ((1 - density)^64 >=
 * 0.05, i.e. density <= 4.6%); else 0.  Structured zeros (zero borders, dead
 * channels) skip more than this estimate: a caller that knows its data may set
 * mode 1 directly (results are identical either way).  Host only.  Returns -1
 * when an argument is invalid (nnz outside [0, element count]). */
DMLNN_API int conv2d_zero_skip_choice(dmlnn_dtype dtype, int pass, long long nnz, int N, int C,
                                      int Hin, int Win, int F, int Hf, int Wf, int stride,
                                      int pad);

/* --------------------------------------------------------- bias_add_relu ----
 * Paper: Section 3, "Tensor Representation" (broadcasting of vectors over
 * matrices) and the affine layer of Section 2 (a bias row added to X W).
 *   out[n, c*HW + q] = relu ? max(X[n,c*HW+q] + b[c], 0) : X[n,c*HW+q] + b[c]
 * X and out are N x (C*HW); b has C entries or is NULL.  out may equal X
 * (in place). */
DMLNN_API int bias_add_relu(dmlnn_dtype dtype, const void *X, const void *b, void *out,
                  int N, int C, int HW, int relu, void *stream);

/* ------------------------------------------------------------ max_pool2d ----
 * Paper: Section 3, "Builtin NN Functions" (pooling and its backward).
 * Window Hf x Wf, stride, pad; padded cells count as -infinity.  Requires
 * pad < Hf and pad < Wf (every window then holds at least one input cell).
 * X is N x (C*Hin*Win); out and argmax are N x (C*Hout*Wout).
 * argmax holds the in-row column index c*Hin*Win + h*Win + w of the first
 * maximum met scanning the window row by row (ties: first wins; +0 == -0).
 * NaN inputs give undefined results. */
DMLNN_API int max_pool2d_fwd(dmlnn_dtype dtype, const void *X, void *out, int32_t *argmax,
                   int N, int C, int Hin, int Win, int Hf, int Wf, int stride, int pad,
                   void *stream);

/* dX[n,k] = sum of dout[n,o] over the outputs o of row n with argmax[n,o] == k,
 * 0 elsewhere.  dout and argmax are N x (C*Hout*Wout); dX is N x (C*Hin*Win).
 * argmax must come from max_pool2d_fwd with the same sizes. */
DMLNN_API int max_pool2d_bwd(dmlnn_dtype dtype, const void *dout, const int32_t *argmax, void *dX,
                   int N, int C, int Hin, int Win, int Hf, int Wf, int stride, int pad,
                   void *stream);

/* ------------------------------------------------------ conv2d_forward_pool ----
 * Paper: Section "Future Work" (vertical fusion across layers); the layers are
 * Section 2's conv2d -> relu -> max_pool2d.  One call computes
 *   c = relu?(conv2d(X, W) + b)                      (as conv2d_forward)
 *   pooled, argmax = max_pool2d_fwd(c, F, Hout, Wout, pool_h, pool_w, pool_stride, pool_pad)
 * pooled and argmax are N x (F*Hp*Wp); argmax is the in-row index of each window's
 * first maximum within a row of c (as max_pool2d_fwd).  c is written to out
 * when out is not NULL.  When pool_pad == 0 and pool_stride >= pool_h the pool
 * runs in the convolution's epilogue and c need not be stored (out may be NULL);
 * otherwise the call runs the two steps back to back and out is required
 * (DMLNN_ERR_ARG if NULL). */
DMLNN_API int conv2d_forward_pool(dmlnn_dtype dtype, const void *X, const void *W, const void *b,
                                  void *out, void *pooled, int32_t *argmax, int N, int C, int Hin,
                                  int Win, int F, int Hf, int Wf, int stride, int pad, int relu,
                                  int pool_h, int pool_w, int pool_stride, int pool_pad,
                                  void *stream);

/* ------------------------------------------------------- conv2d_forward_csr ----
 * Paper: Section 3, "Sparse Operations" (the sparse-input / dense-filter conv2d
 * operator, chosen by the number of non-zeros).  Same result as conv2d_forward
 * with X given in CSR form: X is the N x (C*Hin*Win) matrix with row n holding
 * the values vals[rowptr[n] .. rowptr[n+1]) at columns colidx[...] (in-row index
 * c*Hin*Win + h*Win + w, strictly increasing within a row); rowptr has N+1
 * entries with rowptr[0] = 0 and rowptr[N] = nnz.  All arrays live in device
 * memory; row_index is a caller workspace of N*C*Hin + 1 int32 (overwritten).
 * The kernel stages each input window from the CSR arrays (only non-zeros are
 * read); entries that break the format are ignored rather than read or written
 * out of bounds.  Below 5% density it uses the zero-fragment skip. */
DMLNN_API int conv2d_forward_csr(dmlnn_dtype dtype, const int32_t *rowptr, const int32_t *colidx,
                                 const void *vals, int nnz, int32_t *row_index, const void *W,
                                 const void *b, void *out, int N, int C, int Hin, int Win, int F,
                                 int Hf, int Wf, int stride, int pad, int relu, void *stream);

/* ----------------------------------------------------- conv2d_forward_multi ----
 * Paper: Section "Future Work" (horizontal fusion for shared inputs: several
 * conv operators consuming the same input reuse one im2col intermediate).
 * nbanks (1..8) filter banks with the same Hf, Wf, stride and pad run over one
 * input X as one implicit GEMM whose rows are the banks' filters stacked:
 *   outs[b] = relu?(conv2d(X, W_b) + b_b)        (each as conv2d_forward)
 * Wcat is the banks' filters stacked row-wise ((sum Fs) x C*Hf*Wf), bcat their
 * biases stacked (NULL for none); outs (host array of nbanks device pointers)
 * and Fs (host array of nbanks filter counts) are read during the call only.
 * outs[b] is N x (Fs[b]*Hout*Wout).  Each input tile is staged once for every
 * 64 stacked filters. */
DMLNN_API int conv2d_forward_multi(dmlnn_dtype dtype, const void *X, const void *Wcat,
                                   const void *bcat, void *const *outs, const int *Fs,
                                   int nbanks, int N, int C, int Hin, int Win, int Hf, int Wf,
                                   int stride, int pad, int relu, void *stream);

/* ------------------------------------------------------ max_pool2d_bwd_relu ----
 * The backward of relu -> max_pool2d with the relu mask folded in, so that the
 * conv backward passes can take the result as dout with out_fwd = NULL (and the
 * conv output of the forward need not be kept):
 *   dX[n,k] = sum of dout[n,o] over outputs o with argmax[n,o] == k and pooled[n,o] > 0.
 * (The cell an output routes to holds the pooled value, so its relu mask is
 * pooled > 0.)  Sizes and argmax as max_pool2d_bwd; pooled is N x (C*Hout*Wout). */
DMLNN_API int max_pool2d_bwd_relu(dmlnn_dtype dtype, const void *dout, const int32_t *argmax,
                                  const void *pooled, void *dX, int N, int C, int Hin, int Win,
                                  int Hf, int Wf, int stride, int pad, void *stream);

/* ------------------------------------------- conv2d backward from a pool ----
 * Paper: Section "Future Work" (vertical fusion across layers); the layers are
 * Section 2's conv2d -> relu -> max_pool2d, run forward by conv2d_forward_pool.
 * The conv backward passes take the pool's upstream gradient directly: the
 * conv's output gradient
 *   g[n,f,oh,ow] = dpool[n,o] if argmax[n,o] == f*Hout*Wout + oh*Wout + ow and
 *                  pooled[n,o] > 0, for the window o that covers (oh, ow); else 0
 * (the result of max_pool2d_bwd_relu) is built while the kernels stage it and
 * is never stored.  Requires windows that do not overlap and no pool padding
 * (pool_pad == 0, pool_stride >= pool_h and >= pool_w; for other pools run
 * max_pool2d_bwd_relu and the plain calls) and Hout, Wout < 65536; else
 * DMLNN_ERR_ARG.  dpool, argmax and pooled are N x (F*Hp*Wp) with
 * Hp = conv2d_out_dim(Hout, pool_h, pool_stride, 0) (likewise Wp); argmax and
 * pooled are those of the forward.  Other arguments, outputs and the workspace
 * as in conv2d_backward_filter / conv2d_backward_data (same workspace size);
 * the zero-skip mode has no effect on these calls. */
DMLNN_API int conv2d_backward_filter_pooled(dmlnn_dtype dtype, const void *X, const void *dpool,
                                            const int32_t *argmax, const void *pooled, void *dW,
                                            void *db, int N, int C, int Hin, int Win, int F,
                                            int Hf, int Wf, int stride, int pad, int pool_h,
                                            int pool_w, int pool_stride, int pool_pad,
                                            void *workspace, size_t workspace_bytes,
                                            void *stream);

DMLNN_API int conv2d_backward_data_pooled(dmlnn_dtype dtype, const void *W, const void *dpool,
                                          const int32_t *argmax, const void *pooled, void *dX,
                                          int N, int C, int Hin, int Win, int F, int Hf, int Wf,
                                          int stride, int pad, int pool_h, int pool_w,
                                          int pool_stride, int pool_pad, void *stream);

/* ----------------------------------------------------------------- affine ----
 * Paper: Section 2 (the affine layer of the softmax-classifier example: the
 * product X W plus a bias row; its backward returns dX, dW, db in that order).
 * X is N x D, W is D x M, b is 1 x M, out is N x M, all row-major.
 *
 * Workspace (both calls): optional.  Products too small to fill the GPU by
 * their output tiles alone (few output rows and columns, a long reduction,
 * e.g. a batch-64 forward with D = 3136, M = 512) split the reduction over
 * blocks and add the partial products in a second, fixed-order pass; the
 * partials need up to affine_workspace_size(...) bytes.  With NULL (or fewer
 * bytes) the call splits less (at most what fits) and is still correct.  The
 * result is deterministic for a given workspace size: the split count, and so
 * the order of the additions, depends only on the sizes and workspace_bytes.
 * The workspace must be element aligned and must not overlap the call's
 * tensors (DMLNN_ERR_ARG); its contents on entry are ignored and on return are
 * undefined.  Calls that may run at the same time need separate workspaces.
 * Returns 0 for invalid arguments. */
DMLNN_API size_t affine_workspace_size(dmlnn_dtype dtype, int N, int D, int M);

/* Host-only plan query (no device access), like conv2d_plan: the launch shape
 * one affine product takes for these sizes and workspace_bytes.  product: 0 =
 * out = X W (M_out = N rows, N_out = M columns, reduction D), 1 = dX = g W^T,
 * 2 = dW = X^T g.  *tile: the edge of a block's output tile (16 or 32);
 * *waves: waves per block, each a k range of that tile; *splits: blocks per
 * tile along k (partials in the workspace when above 1).  Returns
 * DMLNN_ERR_ARG for invalid sizes or product, DMLNN_ERR_NULL for a NULL
 * output pointer. */
DMLNN_API int affine_plan(dmlnn_dtype dtype, int product, int N, int D, int M,
                          size_t workspace_bytes, int *tile, int *waves, int *splits);

/* out = X W + b, then max(., 0) if relu.  b may be NULL. */
DMLNN_API int affine_fwd(dmlnn_dtype dtype, const void *X, const void *W, const void *b, void *out,
                         int N, int D, int M, int relu, void *workspace,
                         size_t workspace_bytes, void *stream);

/* g = dout (masked to out_fwd > 0 when out_fwd != NULL);
 *   dX = g W^T (N x D), dW = X^T g (D x M), db = column sums of g (1 x M).
 * relu_input = 1 when X is the output of a relu: dX is then also multiplied
 * by (X > 0), the relu backward of the layer below folded into the product
 * (paper, Section "Future Work": vertical fusion across layers), so that
 * layer's backward can take dX with out_fwd = NULL and read no mask; dX may
 * then not overlap X.  relu_input = 0: dX as above.
 * Each output may be NULL (not computed), but not all three: the products are
 * independent, so a caller may compute them in separate calls on separate
 * streams (each with its own workspace).  The products of one call run one
 * after another on `stream` and share the workspace.  DMLNN_ERR_NULL when
 * dout, X or W is NULL or no output is given. */
DMLNN_API int affine_bwd(dmlnn_dtype dtype, const void *dout, const void *X, const void *W,
                         const void *out_fwd, void *dX, void *dW, void *db, int N, int D, int M,
                         int relu_input, void *workspace, size_t workspace_bytes, void *stream);

/* ----------------------------------------------------------- softmax_xent ----
 * Paper: Section 2 (the softmax-classifier example chains the softmax
 * forward, the cross-entropy backward and the softmax backward); one fused
 * pass with the same result.  Per row: p = exp(s - max s) / sum exp(s - max s);
 *   loss    = -(1/N) sum_{n,k} Y[n,k] * log p[n,k]   (one device scalar)
 *   dscores = (p * sum_k Y[n,k] - Y) / N
 * scores, Y, probs, dscores are N x K; probs may be NULL; loss points to one
 * element of dtype in device memory.
 * workspace (optional, workspace_bytes long): without one, a single block of
 * 1024 threads does the whole call, which suits small batches.  With one, the
 * rows are spread over as many blocks as the workspace has elements, up to the
 * number softmax_xent_workspace_size asks room for (2048 at most).  Each block
 * writes its share of the loss there, and a second pass adds the shares in
 * block order.  The result is deterministic for a given block count, which
 * depends only on N, K and workspace_bytes.  The one-block and many-block forms
 * add the row losses in different orders, so the last bits of the loss can
 * differ between them; dscores and probs are the same in both.  The workspace
 * must be element aligned and overlap none of the call's tensors (DMLNN_ERR_ARG);
 * its contents on entry are ignored.  Calls that may run at the same time need
 * separate workspaces. */
DMLNN_API int softmax_xent(dmlnn_dtype dtype, const void *scores, const void *Y, void *probs,
                 void *dscores, void *loss, int N, int K, void *workspace,
                 size_t workspace_bytes, void *stream);

/* Bytes of workspace softmax_xent uses at most for these sizes: one element of
 * dtype per block.  A block takes 16 x (64 / sw) rows, sw being the smallest
 * power of two >= K (at most 64), so the size is 0 when one block covers all N
 * rows (for K = 10, N <= 64).  Returns 0 for invalid arguments. */
DMLNN_API size_t softmax_xent_workspace_size(dmlnn_dtype dtype, int N, int K);

/* ------------------------------------------------------------- softmax_fwd ----
 * Paper: Section 2 (the softmax layer's forward), used alone for forward-only
 * scoring.  Row-wise, max-shifted:
 *   probs[n,k] = exp(scores[n,k] - max_k scores[n,:]) / sum_k exp(...)
 * scores and probs are N x K (probs may not alias scores). */
DMLNN_API int softmax_fwd(dmlnn_dtype dtype, const void *scores, void *probs, int N, int K,
                          void *stream);

/* ---------------------------------------------------- sgd_momentum_update ----
 * Paper: Section 2 (SGD with momentum is one of the NN library's optimizers;
 * the example's plain gradient step is the case mu = 0).
 *   v <- mu*v - lr*grad;  theta <- theta + v     (elementwise, in place)
 * theta, grad and v hold n elements. */
DMLNN_API int sgd_momentum_update(dmlnn_dtype dtype, void *theta, const void *grad, void *v,
                        double lr, double mu, long long n, void *stream);

/* ------------------------------------------------------------ optimizers ----
 * Paper: Section 2, "NN Library" (the library ships six optimizers: Adagrad,
 * Adam, RMSprop, SGD, SGD with momentum, SGD with Nesterov momentum).  The
 * paper names them without formulas; each update below is the published
 * method's usual statement (see the per-call comments).  All are elementwise
 * and in place over n elements of dtype; theta, grad and the state buffers are
 * caller-owned device memory, the state starts at zero and persists between
 * calls; arithmetic is done in dtype.  Returns DMLNN_ERR_NULL for a missing
 * buffer and DMLNN_ERR_ARG for n outside [1, INT_MAX] or a hyper-parameter
 * outside its stated range; nothing is launched then. */

/* Plain SGD (the gradient step of the paper's softmax-classifier example):
 *   theta <- theta - lr*grad */
DMLNN_API int sgd_update(dmlnn_dtype dtype, void *theta, const void *grad, double lr,
                         long long n, void *stream);

/* SGD with Nesterov momentum, in the form that keeps the current parameters:
 *   v' = mu*v - lr*grad;  theta <- theta - mu*v + (1 + mu)*v';  v <- v' */
DMLNN_API int sgd_nesterov_update(dmlnn_dtype dtype, void *theta, const void *grad, void *v,
                                  double lr, double mu, long long n, void *stream);

/* Adagrad: cache <- cache + grad^2;  theta <- theta - lr*grad / (sqrt(cache) + eps).
 * eps >= 0. */
DMLNN_API int adagrad_update(dmlnn_dtype dtype, void *theta, const void *grad, void *cache,
                             double lr, double eps, long long n, void *stream);

/* RMSprop: cache <- decay*cache + (1 - decay)*grad^2;
 *          theta <- theta - lr*grad / (sqrt(cache) + eps).   0 <= decay <= 1, eps >= 0. */
DMLNN_API int rmsprop_update(dmlnn_dtype dtype, void *theta, const void *grad, void *cache,
                             double lr, double decay, double eps, long long n, void *stream);

/* Adam, step t >= 1 (the caller counts steps from 1):
 *   m <- beta1*m + (1 - beta1)*grad;  v <- beta2*v + (1 - beta2)*grad^2;
 *   theta <- theta - lr_t * m / (sqrt(v) + eps),  lr_t = lr*sqrt(1 - beta2^t)/(1 - beta1^t)
 * (the bias correction folded into the step size).  0 <= beta1, beta2 < 1, eps >= 0. */
DMLNN_API int adam_update(dmlnn_dtype dtype, void *theta, const void *grad, void *m, void *v,
                          double lr, double beta1, double beta2, double eps, long long t,
                          long long n, void *stream);

/* --------------------------------------------------------- count_nonzero ----
 * Paper: Section 3, "Sparse Operations" (the number of non-zeros of every
 * intermediate drives the choice of operator).  Writes the number of entries
 * of X (n elements) different from zero to *out_dev (one int64 in device
 * memory). */
DMLNN_API int count_nonzero(dmlnn_dtype dtype, const void *X, long long n, long long *out_dev,
                  void *stream);

/* Human-readable description of the last failed call on this host thread
 * ("" if none).  The string stays valid until the next call on the thread. */
DMLNN_API const char *dmlnn_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* DMLNN_H */
