// C ABI of libdmlnn.so (declared in include/dmlnn.h): argument validation on the
// host, then dispatch to the kernel launchers.  Nothing here allocates device
// memory.  Validation happens before any HIP runtime call, so bad arguments are
// reported without a GPU and without launching anything.
#include <atomic>
#include <climits>
#include <cstdarg>
#include <cstdio>
#include <cstdlib>
#include <cmath>
#include <cstdint>
#include <initializer_list>
#include <utility>
#include <cstring>
#include <mutex>

#include "../../include/dmlnn.h"
#include "common.hpp"
#include "internal.hpp"

namespace {

thread_local char g_err[512] = "";
std::atomic<int> g_zero_skip{-1};

// Device scratch of conv2d_backward_filter_noalloc: one array per GPU (each
// device holds its own copy of a __device__ variable), reserved when the code
// object is loaded on that GPU.  In host code `scratch` names a host-side
// stand-in, never the device memory: its device address is looked up once per
// device with hipGetSymbolAddress and only that address is used.
static __device__ __align__(256) unsigned char scratch[DMLNN_NOALLOC_SCRATCH_BYTES];

int fail(int code, const char *fmt, ...)
{
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(g_err, sizeof(g_err), fmt, ap);
    va_end(ap);
    return code;
}

int zero_skip_mode()
{
    int m = g_zero_skip.load(std::memory_order_relaxed);
    if (m < 0) {
        const char *e = getenv("DMLNN_ZERO_SKIP");
        m = (e && (strcmp(e, "1") == 0 || strcmp(e, "on") == 0)) ? 1 : 0;
        int expected = -1;
        g_zero_skip.compare_exchange_strong(expected, m);
        m = g_zero_skip.load(std::memory_order_relaxed);
    }
    return m;
}

bool dtype_ok(int dt) { return dt == DMLNN_F64 || dt == DMLNN_F32; }

constexpr long long kMaxElems = (long long)INT_MAX;

bool count_ok(long long a, long long b) { return a >= 1 && b >= 1 && a * b <= kMaxElems; }

// The kernels are built for gfx950 only; check the current device once per id.
int device_check()
{
    static std::mutex mu;
    static int state[64] = {0};  // 0 unknown, 1 ok, 2 bad
    int dev = -1;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess || dev < 0 || dev >= 64)
        return fail(DMLNN_ERR_DEVICE, "no usable HIP device (%s)", hipGetErrorString(e));
    std::lock_guard<std::mutex> lk(mu);
    if (state[dev] == 0) {
        hipDeviceProp_t prop;
        e = hipGetDeviceProperties(&prop, dev);
        if (e != hipSuccess)
            return fail(DMLNN_ERR_DEVICE, "hipGetDeviceProperties failed: %s", hipGetErrorString(e));
        state[dev] = strncmp(prop.gcnArchName, "gfx950", 6) == 0 ? 1 : 2;
        if (state[dev] == 2)
            return fail(DMLNN_ERR_DEVICE, "device %d is %s; libdmlnn is built for gfx950", dev,
                        prop.gcnArchName);
    }
    if (state[dev] != 1) return fail(DMLNN_ERR_DEVICE, "device %d is not gfx950", dev);
    return DMLNN_OK;
}

// Device address of this device's scratch array (looked up on the first call
// on each device, with that device current), or null after a failed lookup.
void *scratch_ptr(int &status)
{
    static std::mutex mu;
    static void *ptr[64] = {nullptr};
    int dev = -1;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess || dev < 0 || dev >= 64) {
        status = fail(DMLNN_ERR_DEVICE, "no usable HIP device (%s)", hipGetErrorString(e));
        return nullptr;
    }
    std::lock_guard<std::mutex> lk(mu);
    if (!ptr[dev]) {
        void *p = nullptr;
        e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess || !p) {
            status = fail(DMLNN_ERR_DEVICE, "scratch lookup on device %d failed: %s", dev,
                          hipGetErrorString(e));
            return nullptr;
        }
        ptr[dev] = p;
    }
    status = DMLNN_OK;
    return ptr[dev];
}

int launched(hipError_t e, const char *what)
{
    if (e != hipSuccess) return fail(DMLNN_ERR_LAUNCH, "%s: launch failed: %s", what, hipGetErrorString(e));
    g_err[0] = '\0';
    return DMLNN_OK;
}

int conv_dims(dmlnn::ConvDims &d, int N, int C, int Hin, int Win, int F, int Hf, int Wf, int stride,
              int pad)
{
    if (N < 1 || C < 1 || Hin < 1 || Win < 1 || F < 1 || Hf < 1 || Wf < 1)
        return fail(DMLNN_ERR_ARG, "sizes must be >= 1 (N=%d C=%d Hin=%d Win=%d F=%d Hf=%d Wf=%d)",
                    N, C, Hin, Win, F, Hf, Wf);
    if (stride < 1 || pad < 0) return fail(DMLNN_ERR_ARG, "stride must be >= 1 and pad >= 0");
    d.N = N;
    d.C = C;
    d.Hin = Hin;
    d.Win = Win;
    d.F = F;
    d.Hf = Hf;
    d.Wf = Wf;
    d.stride = stride;
    d.pad = pad;
    d.Hout = conv2d_out_dim(Hin, Hf, stride, pad);
    d.Wout = conv2d_out_dim(Win, Wf, stride, pad);
    if (d.Hout < 1 || d.Wout < 1)
        return fail(DMLNN_ERR_ARG, "no window fits: Hout=%d Wout=%d", d.Hout, d.Wout);
    if (!count_ok(N, (long long)C * Hin * Win) || !count_ok(N, (long long)F * d.Hout * d.Wout) ||
        !count_ok(F, (long long)C * Hf * Wf) || (long long)Hin + 2LL * pad > INT_MAX / 4 ||
        (long long)Win + 2LL * pad > INT_MAX / 4)
        return fail(DMLNN_ERR_ARG, "tensor too large (element counts must be < 2^31)");
    return DMLNN_OK;
}

}  // namespace

extern "C" {

int conv2d_out_dim(int Hin, int Hf, int stride, int pad)
{
    if (Hin < 1 || Hf < 1 || stride < 1 || pad < 0) return 0;
    long long span = (long long)Hin + 2LL * pad - Hf;
    if (span < 0) return 0;
    long long r = span / stride + 1;
    return r > INT_MAX ? 0 : (int)r;
}

const char *dmlnn_last_error(void) { return g_err; }

int dmlnn_set_zero_skip(int mode)
{
    if (mode != 0 && mode != 1) return -1;
    int prev = zero_skip_mode();
    g_zero_skip.store(mode);
    return prev;
}

int conv2d_forward(dmlnn_dtype dtype, const void *X, const void *W, const void *b, void *out,
                   int N, int C, int Hin, int Win, int F, int Hf, int Wf, int stride, int pad,
                   int relu, void *stream)
{
    if (!dtype_ok(dtype)) return fail(DMLNN_ERR_DTYPE, "conv2d_forward: bad dtype %d", (int)dtype);
    if (!X || !W || !out) return fail(DMLNN_ERR_NULL, "conv2d_forward: X, W and out are required");
    if (relu != 0 && relu != 1) return fail(DMLNN_ERR_ARG, "conv2d_forward: relu must be 0 or 1");
    dmlnn::ConvDims d;
    if (int r = conv_dims(d, N, C, Hin, Win, F, Hf, Wf, stride, pad)) return r;
    if (int r = device_check()) return r;
    return launched(dmlnn::launch_conv_forward(dtype, X, W, b, out, d, relu, zero_skip_mode(),
                                               (hipStream_t)stream),
                    "conv2d_forward");
}

size_t conv2d_backward_filter_workspace_size(dmlnn_dtype dtype, int N, int C, int Hin, int Win,
                                             int F, int Hf, int Wf, int stride, int pad)
{
    if (!dtype_ok(dtype)) return 0;
    dmlnn::ConvDims d;
    if (conv_dims(d, N, C, Hin, Win, F, Hf, Wf, stride, pad)) return 0;
    return dmlnn::conv_wgrad_workspace_bytes(dtype, d);
}

int conv2d_backward_filter(dmlnn_dtype dtype, const void *X, const void *dout, const void *out_fwd,
                           void *dW, void *db, int N, int C, int Hin, int Win, int F, int Hf,
                           int Wf, int stride, int pad, void *workspace, size_t workspace_bytes,
                           void *stream)
{
    if (!dtype_ok(dtype))
        return fail(DMLNN_ERR_DTYPE, "conv2d_backward_filter: bad dtype %d", (int)dtype);
    if (!X || !dout || !dW)
        return fail(DMLNN_ERR_NULL, "conv2d_backward_filter: X, dout and dW are required");
    dmlnn::ConvDims d;
    if (int r = conv_dims(d, N, C, Hin, Win, F, Hf, Wf, stride, pad)) return r;
    const size_t need = dmlnn::conv_wgrad_workspace_bytes(dtype, d);
    if (need == 0) return fail(DMLNN_ERR_ARG, "conv2d_backward_filter: no tiling fits these sizes");
    if (!workspace || workspace_bytes < need)
        return fail(DMLNN_ERR_WORKSPACE, "conv2d_backward_filter: workspace of %zu bytes needed, %zu given",
                    need, workspace ? workspace_bytes : (size_t)0);
    if (int r = device_check()) return r;
    return launched(dmlnn::launch_conv_backward_filter(dtype, X, dout, out_fwd, dW, db, d, workspace,
                                                       zero_skip_mode(), (hipStream_t)stream),
                    "conv2d_backward_filter");
}

// Whether the byte ranges [a, a + na) and [b, b + nb) share a byte.
static bool overlaps(const void *a, size_t na, const void *b, size_t nb)
{
    const uintptr_t x = (uintptr_t)a, y = (uintptr_t)b;
    return x < y + nb && y < x + na;
}

int conv2d_backward_filter_emit(dmlnn_dtype dtype, const void *X, const void *dout,
                                const void *out_fwd, void *dW, void *db, void *g_out, int N,
                                int C, int Hin, int Win, int F, int Hf, int Wf, int stride,
                                int pad, void *workspace, size_t workspace_bytes, void *stream)
{
    const char *name = "conv2d_backward_filter_emit";
    if (!dtype_ok(dtype)) return fail(DMLNN_ERR_DTYPE, "%s: bad dtype %d", name, (int)dtype);
    if (!X || !dout || !dW || !g_out)
        return fail(DMLNN_ERR_NULL, "%s: X, dout, dW and g_out are required", name);
    dmlnn::ConvDims d;
    if (int r = conv_dims(d, N, C, Hin, Win, F, Hf, Wf, stride, pad)) return r;
    const size_t need = dmlnn::conv_wgrad_workspace_bytes(dtype, d);
    if (need == 0) return fail(DMLNN_ERR_ARG, "%s: no tiling fits these sizes", name);
    if (!workspace || workspace_bytes < need)
        return fail(DMLNN_ERR_WORKSPACE, "%s: workspace of %zu bytes needed, %zu given", name,
                    need, workspace ? workspace_bytes : (size_t)0);
    // g_out may be dout itself (each element is read and written by one
    // thread, and masking is idempotent), but no other operand
    const size_t esz = dtype == DMLNN_F64 ? 8 : 4;
    const size_t gbytes = (size_t)N * F * d.Hout * d.Wout * esz;
    const size_t xbytes = (size_t)N * C * Hin * Win * esz, wbytes = (size_t)F * C * Hf * Wf * esz;
    if (overlaps(g_out, gbytes, X, xbytes) || overlaps(g_out, gbytes, dW, wbytes) ||
        (db && overlaps(g_out, gbytes, db, (size_t)F * esz)) ||
        overlaps(g_out, gbytes, workspace, workspace_bytes) ||
        (out_fwd && out_fwd != dout && overlaps(g_out, gbytes, out_fwd, gbytes)))
        return fail(DMLNN_ERR_ARG, "%s: g_out overlaps another operand", name);
    if (int r = device_check()) return r;
    return launched(dmlnn::launch_conv_backward_filter(dtype, X, dout, out_fwd, dW, db, d, workspace,
                                                       zero_skip_mode(), (hipStream_t)stream,
                                                       nullptr, g_out),
                    name);
}

int conv2d_backward_filter_noalloc(dmlnn_dtype dtype, const void *X, const void *dout,
                                   const void *out_fwd, void *dW, void *db, int N, int C, int Hin,
                                   int Win, int F, int Hf, int Wf, int stride, int pad,
                                   void *stream)
{
    if (!dtype_ok(dtype))
        return fail(DMLNN_ERR_DTYPE, "conv2d_backward_filter_noalloc: bad dtype %d", (int)dtype);
    if (!X || !dout || !dW)
        return fail(DMLNN_ERR_NULL, "conv2d_backward_filter_noalloc: X, dout and dW are required");
    dmlnn::ConvDims d;
    if (int r = conv_dims(d, N, C, Hin, Win, F, Hf, Wf, stride, pad)) return r;
    const size_t need = dmlnn::conv_wgrad_workspace_bytes(dtype, d);
    if (need == 0)
        return fail(DMLNN_ERR_ARG, "conv2d_backward_filter_noalloc: no tiling fits these sizes");
    if (need > (size_t)DMLNN_NOALLOC_SCRATCH_BYTES)
        return fail(DMLNN_ERR_WORKSPACE,
                    "conv2d_backward_filter_noalloc: these sizes need %zu bytes of scratch, above "
                    "the library's %u; use conv2d_backward_filter with a workspace",
                    need, (unsigned)DMLNN_NOALLOC_SCRATCH_BYTES);
    if (int r = device_check()) return r;
    int status = DMLNN_OK;
    void *ws = scratch_ptr(status);
    if (!ws) return status;
    return launched(dmlnn::launch_conv_backward_filter(dtype, X, dout, out_fwd, dW, db, d, ws,
                                                       zero_skip_mode(), (hipStream_t)stream),
                    "conv2d_backward_filter_noalloc");
}

int conv2d_backward_data(dmlnn_dtype dtype, const void *W, const void *dout, const void *out_fwd,
                         void *dX, int N, int C, int Hin, int Win, int F, int Hf, int Wf, int stride,
                         int pad, void *stream)
{
    if (!dtype_ok(dtype))
        return fail(DMLNN_ERR_DTYPE, "conv2d_backward_data: bad dtype %d", (int)dtype);
    if (!W || !dout || !dX)
        return fail(DMLNN_ERR_NULL, "conv2d_backward_data: W, dout and dX are required");
    dmlnn::ConvDims d;
    if (int r = conv_dims(d, N, C, Hin, Win, F, Hf, Wf, stride, pad)) return r;
    if (int r = device_check()) return r;
    return launched(dmlnn::launch_conv_backward_data(dtype, W, dout, out_fwd, dX, d,
                                                     zero_skip_mode(), (hipStream_t)stream),
                    "conv2d_backward_data");
}

static int pool_dims(int N, int C, int Hin, int Win, int Hf, int Wf, int stride, int pad, int &Hout,
                     int &Wout);

static int plan_query(const char *name, dmlnn_dtype dtype, int pass, int form, int pool_h,
                      int pool_w, int pool_stride, int pool_pad, int N, int C, int Hin, int Win,
                      int F, int Hf, int Wf, int stride, int pad, int zero_skip,
                      dmlnn_conv_plan *plan)
{
    if (!dtype_ok(dtype)) return fail(DMLNN_ERR_DTYPE, "%s: bad dtype %d", name, (int)dtype);
    if (!plan) return fail(DMLNN_ERR_NULL, "%s: plan is required", name);
    if (pass < DMLNN_PASS_FORWARD || pass > DMLNN_PASS_BACKWARD_DATA)
        return fail(DMLNN_ERR_ARG, "%s: bad pass %d", name, pass);
    if (zero_skip != 0 && zero_skip != 1)
        return fail(DMLNN_ERR_ARG, "%s: zero_skip must be 0 or 1", name);
    dmlnn::ConvDims d;
    if (int r = conv_dims(d, N, C, Hin, Win, F, Hf, Wf, stride, pad)) return r;
    const bool fwd = pass == DMLNN_PASS_FORWARD;
    switch (form) {
    case DMLNN_FORM_PLAIN: break;
    case DMLNN_FORM_POOL_EPILOGUE:
    case DMLNN_FORM_POOLED_SOURCE: {
        if (fwd != (form == DMLNN_FORM_POOL_EPILOGUE))
            return fail(DMLNN_ERR_ARG, "%s: form %d does not apply to pass %d", name, form, pass);
        int Hp, Wp;
        if (int r = pool_dims(N, F, d.Hout, d.Wout, pool_h, pool_w, pool_stride, pool_pad, Hp, Wp))
            return r;
        if (form == DMLNN_FORM_POOLED_SOURCE &&
            (pool_pad != 0 || pool_stride < pool_h || pool_stride < pool_w))
            return fail(DMLNN_ERR_ARG, "%s: a pooled source needs unpadded windows that do not "
                        "overlap", name);
        break;
    }
    case DMLNN_FORM_CSR_INPUT:
    case DMLNN_FORM_BANKS:
        if (!fwd)
            return fail(DMLNN_ERR_ARG, "%s: form %d does not apply to pass %d", name, form, pass);
        break;
    default: return fail(DMLNN_ERR_ARG, "%s: bad form %d", name, form);
    }
    dmlnn::ConvPlanInfo info;
    if (dmlnn::conv_plan_info(dtype, pass, d, zero_skip, form, pool_h, pool_w, pool_stride,
                              pool_pad, info) != hipSuccess)
        return fail(DMLNN_ERR_ARG, "%s: no tiling fits these sizes", name);
    memset(plan, 0, sizeof(*plan));
    plan->kernel = info.kernel;
    plan->zero_skip = zero_skip && info.kernel != dmlnn::kConvSmallM &&
                      info.kernel != dmlnn::kConvResident &&
                      info.kernel != dmlnn::kWgradPoolSparse && form != DMLNN_FORM_POOLED_SOURCE;
    plan->tile_m = info.tile_m;
    plan->tile_pixels = info.tile_pixels;
    plan->blocks = info.blocks;
    plan->chunk = info.chunk;
    plan->k_split = info.k_split;
    plan->splits = info.splits;
    plan->window_width = info.window_width;
    plan->window_rows = info.window_rows;
    plan->lds_bytes = info.lds;
    plan->workspace_bytes =
        pass == DMLNN_PASS_BACKWARD_FILTER ? dmlnn::conv_wgrad_workspace_bytes(dtype, d) : 0;
    plan->tile_stride = info.tile_stride;
    plan->k_chunk = info.k_chunk;
    plan->slice_stride = info.slice_stride;
    plan->stage_bytes = info.stage_bytes;
    plan->window_bytes = info.window_bytes;
    plan->slice_bytes = info.slice_bytes;
    plan->slice_vec = info.slice_vec;
    plan->g_stride = info.g_stride;
    plan->row_slices = info.row_slices;
    plan->pipelined = info.pipelined;
    plan->fused = info.fused;
    plan->row_staged = info.row_staged;
    g_err[0] = '\0';
    return DMLNN_OK;
}

int conv2d_plan(dmlnn_dtype dtype, int pass, int N, int C, int Hin, int Win, int F, int Hf, int Wf,
                int stride, int pad, int zero_skip, dmlnn_conv_plan *plan)
{
    return plan_query("conv2d_plan", dtype, pass, DMLNN_FORM_PLAIN, 0, 0, 0, 0, N, C, Hin, Win, F,
                      Hf, Wf, stride, pad, zero_skip, plan);
}

int conv2d_plan_fused(dmlnn_dtype dtype, int pass, int form, int pool_h, int pool_w,
                      int pool_stride, int pool_pad, int N, int C, int Hin, int Win, int F, int Hf,
                      int Wf, int stride, int pad, int zero_skip, dmlnn_conv_plan *plan)
{
    return plan_query("conv2d_plan_fused", dtype, pass, form, pool_h, pool_w, pool_stride,
                      pool_pad, N, C, Hin, Win, F, Hf, Wf, stride, pad, zero_skip, plan);
}

int conv2d_zero_skip_choice(dmlnn_dtype dtype, int pass, long long nnz, int N, int C, int Hin,
                            int Win, int F, int Hf, int Wf, int stride, int pad)
{
    if (!dtype_ok(dtype) || pass < DMLNN_PASS_FORWARD || pass > DMLNN_PASS_BACKWARD_DATA) return -1;
    dmlnn::ConvDims d;
    if (conv_dims(d, N, C, Hin, Win, F, Hf, Wf, stride, pad)) return -1;
    const long long n = pass == DMLNN_PASS_BACKWARD_DATA ? (long long)N * F * d.Hout * d.Wout
                                                         : (long long)N * C * Hin * Win;
    if (nnz < 0 || nnz > n) return -1;
    // the kernel the pass takes in the dense mode: when it has no skip form (the
    // vector-ALU small-M kernel, the filter-resident forward), the skip mode
    // would swap it for a different kernel, not skip its work
    dmlnn::ConvPlanInfo info;
    if (dmlnn::conv_plan_info(dtype, pass, d, 0, 0, 0, 0, 0, 0, info) != hipSuccess) return -1;
    if (info.kernel == dmlnn::kConvSmallM || info.kernel == dmlnn::kConvResident) return 0;
    // expected share of all-zero 64-value fragments under independent zeros
    const double density = (double)nnz / (double)n;
    return pow(1.0 - density, 64.0) >= 0.05 ? 1 : 0;
}

int bias_add_relu(dmlnn_dtype dtype, const void *X, const void *b, void *out, int N, int C, int HW,
                  int relu, void *stream)
{
    if (!dtype_ok(dtype)) return fail(DMLNN_ERR_DTYPE, "bias_add_relu: bad dtype %d", (int)dtype);
    if (!X || !out) return fail(DMLNN_ERR_NULL, "bias_add_relu: X and out are required");
    if (N < 1 || C < 1 || HW < 1 || !count_ok(N, (long long)C * HW))
        return fail(DMLNN_ERR_ARG, "bias_add_relu: bad sizes N=%d C=%d HW=%d", N, C, HW);
    if (relu != 0 && relu != 1) return fail(DMLNN_ERR_ARG, "bias_add_relu: relu must be 0 or 1");
    if (int r = device_check()) return r;
    return launched(dmlnn::launch_bias_add_relu(dtype, X, b, out, N, C, HW, relu, (hipStream_t)stream),
                    "bias_add_relu");
}

static int pool_dims(int N, int C, int Hin, int Win, int Hf, int Wf, int stride, int pad, int &Hout,
                     int &Wout)
{
    if (N < 1 || C < 1 || Hin < 1 || Win < 1 || Hf < 1 || Wf < 1 || stride < 1 || pad < 0)
        return fail(DMLNN_ERR_ARG, "max_pool2d: sizes must be >= 1, stride >= 1, pad >= 0");
    if (pad >= Hf || pad >= Wf) return fail(DMLNN_ERR_ARG, "max_pool2d: pad must be < Hf and < Wf");
    Hout = conv2d_out_dim(Hin, Hf, stride, pad);
    Wout = conv2d_out_dim(Win, Wf, stride, pad);
    if (Hout < 1 || Wout < 1) return fail(DMLNN_ERR_ARG, "max_pool2d: no window fits");
    if (!count_ok(N, (long long)C * Hin * Win) || !count_ok(N, (long long)C * Hout * Wout))
        return fail(DMLNN_ERR_ARG, "max_pool2d: tensor too large");
    return DMLNN_OK;
}

int max_pool2d_fwd(dmlnn_dtype dtype, const void *X, void *out, int32_t *argmax, int N, int C,
                   int Hin, int Win, int Hf, int Wf, int stride, int pad, void *stream)
{
    if (!dtype_ok(dtype)) return fail(DMLNN_ERR_DTYPE, "max_pool2d_fwd: bad dtype %d", (int)dtype);
    if (!X || !out || !argmax) return fail(DMLNN_ERR_NULL, "max_pool2d_fwd: X, out, argmax are required");
    int Hout, Wout;
    if (int r = pool_dims(N, C, Hin, Win, Hf, Wf, stride, pad, Hout, Wout)) return r;
    if (int r = device_check()) return r;
    return launched(dmlnn::launch_max_pool_fwd(dtype, X, out, argmax, N, C, Hin, Win, Hf, Wf, stride,
                                               pad, Hout, Wout, (hipStream_t)stream),
                    "max_pool2d_fwd");
}

int max_pool2d_bwd(dmlnn_dtype dtype, const void *dout, const int32_t *argmax, void *dX, int N,
                   int C, int Hin, int Win, int Hf, int Wf, int stride, int pad, void *stream)
{
    if (!dtype_ok(dtype)) return fail(DMLNN_ERR_DTYPE, "max_pool2d_bwd: bad dtype %d", (int)dtype);
    if (!dout || !argmax || !dX) return fail(DMLNN_ERR_NULL, "max_pool2d_bwd: dout, argmax, dX are required");
    int Hout, Wout;
    if (int r = pool_dims(N, C, Hin, Win, Hf, Wf, stride, pad, Hout, Wout)) return r;
    if (int r = device_check()) return r;
    return launched(dmlnn::launch_max_pool_bwd(dtype, dout, argmax, nullptr, dX, N, C, Hin, Win,
                                               Hf, Wf, stride, pad, Hout, Wout,
                                               (hipStream_t)stream),
                    "max_pool2d_bwd");
}

int conv2d_forward_multi(dmlnn_dtype dtype, const void *X, const void *Wcat, const void *bcat,
                         void *const *outs, const int *Fs, int nbanks, int N, int C, int Hin,
                         int Win, int Hf, int Wf, int stride, int pad, int relu, void *stream)
{
    if (!dtype_ok(dtype)) return fail(DMLNN_ERR_DTYPE, "conv2d_forward_multi: bad dtype %d", (int)dtype);
    if (!X || !Wcat || !outs || !Fs)
        return fail(DMLNN_ERR_NULL, "conv2d_forward_multi: X, Wcat, outs and Fs are required");
    if (nbanks < 1 || nbanks > 8)
        return fail(DMLNN_ERR_ARG, "conv2d_forward_multi: nbanks=%d outside [1, 8]", nbanks);
    long long Ftot = 0;
    for (int b = 0; b < nbanks; ++b) {
        if (Fs[b] < 1) return fail(DMLNN_ERR_ARG, "conv2d_forward_multi: bank %d has F=%d", b, Fs[b]);
        if (!outs[b]) return fail(DMLNN_ERR_NULL, "conv2d_forward_multi: outs[%d] is NULL", b);
        Ftot += Fs[b];
    }
    if (Ftot > INT_MAX) return fail(DMLNN_ERR_ARG, "conv2d_forward_multi: too many filters");
    dmlnn::ConvDims d;
    if (int r = conv_dims(d, N, C, Hin, Win, (int)Ftot, Hf, Wf, stride, pad)) return r;
    if (int r = device_check()) return r;
    const hipStream_t s = (hipStream_t)stream;
    hipError_t e = dmlnn::launch_conv_forward_multi(dtype, X, Wcat, bcat, outs, Fs, nbanks, d,
                                                    relu, zero_skip_mode(), s);
    if (e == hipErrorNotSupported) {
        // The register-staged path has no per-bank epilogue: one launch per bank.
        (void)hipGetLastError();
        const size_t tsz = dtype == DMLNN_F64 ? 8 : 4;
        const size_t K = (size_t)C * Hf * Wf;
        long long off = 0;
        e = hipSuccess;
        for (int b = 0; b < nbanks && e == hipSuccess; ++b) {
            dmlnn::ConvDims db = d;
            db.F = Fs[b];
            const char *wb = (const char *)Wcat + (size_t)off * K * tsz;
            const char *bb = bcat ? (const char *)bcat + (size_t)off * tsz : nullptr;
            e = dmlnn::launch_conv_forward(dtype, X, wb, bb, outs[b], db, relu, zero_skip_mode(), s);
            off += Fs[b];
        }
    }
    return launched(e, "conv2d_forward_multi");
}

int conv2d_forward_csr(dmlnn_dtype dtype, const int32_t *rowptr, const int32_t *colidx,
                       const void *vals, int nnz, int32_t *row_index, const void *W,
                       const void *b, void *out, int N, int C, int Hin, int Win, int F, int Hf,
                       int Wf, int stride, int pad, int relu, void *stream)
{
    if (!dtype_ok(dtype)) return fail(DMLNN_ERR_DTYPE, "conv2d_forward_csr: bad dtype %d", (int)dtype);
    if (!rowptr || !row_index || !W || !out || (nnz > 0 && (!colidx || !vals)))
        return fail(DMLNN_ERR_NULL,
                    "conv2d_forward_csr: rowptr, row_index, W, out (and colidx, vals if nnz > 0) "
                    "are required");
    if (nnz < 0) return fail(DMLNN_ERR_ARG, "conv2d_forward_csr: bad nnz=%d", nnz);
    dmlnn::ConvDims d;
    if (int r = conv_dims(d, N, C, Hin, Win, F, Hf, Wf, stride, pad)) return r;
    if (nnz > (long long)N * C * Hin * Win)
        return fail(DMLNN_ERR_ARG, "conv2d_forward_csr: nnz=%d exceeds the matrix size", nnz);
    if (int r = device_check()) return r;
    // nnz-driven choice: below 5% density whole MFMA fragments of the staged
    // window are likely zero, so the ballot-skip kernel is used.
    const int skip = zero_skip_mode() || (long long)nnz * 20 < (long long)N * C * Hin * Win;
    return launched(dmlnn::launch_conv_forward_csr(dtype, rowptr, colidx, vals, nnz, row_index, W,
                                                   b, out, d, relu, skip, (hipStream_t)stream),
                    "conv2d_forward_csr");
}

int max_pool2d_bwd_relu(dmlnn_dtype dtype, const void *dout, const int32_t *argmax,
                        const void *pooled, void *dX, int N, int C, int Hin, int Win, int Hf,
                        int Wf, int stride, int pad, void *stream)
{
    if (!dtype_ok(dtype)) return fail(DMLNN_ERR_DTYPE, "max_pool2d_bwd_relu: bad dtype %d", (int)dtype);
    if (!dout || !argmax || !pooled || !dX)
        return fail(DMLNN_ERR_NULL, "max_pool2d_bwd_relu: dout, argmax, pooled, dX are required");
    int Hout, Wout;
    if (int r = pool_dims(N, C, Hin, Win, Hf, Wf, stride, pad, Hout, Wout)) return r;
    if (int r = device_check()) return r;
    return launched(dmlnn::launch_max_pool_bwd(dtype, dout, argmax, pooled, dX, N, C, Hin, Win,
                                               Hf, Wf, stride, pad, Hout, Wout,
                                               (hipStream_t)stream),
                    "max_pool2d_bwd_relu");
}

int conv2d_forward_pool(dmlnn_dtype dtype, const void *X, const void *W, const void *b, void *out,
                        void *pooled, int32_t *argmax, int N, int C, int Hin, int Win, int F,
                        int Hf, int Wf, int stride, int pad, int relu, int pool_h, int pool_w,
                        int pool_stride, int pool_pad, void *stream)
{
    if (!dtype_ok(dtype)) return fail(DMLNN_ERR_DTYPE, "conv2d_forward_pool: bad dtype %d", (int)dtype);
    if (!X || !W || !pooled || !argmax)
        return fail(DMLNN_ERR_NULL, "conv2d_forward_pool: X, W, pooled and argmax are required");
    dmlnn::ConvDims d;
    if (int r = conv_dims(d, N, C, Hin, Win, F, Hf, Wf, stride, pad)) return r;
    int Hp, Wp;
    if (int r = pool_dims(N, F, d.Hout, d.Wout, pool_h, pool_w, pool_stride, pool_pad, Hp, Wp))
        return r;
    if (int r = device_check()) return r;
    const hipStream_t s = (hipStream_t)stream;
    hipError_t e = hipErrorNotSupported;
    if (pool_pad == 0)
        e = dmlnn::launch_conv_forward_pool(dtype, X, W, b, out, pooled, argmax, d, relu, pool_h,
                                            pool_w, pool_stride, Hp, Wp, zero_skip_mode(), s);
    if (e == hipErrorNotSupported) {
        // Unfused: the conv output is needed as the pool's input.
        if (!out)
            return fail(DMLNN_ERR_ARG,
                        "conv2d_forward_pool: this pooling (%dx%d stride %d pad %d after a "
                        "%dx%d output) is not fusable; pass the conv output buffer",
                        pool_h, pool_w, pool_stride, pool_pad, d.Hout, d.Wout);
        (void)hipGetLastError();
        e = dmlnn::launch_conv_forward(dtype, X, W, b, out, d, relu, zero_skip_mode(), s);
        if (e == hipSuccess)
            e = dmlnn::launch_max_pool_fwd(dtype, out, pooled, argmax, N, F, d.Hout, d.Wout,
                                           pool_h, pool_w, pool_stride, pool_pad, Hp, Wp, s);
    }
    return launched(e, "conv2d_forward_pool");
}

// Validation shared by the two pooled backward calls: the pool after the conv
// must have windows that do not overlap and no padding.
static int pooled_src(const char *name, const dmlnn::ConvDims &d, const void *dpool,
                      const int32_t *argmax, const void *pooled, int ph, int pw, int ps, int pp,
                      dmlnn::PoolSrc &src)
{
    int Hp, Wp;
    if (int r = pool_dims(d.N, d.F, d.Hout, d.Wout, ph, pw, ps, pp, Hp, Wp)) return r;
    if (pp != 0 || ps < ph || ps < pw)
        return fail(DMLNN_ERR_ARG,
                    "%s: the pool windows (%dx%d stride %d pad %d) overlap or are padded; run "
                    "max_pool2d_bwd_relu and the plain conv backward call instead",
                    name, ph, pw, ps, pp);
    if (d.Hout >= 65536 || d.Wout >= 65536)
        return fail(DMLNN_ERR_ARG, "%s: conv output of %dx%d is too large", name, d.Hout, d.Wout);
    src.dpool = dpool;
    src.argmax = argmax;
    src.pooled = pooled;
    src.PH = ph;
    src.PW = pw;
    src.PS = ps;
    src.Hp = Hp;
    src.Wp = Wp;
    src.magic_ps = dmlnn::host_magic(ps);
    return DMLNN_OK;
}

int conv2d_backward_filter_pooled(dmlnn_dtype dtype, const void *X, const void *dpool,
                                  const int32_t *argmax, const void *pooled, void *dW, void *db,
                                  int N, int C, int Hin, int Win, int F, int Hf, int Wf, int stride,
                                  int pad, int pool_h, int pool_w, int pool_stride, int pool_pad,
                                  void *workspace, size_t workspace_bytes, void *stream)
{
    const char *name = "conv2d_backward_filter_pooled";
    if (!dtype_ok(dtype)) return fail(DMLNN_ERR_DTYPE, "%s: bad dtype %d", name, (int)dtype);
    if (!X || !dpool || !argmax || !pooled || !dW)
        return fail(DMLNN_ERR_NULL, "%s: X, dpool, argmax, pooled and dW are required", name);
    dmlnn::ConvDims d;
    if (int r = conv_dims(d, N, C, Hin, Win, F, Hf, Wf, stride, pad)) return r;
    dmlnn::PoolSrc src;
    if (int r = pooled_src(name, d, dpool, argmax, pooled, pool_h, pool_w, pool_stride, pool_pad,
                           src))
        return r;
    const size_t need = dmlnn::conv_wgrad_workspace_bytes(dtype, d);
    if (need == 0) return fail(DMLNN_ERR_ARG, "%s: no tiling fits these sizes", name);
    if (!workspace || workspace_bytes < need)
        return fail(DMLNN_ERR_WORKSPACE, "%s: workspace of %zu bytes needed, %zu given", name,
                    need, workspace ? workspace_bytes : (size_t)0);
    if (int r = device_check()) return r;
    return launched(dmlnn::launch_conv_backward_filter(dtype, X, nullptr, nullptr, dW, db, d,
                                                       workspace, 0, (hipStream_t)stream, &src),
                    name);
}

int conv2d_backward_data_pooled(dmlnn_dtype dtype, const void *W, const void *dpool,
                                const int32_t *argmax, const void *pooled, void *dX, int N, int C,
                                int Hin, int Win, int F, int Hf, int Wf, int stride, int pad,
                                int pool_h, int pool_w, int pool_stride, int pool_pad, void *stream)
{
    const char *name = "conv2d_backward_data_pooled";
    if (!dtype_ok(dtype)) return fail(DMLNN_ERR_DTYPE, "%s: bad dtype %d", name, (int)dtype);
    if (!W || !dpool || !argmax || !pooled || !dX)
        return fail(DMLNN_ERR_NULL, "%s: W, dpool, argmax, pooled and dX are required", name);
    dmlnn::ConvDims d;
    if (int r = conv_dims(d, N, C, Hin, Win, F, Hf, Wf, stride, pad)) return r;
    dmlnn::PoolSrc src;
    if (int r = pooled_src(name, d, dpool, argmax, pooled, pool_h, pool_w, pool_stride, pool_pad,
                           src))
        return r;
    if (int r = device_check()) return r;
    return launched(dmlnn::launch_conv_backward_data(dtype, W, nullptr, nullptr, dX, d, 0,
                                                     (hipStream_t)stream, &src),
                    name);
}

size_t affine_workspace_size(dmlnn_dtype dtype, int N, int D, int M)
{
    if (!dtype_ok(dtype) || !count_ok(N, D) || !count_ok(D, M) || !count_ok(N, M)) return 0;
    return dmlnn::affine_workspace_bytes(dtype, N, D, M);
}

int affine_plan(dmlnn_dtype dtype, int product, int N, int D, int M, size_t workspace_bytes,
                int *tile, int *waves, int *splits)
{
    if (!dtype_ok(dtype)) return fail(DMLNN_ERR_DTYPE, "affine_plan: bad dtype %d", (int)dtype);
    if (!tile || !waves || !splits) return fail(DMLNN_ERR_NULL, "affine_plan: NULL output");
    if (!count_ok(N, D) || !count_ok(D, M) || !count_ok(N, M) || product < 0 || product > 2)
        return fail(DMLNN_ERR_ARG, "affine_plan: bad product %d or sizes N=%d D=%d M=%d",
                    product, N, D, M);
    const size_t el = dtype == DMLNN_F64 ? 8 : 4;
    // (rows, columns, reduction) of the product
    const int r = product == 2 ? D : N, c = product == 1 ? D : M, k = product == 0 ? D
                                                                 : (product == 1 ? M : N);
    const dmlnn::GemmPlan p = dmlnn::gemm_plan(r, c, k, el, workspace_bytes);
    *tile = 16 * p.wt;
    *waves = p.nk;
    *splits = p.splits;
    return DMLNN_OK;
}

// An affine workspace is optional; when given it must be element aligned and
// must not overlap the tensors the call reads or writes.
static int workspace_ok(const char *name, dmlnn_dtype dtype, void *ws, size_t ws_bytes,
                        std::initializer_list<std::pair<const void *, size_t>> tensors)
{
    if (!ws || ws_bytes == 0) return DMLNN_OK;
    const size_t esz = dtype == DMLNN_F64 ? 8 : 4;
    if ((uintptr_t)ws % esz) return fail(DMLNN_ERR_ARG, "%s: workspace is not element aligned", name);
    for (const auto &t : tensors)
        if (t.first && overlaps(ws, ws_bytes, t.first, t.second))
            return fail(DMLNN_ERR_ARG, "%s: workspace overlaps a tensor of the call", name);
    return DMLNN_OK;
}

int affine_fwd(dmlnn_dtype dtype, const void *X, const void *W, const void *b, void *out, int N,
               int D, int M, int relu, void *workspace, size_t workspace_bytes, void *stream)
{
    if (!dtype_ok(dtype)) return fail(DMLNN_ERR_DTYPE, "affine_fwd: bad dtype %d", (int)dtype);
    if (!X || !W || !out) return fail(DMLNN_ERR_NULL, "affine_fwd: X, W and out are required");
    if (!count_ok(N, D) || !count_ok(D, M) || !count_ok(N, M))
        return fail(DMLNN_ERR_ARG, "affine_fwd: bad sizes N=%d D=%d M=%d", N, D, M);
    if (relu != 0 && relu != 1) return fail(DMLNN_ERR_ARG, "affine_fwd: relu must be 0 or 1");
    const size_t esz = dtype == DMLNN_F64 ? 8 : 4;
    if (int r = workspace_ok("affine_fwd", dtype, workspace, workspace_bytes,
                                    {{X, (size_t)N * D * esz}, {W, (size_t)D * M * esz},
                                     {b, (size_t)M * esz}, {out, (size_t)N * M * esz}}))
        return r;
    if (int r = device_check()) return r;
    return launched(dmlnn::launch_affine_fwd(dtype, X, W, b, out, N, D, M, relu, workspace,
                                             workspace_bytes, (hipStream_t)stream),
                    "affine_fwd");
}

int affine_bwd(dmlnn_dtype dtype, const void *dout, const void *X, const void *W,
               const void *out_fwd, void *dX, void *dW, void *db, int N, int D, int M,
               int relu_input, void *workspace, size_t workspace_bytes, void *stream)
{
    if (!dtype_ok(dtype)) return fail(DMLNN_ERR_DTYPE, "affine_bwd: bad dtype %d", (int)dtype);
    if (!dout || !X || !W) return fail(DMLNN_ERR_NULL, "affine_bwd: dout, X and W are required");
    if (!dX && !dW && !db) return fail(DMLNN_ERR_NULL, "affine_bwd: no output (dX, dW, db all NULL)");
    if (!count_ok(N, D) || !count_ok(D, M) || !count_ok(N, M))
        return fail(DMLNN_ERR_ARG, "affine_bwd: bad sizes N=%d D=%d M=%d", N, D, M);
    if (relu_input != 0 && relu_input != 1)
        return fail(DMLNN_ERR_ARG, "affine_bwd: relu_input must be 0 or 1");
    const size_t esz = dtype == DMLNN_F64 ? 8 : 4;
    if (int r = workspace_ok("affine_bwd", dtype, workspace, workspace_bytes,
                                    {{dout, (size_t)N * M * esz}, {X, (size_t)N * D * esz},
                                     {W, (size_t)D * M * esz}, {out_fwd, (size_t)N * M * esz},
                                     {dX, (size_t)N * D * esz}, {dW, (size_t)D * M * esz},
                                     {db, (size_t)M * esz}}))
        return r;
    if (dX && relu_input && overlaps(dX, (size_t)N * D * esz, X, (size_t)N * D * esz))
        return fail(DMLNN_ERR_ARG, "affine_bwd: with relu_input, dX may not overlap X");
    if (int r = device_check()) return r;
    return launched(dmlnn::launch_affine_bwd(dtype, dout, X, W, out_fwd, dX, dW, db, N, D, M,
                                             relu_input, workspace, workspace_bytes,
                                             (hipStream_t)stream),
                    "affine_bwd");
}

size_t softmax_xent_workspace_size(dmlnn_dtype dtype, int N, int K)
{
    if (!dtype_ok(dtype) || !count_ok(N, K)) return 0;
    return dmlnn::softmax_xent_workspace_bytes(dtype, N, K);
}

int softmax_xent(dmlnn_dtype dtype, const void *scores, const void *Y, void *probs, void *dscores,
                 void *loss, int N, int K, void *workspace, size_t workspace_bytes, void *stream)
{
    if (!dtype_ok(dtype)) return fail(DMLNN_ERR_DTYPE, "softmax_xent: bad dtype %d", (int)dtype);
    if (!scores || !Y || !dscores || !loss)
        return fail(DMLNN_ERR_NULL, "softmax_xent: scores, Y, dscores and loss are required");
    if (!count_ok(N, K)) return fail(DMLNN_ERR_ARG, "softmax_xent: bad sizes N=%d K=%d", N, K);
    const size_t esz = dtype == DMLNN_F64 ? 8 : 4, nk = (size_t)N * K * esz;
    if (int r = workspace_ok("softmax_xent", dtype, workspace, workspace_bytes,
                             {{scores, nk}, {Y, nk}, {probs, nk}, {dscores, nk}, {loss, esz}}))
        return r;
    if (int r = device_check()) return r;
    return launched(dmlnn::launch_softmax_xent(dtype, scores, Y, probs, dscores, loss, N, K,
                                               workspace, workspace_bytes, (hipStream_t)stream),
                    "softmax_xent");
}

int softmax_fwd(dmlnn_dtype dtype, const void *scores, void *probs, int N, int K, void *stream)
{
    if (!dtype_ok(dtype)) return fail(DMLNN_ERR_DTYPE, "softmax_fwd: bad dtype %d", (int)dtype);
    if (!scores || !probs) return fail(DMLNN_ERR_NULL, "softmax_fwd: scores and probs are required");
    if (!count_ok(N, K)) return fail(DMLNN_ERR_ARG, "softmax_fwd: bad sizes N=%d K=%d", N, K);
    if (scores == probs) return fail(DMLNN_ERR_ARG, "softmax_fwd: probs may not alias scores");
    if (int r = device_check()) return r;
    return launched(dmlnn::launch_softmax(dtype, scores, probs, N, K, (hipStream_t)stream),
                    "softmax_fwd");
}

int sgd_momentum_update(dmlnn_dtype dtype, void *theta, const void *grad, void *v, double lr,
                        double mu, long long n, void *stream)
{
    if (!dtype_ok(dtype)) return fail(DMLNN_ERR_DTYPE, "sgd_momentum_update: bad dtype %d", (int)dtype);
    if (!theta || !grad || !v) return fail(DMLNN_ERR_NULL, "sgd_momentum_update: theta, grad, v are required");
    if (n < 1 || n > kMaxElems) return fail(DMLNN_ERR_ARG, "sgd_momentum_update: bad n=%lld", n);
    if (int r = device_check()) return r;
    return launched(dmlnn::launch_sgd_momentum(dtype, theta, grad, v, lr, mu, n, (hipStream_t)stream),
                    "sgd_momentum_update");
}

static int optim_common(const char *name, dmlnn_dtype dtype, const void *theta, const void *grad,
                        const void *s1, const void *s2, long long n)
{
    if (!dtype_ok(dtype)) return fail(DMLNN_ERR_DTYPE, "%s: bad dtype %d", name, (int)dtype);
    if (!theta || !grad || !s1 || !s2)
        return fail(DMLNN_ERR_NULL, "%s: theta, grad and the state buffers are required", name);
    if (n < 1 || n > kMaxElems) return fail(DMLNN_ERR_ARG, "%s: bad n=%lld", name, n);
    return DMLNN_OK;
}

int sgd_update(dmlnn_dtype dtype, void *theta, const void *grad, double lr, long long n,
               void *stream)
{
    if (int r = optim_common("sgd_update", dtype, theta, grad, theta, theta, n)) return r;
    if (int r = device_check()) return r;
    return launched(dmlnn::launch_sgd(dtype, theta, grad, lr, n, (hipStream_t)stream),
                    "sgd_update");
}

int sgd_nesterov_update(dmlnn_dtype dtype, void *theta, const void *grad, void *v, double lr,
                        double mu, long long n, void *stream)
{
    if (int r = optim_common("sgd_nesterov_update", dtype, theta, grad, v, v, n)) return r;
    if (int r = device_check()) return r;
    return launched(dmlnn::launch_sgd_nesterov(dtype, theta, grad, v, lr, mu, n,
                                               (hipStream_t)stream),
                    "sgd_nesterov_update");
}

int adagrad_update(dmlnn_dtype dtype, void *theta, const void *grad, void *cache, double lr,
                   double eps, long long n, void *stream)
{
    if (int r = optim_common("adagrad_update", dtype, theta, grad, cache, cache, n)) return r;
    if (!(eps >= 0.0)) return fail(DMLNN_ERR_ARG, "adagrad_update: eps must be >= 0");
    if (int r = device_check()) return r;
    return launched(dmlnn::launch_adagrad(dtype, theta, grad, cache, lr, eps, n,
                                          (hipStream_t)stream),
                    "adagrad_update");
}

int rmsprop_update(dmlnn_dtype dtype, void *theta, const void *grad, void *cache, double lr,
                   double decay, double eps, long long n, void *stream)
{
    if (int r = optim_common("rmsprop_update", dtype, theta, grad, cache, cache, n)) return r;
    if (!(decay >= 0.0 && decay <= 1.0) || !(eps >= 0.0))
        return fail(DMLNN_ERR_ARG, "rmsprop_update: need 0 <= decay <= 1 and eps >= 0");
    if (int r = device_check()) return r;
    return launched(dmlnn::launch_rmsprop(dtype, theta, grad, cache, lr, decay, eps, n,
                                          (hipStream_t)stream),
                    "rmsprop_update");
}

int adam_update(dmlnn_dtype dtype, void *theta, const void *grad, void *m, void *v, double lr,
                double beta1, double beta2, double eps, long long t, long long n, void *stream)
{
    if (int r = optim_common("adam_update", dtype, theta, grad, m, v, n)) return r;
    if (!(beta1 >= 0.0 && beta1 < 1.0) || !(beta2 >= 0.0 && beta2 < 1.0) || !(eps >= 0.0))
        return fail(DMLNN_ERR_ARG, "adam_update: need 0 <= beta1, beta2 < 1 and eps >= 0");
    if (t < 1) return fail(DMLNN_ERR_ARG, "adam_update: step t=%lld must be >= 1", t);
    if (int r = device_check()) return r;
    return launched(dmlnn::launch_adam(dtype, theta, grad, m, v, lr, beta1, beta2, eps, t, n,
                                       (hipStream_t)stream),
                    "adam_update");
}

int count_nonzero(dmlnn_dtype dtype, const void *X, long long n, long long *out_dev, void *stream)
{
    if (!dtype_ok(dtype)) return fail(DMLNN_ERR_DTYPE, "count_nonzero: bad dtype %d", (int)dtype);
    if (!X || !out_dev) return fail(DMLNN_ERR_NULL, "count_nonzero: X and out_dev are required");
    if (n < 1 || n > kMaxElems) return fail(DMLNN_ERR_ARG, "count_nonzero: bad n=%lld", n);
    if (int r = device_check()) return r;
    return launched(dmlnn::launch_count_nonzero(dtype, X, n, out_dev, (hipStream_t)stream),
                    "count_nonzero");
}

}  // extern "C"
