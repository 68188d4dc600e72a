/*
 * Reference oracle for the DML-style conv2d layer and its neighbours.
 *
 * TEST INFRASTRUCTURE ONLY.  This file is a plain, slow, obviously-correct CPU
 * implementation of what the GPU path computes.  Only the test-suite, the smoke
 * check and the CPU-baseline leg of the benchmark may load it.  It shares no
 * code, header, table or helper with the HIP library, and the HIP library never
 * calls it.
 *
 * Everything is computed in double precision with the textbook definitions, in
 * a fixed summation order stated per function.  OpenMP parallelises only over
 * independent output elements, so results do not depend on the thread count.
 *
 * Data layout (paper, Section 3 "Tensor Representation"): a 4-d tensor
 * [N, C, H, W] is an N x (C*H*W) matrix: the dimensions after the first are
 * folded into the column index.  Reading used here: row-major in the listed order,
 * i.e. column index c*H*W + h*W + w.  Filters are F x (C*Hf*Wf) with column
 * c*Hf*Wf + i*Wf + j; the conv bias has one entry per filter.
 *
 * Every function below is pinned by tests that do not re-type its formula
 * (library routines, closed forms, invariants, finite differences); see the
 * test files named test_oracle_*.py.
 */
#include <math.h>
#include <stdint.h>
#include <stddef.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

/* ------------------------------------------------------------------------- */
/* threading control (used to report the CPU baseline's core count)          */
/* ------------------------------------------------------------------------- */
void oracle_set_threads(int n)
{
#ifdef _OPENMP
    if (n > 0) omp_set_num_threads(n);
#else
    (void)n;
#endif
}

int oracle_get_threads(void)
{
#ifdef _OPENMP
    return omp_get_max_threads();
#else
    return 1;
#endif
}

/* ------------------------------------------------------------------------- */
/* conv2d (paper, Section 3 "Builtin NN Functions": convolution and its       */
/* backward functions are builtins; Section 3 "Sparse Operations": computed   */
/* by lowering, i.e. stored filter matrix times the patch matrix, which is    */
/* cross-correlation without a filter flip).                                  */
/* ------------------------------------------------------------------------- */

/* Output size with symmetric zero padding p and stride s: floor((H+2p-Hf)/s)+1.
 * Returns <= 0 when no window fits. */
int oracle_conv2d_out_dim(int Hin, int Hf, int stride, int pad)
{
    if (Hin < 1 || Hf < 1 || stride < 1 || pad < 0) return 0;
    int span = Hin + 2 * pad - Hf;
    if (span < 0) return 0;
    return span / stride + 1;
}

/* Zero-padded input value xpad(n,c,h,w): x inside the image, 0 outside. */
static double xpad(const double *X, int C, int Hin, int Win,
                   int n, int c, int h, int w)
{
    if (h < 0 || h >= Hin || w < 0 || w >= Win) return 0.0;
    return X[(size_t)n * C * Hin * Win + (size_t)c * Hin * Win + (size_t)h * Win + w];
}

/* Pre-activation of one output element:
 *   pre(n,f,oh,ow) = b[f] + sum_{c,i,j} W[f,c,i,j] * xpad(n,c,oh*s+i-p,ow*s+j-p)
 * Summation order: c outer, i, j inner, starting from 0; the bias is added last. */
double oracle_conv2d_forward_pre_elem(const double *X, const double *W, const double *b,
                                      int C, int Hin, int Win, int Hf, int Wf,
                                      int stride, int pad,
                                      int n, int f, int oh, int ow)
{
    double acc = 0.0;
    for (int c = 0; c < C; ++c)
        for (int i = 0; i < Hf; ++i)
            for (int j = 0; j < Wf; ++j) {
                double wv = W[(size_t)f * C * Hf * Wf + (size_t)c * Hf * Wf + (size_t)i * Wf + j];
                double xv = xpad(X, C, Hin, Win, n, c, oh * stride + i - pad, ow * stride + j - pad);
                acc += wv * xv;
            }
    return acc + (b ? b[f] : 0.0);
}

/* relu(x) = max(0, x); a non-positive input gives +0.0 (strict comparison). */
static double relu(double x) { return x > 0.0 ? x : 0.0; }

/* out[n, f*Hout*Wout + oh*Wout + ow] = relu?(pre(n,f,oh,ow)); b may be NULL. */
void oracle_conv2d_forward(const double *X, const double *W, const double *b, double *out,
                           int N, int C, int Hin, int Win, int F, int Hf, int Wf,
                           int stride, int pad, int do_relu)
{
    int Hout = oracle_conv2d_out_dim(Hin, Hf, stride, pad);
    int Wout = oracle_conv2d_out_dim(Win, Wf, stride, pad);
    long long total = (long long)N * F * Hout * Wout;
#pragma omp parallel for schedule(static)
    for (long long e = 0; e < total; ++e) {
        int ow = (int)(e % Wout);
        int oh = (int)((e / Wout) % Hout);
        int f = (int)((e / ((long long)Wout * Hout)) % F);
        int n = (int)(e / ((long long)Wout * Hout * F));
        double pre = oracle_conv2d_forward_pre_elem(X, W, b, C, Hin, Win, Hf, Wf, stride, pad,
                                                    n, f, oh, ow);
        out[e] = do_relu ? relu(pre) : pre;
    }
}

/* Upstream gradient after the relu: g = dout where out_fwd > 0, else 0.
 * out_fwd == NULL means the layer had no relu (g = dout). relu'(0) = 0. */
static double masked_grad(const double *dout, const double *out_fwd, size_t idx)
{
    if (out_fwd && !(out_fwd[idx] > 0.0)) return 0.0;
    return dout[idx];
}

/* dW[f,c,i,j] = sum_{n,oh,ow} g(n,f,oh,ow) * xpad(n,c,oh*s+i-p,ow*s+j-p)
 * Summation order: n outer, then oh, then ow. */
double oracle_conv2d_backward_filter_elem(const double *X, const double *dout,
                                          const double *out_fwd,
                                          int N, int C, int Hin, int Win, int F,
                                          int Hf, int Wf, int stride, int pad,
                                          int f, int c, int i, int j)
{
    int Hout = oracle_conv2d_out_dim(Hin, Hf, stride, pad);
    int Wout = oracle_conv2d_out_dim(Win, Wf, stride, pad);
    double acc = 0.0;
    for (int n = 0; n < N; ++n)
        for (int oh = 0; oh < Hout; ++oh)
            for (int ow = 0; ow < Wout; ++ow) {
                size_t gi = (size_t)n * F * Hout * Wout + (size_t)f * Hout * Wout
                          + (size_t)oh * Wout + ow;
                double g = masked_grad(dout, out_fwd, gi);
                acc += g * xpad(X, C, Hin, Win, n, c, oh * stride + i - pad, ow * stride + j - pad);
            }
    return acc;
}

/* db[f] = sum_{n,oh,ow} g(n,f,oh,ow), in n, oh, ow order. */
double oracle_conv2d_backward_bias_elem(const double *dout, const double *out_fwd,
                                        int N, int F, int Hout, int Wout, int f)
{
    double acc = 0.0;
    for (int n = 0; n < N; ++n)
        for (int q = 0; q < Hout * Wout; ++q)
            acc += masked_grad(dout, out_fwd, (size_t)n * F * Hout * Wout + (size_t)f * Hout * Wout + q);
    return acc;
}

void oracle_conv2d_backward_filter(const double *X, const double *dout, const double *out_fwd,
                                   double *dW, double *db,
                                   int N, int C, int Hin, int Win, int F, int Hf, int Wf,
                                   int stride, int pad)
{
    long long K = (long long)C * Hf * Wf;
    long long total = (long long)F * K;
#pragma omp parallel for schedule(dynamic, 1)
    for (long long e = 0; e < total; ++e) {
        int j = (int)(e % Wf);
        int i = (int)((e / Wf) % Hf);
        int c = (int)((e / ((long long)Wf * Hf)) % C);
        int f = (int)(e / K);
        dW[e] = oracle_conv2d_backward_filter_elem(X, dout, out_fwd, N, C, Hin, Win, F,
                                                   Hf, Wf, stride, pad, f, c, i, j);
    }
    if (db) {
        int Hout = oracle_conv2d_out_dim(Hin, Hf, stride, pad);
        int Wout = oracle_conv2d_out_dim(Win, Wf, stride, pad);
#pragma omp parallel for schedule(static)
        for (int f = 0; f < F; ++f)
            db[f] = oracle_conv2d_backward_bias_elem(dout, out_fwd, N, F, Hout, Wout, f);
    }
}

/* dX[n,c,h,w] = sum_{f,i,j} W[f,c,i,j] * g(n,f,oh,ow) over the (i,j) for which
 * oh = (h+p-i)/s and ow = (w+p-j)/s are exact integers inside the output.
 * Summation order: f outer, then i, then j.  Input positions that no window
 * covers receive 0. */
double oracle_conv2d_backward_data_elem(const double *W, const double *dout,
                                        const double *out_fwd,
                                        int C, int Hin, int Win, int F, int Hf, int Wf,
                                        int stride, int pad, int n, int c, int h, int w)
{
    int Hout = oracle_conv2d_out_dim(Hin, Hf, stride, pad);
    int Wout = oracle_conv2d_out_dim(Win, Wf, stride, pad);
    double acc = 0.0;
    for (int f = 0; f < F; ++f)
        for (int i = 0; i < Hf; ++i)
            for (int j = 0; j < Wf; ++j) {
                int th = h + pad - i, tw = w + pad - j;
                if (th < 0 || tw < 0) continue;
                if (th % stride != 0 || tw % stride != 0) continue;
                int oh = th / stride, ow = tw / stride;
                if (oh >= Hout || ow >= Wout) continue;
                size_t gi = (size_t)n * F * Hout * Wout + (size_t)f * Hout * Wout
                          + (size_t)oh * Wout + ow;
                acc += W[(size_t)f * C * Hf * Wf + (size_t)c * Hf * Wf + (size_t)i * Wf + j]
                     * masked_grad(dout, out_fwd, gi);
            }
    return acc;
}

void oracle_conv2d_backward_data(const double *W, const double *dout, const double *out_fwd,
                                 double *dX, int N, int C, int Hin, int Win, int F,
                                 int Hf, int Wf, int stride, int pad)
{
    long long total = (long long)N * C * Hin * Win;
#pragma omp parallel for schedule(static)
    for (long long e = 0; e < total; ++e) {
        int w = (int)(e % Win);
        int h = (int)((e / Win) % Hin);
        int c = (int)((e / ((long long)Win * Hin)) % C);
        int n = (int)(e / ((long long)Win * Hin * C));
        dX[e] = oracle_conv2d_backward_data_elem(W, dout, out_fwd, C, Hin, Win, F, Hf, Wf,
                                                 stride, pad, n, c, h, w);
    }
}

/* ------------------------------------------------------------------------- */
/* bias_add (+relu): broadcasting a vector over a matrix (Section 3 "Tensor   */
/* Representation"; Section 2's affine layer adds a bias row to X W).       */
/* out[n, c*HW + q] = relu?(X[n, c*HW + q] + b[c]);  b may be NULL.            */
/* ------------------------------------------------------------------------- */
void oracle_bias_add_relu(const double *X, const double *b, double *out,
                          int N, int C, int HW, int do_relu)
{
    long long total = (long long)N * C * HW;
#pragma omp parallel for schedule(static)
    for (long long e = 0; e < total; ++e) {
        int c = (int)((e / HW) % C);
        double v = X[e] + (b ? b[c] : 0.0);
        out[e] = do_relu ? relu(v) : v;
    }
}

/* ------------------------------------------------------------------------- */
/* max_pool2d (Section 3: pooling and its backward are builtins).             */
/* Window Hf x Wf, stride s, padding p; padded cells count as -infinity and   */
/* are never selected.  argmax is the in-row column index c*Hin*Win+h*Win+w   */
/* of the first maximum met scanning the window row by row (i outer, j        */
/* inner), replacing only on a strictly larger value.                          */
/* ------------------------------------------------------------------------- */
void oracle_max_pool2d_fwd(const double *X, double *out, int32_t *argmax,
                           int N, int C, int Hin, int Win, int Hf, int Wf,
                           int stride, int pad)
{
    int Hout = oracle_conv2d_out_dim(Hin, Hf, stride, pad);
    int Wout = oracle_conv2d_out_dim(Win, Wf, stride, pad);
    long long total = (long long)N * C * Hout * Wout;
#pragma omp parallel for schedule(static)
    for (long long e = 0; e < total; ++e) {
        int ow = (int)(e % Wout);
        int oh = (int)((e / Wout) % Hout);
        int c = (int)((e / ((long long)Wout * Hout)) % C);
        int n = (int)(e / ((long long)Wout * Hout * C));
        const double *row = X + (size_t)n * C * Hin * Win;
        double best = -INFINITY;
        int32_t best_idx = -1;
        for (int i = 0; i < Hf; ++i)
            for (int j = 0; j < Wf; ++j) {
                int h = oh * stride + i - pad, w = ow * stride + j - pad;
                if (h < 0 || h >= Hin || w < 0 || w >= Win) continue;
                int32_t col = (int32_t)(c * Hin * Win + h * Win + w);
                if (best_idx < 0 || row[col] > best) {
                    best = row[col];
                    best_idx = col;
                }
            }
        out[e] = best;
        argmax[e] = best_idx;
    }
}

/* dX[n, k] = sum of dout over the outputs of row n whose argmax is k; every
 * other entry is 0.  Scatter in output order, one row at a time. */
void oracle_max_pool2d_bwd(const double *dout, const int32_t *argmax, double *dX,
                           int N, int C, int Hin, int Win, int Hf, int Wf,
                           int stride, int pad)
{
    int Hout = oracle_conv2d_out_dim(Hin, Hf, stride, pad);
    int Wout = oracle_conv2d_out_dim(Win, Wf, stride, pad);
    long long in_cols = (long long)C * Hin * Win;
    long long out_cols = (long long)C * Hout * Wout;
#pragma omp parallel for schedule(static)
    for (int n = 0; n < N; ++n) {
        double *dxr = dX + (size_t)n * in_cols;
        for (long long k = 0; k < in_cols; ++k) dxr[k] = 0.0;
        for (long long o = 0; o < out_cols; ++o)
            dxr[argmax[(size_t)n * out_cols + o]] += dout[(size_t)n * out_cols + o];
    }
}

/* ------------------------------------------------------------------------- */
/* affine (Section 2: the affine layer is X W plus a bias row; its backward   */
/* returns the gradients of X, W and b in that order).  X is N x D, W is      */
/* D x M, b is 1 x M.                                                          */
/* ------------------------------------------------------------------------- */
void oracle_affine_fwd(const double *X, const double *W, const double *b, double *out,
                       int N, int D, int M, int do_relu)
{
    long long total = (long long)N * M;
#pragma omp parallel for schedule(static)
    for (long long e = 0; e < total; ++e) {
        int m = (int)(e % M), n = (int)(e / M);
        double acc = 0.0;
        for (int d = 0; d < D; ++d) acc += X[(size_t)n * D + d] * W[(size_t)d * M + m];
        acc += b ? b[m] : 0.0;
        out[e] = do_relu ? relu(acc) : acc;
    }
}

/* g = dout (masked by out_fwd > 0 when out_fwd is given);
 * dX = g W^T (N x D), dW = X^T g (D x M), db = column sums of g (1 x M).
 * dX may be NULL (first layer). */
void oracle_affine_bwd(const double *dout, const double *X, const double *W,
                       const double *out_fwd, double *dX, double *dW, double *db,
                       int N, int D, int M)
{
    if (dX) {
        long long total = (long long)N * D;
#pragma omp parallel for schedule(static)
        for (long long e = 0; e < total; ++e) {
            int d = (int)(e % D), n = (int)(e / D);
            double acc = 0.0;
            for (int m = 0; m < M; ++m)
                acc += masked_grad(dout, out_fwd, (size_t)n * M + m) * W[(size_t)d * M + m];
            dX[e] = acc;
        }
    }
    long long total = (long long)D * M;
#pragma omp parallel for schedule(static)
    for (long long e = 0; e < total; ++e) {
        int m = (int)(e % M), d = (int)(e / M);
        double acc = 0.0;
        for (int n = 0; n < N; ++n)
            acc += X[(size_t)n * D + d] * masked_grad(dout, out_fwd, (size_t)n * M + m);
        dW[e] = acc;
    }
    for (int m = 0; m < M; ++m) {
        double acc = 0.0;
        for (int n = 0; n < N; ++n) acc += masked_grad(dout, out_fwd, (size_t)n * M + m);
        db[m] = acc;
    }
}

/* ------------------------------------------------------------------------- */
/* softmax + cross-entropy (Section 2: the classifier example chains the     */
/* softmax forward, the cross-entropy backward and the softmax backward).      */
/* Readings: the loss is the mean over the N rows; log-sum-exp is shifted by   */
/* the row maximum.                                                            */
/* ------------------------------------------------------------------------- */

/* Fused closed form.  For each row: m = max s, lse = m + log sum exp(s - m),
 * p = exp(s - lse), row loss = -sum_k y (s - lse), ds = (p * sum_k y - y) / N.
 * Returns loss = (1/N) * sum of row losses (rows added in order).
 * probs may be NULL. */
double oracle_softmax_xent(const double *S, const double *Y, double *probs, double *dS,
                           int N, int K)
{
    double total = 0.0;
    for (int n = 0; n < N; ++n) {
        const double *s = S + (size_t)n * K;
        const double *y = Y + (size_t)n * K;
        double m = s[0];
        for (int k = 1; k < K; ++k) if (s[k] > m) m = s[k];
        double se = 0.0;
        for (int k = 0; k < K; ++k) se += exp(s[k] - m);
        double lse = m + log(se);
        double ysum = 0.0, rl = 0.0;
        for (int k = 0; k < K; ++k) {
            ysum += y[k];
            rl -= y[k] * (s[k] - lse);
        }
        for (int k = 0; k < K; ++k) {
            double p = exp(s[k] - m) / se;
            if (probs) probs[(size_t)n * K + k] = p;
            dS[(size_t)n * K + k] = (p * ysum - y[k]) / N;
        }
        total += rl;
    }
    return total / N;
}

/* The unfused chain in the order of the paper's listing (used to pin the fused
 * closed form to the paper's composition). */
void oracle_softmax_forward(const double *S, double *P, int N, int K)
{
    for (int n = 0; n < N; ++n) {
        const double *s = S + (size_t)n * K;
        double m = s[0];
        for (int k = 1; k < K; ++k) if (s[k] > m) m = s[k];
        double se = 0.0;
        for (int k = 0; k < K; ++k) se += exp(s[k] - m);
        for (int k = 0; k < K; ++k) P[(size_t)n * K + k] = exp(s[k] - m) / se;
    }
}

/* loss = -(1/N) sum y log p;  dprobs = -y / (N p). */
double oracle_xent_forward(const double *P, const double *Y, int N, int K)
{
    double total = 0.0;
    for (int n = 0; n < N; ++n)
        for (int k = 0; k < K; ++k)
            if (Y[(size_t)n * K + k] != 0.0)
                total -= Y[(size_t)n * K + k] * log(P[(size_t)n * K + k]);
    return total / N;
}

void oracle_xent_backward(const double *P, const double *Y, double *dP, int N, int K)
{
    for (long long e = 0; e < (long long)N * K; ++e)
        dP[e] = -Y[e] / ((double)N * P[e]);
}

/* Softmax Jacobian-vector product: dS = p * (dP - rowsum(dP * p)). */
void oracle_softmax_backward(const double *dP, const double *P, double *dS, int N, int K)
{
    for (int n = 0; n < N; ++n) {
        double dot = 0.0;
        for (int k = 0; k < K; ++k) dot += dP[(size_t)n * K + k] * P[(size_t)n * K + k];
        for (int k = 0; k < K; ++k)
            dS[(size_t)n * K + k] = P[(size_t)n * K + k] * (dP[(size_t)n * K + k] - dot);
    }
}

/* ------------------------------------------------------------------------- */
/* SGD with momentum (Section 2 names it among the optimizers; the example's  */
/* plain gradient step is the case mu = 0).                                    */
/* Reading: v <- mu*v - lr*g;  theta <- theta + v                              */
/* ------------------------------------------------------------------------- */
void oracle_sgd_momentum_update(double *theta, const double *grad, double *v,
                                double lr, double mu, long long n)
{
#pragma omp parallel for schedule(static)
    for (long long e = 0; e < n; ++e) {
        v[e] = mu * v[e] - lr * grad[e];
        theta[e] = theta[e] + v[e];
    }
}

/* ------------------------------------------------------------------------- */
/* The other optimizers (Section 2 names Adagrad, Adam, RMSprop, SGD and SGD   */
/* with Nesterov momentum; it prints no formulas).  Readings, one step each:   */
/*   SGD:      theta <- theta - lr*g                                           */
/*   Nesterov: v' = mu*v - lr*g; theta <- theta - mu*v + (1+mu)*v'; v <- v'    */
/*             (Nesterov's look-ahead step rewritten on the current iterate)   */
/*   Adagrad:  c <- c + g^2; theta <- theta - lr*g/(sqrt(c) + eps)   (Duchi et */
/*             al.)                                                            */
/*   RMSprop:  c <- rho*c + (1-rho)*g^2; theta <- theta - lr*g/(sqrt(c) + eps) */
/*             (Tieleman and Hinton)                                          */
/*   Adam:     m <- b1*m + (1-b1)*g; v <- b2*v + (1-b2)*g^2;                   */
/*             theta <- theta - a_t*m/(sqrt(v) + eps),                         */
/*             a_t = lr*sqrt(1-b2^t)/(1-b1^t)  (Kingma and Ba, with the bias   */
/*             corrections folded into the step size), t = 1, 2, ...           */
/* ------------------------------------------------------------------------- */
void oracle_sgd_update(double *theta, const double *g, double lr, long long n)
{
#pragma omp parallel for schedule(static)
    for (long long e = 0; e < n; ++e) theta[e] = theta[e] - lr * g[e];
}

void oracle_sgd_nesterov_update(double *theta, const double *g, double *v, double lr,
                                double mu, long long n)
{
#pragma omp parallel for schedule(static)
    for (long long e = 0; e < n; ++e) {
        double v_prev = v[e];
        v[e] = mu * v_prev - lr * g[e];
        theta[e] = theta[e] - mu * v_prev + (1.0 + mu) * v[e];
    }
}

void oracle_adagrad_update(double *theta, const double *g, double *c, double lr, double eps,
                           long long n)
{
#pragma omp parallel for schedule(static)
    for (long long e = 0; e < n; ++e) {
        c[e] = c[e] + g[e] * g[e];
        theta[e] = theta[e] - lr * g[e] / (sqrt(c[e]) + eps);
    }
}

void oracle_rmsprop_update(double *theta, const double *g, double *c, double lr, double rho,
                           double eps, long long n)
{
#pragma omp parallel for schedule(static)
    for (long long e = 0; e < n; ++e) {
        c[e] = rho * c[e] + (1.0 - rho) * g[e] * g[e];
        theta[e] = theta[e] - lr * g[e] / (sqrt(c[e]) + eps);
    }
}

void oracle_adam_update(double *theta, const double *g, double *m, double *v, double lr,
                        double b1, double b2, double eps, long long t, long long n)
{
    double a_t = lr * sqrt(1.0 - pow(b2, (double)t)) / (1.0 - pow(b1, (double)t));
#pragma omp parallel for schedule(static)
    for (long long e = 0; e < n; ++e) {
        m[e] = b1 * m[e] + (1.0 - b1) * g[e];
        v[e] = b2 * v[e] + (1.0 - b2) * g[e] * g[e];
        theta[e] = theta[e] - a_t * m[e] / (sqrt(v[e]) + eps);
    }
}

/* Number of entries different from zero (the paper tracks non-zero counts of
 * every intermediate; Section 3 "Sparse Operations"). */
long long oracle_count_nonzero(const double *X, long long n)
{
    long long cnt = 0;
    for (long long e = 0; e < n; ++e) cnt += (X[e] != 0.0);
    return cnt;
}
