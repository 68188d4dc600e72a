/* Drives every oracle entry point over edge-case shapes on buffers of exactly
 * the documented sizes, for a build under AddressSanitizer and
 * UndefinedBehaviorSanitizer: an index outside a tensor, a signed overflow or
 * a use of an unset value aborts the run.  It also checks that each element
 * function equals the tensor it is part of, bit for bit.  Exit status 0: all
 * passes ran clean. */
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

int oracle_conv2d_out_dim(int, int, int, int);
double oracle_conv2d_forward_pre_elem(const double *, const double *, const double *, int, int,
                                      int, int, int, int, int, int, int, int, int);
void oracle_conv2d_forward(const double *, const double *, const double *, double *, int, int,
                           int, int, int, int, int, int, int, int);
double oracle_conv2d_backward_filter_elem(const double *, const double *, const double *, int,
                                          int, int, int, int, int, int, int, int, int, int, int,
                                          int);
double oracle_conv2d_backward_bias_elem(const double *, const double *, int, int, int, int, int);
void oracle_conv2d_backward_filter(const double *, const double *, const double *, double *,
                                   double *, int, int, int, int, int, int, int, int, int);
double oracle_conv2d_backward_data_elem(const double *, const double *, const double *, int, int,
                                        int, int, int, int, int, int, int, int, int, int);
void oracle_conv2d_backward_data(const double *, const double *, const double *, double *, int,
                                 int, int, int, int, int, int, int, int);
void oracle_bias_add_relu(const double *, const double *, double *, int, int, int, int);
void oracle_max_pool2d_fwd(const double *, double *, int32_t *, int, int, int, int, int, int, int,
                           int);
void oracle_max_pool2d_bwd(const double *, const int32_t *, double *, int, int, int, int, int, int,
                           int, int);
void oracle_affine_fwd(const double *, const double *, const double *, double *, int, int, int,
                       int);
void oracle_affine_bwd(const double *, const double *, const double *, const double *, double *,
                       double *, double *, int, int, int);
double oracle_softmax_xent(const double *, const double *, double *, double *, int, int);
void oracle_softmax_forward(const double *, double *, int, int);
double oracle_xent_forward(const double *, const double *, int, int);
void oracle_xent_backward(const double *, const double *, double *, int, int);
void oracle_softmax_backward(const double *, const double *, double *, int, int);
void oracle_sgd_momentum_update(double *, const double *, double *, double, double, long long);
void oracle_sgd_update(double *, const double *, double, long long);
void oracle_sgd_nesterov_update(double *, const double *, double *, double, double, long long);
void oracle_adagrad_update(double *, const double *, double *, double, double, long long);
void oracle_rmsprop_update(double *, const double *, double *, double, double, double, long long);
void oracle_adam_update(double *, const double *, double *, double *, double, double, double,
                        double, long long, long long);
long long oracle_count_nonzero(const double *, long long);

static unsigned long long rng_state = 88172645463325252ull;
static double urand(void) /* xorshift64, uniform in [-1, 1), a quarter of the draws exactly 0 */
{
    rng_state ^= rng_state << 13;
    rng_state ^= rng_state >> 7;
    rng_state ^= rng_state << 17;
    if ((rng_state & 3) == 0) return 0.0;
    return (double)(rng_state >> 11) / 4503599627370496.0 - 1.0;
}

static double *vec(long long n)
{
    double *p = (double *)malloc((size_t)(n > 0 ? n : 1) * sizeof(double));
    for (long long i = 0; i < n; ++i) p[i] = urand();
    return p;
}

static int fail(const char *what, int k)
{
    fprintf(stderr, "oracle_check: %s (case %d)\n", what, k);
    return 1;
}

int main(void)
{
    /* N, C, Hin, Win, F, Hf, Wf, stride, pad */
    static const int conv[][9] = {
        {1, 1, 1, 1, 1, 1, 1, 1, 0},   {2, 3, 5, 6, 2, 3, 3, 1, 3},  /* pad >= filter */
        {1, 2, 9, 7, 3, 2, 3, 2, 0},   /* uncovered border cells */
        {2, 2, 8, 5, 3, 3, 1, 3, 1},   {1, 1, 4, 4, 2, 4, 4, 1, 0},  /* stride 3; whole image */
        {2, 4, 7, 9, 5, 5, 5, 1, 2},   {1, 3, 11, 10, 2, 3, 3, 4, 1}, /* LeNet-like; stride 4 */
    };
    int bad = 0;
    for (int k = 0; k < (int)(sizeof(conv) / sizeof(conv[0])); ++k) {
        const int N = conv[k][0], C = conv[k][1], H = conv[k][2], Wd = conv[k][3], F = conv[k][4];
        const int Hf = conv[k][5], Wf = conv[k][6], s = conv[k][7], p = conv[k][8];
        const int Ho = oracle_conv2d_out_dim(H, Hf, s, p), Wo = oracle_conv2d_out_dim(Wd, Wf, s, p);
        if (Ho < 1 || Wo < 1) return fail("out_dim", k);
        const long long nx = (long long)N * C * H * Wd, nw = (long long)F * C * Hf * Wf;
        const long long no = (long long)N * F * Ho * Wo;
        double *X = vec(nx), *W = vec(nw), *b = vec(F), *out = vec(no), *dout = vec(no);
        double *dW = vec(nw), *db = vec(F), *dX = vec(nx);
        oracle_conv2d_forward(X, W, b, out, N, C, H, Wd, F, Hf, Wf, s, p, 1);
        for (int n = 0; n < N; ++n)
            for (int f = 0; f < F; ++f)
                for (int oh = 0; oh < Ho; ++oh)
                    for (int ow = 0; ow < Wo; ++ow) {
                        double v = oracle_conv2d_forward_pre_elem(X, W, b, C, H, Wd, Hf, Wf, s, p,
                                                                  n, f, oh, ow);
                        v = v > 0.0 ? v : 0.0;
                        if (v != out[(((long long)n * F + f) * Ho + oh) * Wo + ow])
                            bad |= fail("forward element", k);
                    }
        for (int masked = 0; masked < 2; ++masked) {
            const double *m = masked ? out : NULL;
            oracle_conv2d_backward_filter(X, dout, m, dW, db, N, C, H, Wd, F, Hf, Wf, s, p);
            oracle_conv2d_backward_data(W, dout, m, dX, N, C, H, Wd, F, Hf, Wf, s, p);
            for (int f = 0; f < F; ++f) {
                if (db[f] != oracle_conv2d_backward_bias_elem(dout, m, N, F, Ho, Wo, f))
                    bad |= fail("bias element", k);
                for (int c = 0; c < C; ++c)
                    for (int i = 0; i < Hf; ++i)
                        for (int j = 0; j < Wf; ++j)
                            if (dW[((f * C + c) * Hf + i) * Wf + j] !=
                                oracle_conv2d_backward_filter_elem(X, dout, m, N, C, H, Wd, F, Hf,
                                                                   Wf, s, p, f, c, i, j))
                                bad |= fail("filter element", k);
            }
            for (int n = 0; n < N; ++n)
                for (int c = 0; c < C; ++c)
                    for (int h = 0; h < H; ++h)
                        for (int w = 0; w < Wd; ++w)
                            if (dX[(((long long)n * C + c) * H + h) * Wd + w] !=
                                oracle_conv2d_backward_data_elem(W, dout, m, C, H, Wd, F, Hf, Wf,
                                                                 s, p, n, c, h, w))
                                bad |= fail("data element", k);
        }
        oracle_bias_add_relu(X, b, dX, N, 1, (int)(nx / N), 0);
        free(X); free(W); free(b); free(out); free(dout); free(dW); free(db); free(dX);
    }
    /* pools: N, C, H, W, Hf, Wf, stride, pad (overlapping, padded, gaps, trailing cells) */
    static const int pool[][8] = {{2, 3, 6, 7, 2, 2, 2, 0}, {1, 2, 7, 9, 3, 3, 2, 1},
                                  {2, 2, 6, 5, 2, 3, 1, 1}, {1, 2, 10, 11, 3, 3, 3, 0},
                                  {2, 3, 8, 8, 2, 2, 3, 0}, {1, 1, 1, 1, 1, 1, 1, 0}};
    for (int k = 0; k < (int)(sizeof(pool) / sizeof(pool[0])); ++k) {
        const int N = pool[k][0], C = pool[k][1], H = pool[k][2], Wd = pool[k][3];
        const int Hf = pool[k][4], Wf = pool[k][5], s = pool[k][6], p = pool[k][7];
        const int Ho = oracle_conv2d_out_dim(H, Hf, s, p), Wo = oracle_conv2d_out_dim(Wd, Wf, s, p);
        const long long nx = (long long)N * C * H * Wd, no = (long long)N * C * Ho * Wo;
        double *X = vec(nx), *out = vec(no), *dout = vec(no), *dX = vec(nx);
        int32_t *idx = (int32_t *)malloc((size_t)no * sizeof(int32_t));
        oracle_max_pool2d_fwd(X, out, idx, N, C, H, Wd, Hf, Wf, s, p);
        for (long long e = 0; e < no; ++e)
            if (idx[e] < 0 || idx[e] >= C * H * Wd) bad |= fail("pool argmax range", k);
        oracle_max_pool2d_bwd(dout, idx, dX, N, C, H, Wd, Hf, Wf, s, p);
        free(X); free(out); free(dout); free(dX); free(idx);
    }
    /* affine, softmax / cross-entropy, optimizers, count */
    {
        const int N = 5, D = 7, M = 3;
        double *X = vec(N * D), *W = vec(D * M), *b = vec(M), *o = vec(N * M), *g = vec(N * M);
        double *dX = vec(N * D), *dW = vec(D * M), *db = vec(M);
        oracle_affine_fwd(X, W, b, o, N, D, M, 1);
        oracle_affine_bwd(g, X, W, o, dX, dW, db, N, D, M);
        oracle_affine_bwd(g, X, W, NULL, dX, dW, db, N, D, M);
        double *S = vec(N * M), *Y = vec(N * M), *P = vec(N * M), *dS = vec(N * M), *dP = vec(N * M);
        for (int e = 0; e < N * M; ++e) Y[e] = (e % M) == (e / M) % M ? 1.0 : 0.0;
        const double l1 = oracle_softmax_xent(S, Y, P, dS, N, M);
        oracle_softmax_forward(S, P, N, M);
        const double l2 = oracle_xent_forward(P, Y, N, M);
        oracle_xent_backward(P, Y, dP, N, M);
        oracle_softmax_backward(dP, P, dS, N, M);
        if (!isfinite(l1) || !isfinite(l2)) bad |= fail("softmax loss", 0);
        const long long n = 11;
        double *th = vec(n), *gr = vec(n), *v = vec(n), *c2 = vec(n);
        for (long long i = 0; i < n; ++i) { v[i] = 0.0; c2[i] = 0.0; }
        oracle_sgd_momentum_update(th, gr, v, 0.01, 0.9, n);
        oracle_sgd_update(th, gr, 0.01, n);
        oracle_sgd_nesterov_update(th, gr, v, 0.01, 0.9, n);
        oracle_adagrad_update(th, gr, c2, 0.01, 1e-8, n);
        oracle_rmsprop_update(th, gr, c2, 0.01, 0.9, 1e-8, n);
        for (long long i = 0; i < n; ++i) { v[i] = 0.0; c2[i] = 0.0; }
        oracle_adam_update(th, gr, v, c2, 1e-3, 0.9, 0.999, 1e-8, 1, n);
        if (oracle_count_nonzero(X, N * D) < 0) bad |= fail("count", 0);
        free(X); free(W); free(b); free(o); free(g); free(dX); free(dW); free(db);
        free(S); free(Y); free(P); free(dS); free(dP); free(th); free(gr); free(v); free(c2);
    }
    if (!bad) printf("oracle_check: all entry points ran clean\n");
    return bad;
}
