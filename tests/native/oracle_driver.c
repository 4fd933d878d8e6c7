/*
 * Test driver of the oracle for the sanitizer builds (AddressSanitizer and
 * UndefinedBehaviorSanitizer on the host): reads one training problem from
 * a binary file, runs it through the oracle's training loops and writes the
 * results, which the test compares with the same oracle loaded without
 * sanitizers.  Test infrastructure only.
 *
 * Input (little endian): int32 n_ops, N, C0, H0, W0, n_stages, T, bf16,
 * nesterov; int32 desc[9*n_ops]; int32 stage_end[n_stages]; int64 n_params;
 * double params0[n_params]; float xs[T*N*C0*H0*W0]; int32 labels[T*N];
 * int32 staleness[T*n_stages]; double lr[T*n_stages].
 * Output: double params[n_params], losses[T]; then the same from a run
 * resumed at step T/2 from the first half's checkpoint (params, losses of
 * the second half), then the loss and gradient of one pass at W^(0).
 */
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>

int orc_train(int n_ops, const int32_t *desc, int N, int C0, int H0, int W0, int n_stages,
              const int32_t *stage_end, const double *params0, int T, const float *xs,
              const int32_t *labels, const int32_t *staleness, const double *lr, double mom,
              double wd, int nesterov, double bn_eps, double bn_mom, int bf16, int stash, double *params_out,
              double *mom_out, double *run_mean, double *run_var, double *losses, int32_t *versions,
              uint64_t dropout_seed);
int orc_train_from(int n_ops, const int32_t *desc, int N, int C0, int H0, int W0, int n_stages,
                   const int32_t *stage_end, int64_t t0, int depth, const double *hist0,
                   const double *mom0, int bn_in, int T, const float *xs, const int32_t *labels,
                   const int32_t *staleness, const double *lr, double mom, double wd, int nesterov,
                   double bn_eps, double bn_mom, int bf16, int stash, int out_depth, double *hist_out,
                   double *mom_out, double *grad_out, double *run_mean, double *run_var,
                   double *losses, int32_t *versions, uint64_t dropout_seed);
int orc_loss_and_grad(int n_ops, const int32_t *desc, int N, int C0, int H0, int W0, int n_stages,
                      const int32_t *stage_end, const double *params, const float *x,
                      const int32_t *labels, double bn_eps, int bf16, double *loss, double *grads_out,
                      double *acts_out, uint64_t dropout_seed, int64_t step);
int orc_param_counts(int n_ops, const int32_t *desc, int N, int C0, int H0, int W0, int n_stages,
                     const int32_t *stage_end, int64_t *out);

static void *rd(FILE *f, size_t size, size_t n)
{
    void *p = malloc(size * (n ? n : 1));
    if (!p || fread(p, size, n, f) != n) {
        fprintf(stderr, "short input\n");
        exit(2);
    }
    return p;
}

int main(int argc, char **argv)
{
    if (argc != 3) {
        fprintf(stderr, "usage: %s input output\n", argv[0]);
        return 2;
    }
    FILE *f = fopen(argv[1], "rb");
    if (!f) return 2;
    int32_t *h = rd(f, sizeof(int32_t), 9);
    const int n_ops = h[0], N = h[1], C0 = h[2], H0 = h[3], W0 = h[4], S = h[5], T = h[6], bf16 = h[7],
              nest = h[8];
    int32_t *desc = rd(f, sizeof(int32_t), (size_t)9 * n_ops);
    int32_t *se = rd(f, sizeof(int32_t), (size_t)S);
    int64_t *np_ = rd(f, sizeof(int64_t), 1);
    const int64_t np = *np_;
    double *p0 = rd(f, sizeof(double), (size_t)np);
    const size_t xn = (size_t)T * N * C0 * H0 * W0;
    float *xs = rd(f, sizeof(float), xn);
    int32_t *labels = rd(f, sizeof(int32_t), (size_t)T * N);
    int32_t *st = rd(f, sizeof(int32_t), (size_t)T * S);
    double *lr = rd(f, sizeof(double), (size_t)T * S);
    fclose(f);

    int64_t *counts = calloc((size_t)S, sizeof(int64_t));
    if (orc_param_counts(n_ops, desc, N, C0, H0, W0, S, se, counts) != 0) return 3;
    int64_t total = 0;
    for (int s = 0; s < S; ++s) total += counts[s];
    if (total != np) return 4;

    double *params = calloc((size_t)np, sizeof(double)), *mom = calloc((size_t)np, sizeof(double));
    double *losses = calloc((size_t)T, sizeof(double));
    int32_t *ver = calloc((size_t)T * S, sizeof(int32_t));
    int n_bn = 0;
    for (int i = 0; i < n_ops; ++i)
        if (desc[9 * i] == 2) n_bn += desc[9 * i + 4];
    double *rm = calloc((size_t)(n_bn + 1), sizeof(double)), *rv = calloc((size_t)(n_bn + 1), sizeof(double));
    if (orc_train(n_ops, desc, N, C0, H0, W0, S, se, p0, T, xs, labels, st, lr, 0.9, 1e-4, nest, 1e-5, 0.1, bf16, 0,
                  params, mom, rm, rv, losses, ver, 77) != 0)
        return 5;

    /* resume at T/2: the first half with the versions the schedule can read
       (depth = max staleness + 1), then the second half */
    int D = 1;
    for (int64_t i = 0; i < (int64_t)T * S; ++i)
        if (st[i] + 1 > D) D = st[i] + 1;
    const int T1 = T / 2, T2 = T - T1;
    double *hist = calloc((size_t)np * D, sizeof(double)), *mom1 = calloc((size_t)np, sizeof(double));
    double *grad = calloc((size_t)np, sizeof(double));
    double *l1 = calloc((size_t)T, sizeof(double));
    int32_t *v1 = calloc((size_t)T * S, sizeof(int32_t));
    double *rm1 = calloc((size_t)(n_bn + 1), sizeof(double)), *rv1 = calloc((size_t)(n_bn + 1), sizeof(double));
    if (orc_train_from(n_ops, desc, N, C0, H0, W0, S, se, 0, 1, p0, NULL, 0, T1, xs, labels, st, lr, 0.9, 1e-4, nest,
                       1e-5, 0.1, bf16, 0, D, hist, mom1, grad, rm1, rv1, l1, v1, 77) != 0)
        return 6;
    double *params2 = calloc((size_t)np, sizeof(double)), *mom2 = calloc((size_t)np, sizeof(double));
    const size_t per_img = (size_t)N * C0 * H0 * W0;
    if (orc_train_from(n_ops, desc, N, C0, H0, W0, S, se, T1, D, hist, mom1, 1, T2, xs + (size_t)T1 * per_img,
                       labels + (size_t)T1 * N, st + (size_t)T1 * S, lr + (size_t)T1 * S, 0.9, 1e-4, nest, 1e-5, 0.1,
                       bf16, 0, 1, params2, mom2, grad, rm1, rv1, l1 + T1, v1 + (size_t)T1 * S, 77) != 0)
        return 7;

    double loss = 0.0;
    double *g0 = calloc((size_t)np, sizeof(double));
    if (orc_loss_and_grad(n_ops, desc, N, C0, H0, W0, S, se, p0, xs, labels, 1e-5, bf16, &loss, g0, NULL, 77, 0) != 0)
        return 8;

    FILE *o = fopen(argv[2], "wb");
    if (!o) return 2;
    fwrite(params, sizeof(double), (size_t)np, o);
    fwrite(losses, sizeof(double), (size_t)T, o);
    fwrite(params2, sizeof(double), (size_t)np, o);
    fwrite(l1, sizeof(double), (size_t)T, o);
    fwrite(&loss, sizeof(double), 1, o);
    fwrite(g0, sizeof(double), (size_t)np, o);
    fclose(o);
    free(h); free(desc); free(se); free(np_); free(p0); free(xs); free(labels); free(st); free(lr); free(counts);
    free(params); free(mom); free(losses); free(ver); free(rm); free(rv); free(hist); free(mom1); free(grad);
    free(l1); free(v1); free(rm1); free(rv1); free(params2); free(mom2); free(g0);
    return 0;
}
