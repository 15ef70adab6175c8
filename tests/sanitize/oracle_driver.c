/* Exercises every exported oracle function (normal, edge and error paths)
 * under AddressSanitizer / UndefinedBehaviorSanitizer.  Test infrastructure:
 * built and run by tests/test_sanitizers.py on the CPU. */
#include <math.h>
#include <stdio.h>
#include <stdlib.h>

int orc_shape(int, int, const int *, int, long long *, long long *);
void orc_activation(int, double, double *, double *);
void orc_conv_forward(const double *, int, int, int, const double *, const double *, int, int, double *);
void orc_conv_wgrad(const double *, int, int, int, const double *, int, int, double *, double *);
void orc_conv_backdata(const double *, int, int, const double *, int, int, int, double *);
int orc_forward_backward(int, int, const int *, int, int, const double *, long long, const float *, int,
                         double *, double *, double *, double *);
int orc_train_sequential(int, int, const int *, int, int, double *, long long, int, const float *,
                         const int *, long long, double, double *, double *);
int orc_grad_sum(int, int, const int *, int, int, const double *, long long, const float *, const int *,
                 long long, double *, double *, double *);
int orc_evaluate(int, int, const int *, int, int, const double *, long long, const float *, const int *,
                 long long, double *, long long *);

static unsigned long long rng = 88172645463325252ull;
static double urand(void) {  /* xorshift64 */
    rng ^= rng << 13; rng ^= rng >> 7; rng ^= rng << 17;
    return (double)(rng >> 11) / 9007199254740992.0;
}
static int fails = 0;
#define CHECK(c) do { if (!(c)) { fprintf(stderr, "check failed line %d: %s\n", __LINE__, #c); ++fails; } } while (0)

static void run_net(const int *ly, int nl, int hw, int n_out) {
    long long dims[7 * 16], np = 0;
    CHECK(orc_shape(hw, hw, ly, nl, dims, &np) == 0 && np > 0);
    double *p = malloc(sizeof(double) * np), *g = malloc(sizeof(double) * np), *gs = malloc(sizeof(double) * np);
    const int n = 5;
    float *x = malloc(sizeof(float) * n * hw * hw);
    int lab[5];
    for (long long i = 0; i < np; ++i) p[i] = 0.3 * (urand() - 0.5);
    for (int i = 0; i < n * hw * hw; ++i) x[i] = urand() < 0.8 ? 0.0f : (float)urand();
    for (int i = 0; i < n; ++i) lab[i] = (int)(urand() * n_out) % n_out;
    double out[256], loss, gap, losses[5], gaps[5];
    long long wrong = -1;
    CHECK(orc_forward_backward(hw, hw, ly, nl, 0, p, np, x, lab[0], out, &loss, g, &gap) == 0);
    CHECK(orc_forward_backward(hw, hw, ly, nl, 1, p, np, x, lab[0], NULL, NULL, NULL, NULL) == 0);
    CHECK(orc_forward_backward(hw, hw, ly, nl, 0, p, np, x, n_out, out, &loss, g, &gap) != 0);  /* bad label */
    CHECK(orc_forward_backward(hw, hw, ly, nl, 0, p, np + 1, x, 0, out, &loss, g, &gap) != 0); /* bad size */
    CHECK(orc_grad_sum(hw, hw, ly, nl, 0, p, np, x, lab, n, gs, losses, gaps) == 0);
    CHECK(orc_grad_sum(hw, hw, ly, nl, 0, p, np, x, lab, 0, gs, NULL, NULL) == 0);
    CHECK(orc_evaluate(hw, hw, ly, nl, 0, p, np, x, lab, n, NULL, &wrong) == 0 && wrong >= 0 && wrong <= n);
    CHECK(orc_train_sequential(hw, hw, ly, nl, 0, p, np, 1, x, lab, n, 1e-2, losses, gaps) == 0);
    CHECK(orc_train_sequential(hw, hw, ly, nl, 0, p, np, 0, x, lab, 0, 1e-2, NULL, NULL) == 0);
    for (long long i = 0; i < np; ++i) CHECK(isfinite(p[i]));
    free(p); free(g); free(gs); free(x);
}

int main(void) {
    const int small[] = {1, 5, 4, 2, 0, 2, 1, 10, 5, 2, 0, 3, 3, 50, 0, 3, 10, 0};
    const int large[] = {1, 20, 4, 2, 0, 2, 1, 60, 3, 1, 100, 6, 2, 0, 2, 3, 150, 0, 3, 10, 0};
    const int tiny[] = {2, 0, 2, 1, 2, 2, 3, 5, 0};
    const int fc[] = {3, 7, 0, 3, 3, 0};
    run_net(small, 6, 29, 10);
    run_net(large, 7, 29, 10);
    run_net(tiny, 3, 6, 5);
    run_net(fc, 2, 5, 3);
    /* shape errors: kernel larger than the map, pool not dividing, unknown kind, empty layers */
    const int bad1[] = {1, 2, 30}, bad2[] = {1, 2, 4, 2, 0, 3}, bad3[] = {7, 2, 4}, bad4[] = {3, 0, 0};
    long long np;
    CHECK(orc_shape(29, 29, bad1, 1, NULL, &np) == -2);
    CHECK(orc_shape(29, 29, bad2, 2, NULL, &np) == -2);
    CHECK(orc_shape(29, 29, bad3, 1, NULL, &np) == -1);
    CHECK(orc_shape(29, 29, bad4, 1, NULL, &np) == -1);
    CHECK(orc_shape(29, 29, NULL, 1, NULL, &np) == -1);
    CHECK(orc_shape(29, 29, bad1, 0, NULL, &np) == -1);
    /* primitives, including a 1x1 map */
    double in[2 * 4 * 4], w[3 * 2 * 2 * 2], b[3], o[3 * 3 * 3], gw[3 * 2 * 2 * 2], gb[3], e[2 * 4 * 4];
    for (int i = 0; i < 32; ++i) in[i] = urand();
    for (int i = 0; i < 24; ++i) w[i] = urand();
    for (int i = 0; i < 3; ++i) b[i] = urand();
    orc_conv_forward(in, 2, 4, 4, w, b, 3, 2, o);
    orc_conv_wgrad(in, 2, 4, 4, o, 3, 2, gw, gb);
    orc_conv_backdata(o, 3, 2, w, 2, 4, 4, e);
    double one[1] = {2.0}, k1[1] = {3.0}, r1[1];
    orc_conv_forward(one, 1, 1, 1, k1, NULL, 1, 1, r1);
    CHECK(r1[0] == 6.0);
    double f, df;
    orc_activation(0, 1e300, &f, &df);
    CHECK(isfinite(f) && df == 0.0);
    orc_activation(1, -3.0, &f, NULL);
    CHECK(f == -3.0);
    if (fails) return 1;
    printf("oracle driver ok\n");
    return 0;
}
