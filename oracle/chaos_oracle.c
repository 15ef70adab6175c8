/*
 * CHAOS oracle -- TEST INFRASTRUCTURE ONLY.
 *
 * A plain, slow, single-threaded CPU implementation of what the CHAOS
 * per-sample back-propagation path computes (Viebke & Pllana, HPCC 2015).
 * Only the tests, the smoke check and the CPU-baseline leg of the benchmark
 * may load it.  It shares no code, header or table with the HIP library.
 *
 * Arithmetic is double throughout; parameters arrive as double arrays.
 * orc_train_sequential() can round the shared weights to fp32 after every
 * update (store_f32 = 1), the precision in which the GPU keeps them.
 *
 * What follows the paper:
 *   - forward propagation, Section II-A: each neuron's input is the weighted
 *     sum of the connected outputs of the previous layer, its output the
 *     activation of that sum; the input layer passes the image through.
 *   - conv / max-pool / fully-connected layers and their sizes, Section II-A
 *     and Table I (every output map is connected to every input map and has
 *     one bias: the weight counts of Table I fix this).
 *   - back-propagation, Section II-A: partial derivatives at the output from
 *     the error against the label, then layer by layer downwards.
 *   - per-layer update of the shared weights after that layer's gradients and
 *     the partial derivatives below it are computed (Section III-A.2,
 *     Controlled Hogwild); with one worker this is per-sample SGD.
 *   - Validation/Testing: forward only, count of wrong predictions (Table II).
 * Readings where the paper is silent (activation, loss, orientation, tie
 * rules) are the ones listed in the design notes and pinned by the tests:
 *   f(z) = 1.7159 tanh(2z/3) on every conv and FC layer incl. the output,
 *   E = 1/2 sum_k (y_k - t_k)^2 against a one-hot target,
 *   conv = cross-correlation, valid, stride 1,
 *   max-pool = non-overlapping k x k, argmax = first maximum in row-major
 *   window order, the update w <- w - lr * g (lr = the paper's decay lambda),
 *   prediction = lowest index among equal maxima.
 *
 * act = 0 selects the scaled tanh, act = 1 the identity (used by pins only).
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#define ORC_OK 0
#define ORC_EINVAL (-1)
#define ORC_ESHAPE (-2)
#define ORC_ENOMEM (-3)

#define ORC_CONV 1
#define ORC_POOL 2
#define ORC_FC 3

#define ORC_MAX_LAYERS 32

static const double ACT_A = 1.7159;
static const double ACT_B = 2.0 / 3.0;

typedef struct {
    int kind, maps, k;
    int cin, hin, win;   /* input shape (FC: cin = flattened size, hin = win = 1) */
    int cout, hout, wout;
    long long woff;      /* offset of W in the parameter vector */
    long long nw;        /* number of weights, bias excluded */
    long long boff;      /* offset of the biases */
    long long nb;
} orc_stage;

typedef struct {
    int n;
    orc_stage s[ORC_MAX_LAYERS];
    long long n_params;
    int in_size, out_size;
} orc_net;

/* ---- net construction: Table I shapes ------------------------------------ */
static int build_net(int in_h, int in_w, const int *layers, int n_layers, orc_net *net)
{
    if (!layers || n_layers < 1 || n_layers > ORC_MAX_LAYERS || in_h < 1 || in_w < 1)
        return ORC_EINVAL;
    int c = 1, h = in_h, w = in_w;
    long long off = 0;
    net->n = n_layers;
    net->in_size = in_h * in_w;
    for (int l = 0; l < n_layers; ++l) {
        orc_stage *st = &net->s[l];
        st->kind = layers[3 * l];
        st->maps = layers[3 * l + 1];
        st->k = layers[3 * l + 2];
        st->cin = c; st->hin = h; st->win = w;
        st->nw = st->nb = 0;
        st->woff = st->boff = off;
        if (st->kind == ORC_CONV) {
            if (st->maps < 1 || st->k < 1) return ORC_EINVAL;
            if (st->k > h || st->k > w) return ORC_ESHAPE;
            st->cout = st->maps; st->hout = h - st->k + 1; st->wout = w - st->k + 1;
            st->nw = (long long)st->maps * c * st->k * st->k;
            st->nb = st->maps;
        } else if (st->kind == ORC_POOL) {
            if (st->k < 1) return ORC_EINVAL;
            if (h % st->k || w % st->k) return ORC_ESHAPE;
            st->cout = c; st->hout = h / st->k; st->wout = w / st->k;
        } else if (st->kind == ORC_FC) {
            if (st->maps < 1) return ORC_EINVAL;
            st->cin = c * h * w; st->hin = 1; st->win = 1;
            st->cout = st->maps; st->hout = 1; st->wout = 1;
            st->nw = (long long)st->maps * st->cin;
            st->nb = st->maps;
        } else {
            return ORC_EINVAL;
        }
        st->woff = off;
        st->boff = off + st->nw;
        off += st->nw + st->nb;
        c = st->cout; h = st->hout; w = st->wout;
    }
    net->n_params = off;
    net->out_size = c * h * w;
    return ORC_OK;
}

static long long stage_in_size(const orc_stage *st) { return (long long)st->cin * st->hin * st->win; }
static long long stage_out_size(const orc_stage *st) { return (long long)st->cout * st->hout * st->wout; }

/* Shape walk exported for the tests: per layer cin,hin,win,cout,hout,wout,
 * n_weights(+bias).  Returns a status code. */
int orc_shape(int in_h, int in_w, const int *layers, int n_layers,
              long long *dims_out, long long *n_params_out)
{
    orc_net net;
    int rc = build_net(in_h, in_w, layers, n_layers, &net);
    if (rc) return rc;
    if (dims_out) {
        for (int l = 0; l < n_layers; ++l) {
            const orc_stage *st = &net.s[l];
            long long *d = dims_out + 7 * l;
            d[0] = st->cin; d[1] = st->hin; d[2] = st->win;
            d[3] = st->cout; d[4] = st->hout; d[5] = st->wout;
            d[6] = st->nw + st->nb;
        }
    }
    if (n_params_out) *n_params_out = net.n_params;
    return ORC_OK;
}

/* ---- activation ---------------------------------------------------------- */
static double act_f(int act, double z) { return act ? z : ACT_A * tanh(ACT_B * z); }
static double act_df(int act, double z)
{
    if (act) return 1.0;
    double t = tanh(ACT_B * z);
    return ACT_A * ACT_B * (1.0 - t * t);
}

/* f and f' at z for the closed-form pins. */
void orc_activation(int act, double z, double *f, double *df)
{
    if (f) *f = act_f(act, z);
    if (df) *df = act_df(act, z);
}

/* ---- single-layer primitives (also exported for the hand-worked pins) ---- */

/* out[o][p][q] = b[o] + sum_{c,u,v} w[o][c][u][v] * in[c][p+u][q+v] */
void orc_conv_forward(const double *in, int C, int H, int W, const double *w, const double *b,
                      int O, int K, double *out)
{
    int Ho = H - K + 1, Wo = W - K + 1;
    for (int o = 0; o < O; ++o)
        for (int p = 0; p < Ho; ++p)
            for (int q = 0; q < Wo; ++q) {
                double s = b ? b[o] : 0.0;
                for (int c = 0; c < C; ++c)
                    for (int u = 0; u < K; ++u)
                        for (int v = 0; v < K; ++v)
                            s += w[((o * C + c) * K + u) * K + v] * in[(c * H + p + u) * W + q + v];
                out[(o * Ho + p) * Wo + q] = s;
            }
}

/* gw[o][c][u][v] = sum_{p,q} d[o][p][q] * in[c][p+u][q+v];  gb[o] = sum_{p,q} d[o][p][q] */
void orc_conv_wgrad(const double *in, int C, int H, int W, const double *d, int O, int K,
                    double *gw, double *gb)
{
    int Ho = H - K + 1, Wo = W - K + 1;
    for (int o = 0; o < O; ++o) {
        for (int c = 0; c < C; ++c)
            for (int u = 0; u < K; ++u)
                for (int v = 0; v < K; ++v) {
                    double s = 0.0;
                    for (int p = 0; p < Ho; ++p)
                        for (int q = 0; q < Wo; ++q)
                            s += d[(o * Ho + p) * Wo + q] * in[(c * H + p + u) * W + q + v];
                    gw[((o * C + c) * K + u) * K + v] = s;
                }
        if (gb) {
            double s = 0.0;
            for (int p = 0; p < Ho; ++p)
                for (int q = 0; q < Wo; ++q) s += d[(o * Ho + p) * Wo + q];
            gb[o] = s;
        }
    }
}

/* e_in[c][r][s] = sum_o sum_{u,v} w[o][c][u][v] * d[o][r-u][s-v], terms with
 * (r-u, s-v) inside the output map only. */
void orc_conv_backdata(const double *d, int O, int K, const double *w, int C, int H, int W,
                       double *e_in)
{
    int Ho = H - K + 1, Wo = W - K + 1;
    for (int c = 0; c < C; ++c)
        for (int r = 0; r < H; ++r)
            for (int s = 0; s < W; ++s) {
                double acc = 0.0;
                for (int o = 0; o < O; ++o)
                    for (int u = 0; u < K; ++u) {
                        int p = r - u;
                        if (p < 0 || p >= Ho) continue;
                        for (int v = 0; v < K; ++v) {
                            int q = s - v;
                            if (q < 0 || q >= Wo) continue;
                            acc += w[((o * C + c) * K + u) * K + v] * d[(o * Ho + p) * Wo + q];
                        }
                    }
                e_in[(c * H + r) * W + s] = acc;
            }
}

/* Non-overlapping k x k max; arg[...] = flat index into `in` of the first
 * maximum in row-major window order.  gap (optional) = smallest positive
 * relative distance between the maximum and the runner-up over all windows. */
static void pool_forward(const double *in, int C, int H, int W, int k, double *out, int *arg,
                         double *gap)
{
    int Ho = H / k, Wo = W / k;
    for (int c = 0; c < C; ++c)
        for (int P = 0; P < Ho; ++P)
            for (int Q = 0; Q < Wo; ++Q) {
                int best = (c * H + P * k) * W + Q * k;
                double m = in[best];
                for (int u = 0; u < k; ++u)
                    for (int v = 0; v < k; ++v) {
                        int idx = (c * H + P * k + u) * W + Q * k + v;
                        if (in[idx] > m) { m = in[idx]; best = idx; }
                    }
                out[(c * Ho + P) * Wo + Q] = m;
                arg[(c * Ho + P) * Wo + Q] = best;
                if (gap) {
                    double second = -INFINITY;
                    for (int u = 0; u < k; ++u)
                        for (int v = 0; v < k; ++v) {
                            int idx = (c * H + P * k + u) * W + Q * k + v;
                            if (idx != best && in[idx] > second) second = in[idx];
                        }
                    if (k > 1) {
                        double den = fabs(m) > 1e-30 ? fabs(m) : 1e-30;
                        double g = (m - second) / den;
                        if (g > 0.0 && g < *gap) *gap = g;
                    }
                }
            }
}

/* ---- whole-net workspace ------------------------------------------------- */
typedef struct {
    double *a[ORC_MAX_LAYERS + 1];  /* a[0] = input, a[l+1] = output of layer l */
    double *z[ORC_MAX_LAYERS];      /* pre-activation of conv/fc layers */
    int *arg[ORC_MAX_LAYERS];       /* pool argmax */
    double *e0, *e1;                /* gradient of E w.r.t. a layer's output */
    double *gw;                     /* one layer's weight+bias gradient */
    long long emax, gmax;
} orc_ws;

static void ws_free(orc_ws *ws)
{
    for (int i = 0; i <= ORC_MAX_LAYERS; ++i) free(ws->a[i]);
    for (int i = 0; i < ORC_MAX_LAYERS; ++i) { free(ws->z[i]); free(ws->arg[i]); }
    free(ws->e0); free(ws->e1); free(ws->gw);
    memset(ws, 0, sizeof(*ws));
}

static int ws_alloc(const orc_net *net, orc_ws *ws)
{
    memset(ws, 0, sizeof(*ws));
    ws->a[0] = calloc((size_t)net->in_size, sizeof(double));
    if (!ws->a[0]) return ORC_ENOMEM;
    long long emax = net->in_size, gmax = 1;
    for (int l = 0; l < net->n; ++l) {
        const orc_stage *st = &net->s[l];
        long long no = stage_out_size(st);
        ws->a[l + 1] = calloc((size_t)no, sizeof(double));
        if (!ws->a[l + 1]) { ws_free(ws); return ORC_ENOMEM; }
        if (st->kind == ORC_POOL) {
            ws->arg[l] = calloc((size_t)no, sizeof(int));
            if (!ws->arg[l]) { ws_free(ws); return ORC_ENOMEM; }
        } else {
            ws->z[l] = calloc((size_t)no, sizeof(double));
            if (!ws->z[l]) { ws_free(ws); return ORC_ENOMEM; }
        }
        if (no > emax) emax = no;
        if (stage_in_size(st) > emax) emax = stage_in_size(st);
        if (st->nw + st->nb > gmax) gmax = st->nw + st->nb;
    }
    ws->emax = emax; ws->gmax = gmax;
    ws->e0 = calloc((size_t)emax, sizeof(double));
    ws->e1 = calloc((size_t)emax, sizeof(double));
    ws->gw = calloc((size_t)gmax, sizeof(double));
    if (!ws->e0 || !ws->e1 || !ws->gw) { ws_free(ws); return ORC_ENOMEM; }
    return ORC_OK;
}

/* Forward propagation (Section II-A): a[0] = image, then layer by layer. */
static void forward(const orc_net *net, int act, const double *params, const float *x,
                    orc_ws *ws, double *gap)
{
    for (int i = 0; i < net->in_size; ++i) ws->a[0][i] = (double)x[i];
    for (int l = 0; l < net->n; ++l) {
        const orc_stage *st = &net->s[l];
        const double *in = ws->a[l];
        double *out = ws->a[l + 1];
        long long no = stage_out_size(st);
        if (st->kind == ORC_CONV) {
            orc_conv_forward(in, st->cin, st->hin, st->win, params + st->woff, params + st->boff,
                             st->cout, st->k, ws->z[l]);
        } else if (st->kind == ORC_FC) {
            const double *w = params + st->woff, *b = params + st->boff;
            for (int j = 0; j < st->cout; ++j) {
                double s = b[j];
                for (int i = 0; i < st->cin; ++i) s += w[(long long)j * st->cin + i] * in[i];
                ws->z[l][j] = s;
            }
        } else {
            pool_forward(in, st->cin, st->hin, st->win, st->k, out, ws->arg[l], gap);
            continue;
        }
        for (long long i = 0; i < no; ++i) out[i] = act_f(act, ws->z[l][i]);
    }
}

/* E = 1/2 sum_k (y_k - t_k)^2 with t = one-hot(label). */
static double loss_and_top_error(const orc_net *net, const orc_ws *ws, int label, double *e)
{
    const double *y = ws->a[net->n];
    double E = 0.0;
    for (int k = 0; k < net->out_size; ++k) {
        double t = (k == label) ? 1.0 : 0.0;
        double d = y[k] - t;
        E += 0.5 * d * d;
        if (e) e[k] = d;
    }
    return E;
}

/* Back-propagation (Section II-A) with the per-layer update of Controlled
 * Hogwild (Section III-A.2).  On entry ws->e0 holds dE/dy at the output.
 * For each layer from the top: delta = e * f'(z) (conv/FC), gradient of its
 * weights and biases, dE/d(input) with the layer's weights as they were
 * before its update, then (lr != 0) the update of that layer.  grad (if not
 * NULL) receives the full gradient in the canonical layout. */
static void backward(const orc_net *net, int act, double *params, double lr, int store_f32,
                     orc_ws *ws, double *grad)
{
    double *e = ws->e0, *e_prev = ws->e1;
    for (int l = net->n - 1; l >= 0; --l) {
        const orc_stage *st = &net->s[l];
        const double *in = ws->a[l];
        long long no = stage_out_size(st), ni = stage_in_size(st);
        int has_below = l > 0;  /* the layer below is not the input image */
        if (st->kind == ORC_POOL) {
            if (has_below) {
                for (long long i = 0; i < ni; ++i) e_prev[i] = 0.0;
                for (long long i = 0; i < no; ++i) e_prev[ws->arg[l][i]] += e[i];
            }
        } else {
            for (long long i = 0; i < no; ++i) e[i] *= act_df(act, ws->z[l][i]);  /* delta */
            double *w = params + st->woff;
            double *gw = ws->gw, *gb = ws->gw + st->nw;
            if (st->kind == ORC_CONV) {
                orc_conv_wgrad(in, st->cin, st->hin, st->win, e, st->cout, st->k, gw, gb);
                if (has_below)
                    orc_conv_backdata(e, st->cout, st->k, w, st->cin, st->hin, st->win, e_prev);
            } else {
                for (int j = 0; j < st->cout; ++j) {
                    for (int i = 0; i < st->cin; ++i) gw[(long long)j * st->cin + i] = e[j] * in[i];
                    gb[j] = e[j];
                }
                if (has_below)
                    for (int i = 0; i < st->cin; ++i) {
                        double s = 0.0;
                        for (int j = 0; j < st->cout; ++j) s += w[(long long)j * st->cin + i] * e[j];
                        e_prev[i] = s;
                    }
            }
            long long ng = st->nw + st->nb;
            if (grad) memcpy(grad + st->woff, ws->gw, (size_t)ng * sizeof(double));
            if (lr != 0.0) {
                for (long long i = 0; i < ng; ++i) {
                    double v = params[st->woff + i] - lr * ws->gw[i];
                    params[st->woff + i] = store_f32 ? (double)(float)v : v;
                }
            }
        }
        double *t = e; e = e_prev; e_prev = t;
    }
}

static int check_label(const orc_net *net, int label)
{
    return (label < 0 || label >= net->out_size) ? ORC_EINVAL : ORC_OK;
}

/* One sample at fixed weights: outputs, loss, gradient, smallest positive
 * relative max-pool gap (NULL = skip each). */
int orc_forward_backward(int in_h, int in_w, const int *layers, int n_layers, int act,
                         const double *params, long long n_params, const float *x, int label,
                         double *out, double *loss, double *grad, double *min_gap)
{
    orc_net net;
    int rc = build_net(in_h, in_w, layers, n_layers, &net);
    if (rc) return rc;
    if (n_params != net.n_params || !params || !x) return ORC_EINVAL;
    if ((rc = check_label(&net, label))) return rc;
    orc_ws ws;
    if ((rc = ws_alloc(&net, &ws))) return rc;
    double gap = INFINITY;
    forward(&net, act, params, x, &ws, &gap);
    double E = loss_and_top_error(&net, &ws, label, ws.e0);
    if (out) memcpy(out, ws.a[net.n], (size_t)net.out_size * sizeof(double));
    if (loss) *loss = E;
    if (min_gap) *min_gap = gap;
    if (grad) backward(&net, act, (double *)params, 0.0, 0, &ws, grad);
    ws_free(&ws);
    return ORC_OK;
}

/* Sequential per-sample SGD over x[0..n) in index order: for each sample a
 * forward pass, the loss, then back-propagation with the per-layer update
 * w <- w - lr * g.  params is updated in place; loss_out[i] (optional) is the
 * loss of sample i before its update, gap_out[i] (optional) the smallest
 * positive relative max-pool gap of its forward pass. */
int orc_train_sequential(int in_h, int in_w, const int *layers, int n_layers, int act,
                         double *params, long long n_params, int store_f32, const float *x,
                         const int *labels, long long n, double lr, double *loss_out,
                         double *gap_out)
{
    orc_net net;
    int rc = build_net(in_h, in_w, layers, n_layers, &net);
    if (rc) return rc;
    if (n_params != net.n_params || !params || n < 0 || (n > 0 && (!x || !labels))) return ORC_EINVAL;
    for (long long i = 0; i < n; ++i)
        if ((rc = check_label(&net, labels[i]))) return rc;
    orc_ws ws;
    if ((rc = ws_alloc(&net, &ws))) return rc;
    for (long long i = 0; i < n; ++i) {
        double gap = INFINITY;
        forward(&net, act, params, x + i * net.in_size, &ws, &gap);
        double E = loss_and_top_error(&net, &ws, labels[i], ws.e0);
        if (loss_out) loss_out[i] = E;
        if (gap_out) gap_out[i] = gap;
        backward(&net, act, params, lr, store_f32, &ws, NULL);
    }
    ws_free(&ws);
    return ORC_OK;
}

/* Frozen-weight gradient sum G = sum_i grad E_i(W) over x[0..n), accumulated
 * in double in sample order.  loss_out (optional) per-sample loss; gap_out
 * (optional) per sample the smallest positive relative max-pool gap of its
 * forward pass (a diagnostic for the comparison with fp32 results; it does
 * not enter the sum). */
int orc_grad_sum(int in_h, int in_w, const int *layers, int n_layers, int act,
                 const double *params, long long n_params, const float *x, const int *labels,
                 long long n, double *grad_sum, double *loss_out, double *gap_out)
{
    orc_net net;
    int rc = build_net(in_h, in_w, layers, n_layers, &net);
    if (rc) return rc;
    if (n_params != net.n_params || !params || !grad_sum || n < 0) return ORC_EINVAL;
    for (long long i = 0; i < n; ++i)
        if ((rc = check_label(&net, labels[i]))) return rc;
    orc_ws ws;
    if ((rc = ws_alloc(&net, &ws))) return rc;
    double *g = calloc((size_t)net.n_params, sizeof(double));
    if (!g) { ws_free(&ws); return ORC_ENOMEM; }
    memset(grad_sum, 0, (size_t)net.n_params * sizeof(double));
    for (long long i = 0; i < n; ++i) {
        double gap = INFINITY;
        forward(&net, act, params, x + i * net.in_size, &ws, &gap);
        double E = loss_and_top_error(&net, &ws, labels[i], ws.e0);
        if (loss_out) loss_out[i] = E;
        if (gap_out) gap_out[i] = gap;
        backward(&net, act, (double *)params, 0.0, 0, &ws, g);
        for (long long p = 0; p < net.n_params; ++p) grad_sum[p] += g[p];
    }
    free(g);
    ws_free(&ws);
    return ORC_OK;
}

/* Validation / Testing (Section III-A.1, Table II): forward only, predicted
 * class = lowest index among the maximal outputs, count of predictions that
 * differ from the label.  out (optional) [n][n_out]. */
int orc_evaluate(int in_h, int in_w, const int *layers, int n_layers, int act,
                 const double *params, long long n_params, const float *x, const int *labels,
                 long long n, double *out, long long *n_wrong)
{
    orc_net net;
    int rc = build_net(in_h, in_w, layers, n_layers, &net);
    if (rc) return rc;
    if (n_params != net.n_params || !params || n < 0 || !n_wrong) return ORC_EINVAL;
    orc_ws ws;
    if ((rc = ws_alloc(&net, &ws))) return rc;
    long long wrong = 0;
    for (long long i = 0; i < n; ++i) {
        forward(&net, act, params, x + i * net.in_size, &ws, NULL);
        const double *y = ws.a[net.n];
        int best = 0;
        for (int k = 1; k < net.out_size; ++k)
            if (y[k] > y[best]) best = k;
        if (best != labels[i]) ++wrong;
        if (out) memcpy(out + i * net.out_size, y, (size_t)net.out_size * sizeof(double));
    }
    *n_wrong = wrong;
    ws_free(&ws);
    return ORC_OK;
}
