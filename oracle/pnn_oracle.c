/*
 * pnn_oracle.c -- CPU oracle for the parallel neural network (PNN) of
 * Kalwarowskyj & Schikuta, "Parallel Neural Networks in Golang".
 *
 * TEST INFRASTRUCTURE ONLY.  This file is the plain, slow reference the GPU library is
 * checked against.  Only the test suite, the package smoke check and the CPU-baseline
 * leg of the benchmark may load it; the GPU library shares no code with it.
 *
 * Precision: the paper's implementation uses Gonum matrices of float64 (section
 * "Implementation Details"), so every value here is a double.  The one exception is the
 * bf16-mixed precision mode, where the configuration itself fixes rounding points:
 * GEMM operands (inputs, hidden activations, weights, deltas) are rounded to bfloat16
 * (round to nearest even) and everything else stays in double.
 *
 * Parameter layout of one network (flat): W1, b1, W2, b2, ..., W_l row-major
 * [sizes[l]][sizes[l-1]], b_l [sizes[l]].
 *
 * Readings of points the paper leaves open (each one is listed with its reason in the
 * design notes of the repository):
 *  - eq. (1) puts the bias inside the sum over j; eq. (2) adds it once.  Added once.
 *  - the rectifier derivative at z = 0 is 1: eq. (4) puts z = 0 in the linear branch.
 *  - sigmoid output with the quadratic loss uses eq. (9) literally:
 *    delta^L = (x^L - e) * x^L (1 - x^L); the cross-entropy flag uses eq. (10),
 *    delta^L = x^L - e, for softmax or sigmoid outputs.
 *  - mini-batch updates use eta / B_t with B_t the actual size of the batch (the last
 *    batch of a shard may be short); samples are visited in shard order, no shuffling.
 *  - shards are contiguous; the first N mod K shards hold one extra sample.
 *  - the merge is the exact mean: sum in long double with k ascending, divided by K.
 */
#include <math.h>
#include <pthread.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

enum { OR_SIGMOID = 0, OR_TANH = 1, OR_RELU = 2, OR_LEAKY_RELU = 3, OR_SOFTMAX = 4 };
enum { OR_LOSS_MSE = 0, OR_LOSS_XENT = 1 };
enum { OR_EXACT = 0, OR_BF16 = 1 };

#define OR_MAX_LAYERS 8

typedef struct {
    int32_t n_layers;                 /* number of weight layers L */
    int32_t sizes[OR_MAX_LAYERS + 1]; /* sizes[0] inputs ... sizes[L] outputs */
    int32_t act[OR_MAX_LAYERS];       /* activation of weight layer l+1 */
    int32_t loss;
    int32_t precision;
    int32_t replicas;                 /* K child networks */
    int32_t batch;                    /* B; 1 = per-sample stochastic gradient descent */
    float lr;                         /* eta */
} or_config;

/* ---------------------------------------------------------------------------------- */
/* layout                                                                              */

static int64_t w_off(const or_config* c, int l) /* offset of W_{l+1} */
{
    int64_t o = 0;
    for (int i = 0; i < l; ++i) o += (int64_t)c->sizes[i + 1] * c->sizes[i] + c->sizes[i + 1];
    return o;
}
static int64_t b_off(const or_config* c, int l) { return w_off(c, l) + (int64_t)c->sizes[l + 1] * c->sizes[l]; }

int64_t or_param_count(const or_config* c) { return w_off(c, c->n_layers); }

static int max_width(const or_config* c)
{
    int m = 0;
    for (int l = 0; l <= c->n_layers; ++l) if (c->sizes[l] > m) m = c->sizes[l];
    return m;
}

/* Dataset split (section "Implementation Details": the dataset is split according to the
 * number of child networks).  Contiguous slices; the first N mod K slices get one more. */
void or_shard(int64_t n, int32_t k_total, int32_t k, int64_t* start, int64_t* len)
{
    int64_t q = n / k_total, r = n % k_total;
    *len = q + (k < r ? 1 : 0);
    *start = (int64_t)k * q + (k < r ? k : r);
}

/* ---------------------------------------------------------------------------------- */
/* bfloat16 rounding (round to nearest, ties to even) of a double to 8 significant bits */

double or_round_bf16(double v)
{
    if (v == 0.0 || !isfinite(v)) return v;
    int e;
    frexp(v, &e);            /* |v| = m * 2^e, 0.5 <= m < 1 */
    if (e < -125) e = -125;  /* below the smallest normal the quantum stays 2^-133 */
    double q = ldexp(1.0, e - 8);
    return nearbyint(v / q) * q; /* default rounding mode: nearest, ties to even */
}

static double rnd(const or_config* c, double v) { return c->precision == OR_BF16 ? or_round_bf16(v) : v; }

/* ---------------------------------------------------------------------------------- */
/* activations: eq. (4) rectifier, eq. (5) softmax; sigmoid and tanh are named only in
 * section "Activation Functions ..." and use their textbook forms.                     */

static double act_scalar(int a, double z)
{
    switch (a) {
    case OR_SIGMOID: return 1.0 / (1.0 + exp(-z));
    case OR_TANH: return tanh(z);
    case OR_RELU: return z < 0.0 ? 0.0 : z;
    case OR_LEAKY_RELU: return z < 0.0 ? 0.01 * z : z;
    default: return z;
    }
}

/* phi'(z), written with the activation value x = phi(z) where that is the usual form */
static double act_deriv(int a, double z, double x)
{
    switch (a) {
    case OR_SIGMOID: return x * (1.0 - x);
    case OR_TANH: return 1.0 - x * x;
    case OR_RELU: return z < 0.0 ? 0.0 : 1.0;
    case OR_LEAKY_RELU: return z < 0.0 ? 0.01 : 1.0;
    default: return 1.0;
    }
}

/* ---------------------------------------------------------------------------------- */
/* one sample: forward, output error, hidden errors                                    */

typedef struct {
    double* z[OR_MAX_LAYERS + 1]; /* z[l] for l = 1..L */
    double* x[OR_MAX_LAYERS + 1]; /* x[0] input, x[l] activation of layer l */
    double* d[OR_MAX_LAYERS + 1]; /* delta[l] */
} or_work;

static void work_alloc(const or_config* c, or_work* w)
{
    for (int l = 0; l <= c->n_layers; ++l) {
        w->z[l] = (double*)calloc((size_t)c->sizes[l], sizeof(double));
        w->x[l] = (double*)calloc((size_t)c->sizes[l], sizeof(double));
        w->d[l] = (double*)calloc((size_t)c->sizes[l], sizeof(double));
    }
}
static void work_free(const or_config* c, or_work* w)
{
    for (int l = 0; l <= c->n_layers; ++l) { free(w->z[l]); free(w->x[l]); free(w->d[l]); }
}

/* Forward propagation, eq. (2)-(3): z^l = W^l x^{l-1} + b^l, x^l = phi(z^l).
 * `wts` holds the weights used as operands (the bf16 shadow in bf16 mode), `th` the
 * master parameters (biases are always taken from the master). */
static void forward(const or_config* c, const double* wts, const double* th, const float* in, or_work* w)
{
    const int L = c->n_layers;
    for (int i = 0; i < c->sizes[0]; ++i) w->x[0][i] = rnd(c, (double)in[i]);
    for (int l = 1; l <= L; ++l) {
        const int n_in = c->sizes[l - 1], n_out = c->sizes[l];
        const double* W = wts + w_off(c, l - 1);
        const double* b = th + b_off(c, l - 1);
        for (int k = 0; k < n_out; ++k) {
            double s = 0.0;
            for (int j = 0; j < n_in; ++j) s += W[(int64_t)k * n_in + j] * w->x[l - 1][j];
            w->z[l][k] = s + b[k];
        }
        if (c->act[l - 1] == OR_SOFTMAX) {
            /* eq. (5); max(z) is subtracted first, which leaves every quotient unchanged */
            double m = w->z[l][0];
            for (int k = 1; k < n_out; ++k) if (w->z[l][k] > m) m = w->z[l][k];
            double sum = 0.0;
            for (int k = 0; k < n_out; ++k) sum += exp(w->z[l][k] - m);
            for (int k = 0; k < n_out; ++k) w->x[l][k] = exp(w->z[l][k] - m) / sum;
        } else {
            for (int k = 0; k < n_out; ++k) w->x[l][k] = act_scalar(c->act[l - 1], w->z[l][k]);
        }
        /* hidden activations are GEMM operands of the next layer and of the weight
         * gradient; in bf16 mode they are stored rounded */
        if (l < L)
            for (int k = 0; k < n_out; ++k) w->x[l][k] = rnd(c, w->x[l][k]);
    }
}

/* Output error and back-propagation, eq. (9)-(11). */
static void backward(const or_config* c, const double* wts, int label, or_work* w)
{
    const int L = c->n_layers, n_out = c->sizes[L];
    for (int k = 0; k < n_out; ++k) {
        const double e = (k == label) ? 1.0 : 0.0;
        double d;
        if (c->loss == OR_LOSS_XENT)
            d = w->x[L][k] - e; /* eq. (10) */
        else                    /* eq. (9) with C = 1/2 sum (x - e)^2 */
            d = (w->x[L][k] - e) * act_deriv(c->act[L - 1], w->z[L][k], w->x[L][k]);
        w->d[L][k] = rnd(c, d);
    }
    for (int l = L - 1; l >= 1; --l) { /* eq. (11): delta^l = (W^{l+1})^T delta^{l+1} (.) phi'(z^l) */
        const int n_here = c->sizes[l], n_next = c->sizes[l + 1];
        const double* W = wts + w_off(c, l);
        for (int j = 0; j < n_here; ++j) {
            double s = 0.0;
            for (int k = 0; k < n_next; ++k) s += W[(int64_t)k * n_here + j] * w->d[l + 1][k];
            w->d[l][j] = rnd(c, s * act_deriv(c->act[l - 1], w->z[l][j], w->x[l][j]));
        }
    }
}

/* Accumulate dC/dW_kj = delta_k x_j^{l-1} and dC/db_k = delta_k, eq. (7)-(8), (12)-(13). */
static void accumulate(const or_config* c, const or_work* w, double* grad)
{
    for (int l = 1; l <= c->n_layers; ++l) {
        const int n_in = c->sizes[l - 1], n_out = c->sizes[l];
        double* gW = grad + w_off(c, l - 1);
        double* gb = grad + b_off(c, l - 1);
        for (int k = 0; k < n_out; ++k) {
            for (int j = 0; j < n_in; ++j) gW[(int64_t)k * n_in + j] += w->d[l][k] * w->x[l - 1][j];
            gb[k] += w->d[l][k];
        }
    }
}

/* weights used as GEMM operands: the master itself, or its bf16 rounding */
static void make_operand_weights(const or_config* c, const double* th, double* wts)
{
    const int64_t P = or_param_count(c);
    memcpy(wts, th, (size_t)P * sizeof(double));
    if (c->precision == OR_BF16)
        for (int l = 0; l < c->n_layers; ++l) {
            double* W = wts + w_off(c, l);
            const int64_t n = (int64_t)c->sizes[l + 1] * c->sizes[l];
            for (int64_t i = 0; i < n; ++i) W[i] = or_round_bf16(W[i]);
        }
}

/* ---------------------------------------------------------------------------------- */
/* Training of one child network on its slice (section "Gradient Descent": stochastic,
 * batch and mini-batch gradient descent; the batch's gradients are averaged before the
 * update, and the changes are added to the old weights and biases).                   */

static void train_network(const or_config* c, double* th, const float* X, const int32_t* y, int64_t n)
{
    const int64_t P = or_param_count(c);
    const int n0 = c->sizes[0];
    double* grad = (double*)malloc((size_t)P * sizeof(double));
    double* wts = (double*)malloc((size_t)P * sizeof(double));
    or_work w;
    work_alloc(c, &w);
    const double eta = (double)c->lr;
    for (int64_t b0 = 0; b0 < n; b0 += c->batch) {
        const int64_t bt = (n - b0 < c->batch) ? (n - b0) : c->batch;
        memset(grad, 0, (size_t)P * sizeof(double));
        make_operand_weights(c, th, wts); /* every sample of the batch sees the pre-batch weights */
        for (int64_t s = b0; s < b0 + bt; ++s) {
            forward(c, wts, th, X + s * n0, &w);
            backward(c, wts, y[s], &w);
            accumulate(c, &w, grad);
        }
        const double scale = eta / (double)bt;
        for (int64_t i = 0; i < P; ++i) th[i] -= scale * grad[i];
    }
    work_free(c, &w);
    free(wts);
    free(grad);
}

typedef struct {
    const or_config* c;
    double* theta;
    const float* X;
    const int32_t* y;
    int64_t n;
    int first, stride;
} or_job;

static void* train_job(void* arg)
{
    or_job* j = (or_job*)arg;
    const int64_t P = or_param_count(j->c);
    for (int k = j->first; k < j->c->replicas; k += j->stride) {
        int64_t s, len;
        or_shard(j->n, j->c->replicas, k, &s, &len);
        train_network(j->c, j->theta + (int64_t)k * P, j->X + s * j->c->sizes[0], j->y + s, len);
    }
    return NULL;
}

/* One epoch of PNN training (section "Implementation Details"): split the data, train each
 * child network on its own slice, one thread per child network up to `threads` at once,
 * mirroring one goroutine per child network.  theta holds K parameter vectors. */
void or_train_epoch(const or_config* c, double* theta, const float* X, const int32_t* y, int64_t n,
                    int32_t threads)
{
    if (threads < 1) threads = 1;
    if (threads > c->replicas) threads = c->replicas;
    pthread_t* tid = (pthread_t*)malloc(sizeof(pthread_t) * (size_t)threads);
    or_job* jobs = (or_job*)malloc(sizeof(or_job) * (size_t)threads);
    for (int t = 0; t < threads; ++t) {
        jobs[t] = (or_job){c, theta, X, y, n, t, threads};
        pthread_create(&tid[t], NULL, train_job, &jobs[t]);
    }
    for (int t = 0; t < threads; ++t) pthread_join(tid[t], NULL);
    free(jobs);
    free(tid);
}

/* Train a subset of the child networks (replica ids in `ids`), for sampled checks. */
void or_train_replicas(const or_config* c, double* theta_sub, const int32_t* ids, int32_t n_ids,
                       const float* X, const int32_t* y, int64_t n)
{
    const int64_t P = or_param_count(c);
    for (int i = 0; i < n_ids; ++i) {
        int64_t s, len;
        or_shard(n, c->replicas, ids[i], &s, &len);
        train_network(c, theta_sub + (int64_t)i * P, X + s * c->sizes[0], y + s, len);
    }
}

/* Combination by averaging (section "Implementation Details"): each parameter of the
 * combined network is the sum of the K child networks' values divided by K.  Summation in long
 * double, k ascending, then the division by K. */
void or_merge(const or_config* c, const double* theta, double* merged)
{
    const int64_t P = or_param_count(c);
    for (int64_t i = 0; i < P; ++i) {
        long double s = 0.0L;
        for (int k = 0; k < c->replicas; ++k) s += (long double)theta[(int64_t)k * P + i];
        merged[i] = (double)(s / (long double)c->replicas);
    }
}

/* Weighted combination (sections "Parallel Neuronal Networks" and "Findings and Conclusion"
 * leave combination functions other than the average open without defining one; this is the
 * weighted mean): merged = sum_k w_k theta_k / sum_k w_k, the sums in long double with k
 * ascending.  w: K non-negative weights with a positive sum. */
void or_merge_weighted(const or_config* c, const double* theta, const double* w, double* merged)
{
    const int64_t P = or_param_count(c);
    long double ws = 0.0L;
    for (int k = 0; k < c->replicas; ++k) ws += (long double)w[k];
    for (int64_t i = 0; i < P; ++i) {
        long double s = 0.0L;
        for (int k = 0; k < c->replicas; ++k) s += (long double)w[k] * (long double)theta[(int64_t)k * P + i];
        merged[i] = (double)(s / ws);
    }
}

/* Forward pass of one network over n samples; out [n][sizes[L]] receives x^L. */
void or_forward(const or_config* c, const double* th, const float* X, int64_t n, double* out)
{
    const int64_t P = or_param_count(c);
    const int L = c->n_layers;
    double* wts = (double*)malloc((size_t)P * sizeof(double));
    make_operand_weights(c, th, wts);
    or_work w;
    work_alloc(c, &w);
    for (int64_t s = 0; s < n; ++s) {
        forward(c, wts, th, X + s * c->sizes[0], &w);
        memcpy(out + s * c->sizes[L], w.x[L], sizeof(double) * (size_t)c->sizes[L]);
    }
    work_free(c, &w);
    free(wts);
}

/* Classification (section "Fundamentals": one output neuron per class): the predicted class
 * is the index of the largest output, the lowest index on ties.  Returns the number of
 * correct predictions when labels are given. */
int64_t or_predict(const or_config* c, const double* th, const float* X, int64_t n, const int32_t* y,
                   int32_t* pred)
{
    const int n_out = c->sizes[c->n_layers];
    double* out = (double*)malloc(sizeof(double) * (size_t)n_out * (size_t)n);
    or_forward(c, th, X, n, out);
    int64_t correct = 0;
    for (int64_t s = 0; s < n; ++s) {
        int best = 0;
        for (int k = 1; k < n_out; ++k) if (out[s * n_out + k] > out[s * n_out + best]) best = k;
        if (pred) pred[s] = best;
        if (y && y[s] == best) ++correct;
    }
    free(out);
    return correct;
}

/* Mean cost over n samples: quadratic 1/2 sum (x - e)^2, or cross-entropy eq. (6) for a
 * softmax output; for a sigmoid output with the cross-entropy flag the matching cost is
 * -sum [e log x + (1 - e) log(1 - x)], whose output error is x - e. */
double or_cost(const or_config* c, const double* th, const float* X, const int32_t* y, int64_t n)
{
    const int L = c->n_layers, n_out = c->sizes[L];
    double* out = (double*)malloc(sizeof(double) * (size_t)n_out * (size_t)n);
    or_forward(c, th, X, n, out);
    double total = 0.0;
    for (int64_t s = 0; s < n; ++s)
        for (int k = 0; k < n_out; ++k) {
            const double x = out[s * n_out + k], e = (k == y[s]) ? 1.0 : 0.0;
            if (c->loss == OR_LOSS_MSE)
                total += 0.5 * (x - e) * (x - e);
            else if (c->act[L - 1] == OR_SOFTMAX)
                total += -e * log(x);
            else
                total += -(e * log(x) + (1.0 - e) * log(1.0 - x));
        }
    free(out);
    return total / (double)n;
}

/* Mean gradient of the cost over n samples at fixed parameters (back-propagation). */
void or_gradient(const or_config* c, const double* th, const float* X, const int32_t* y, int64_t n,
                 double* grad)
{
    const int64_t P = or_param_count(c);
    double* wts = (double*)malloc((size_t)P * sizeof(double));
    make_operand_weights(c, th, wts);
    memset(grad, 0, (size_t)P * sizeof(double));
    or_work w;
    work_alloc(c, &w);
    for (int64_t s = 0; s < n; ++s) {
        forward(c, wts, th, X + s * c->sizes[0], &w);
        backward(c, wts, y[s], &w);
        accumulate(c, &w, grad);
    }
    for (int64_t i = 0; i < P; ++i) grad[i] /= (double)n;
    work_free(c, &w);
    free(wts);
}

/* Per-sample intermediate values of one forward/backward pass (for worked examples):
 * z, x and delta of every layer, concatenated layer by layer (layers 1..L). */
void or_trace(const or_config* c, const double* th, const float* x_in, int32_t label, double* z_out,
              double* x_out, double* d_out)
{
    const int64_t P = or_param_count(c);
    double* wts = (double*)malloc((size_t)P * sizeof(double));
    make_operand_weights(c, th, wts);
    or_work w;
    work_alloc(c, &w);
    forward(c, wts, th, x_in, &w);
    backward(c, wts, label, &w);
    int64_t o = 0;
    for (int l = 1; l <= c->n_layers; ++l) {
        for (int k = 0; k < c->sizes[l]; ++k) {
            z_out[o + k] = w.z[l][k];
            x_out[o + k] = w.x[l][k];
            d_out[o + k] = w.d[l][k];
        }
        o += c->sizes[l];
    }
    work_free(c, &w);
    free(wts);
    (void)max_width;
}
