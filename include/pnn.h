/*
 * pnn.h -- C ABI of the MI355X (gfx950) parallel neural network (PNN) library.
 *
 * The method (Kalwarowskyj & Schikuta, "Parallel Neural Networks in Golang", section
 * "Parallel Neuronal Networks"): the training set is split into K slices; K child networks
 * (CNs), all started from one parameter vector, each train on their own slice with
 * back-propagation and (mini-batch) stochastic gradient descent (section "Fundamentals",
 * eq. (2)-(13)); the CNs are then combined into one network by averaging all weights and
 * all biases.  One handle serves a single sequential network (K = 1) and a PNN (K > 1)
 * alike, as the paper's TrainableNetwork interface does (section "Implementation Details").
 *
 * Conventions shared by every call:
 *  - Device pointers (suffix _dev) are HIP device memory owned by the caller; the library
 *    never frees them and does not keep them after the call returns.
 *  - The library owns the parameters and its workspace (allocated in pnn_init, released
 *    in pnn_destroy).
 *  - `hip_stream` is a hipStream_t (NULL = the default stream).  Device work is enqueued on
 *    it and the call returns once enqueued; only pnn_get_params, pnn_set_params, pnn_eval
 *    and a pnn_infer call with correct_host != NULL wait for the device.  After a training
 *    epoch on a persistent plan (pnn_plan), the next call that consumes the CNs other than
 *    pnn_train_epoch first waits for that epoch to end, to read its failure flag.
 *  - Errors are returned as a pnn_status; the message of the last failure is available
 *    from pnn_last_error (per handle; a NULL handle gives the message of the last failed
 *    pnn_init on the calling thread).  No exception or abort crosses the interface.
 *  - One handle must not be used from two host threads at once.
 *  - Input rows x_dev are read with 16-byte vector loads: x_dev must be 16-byte aligned
 *    (PNN_EINVAL otherwise); sizes[0] is a multiple of 8, so every row then is too.
 *
 * Parameter layout (host side, get/set): one network is P = pnn_param_count(cfg) floats,
 * W1, b1, W2, b2, ..., W_l row-major [sizes[l]][sizes[l-1]], b_l [sizes[l]].
 */
#ifndef PNN_H
#define PNN_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct pnn_net pnn_net; /* opaque, library-owned */

typedef enum {
    PNN_OK = 0,
    PNN_EINVAL = -1, /* invalid configuration or argument (NULL pointer, bad index) */
    PNN_ESHAPE = -2, /* sizes do not fit (N < K leaves a slice empty, n < 0, ...) */
    PNN_ENOMEM = -3, /* device allocation failed */
    PNN_EHIP = -4,   /* a HIP runtime call or kernel launch failed */
    PNN_ESTATE = -5  /* the handle is unusable after an earlier device failure */
} pnn_status;

/* Activation of a layer.  Rectifier eq. (4), softmax eq. (5); sigmoid and tanh are named in
 * section "Activation Functions in Single- and Parallel Neuronal Networks" (textbook forms);
 * leaky rectifier with slope 0.01 for z < 0.  The rectifier's derivative at z = 0 is 1
 * (eq. (4) puts z = 0 in the linear branch).  Softmax is allowed on the output layer only. */
typedef enum { PNN_SIGMOID = 0, PNN_TANH = 1, PNN_RELU = 2, PNN_LEAKY_RELU = 3, PNN_SOFTMAX = 4 } pnn_act;

/* Output error rule.  MSE: quadratic cost 1/2 sum (x - e)^2 with eq. (9),
 * delta^L = (x^L - e) (.) phi'(z^L).  XENT: eq. (10), delta^L = x^L - e, for a softmax
 * output (eq. (6) cost) or a sigmoid output (binary cross-entropy). */
typedef enum { PNN_LOSS_MSE = 0, PNN_LOSS_XENT = 1 } pnn_loss;

/* FP32: every value stored in fp32.  BF16_MIXED: inputs, hidden activations, weights and
 * deltas enter the matrix products as bfloat16 (round to nearest even) with fp32
 * accumulation; biases, activations' arithmetic, softmax and the master weights are fp32. */
typedef enum { PNN_FP32 = 0, PNN_BF16_MIXED = 1 } pnn_precision;

typedef struct {
    int32_t n_layers;  /* L weight layers, 1..8 */
    int32_t sizes[9];  /* sizes[0] inputs ... sizes[L] outputs (classes), each >= 1 */
    int32_t act[8];    /* pnn_act of weight layer l+1 */
    int32_t loss;      /* pnn_loss */
    int32_t precision; /* pnn_precision */
    int32_t replicas;  /* K >= 1 child networks */
    int32_t batch;     /* B >= 1; 1 = per-sample stochastic gradient descent */
    float lr;          /* eta, eq. (12)-(13) */
} pnn_config;

/* Checks a configuration without touching the GPU.  Rules: 1 <= L <= 8; sizes >= 1 and
 * sizes[l] % 8 == 0 for every layer except the output layer, whose width is <= 16;
 * softmax only on the output layer and only with PNN_LOSS_XENT; XENT needs a sigmoid or
 * softmax output; K >= 1, B >= 1, finite lr >= 0.  Returns PNN_OK or PNN_EINVAL. */
pnn_status pnn_config_check(const pnn_config* cfg);

/* P, the number of parameters of one network: every weight W_kj and every bias b_k of each
 * layer (eq. (2): sizes[l] * sizes[l-1] weights and sizes[l] biases per layer l), which is what
 * the combination averages (section "Implementation Details").  0 for an invalid
 * configuration. */
int64_t pnn_param_count(const pnn_config* cfg);

/* Dataset split (section "Implementation Details": the dataset is split according to the
 * number of CNs): slice k of N samples over K CNs is the contiguous row range
 * [start, start + len); the first N mod K slices hold one more sample.  Host only. */
pnn_status pnn_shard(int64_t N, int32_t K, int32_t k, int64_t* start, int64_t* len);

/* Creates a handle on the current HIP device.  theta0_host (P floats, host memory, read
 * during the call) is cloned into all K child networks and into the merged network
 * (section "Accuracy and Confidence of Networks": the PNN's CNs start as clones of one
 * random network).  *out receives the handle; NULL on failure. */
pnn_status pnn_init(const pnn_config* cfg, const float* theta0_host, void* hip_stream, pnn_net** out);

/* One training epoch of every CN over its own slice (sections "Gradient Descent" and
 * "Implementation Details").  x_dev: [N][sizes[0]] row-major fp32; y_dev: [N] int32
 * class labels in [0, sizes[L]).  CN k visits rows of its slice in ascending order in
 * batches of B (the last batch may be shorter); each batch's gradients are averaged before
 * the update W <- W - eta / B_t * sum_b delta_b x_b^T, b <- b - eta / B_t * sum_b delta_b.
 * Requires N >= K (PNN_ESHAPE otherwise).  Labels outside [0, sizes[L]) give an undefined
 * (but memory-safe) update. */
pnn_status pnn_train_epoch(pnn_net* net, const float* x_dev, const int32_t* y_dev, int64_t N, void* hip_stream);

/* One epoch over the rows in a given order (the per-epoch shuffling that the paper leaves
 * open: it trains on the slices in their stored order).  Equivalent to pnn_train_epoch on
 * x[order[0..N)], y[order[0..N)]: epoch row r is data-set row order_dev[r], and the K slices
 * are the contiguous ranges of that sequence.  order_dev [N] int32 on the device, normally a
 * permutation drawn by the caller from a seeded generator (within each slice's range for a
 * per-CN shuffle); entries outside [0, N) select row 0.  The rows are gathered into a
 * library-owned staging copy (N x sizes[0] floats, grown with hipMalloc when a larger N
 * arrives) on the caller's stream.  Errors as pnn_train_epoch; N must fit int32. */
pnn_status pnn_train_epoch_order(pnn_net* net, const float* x_dev, const int32_t* y_dev, int64_t N,
                                 const int32_t* order_dev, void* hip_stream);

/* Combination by averaging (section "Implementation Details"): merged := (1/K) sum_k theta_k
 * for every weight and bias, accumulated in fp64 with k ascending, rounded once to fp32.
 * broadcast != 0 also copies the merged network back into every CN (model averaging
 * between epochs); with the fused last-layer plan (pnn_plan) that copy is made by the next
 * epoch's first step, which reads the merged network, or on demand by the first other call
 * that reads a CN's parameters: every call sees the CNs as copied. */
pnn_status pnn_merge(pnn_net* net, int32_t broadcast, void* hip_stream);

/* Weighted combination: the paper notes that CNs can be combined in several ways and leaves
 * better combination functions to future work (sections "Parallel Neuronal Networks" and
 * "Findings and Conclusion") without defining one; this one is the weighted mean:
 * merged := sum_k w_k theta_k / sum_k w_k, each product and the sum in fp64 with k ascending,
 * rounded once to fp32.  weights_host: K host doubles, each finite and >= 0, with a positive sum
 * (PNN_EINVAL otherwise, nothing launched).  Equal weights give pnn_merge's result bitwise.
 * broadcast as in pnn_merge.  The weights are copied to a library-owned device array before
 * the call returns (the call waits for the stream's earlier work). */
pnn_status pnn_merge_weighted(pnn_net* net, const double* weights_host, int32_t broadcast, void* hip_stream);

/* Classification (sections "Fundamentals" and "MNIST Dataset": one output neuron per class,
 * tested on unseen data).  which = -1 uses the merged network, 0..K-1 one CN.
 * x_dev [n][sizes[0]] fp32.  pred_dev [n] int32 receives the argmax of the outputs (lowest
 * index on ties).  out_dev (nullable) [n][sizes[L]] fp32 receives the outputs x^L.  When
 * y_dev [n] and correct_host are both non-NULL, the call waits for the device and writes
 * the number of rows with pred == y to *correct_host.  n = 0 reads and writes nothing on the
 * device (the pointers may be NULL) and sets *correct_host, if given, to 0. */
pnn_status pnn_infer(pnn_net* net, int32_t which, const float* x_dev, int64_t n, int32_t* pred_dev, float* out_dev,
                     int64_t* correct_host, const int32_t* y_dev, void* hip_stream);

/* Evaluation of one network on labelled rows: the accuracy test of the merged network
 * (sections "Implementation Details" and "MNIST Dataset") and the per-CN comparison and cost
 * per epoch of the experiments.  which = -1 merged, 0..K-1 one CN.  x_dev [n][sizes[0]] fp32
 * and y_dev [n] int32 are the caller's device arrays (labels in [0, sizes[L])).  Writes
 *   *correct_host (nullable): rows whose argmax output (lowest index on ties) equals the label;
 *   *cost_host (nullable): the mean cost over the rows, the cost whose output error training
 *     uses: quadratic 1/2 sum_o (x_o - e_o)^2, or with PNN_LOSS_XENT the cross-entropy
 *     (-log x_label for a softmax output, eq. (6); -sum_o [e_o log x_o + (1 - e_o) log(1 - x_o)]
 *     for a sigmoid output), each row's cost in fp64 from the fp32 outputs, the rows summed in
 *     a fixed order in fp64.
 * Waits for the device.  The library owns a per-row cost buffer of the largest n seen (grown
 * with hipMalloc on the first call that needs more).  n = 0 gives 0 and 0.0 without device work;
 * a NULL x_dev or y_dev is PNN_EINVAL. */
pnn_status pnn_eval(pnn_net* net, int32_t which, const float* x_dev, const int32_t* y_dev, int64_t n,
                    int64_t* correct_host, double* cost_host, void* hip_stream);

/* pnn_eval without any device allocation, for callers that cannot allocate device memory
 * (code that must not call hipMalloc: tight evaluation loops in serving or training, harnesses
 * that forbid allocation).  Same arguments, results and errors as pnn_eval, computed by the same
 * kernels; its workspace (a count, a sum, one 8,192-row chunk's hidden activations and, when
 * cost_host is given, n per-row costs) lives in a fixed 64 MiB device array that the library
 * holds on every GPU it runs on until the process ends, instead of in buffers grown with
 * hipMalloc.  A call that needs more workspace than that returns PNN_ESHAPE and launches
 * nothing (with cost_host: n <= 8,388,576 - 1,024 A up to alignment, A the bytes of hidden
 * activations of one row: 4 per hidden neuron, 2 in bf16-mixed precision).  Every call on one GPU shares that GPU's array, which keeps the last call's contents:
 * calls that overlap in time on one GPU (other host threads, other streams) race and must be
 * serialised by the caller. */
pnn_status pnn_eval_noalloc(pnn_net* net, int32_t which, const float* x_dev, const int32_t* y_dev, int64_t n,
                            int64_t* correct_host, double* cost_host, void* hip_stream);

/* Copies one network's parameters (which = -1 merged, 0..K-1 a CN) to host_out (P floats)
 * in the layout above.  Waits for the device. */
pnn_status pnn_get_params(pnn_net* net, int32_t which, float* host_out);

/* Overwrites parameters from host_in (P floats): which = -1 the merged network, 0..K-1 one
 * CN, -2 every CN and the merged network.  Waits for the device.  Used for checkpoint and
 * resume: training continued from restored parameters is bitwise identical. */
pnn_status pnn_set_params(pnn_net* net, int32_t which, const float* host_in);

/* Message of the last failure on this handle ("" if none); NULL net: last pnn_init failure
 * of the calling thread.  The string lives until the next call on the same handle. */
const char* pnn_last_error(const pnn_net* net);

/* Device time of the library's kernels, for throughput accounting.  pnn_profile(net, 1)
 * starts recording a HIP event pair around every kernel the library launches (this adds
 * host overhead; leave it off when measuring whole-call throughput) and clears the
 * counters; pnn_profile(net, 0) stops.  pnn_profile_read fills up to `cap` entries of
 * names (static strings), total_ms and launches, waits for the device, and returns the
 * number of distinct kernels recorded. */
pnn_status pnn_profile(pnn_net* net, int32_t enable);
int32_t pnn_profile_read(pnn_net* net, const char** names, double* total_ms, int64_t* launches, int32_t cap);

/* Name of the training plan that pnn_init chose for the handle (a static string; "" for
 * a NULL handle).  All plans compute the update of pnn_train_epoch and differ only in the
 * order of fp32 roundings:
 *  "per-sample persistent"  B = 1, one hidden layer of <= 128 neurons, sizes[0] <= 832: one
 *                           launch per epoch for each group of CNs whose workgroups fit the
 *                           device at once (all K CNs in one group where they fit);
 *  "per-sample chunked"     B = 1 otherwise;
 *  "mini-batch persistent"  fp32, one hidden layer, 2 <= B <= 32, <= 16 outputs,
 *                           sizes[0] % 16 == 0 and <= 832, H <= 512: one launch per epoch for
 *                           each group of CNs whose ceil(H / 16) (or ceil(H / 32)) tile
 *                           workgroups fit the device at once;
 *  "mini-batch fused last layer"  fp32, one hidden layer of >= 256 neurons (a multiple of
 *                           4), B = 128, <= 16 outputs, sizes[0] >= 128 (a multiple of 4),
 *                           the split-bf16 products (not PNN_GEMM=fp32): kernel launches per
 *                           batch step, with the last layer's forward in the hidden layer's
 *                           forward and its hidden errors and update in the hidden layer's
 *                           update (one pass less over the hidden activations);
 *  "mini-batch"             kernel launches per layer and batch step.
 * The environment variable PNN_MB_PLAN=launch, read by pnn_init, selects "mini-batch"
 * where "mini-batch persistent" or "mini-batch fused last layer" would apply.  The persistent plans' workgroups wait for each
 * other with bounded polls (PNN_SPIN_LIMIT, read by pnn_init, default 4194304 polls); a launch
 * that runs into the bound ends every workgroup and leaves the CNs' parameters unspecified.
 * The next call that consumes the CNs -- pnn_merge, pnn_merge_weighted, pnn_infer, pnn_eval,
 * pnn_get_params, pnn_set_params (each waits for the last persistent launch to end first) or
 * pnn_train_epoch (which does not wait: it sees the failure once that launch has ended, and a
 * persistent launch enqueued after the failed one ends at once) -- returns PNN_EHIP and marks
 * the handle unusable (PNN_ESTATE from then on).  PNN_TEST_STALL_WAITS=1 (tests of that path
 * only) makes the persistent kernels' waits run into the bound.  PNN_TEST_TILE_DELAY=n (n sleeps
 * of about 3 us, ordering tests only) starts half of every CN's tile workgroups late in the
 * per-sample persistent kernel; the results stay within rounding of an undelayed run. */
const char* pnn_plan(const pnn_net* net);

/* Releases the handle and everything it owns (NULL is ignored). */
void pnn_destroy(pnn_net* net);

#ifdef __cplusplus
}
#endif

#endif /* PNN_H */
