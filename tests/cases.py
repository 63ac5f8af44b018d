"""Parity cases shared by the GPU parity tests and the CPU test of the oracle's own sensitivity
to rounding (which shows, for each case, that its comparison bar measures the implementation and
not the amplification of rounding differences)."""
import pnn_inputs as I

# ------------------------------------------------------------------------------------
# full epochs at reduced sizes: ragged last batches / chunks, uneven slices, merges
# (workload, overrides, N, epochs)

EPOCH_CASES = [
    # workload, overrides, N, epochs
    (0, {}, 2000, 1),                                         # 784-16-10, K = 1, at full size
    (1, {}, 4 * 300 + 3, 1),                                  # per-sample chunks with a ragged tail
    (1, dict(replicas=3), 3 * 140 + 1, 2),                    # uneven slices, two epochs
    (2, {}, 16 * 100 + 5, 2),                                 # batches 32,32,32,4/5
    (3, dict(replicas=8), 8 * 150 + 3, 2),                    # bf16, merge + broadcast each epoch
    (3, dict(replicas=6), 6 * 150 + 5, 1),                    # bf16, K not a multiple of 8: two update launches
    (4, dict(replicas=16), 16 * 260 + 7, 2),                  # batches 128,128,4/5, merge each epoch
    (4, dict(replicas=4), 4 * 224 + 2, 2),                    # batches 128, 97/96 (one launch, zero padded)
    # the fused last layer with softmax / cross-entropy over 16 outputs (tanh hidden layer), and
    # with a single sigmoid output; batches 128 + 72/73 and 128 + 5/6
    (4, dict(sizes=(784, 256, 16), acts=(I.TANH, I.SOFTMAX), loss=I.LOSS_XENT, replicas=3), 3 * 200 + 1, 1),
    (4, dict(sizes=(784, 320, 1), replicas=2), 2 * 134 + 1, 1),
    # shards of 257 and 256 samples: the third batch step has one row for two CNs and none for
    # the other two (fused last layer with empty CNs in a step)
    (4, dict(sizes=(784, 256, 10), replicas=4), 4 * 256 + 2, 1),
    (2, dict(sizes=(784, 64, 32, 10), acts=(I.RELU, I.TANH, I.SOFTMAX), loss=I.LOSS_XENT, batch=16,
             replicas=2, merge_every_epoch=True), 2 * 90 + 1, 2),   # deeper fp32 net
    (0, dict(sizes=(784, 32, 16, 10), acts=(I.TANH, I.SIGMOID, I.SIGMOID), replicas=2), 2 * 40, 1),  # B=1, L=3
    (1, dict(acts=(I.RELU, I.SOFTMAX), loss=I.LOSS_XENT, replicas=2), 2 * 150, 1),  # per-sample softmax/xent
    # variants of the paper's first experiment: other activations, a large learning rate,
    # full-batch gradient descent (a batch as large as the slice)
    (1, dict(acts=(I.LEAKY_RELU, I.SOFTMAX), loss=I.LOSS_XENT, replicas=2), 2 * 150, 1),  # per-sample leaky ReLU
    (1, dict(sizes=(784, 64, 10), acts=(I.TANH, I.SIGMOID), replicas=3), 3 * 100 + 2, 1),  # per-sample tanh
    (1, dict(lr=0.6, replicas=2), 2 * 120, 1),                # sigmoid, eta 0.6
    (2, dict(sizes=(784, 96, 10), acts=(I.LEAKY_RELU, I.SOFTMAX), loss=I.LOSS_XENT, batch=8, replicas=4),
     4 * 40 + 3, 2),                                          # mini-batch leaky ReLU / softmax
    (2, dict(batch=101, replicas=4), 4 * 100 + 3, 3),         # full batch: one step per slice and epoch
    # per-sample with more CNs than 16-row tile workgroups fit: 32-row tiles
    (1, dict(replicas=32), 32 * 70 + 5, 1),
    (1, dict(sizes=(784, 64, 10), replicas=60), 60 * 40 + 7, 1),
    # per-sample with more CNs than fit the device at once: 64 CNs of 16-row tiles in 3
    # launches of 21/21/22; 96 CNs of 32-row tiles in 2 launches of 48
    (1, dict(replicas=64), 64 * 40 + 5, 1),
    (1, dict(replicas=96), 96 * 30 + 5, 1),
    # persistent mini-batch plan: a hidden width that leaves the last 16-neuron tile half
    # empty, batches of 7 and a grid that is no multiple of 8; 32-neuron tiles (20 CNs of 256
    # neurons); batches of 2 with ReLU / softmax
    (2, dict(sizes=(784, 56, 10), acts=(I.SIGMOID, I.SIGMOID), batch=7, replicas=5), 5 * 40 + 3, 2),
    (2, dict(replicas=20), 20 * 40 + 3, 1),
    (2, dict(acts=(I.RELU, I.SOFTMAX), loss=I.LOSS_XENT, batch=2, replicas=3), 3 * 30 + 2, 1),
    # edge shapes: the most weight layers (8, mini-batch, every activation); four layers with
    # B = 1 (the generic per-sample path); one weight layer (logistic regression); the widest
    # output layer (16, softmax); a single sigmoid output; a hidden width that leaves the
    # per-sample kernel's last 16-row tile half empty; bf16-mixed with B = 1
    (2, dict(sizes=(784, 64, 56, 48, 40, 32, 24, 16, 10),
             acts=(I.RELU, I.TANH, I.LEAKY_RELU, I.SIGMOID, I.RELU, I.TANH, I.SIGMOID, I.SOFTMAX),
             loss=I.LOSS_XENT, batch=8, replicas=3), 3 * 50 + 2, 1),
    (0, dict(sizes=(784, 40, 24, 16, 10), acts=(I.RELU, I.TANH, I.SIGMOID, I.SIGMOID), replicas=2), 2 * 40 + 1, 1),
    (2, dict(sizes=(784, 10), acts=(I.SOFTMAX,), loss=I.LOSS_XENT, batch=8, replicas=4), 4 * 40 + 3, 2),
    (2, dict(sizes=(784, 64, 16), acts=(I.SIGMOID, I.SOFTMAX), loss=I.LOSS_XENT, batch=16, replicas=4), 4 * 60 + 1, 1),
    (2, dict(sizes=(784, 32, 1), acts=(I.SIGMOID, I.SIGMOID), batch=4, replicas=2), 2 * 40 + 1, 1),
    (1, dict(sizes=(784, 40, 10), replicas=3), 3 * 70 + 1, 1),
    (3, dict(sizes=(784, 64, 10), acts=(I.RELU, I.SOFTMAX), batch=1, replicas=2, merge_every_epoch=False), 2 * 40, 1),
    # persistent mini-batch plan in CN groups (32-neuron tiles): 80 CNs in 3 launches of
    # 26/27/27; 64 CNs in 2 launches of 32, merge + broadcast each epoch
    (2, dict(replicas=80), 80 * 40 + 3, 1),
    (2, dict(replicas=64, merge_every_epoch=True), 64 * 40 + 3, 2),
]

# fp32 epoch cases where the method amplifies rounding differences to the size of the epoch bar
# (tests/test_sensitivity.py: a one-ulp change of the oracle's own start moves some elements by
# half the bar or more, while every layer stays below a tenth of it normwise).  On the GPU they
# are held normwise per layer after the epoch, and elementwise step by step.
SENSITIVE_FP32_CASES = [
    # tanh hidden layer, sigmoid outputs with the cross-entropy error (per-sample)
    (1, dict(sizes=(784, 64, 10), acts=(I.TANH, I.SIGMOID), loss=I.LOSS_XENT, replicas=3), 3 * 100 + 2, 1),
]

# ------------------------------------------------------------------------------------
# the per-sample chunked plan (B = 1, one hidden layer, where the persistent per-sample kernel
# does not fit): overrides of the 784-128-10 per-sample workload and N, one epoch

CHUNKED_CASES = [
    # overrides of the 784-128-10 per-sample workload, N; chunk length T = 64 / 128 / 16 / 32
    (dict(sizes=(784, 256, 10), replicas=2), 2 * 300 + 1),             # 4 full chunks + 44/45
    (dict(sizes=(784, 160, 10), replicas=48), 48 * 200 + 5),           # 48 CNs: 1 chunk + 72/73
    (dict(sizes=(784, 1024, 10), replicas=2), 2 * 50 + 1),             # 3 chunks + 2/3
    (dict(sizes=(784, 384, 10), acts=(I.RELU, I.SOFTMAX), loss=I.LOSS_XENT, replicas=3), 3 * 90 + 2),
]


# ------------------------------------------------------------------------------------
# bf16-mixed epochs: the weight tensors held elementwise after each epoch (all tensors are also
# held normwise per layer).  A tensor is left out where the oracle's own divergence under a
# one-ulp change of its start reaches half the bar (tests/test_sensitivity.py asserts both
# sides); at full size (59 steps per epoch) every tensor is normwise only.
# key: (workload, overrides as sorted items, N, epochs) -> {epoch: tensors}

def case_key(idx, over, N, epochs):
    return (idx, tuple(sorted(over.items())), N, epochs)


BF16_ELEMENTWISE = {
    case_key(3, dict(replicas=8), 8 * 150 + 3, 2): {0: ("W1", "W3", "b3"), 1: ("W3",)},
    case_key(3, dict(replicas=6), 6 * 150 + 5, 1): {0: ("W1", "W3", "b3")},
}
