// pnn.hip -- host orchestration and C ABI of the MI355X PNN library (declared in pnn.h).
//
// Device layout: every network (each of the K CNs and the merged one) is a padded
// parameter block of `pstride` floats; W_l and b_l start at 64-float (256-byte) aligned
// offsets, so every row of every matrix can be read with 16-byte loads.  The K CN blocks
// are contiguous ([K][pstride]).  In bf16-mixed precision a bf16 shadow of every block
// ([K][pstride] plus one for the merged network) holds the weights used as GEMM operands.
//
// Training plans:
//  * per-sample SGD of a one-hidden-layer fp32 network (B = 1, L = 2, hidden <= 1024,
//    outputs <= 16): chunked plan -- Gram matrices of each chunk of T samples, then per
//    chunk P = W1 x_t (GEMM), the T sequential steps (psgd_chunk_kernel), and the rank-T
//    update of W1 (GEMM).
//  * everything else: mini-batch plan -- per batch step, forward GEMMs with fused bias and
//    activation, output layer with fused output error, hidden errors (GEMM with fused
//    phi'), and weight-gradient GEMMs with the SGD update (and bias update) fused into the
//    epilogue.  B = 1 runs this plan with batches of one sample.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <map>
#include <mutex>
#include <string>
#include <vector>

#include "../../include/pnn.h"
#include "kernels.hpp"

using namespace pnn;

// Fixed workspace of pnn_eval_noalloc, for callers that cannot allocate device memory: one
// copy per GPU, held until the process ends.  In host code `scratch` names a host-side stand-in
// of the array, not its device address: host code reaches the memory only through the address
// that hipGetSymbolAddress gives for the current device (scratch_setup, scratch_ptr).
constexpr size_t SCRATCH_BYTES = size_t(64) << 20;
static __device__ __align__(256) unsigned char scratch[SCRATCH_BYTES];

namespace {

thread_local std::string g_init_error;

constexpr int MAX_DEVICES = 64;
std::mutex g_scratch_mu;
void* g_scratch_addr[MAX_DEVICES] = {nullptr};

// device address of the workspace on `dev` (NULL before scratch_setup ran there)
void* scratch_ptr(int dev) {
    if (dev < 0 || dev >= MAX_DEVICES) return nullptr;
    std::lock_guard<std::mutex> g(g_scratch_mu);
    return g_scratch_addr[dev];
}

struct ProfRec {
    const char* name;
    hipEvent_t a, b;
};

}  // namespace

struct pnn_net {
    pnn_config cfg;
    int L = 0;
    int sizes[9] = {0};
    int act[8] = {0};
    int64_t P = 0;        // packed parameters per network
    int64_t pstride = 0;  // padded block
    int64_t off_w[8] = {0}, off_b[8] = {0};
    bool bf16 = false;
    int device = 0;
    bool broken = false;
    std::string err;

    float* theta = nullptr;    // [K][pstride]
    float* merged = nullptr;   // [pstride]
    bf16_t* shadow = nullptr;  // [K][pstride]
    bf16_t* mshadow = nullptr; // [pstride]

    // mini-batch workspace: activations x_l (l = 1..L-1) and errors d_l (l = 1..L), [K][B][s_l]
    void* act_ws[9] = {nullptr};
    void* del_ws[9] = {nullptr};
    // inference workspace: [rows][s_l], l = 1..L-1
    void* inf_ws[9] = {nullptr};
    int inf_rows = 0;
    unsigned long long* d_correct = nullptr;
    double* d_cost = nullptr;     // [cost_rows] per-row costs of an evaluation
    int64_t cost_rows = 0;
    double* d_cost_sum = nullptr;
    double* d_mw = nullptr;       // [K] weights of a weighted combination
    float* ord_x = nullptr;       // [ord_rows][sizes[0]] rows of an epoch in a given order
    int32_t* ord_y = nullptr;
    int64_t ord_rows = 0;

    // chunked per-sample plan
    bool psgd = false;
    int T = 0, ksplit = 1, kchunk = 0;
    float* ppart = nullptr;  // [ksplit][K][T][H]
    float* d1 = nullptr;     // [K][T][H]
    float* gram = nullptr;   // [K][nch][T][T]
    size_t gram_elems = 0;
    // persistent variant: nrb tiles of 16 rows of W1 per CN
    bool persistent = false;
    bool pspecial = false;   // sigmoid / sigmoid / quadratic loss / 10 outputs
    int nrb = 0;             // tile workgroups per CN
    int kgroup = 0;          // CNs per launch of a persistent plan (all K, or groups that fit the CUs)
    int prt = 1;             // 16-row sub-tiles per tile workgroup
    int* flags = nullptr;    // per-sample plan: qready[2][K] (by chunk parity), dready[K], abort
    float* qbuf = nullptr;   // [2][K][T][H]
    float* gramx = nullptr;  // [K][nch-1][T][T]
    size_t gramx_elems = 0;
    size_t psmem = 0;
    // persistent mini-batch plan (one hidden layer, fp32, batches of 2..32 rows): nrb tile
    // workgroups of 16 mrt neurons per CN; flags[K] = abort
    bool mbp = false;
    int mrt = 1;
    unsigned long long* zpart = nullptr;  // [2][K][nrb][32][16] tagged output-sum shares
    size_t zpart_elems = 0;
    unsigned mbp_tag = 1;                 // tag of the next launch's first batch step
    // fp32 products of the large GEMMs on the bf16 matrix cores (three-part split); false:
    // fp32 matrix instructions throughout (PNN_GEMM=fp32, read by pnn_init)
    bool gemm_x3 = true;
    // mini-batch plan with the last layer fused into the split-bf16 products of one hidden
    // layer: output-sum partials [K][ceil(H / 256)][B][16], output errors [K][B][16]
    bool fx3 = false;
    // (fx3) a merge with broadcast left the copy of the merged network into the CNs to the next
    // epoch's first step, which reads the merged slot; anything else that reads a CN's
    // parameters first makes the copy (settle)
    bool bcast_pending = false;
    float* fx3_zpart = nullptr;
    float* fx3_dout = nullptr;
    // bounded waits of the persistent kernels: polls before giving up; and a test hook that
    // makes their waits run into that bound (the mini-batch kernel's readers wait for share
    // tags that are never written, the per-sample kernel's for more tiles than exist)
    long spin_limit = 0;
    unsigned tag_skew = 0;
    int wait_skew = 0;
    int tile_delay = 0;  // PNN_TEST_TILE_DELAY: late tile workgroups in the per-sample kernel
    // the abort flag of the last persistent launch has not been read yet; abort_ev follows
    // that launch on its stream
    bool abort_pending = false;
    hipEvent_t abort_ev = nullptr;

    // profiling
    bool prof = false;
    std::vector<ProfRec> pending;
    std::vector<hipEvent_t> free_events;
    std::map<std::string, std::pair<double, int64_t>> prof_acc;
    std::vector<std::string> prof_names_store;
};

namespace {

pnn_status fail(pnn_net* n, pnn_status s, const char* fmt, ...) {
    char buf[512];
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(buf, sizeof buf, fmt, ap);
    va_end(ap);
    if (n) n->err = buf;
    else g_init_error = buf;
    return s;
}

#define HIP_TRY(net, call)                                                                         \
    do {                                                                                           \
        hipError_t e_ = (call);                                                                    \
        if (e_ != hipSuccess) {                                                                    \
            if (net) (net)->broken = true;                                                         \
            return fail(net, PNN_EHIP, "%s failed: %s", #call, hipGetErrorString(e_));            \
        }                                                                                          \
    } while (0)

int64_t round_up(int64_t v, int64_t m) { return (v + m - 1) / m * m; }

// rows per group of the fused last layer behind a hidden layer of H neurons at batch B: a
// multiple of 16 covering the batch if it can, at most TAIL_GROUP / H and 256; 0 if the
// layer does not fit (H not a multiple of 16, or above TAIL_GROUP / 16)
int tail_rows(int H, int B) {
    if (H <= 0 || H % 16 != 0) return 0;
    const int cap = (int)std::min<int64_t>(TAIL_GROUP / H / 16 * 16, 256);
    if (cap < 16) return 0;
    return (int)std::min<int64_t>(round_up(B, 16), cap);
}

pnn_status check_config(const pnn_config* c, std::string* why) {
    auto bad = [&](const char* m) { if (why) *why = m; return PNN_EINVAL; };
    if (!c) return bad("config is NULL");
    if (c->n_layers < 1 || c->n_layers > 8) return bad("n_layers must be in 1..8");
    for (int l = 0; l <= c->n_layers; ++l)
        if (c->sizes[l] < 1) return bad("every layer size must be >= 1");
    for (int l = 0; l < c->n_layers; ++l)
        if (c->sizes[l] % 8 != 0) return bad("input and hidden layer sizes must be multiples of 8");
    if (c->sizes[c->n_layers] > MAX_OUT) return bad("the output layer may have at most 16 neurons");
    for (int l = 0; l < c->n_layers; ++l) {
        if (c->act[l] < 0 || c->act[l] > 4) return bad("unknown activation");
        if (c->act[l] == PNN_SOFTMAX && l != c->n_layers - 1) return bad("softmax is allowed on the output layer only");
    }
    const int out_act = c->act[c->n_layers - 1];
    if (c->loss != PNN_LOSS_MSE && c->loss != PNN_LOSS_XENT) return bad("unknown loss");
    if (out_act == PNN_SOFTMAX && c->loss != PNN_LOSS_XENT) return bad("a softmax output needs the cross-entropy loss");
    if (c->loss == PNN_LOSS_XENT && out_act != PNN_SOFTMAX && out_act != PNN_SIGMOID)
        return bad("the cross-entropy loss needs a sigmoid or softmax output");
    if (c->precision != PNN_FP32 && c->precision != PNN_BF16_MIXED) return bad("unknown precision");
    if (c->replicas < 1) return bad("replicas must be >= 1");
    if (c->batch < 1) return bad("batch must be >= 1");
    if (!std::isfinite(c->lr) || c->lr < 0.0f) return bad("lr must be finite and >= 0");
    return PNN_OK;
}

int64_t packed_count(const pnn_config* c) {
    int64_t p = 0;
    for (int l = 0; l < c->n_layers; ++l) p += (int64_t)c->sizes[l + 1] * c->sizes[l] + c->sizes[l + 1];
    return p;
}

template <typename T>
pnn_status dev_alloc(pnn_net* n, T** p, size_t elems) {
    if (elems == 0) elems = 1;
    hipError_t e = hipMalloc((void**)p, elems * sizeof(T));
    if (e != hipSuccess) {
        *p = nullptr;
        return fail(n, PNN_ENOMEM, "hipMalloc of %zu bytes failed: %s", elems * sizeof(T), hipGetErrorString(e));
    }
    e = hipMemset(*p, 0, elems * sizeof(T));
    if (e != hipSuccess) return fail(n, PNN_EHIP, "hipMemset failed: %s", hipGetErrorString(e));
    return PNN_OK;
}

// ---------------------------------------------------------------------------------------
// profiling hooks

void prof_begin(pnn_net* n, hipStream_t s, hipEvent_t* ev) {
    if (!n->prof) return;
    if (n->free_events.empty()) {
        hipEvent_t e;
        if (hipEventCreate(&e) != hipSuccess) { *ev = nullptr; return; }
        n->free_events.push_back(e);
    }
    *ev = n->free_events.back();
    n->free_events.pop_back();
    (void)hipEventRecord(*ev, s);
}
void prof_end(pnn_net* n, hipStream_t s, hipEvent_t a, const char* name) {
    if (!n->prof || !a) return;
    if (n->free_events.empty()) {
        hipEvent_t e;
        if (hipEventCreate(&e) != hipSuccess) return;
        n->free_events.push_back(e);
    }
    hipEvent_t b = n->free_events.back();
    n->free_events.pop_back();
    (void)hipEventRecord(b, s);
    n->pending.push_back({name, a, b});
}
void prof_drain(pnn_net* n) {
    for (auto& r : n->pending) {
        (void)hipEventSynchronize(r.b);
        float ms = 0.f;
        (void)hipEventElapsedTime(&ms, r.a, r.b);
        auto& acc = n->prof_acc[r.name];
        acc.first += ms;
        acc.second += 1;
        n->free_events.push_back(r.a);
        n->free_events.push_back(r.b);
    }
    n->pending.clear();
}

// ---------------------------------------------------------------------------------------
// launch helpers

struct Launch {
    pnn_net* n;
    hipStream_t s;
    hipEvent_t ev = nullptr;
    const char* name;
    Launch(pnn_net* n_, hipStream_t s_, const char* nm) : n(n_), s(s_), name(nm) { prof_begin(n, s, &ev); }
    pnn_status done() {
        hipError_t e = hipGetLastError();
        prof_end(n, s, ev, name);
        if (e != hipSuccess) {
            n->broken = true;
            return fail(n, PNN_EHIP, "launch of %s failed: %s", name, hipGetErrorString(e));
        }
        return PNN_OK;
    }
};

GemmArgs gemm_base(const pnn_net* n, int M, int N, int Kd, int64_t n_total, int64_t r0, int step_rows, int sample_dims) {
    GemmArgs g;
    memset(&g, 0, sizeof g);
    g.M = M; g.N = N; g.Kd = Kd;
    g.n_total = n_total;
    g.k_rep = n->cfg.replicas;
    g.zdiv = 1;
    g.r0_base = r0;
    g.r0_step = 0;
    g.step_rows = step_rows;
    g.sample_dims = sample_dims;
    g.ksplit = 1;
    g.kchunk = 1 << 30;
    return g;
}

// profiling name of a launch on the split-bf16 path ("<name>_x3")
const char* x3_name(const char* name) {
    static const char* const names[][2] = {{"fwd_gemm", "fwd_gemm_x3"}, {"upd_gemm", "upd_gemm_x3"},
                                           {"bwd_gemm", "bwd_gemm_x3"}, {"infer_fwd_gemm", "infer_fwd_gemm_x3"},
                                           {"psgd_upd", "psgd_upd_x3"},  {"psgd_p", "psgd_p_x3"},
                                           {"psgd_gram", "psgd_gram_x3"}};
    for (const auto& e : names)
        if (strcmp(e[0], name) == 0) return e[1];
    return name;
}

template <bool BF, typename TA, typename TB, bool A_KC, bool B_KC, int EPI, typename TO>
pnn_status run_gemm(pnn_net* n, hipStream_t s, const GemmArgs& g, int Z, const char* name) {
    // shapes the kernel assumes: 16-byte loads along contiguous dimensions
    const int vec = BF ? 8 : 4;
    if ((A_KC || B_KC) && (g.sample_dims & 4) == 0 && g.Kd % vec != 0)
        return fail(n, PNN_EINVAL, "%s: contraction length %d is not a multiple of %d", name, g.Kd, vec);
    if (g.kchunk % GemmTile<BF>::BK != 0 && g.ksplit > 1)
        return fail(n, PNN_EINVAL, "%s: split chunk %d is not a multiple of the tile depth", name, g.kchunk);
    if ((!A_KC && g.M % 4 != 0) || (!B_KC && g.N % 4 != 0))
        return fail(n, PNN_EINVAL, "%s: M=%d / N=%d not a multiple of 4", name, g.M, g.N);
    // 4-wide loads run along columns of NC operands and along k of KC operands: none of
    // those may be a dimension cut to the rows of a step
    if ((!A_KC && (g.sample_dims & 1)) || (!B_KC && (g.sample_dims & 2)) || ((A_KC || B_KC) && (g.sample_dims & 4)))
        return fail(n, PNN_EINVAL, "%s: vector loads along a sample dimension", name);
    dim3 grid((g.N + 63) / 64, (g.M + 63) / 64, (unsigned)(Z * g.ksplit));
    if (grid.x == 0 || grid.y == 0 || grid.z == 0 || grid.y > 65535 || grid.z > 65535)
        return fail(n, PNN_EINVAL, "%s: bad grid %u x %u x %u", name, grid.x, grid.y, grid.z);
    if constexpr (!BF) {
        const dim3 g128((g.N + 127) / 128, (g.M + 127) / 128, (unsigned)(Z * g.ksplit));
        // the weight update over at most 128 samples of a layer of >= 128 neurons: strips of 128
        // rows of W on the bf16 matrix cores (upd128x3_kernel)
        if constexpr (EPI == EPI_UPD && !A_KC && !B_KC) {
            const int kmax = (g.sample_dims & 4) ? g.step_rows : g.Kd;
            if (n->gemm_x3 && g.M >= 128 && g.N >= 128 && kmax <= U3_KMAX && g.ksplit == 1 && g.shadow == nullptr &&
                g.N % 4 == 0 && g.c_ld % 4 == 0) {
                static const hipError_t attr =
                    hipFuncSetAttribute((const void*)upd128x3_kernel<false>, hipFuncAttributeMaxDynamicSharedMemorySize,
                                        (int)u3_lds_bytes());
                static const hipError_t attr_full =
                    hipFuncSetAttribute((const void*)upd128x3_kernel<true>, hipFuncAttributeMaxDynamicSharedMemorySize,
                                        (int)u3_lds_bytes());
                if (attr != hipSuccess || attr_full != hipSuccess)
                    return fail(n, PNN_EHIP, "%s: hipFuncSetAttribute: %s", name,
                                hipGetErrorString(attr != hipSuccess ? attr : attr_full));
                const dim3 grid_u(1, (g.M + 127) / 128, (unsigned)Z);
                Launch l(n, s, x3_name(name));
                // more than 96 samples: four k-chunks per tile, the compile-time schedule
                if (kmax > 96) upd128x3_kernel<true><<<grid_u, B3_THREADS, u3_lds_bytes(), s>>>(g);
                else upd128x3_kernel<false><<<grid_u, B3_THREADS, u3_lds_bytes(), s>>>(g);
                return l.done();
            }
        }
        // large fp32 shapes with both operands along k and at least 256 columns: 128 x 256 tiles
        // (gemm256x3_kernel)
        if constexpr (A_KC && B_KC && (EPI == EPI_FWD || EPI == EPI_STORE)) {
            if (n->gemm_x3 && g.M >= 128 && g.N >= 256 && g.shadow == nullptr && g.ksplit == 1 && !(g.sample_dims & 4)) {
                static const hipError_t attr = hipFuncSetAttribute((const void*)gemm256x3_kernel<EPI>,
                                                                   hipFuncAttributeMaxDynamicSharedMemorySize,
                                                                   (int)g2_lds_bytes());
                if (attr != hipSuccess) return fail(n, PNN_EHIP, "%s: hipFuncSetAttribute: %s", name, hipGetErrorString(attr));
                Launch l(n, s, x3_name(name));
                gemm256x3_kernel<EPI><<<dim3((g.N + 255) / 256, (g.M + 127) / 128, (unsigned)Z), B3_THREADS, g2_lds_bytes(), s>>>(g);
                return l.done();
            }
        }
        if (g.zpart != nullptr || g.dout != nullptr)
            return fail(n, PNN_EINVAL, "%s: the fused last layer needs the split-bf16 kernels for this shape", name);
        // other large fp32 shapes: 128 x 128 tiles on the bf16 matrix cores, each fp32 operand
        // split into three bf16 parts (gemm128x3_kernel)
        if (n->gemm_x3 && g.M >= 128 && g.N >= 128 && g.shadow == nullptr && (g.ksplit == 1 || g.kchunk % B3_BK == 0)) {
            static const hipError_t attr = hipFuncSetAttribute((const void*)gemm128x3_kernel<A_KC, B_KC, EPI>,
                                                               hipFuncAttributeMaxDynamicSharedMemorySize,
                                                               (int)b3_lds_bytes());
            if (attr != hipSuccess) return fail(n, PNN_EHIP, "%s: hipFuncSetAttribute: %s", name, hipGetErrorString(attr));
            Launch l(n, s, x3_name(name));
            gemm128x3_kernel<A_KC, B_KC, EPI><<<g128, B3_THREADS, b3_lds_bytes(), s>>>(g);
            return l.done();
        }
        // otherwise, with both operands along k (forward, inference): 128 x 128 tiles on the
        // fp32 matrix instructions.  (The weight update, short contraction and a
        // read-modify-write epilogue, keeps the 64 x 64 tiles: more workgroups in flight to
        // cover its epilogue.)
        if (A_KC && B_KC && g.M >= 128 && g.N >= 128 && g.shadow == nullptr) {
            Launch l(n, s, name);
            gemm128_kernel<A_KC, B_KC, EPI><<<g128, 256, 0, s>>>(g);
            return l.done();
        }
    }
    // the bf16 forward product of a training step's batch (at most 64 rows): the waves of a
    // tile split the contraction (gemm_kw_kernel)
    if constexpr (BF && A_KC && B_KC && EPI == EPI_FWD && sizeof(TB) == 2) {
        if (g.M <= 64 && g.ksplit == 1 && g.Kd % 8 == 0 && !(g.sample_dims & 4)) {
            Launch l(n, s, name);
            gemm_kw_kernel<TA, TO><<<grid, 256, 0, s>>>(g);
            return l.done();
        }
    }
    Launch l(n, s, name);
    if (EPI == EPI_UPD && g.Kd <= 64) gemm_kernel<BF, TA, TB, A_KC, B_KC, EPI, TO, EPI == EPI_UPD><<<grid, 256, 0, s>>>(g);
    else gemm_kernel<BF, TA, TB, A_KC, B_KC, EPI, TO><<<grid, 256, 0, s>>>(g);
    return l.done();
}

Operand opnd(const void* p, int64_t zs, int64_t ld, int xrows, int64_t xshift = 0) {
    Operand o;
    o.ptr = p; o.zstride = zs; o.ld = ld; o.xrows = xrows; o.xshift = xshift;
    return o;
}

#define TRY(x) do { pnn_status st_ = (x); if (st_ != PNN_OK) return st_; } while (0)

// ---------------------------------------------------------------------------------------
// mini-batch plan: one batch step of every CN

template <bool BF>
pnn_status minibatch_step(pnn_net* n, const float* X, const int32_t* Y, int64_t N, int64_t r0, hipStream_t s,
                          bool from_merged) {
    typedef typename std::conditional<BF, bf16_t, float>::type TH;  // hidden activations / errors
    const int L = n->L, B = n->cfg.batch, K = n->cfg.replicas;
    const bool fx3 = !BF && n->fx3;  // last layer fused into the split-bf16 products
    // (fx3) every CN starts this step from the merged network, read from its one slot
    from_merged = from_merged && fx3;
    const int64_t ps = n->pstride;
    const void* Wop = BF ? (const void*)n->shadow : (const void*)n->theta;  // operand weights
    const int64_t wz = ps;

    // forward, hidden layers (eq. (2)-(3))
    for (int l = 1; l <= L - 1; ++l) {
        GemmArgs g = gemm_base(n, B, n->sizes[l], n->sizes[l - 1], N, r0, B, 1);
        if (l == 1) g.a = opnd(X, 0, n->sizes[0], 1);
        else g.a = opnd(n->act_ws[l - 1], (int64_t)B * n->sizes[l - 1], n->sizes[l - 1], 0);
        g.b = opnd((const char*)Wop + n->off_w[l - 1] * (BF ? 2 : 4), wz, n->sizes[l - 1], 0);
        g.c = n->act_ws[l]; g.c_z = (int64_t)B * n->sizes[l]; g.c_ld = n->sizes[l];
        g.bias = n->theta + n->off_b[l - 1]; g.bias_z = ps;
        g.act = n->act[l - 1];
        if (!BF && l == 1 && n->ksplit > 1) {
            // few tiles with a long contraction: split it, then sum, bias and activation
            g.c = n->ppart; g.ksplit = n->ksplit; g.kchunk = n->kchunk;
            g.c_split = (int64_t)K * B * n->sizes[1];
            TRY((run_gemm<false, float, float, true, true, EPI_STORE, float>(n, s, g, K, "fwd_gemm")));
            FwdReduceArgs ra;
            memset(&ra, 0, sizeof ra);
            ra.part = n->ppart; ra.split = g.c_split; ra.ksplit = n->ksplit;
            ra.out = (float*)n->act_ws[1];
            ra.bias = n->theta + n->off_b[0]; ra.bias_z = ps;
            ra.N = n->sizes[1]; ra.act = n->act[0];
            ra.n_total = N; ra.k_rep = K; ra.r0 = r0; ra.step_rows = B;
            Launch lr(n, s, "fwd_reduce");
            fwd_reduce_kernel<<<dim3((n->sizes[1] + 255) / 256, B, K), 256, 0, s>>>(ra);
            TRY(lr.done());
            continue;
        }
        if (fx3) {
            g.w2 = n->theta + n->off_w[1]; g.w2_z = ps;
            g.zpart = n->fx3_zpart; g.o2 = n->sizes[2];
            if (from_merged) {
                g.b = opnd(n->merged + n->off_w[0], 0, n->sizes[0], 0);
                g.bias = n->merged + n->off_b[0]; g.bias_z = 0;
                g.w2 = n->merged + n->off_w[1]; g.w2_z = 0;
            }
        }
        if (l == 1) TRY((run_gemm<BF, float, TH, true, true, EPI_FWD, TH>(n, s, g, K, "fwd_gemm")));
        else TRY((run_gemm<BF, TH, TH, true, true, EPI_FWD, TH>(n, s, g, K, "fwd_gemm")));
    }
    if (fx3) {
        // the last layer's outputs and errors from the forward tiles' partial sums
        OutErrArgs a;
        memset(&a, 0, sizeof a);
        a.zpart = n->fx3_zpart; a.ntile = (n->sizes[1] + 255) / 256;
        a.bias = n->theta + n->off_b[1]; a.bias_z = ps;
        if (from_merged) { a.bias = n->merged + n->off_b[1]; a.bias_z = 0; }
        a.O = n->sizes[2]; a.act_out = n->act[1]; a.loss = n->cfg.loss;
        a.n_total = N; a.k_rep = K; a.r0 = r0; a.step_rows = B;
        a.y = Y;
        a.dout = n->fx3_dout;
        Launch lc(n, s, "out_err");
        out_err_kernel<<<dim3((B + 15) / 16, 1, K), 256, 0, s>>>(a);
        TRY(lc.done());
    }
    // a narrow last layer behind a hidden layer: forward, output error, the hidden error
    // behind it and its update in one kernel per CN
    const int Hl = L >= 2 ? n->sizes[L - 1] : 0;
    const int trg = tail_rows(Hl, B);
    const size_t tail_smem = trg > 0 ? (size_t)tail_lds_floats(Hl, trg) * sizeof(float) : 0;
    const bool fuse_tail = !fx3 && L >= 2 && n->sizes[L] <= MAX_OUT && trg > 0 && tail_smem <= 160 * 1024;
    if (fuse_tail) {
        TailArgs a;
        memset(&a, 0, sizeof a);
        a.x = n->act_ws[L - 1]; a.x_z = (int64_t)B * Hl;
        a.wop = (const char*)Wop + n->off_w[L - 1] * (BF ? 2 : 4);
        a.w = n->theta + n->off_w[L - 1];
        a.shadow = BF ? n->shadow + n->off_w[L - 1] : nullptr;
        a.bias = n->theta + n->off_b[L - 1];
        a.w_z = ps; a.bias_z = ps;
        a.d = n->del_ws[L - 1];
        a.H = Hl; a.O = n->sizes[L]; a.act_out = n->act[L - 1]; a.act_hid = n->act[L - 2]; a.loss = n->cfg.loss;
        a.rg = trg;
        a.lr = n->cfg.lr;
        a.n_total = N; a.k_rep = K; a.r0 = r0; a.step_rows = B;
        a.y = Y;
        Launch lc(n, s, "tail");
        if (Hl <= 256) tail_kernel<TH, 1><<<dim3(K), TAIL_THREADS, tail_smem, s>>>(a);
        else if (Hl <= 512) tail_kernel<TH, 2><<<dim3(K), TAIL_THREADS, tail_smem, s>>>(a);
        else tail_kernel<TH, 4><<<dim3(K), TAIL_THREADS, tail_smem, s>>>(a);
        TRY(lc.done());
    }
    // output layer and output error (eq. (3), (5), (9)-(10))
    if (!fuse_tail && !fx3) {
        RowArgs a;
        memset(&a, 0, sizeof a);
        if (L == 1) { a.x = X; a.x_xrows = 1; a.x_ld = n->sizes[0]; }
        else { a.x = n->act_ws[L - 1]; a.x_z = (int64_t)B * n->sizes[L - 1]; a.x_ld = n->sizes[L - 1]; }
        a.w = (const char*)Wop + n->off_w[L - 1] * (BF ? 2 : 4); a.w_z = wz;
        a.bias = n->theta + n->off_b[L - 1]; a.bias_z = ps;
        a.H = n->sizes[L - 1]; a.O = n->sizes[L]; a.act = n->act[L - 1]; a.loss = n->cfg.loss;
        a.n_total = N; a.k_rep = K; a.r0 = r0; a.step_rows = B;
        a.y = Y;
        a.delta = n->del_ws[L]; a.d_z = (int64_t)B * n->sizes[L];
        dim3 grid((B + 3) / 4, 1, K);
        Launch lc(n, s, "out_layer");
        if (L == 1) out_layer_kernel<float, TH, TH, true><<<grid, 256, 0, s>>>(a);
        else out_layer_kernel<TH, TH, TH, true><<<grid, 256, 0, s>>>(a);
        TRY(lc.done());
    }
    // hidden errors, back to front, with the pre-update weights (eq. (11))
    for (int l = L - 1; l >= 1; --l) {
        if ((fuse_tail || fx3) && l == L - 1) continue;  // (in the fused last layer)
        const int Hl = n->sizes[l], On = n->sizes[l + 1];
        if (On <= MAX_OUT) {
            BwdSmallArgs a;
            memset(&a, 0, sizeof a);
            a.dnext = n->del_ws[l + 1]; a.dn_z = (int64_t)B * On;
            a.w = (const char*)Wop + n->off_w[l] * (BF ? 2 : 4); a.w_z = wz;
            a.x = n->act_ws[l]; a.d = n->del_ws[l]; a.xz = (int64_t)B * Hl;
            a.H = Hl; a.O = On; a.act = n->act[l - 1];
            a.n_total = N; a.k_rep = K; a.r0 = r0; a.step_rows = B;
            dim3 grid((Hl + 255) / 256, B, K);
            Launch lc(n, s, "bwd_small");
            bwd_small_kernel<TH, TH><<<grid, 256, 0, s>>>(a);
            TRY(lc.done());
        } else {
            GemmArgs g = gemm_base(n, B, Hl, On, N, r0, B, 1);
            g.a = opnd(n->del_ws[l + 1], (int64_t)B * On, On, 0);
            g.b = opnd((const char*)Wop + n->off_w[l] * (BF ? 2 : 4), wz, Hl, 0);
            g.c = n->del_ws[l]; g.c_z = (int64_t)B * Hl; g.c_ld = Hl;
            g.aux = n->act_ws[l];
            g.act = n->act[l - 1];
            TRY((run_gemm<BF, TH, TH, true, false, EPI_BWD, TH>(n, s, g, K, "bwd_gemm")));
        }
    }
    // updates, eq. (12)-(13) averaged over the batch
    // (bf16, two wide layers before a fused last layer: both weight updates in one launch)
    const bool upd2 = BF && L == 3 && fuse_tail && n->sizes[1] > MAX_OUT && n->sizes[2] > MAX_OUT && B <= 64 &&
                      K % 8 == 0 && n->sizes[0] % 4 == 0 && n->sizes[1] % 4 == 0 && n->sizes[2] % 4 == 0;
    if constexpr (BF) if (upd2) {
        GemmArgs gg[2];
        int gd[2][3];
        for (int l = 1; l <= 2; ++l) {
            const int In = n->sizes[l - 1], Out = n->sizes[l];
            GemmArgs g = gemm_base(n, Out, In, B, N, r0, B, 4);
            g.a = opnd(n->del_ws[l], (int64_t)B * Out, Out, 0);
            if (l == 1) g.b = opnd(X, 0, In, 1);
            else g.b = opnd(n->act_ws[l - 1], (int64_t)B * In, In, 0);
            g.c = n->theta + n->off_w[l - 1]; g.c_z = ps; g.c_ld = In;
            g.ubias = n->theta + n->off_b[l - 1]; g.bias_z = ps;
            g.lr = n->cfg.lr; g.scale_per_batch = 1;
            g.shadow = n->shadow + n->off_w[l - 1];
            gg[l - 1] = g;
            gd[l - 1][0] = (In + 63) / 64; gd[l - 1][1] = (Out + 63) / 64; gd[l - 1][2] = K;
        }
        const int64_t nwg = (int64_t)gd[0][0] * gd[0][1] * K + (int64_t)gd[1][0] * gd[1][1] * K;
        if (nwg > INT32_MAX) return fail(n, PNN_EINVAL, "upd_gemm: %lld workgroups", (long long)nwg);
        Launch lu(n, s, "upd_gemm");
        gemm_upd2_kernel<float, TH><<<(unsigned)nwg, 256, 0, s>>>(gg[0], gg[1], gd[0][0], gd[0][1], gd[0][2],
                                                                  gd[1][0], gd[1][1], gd[1][2]);
        TRY(lu.done());
    }
    for (int l = 1; l <= L; ++l) {
        if ((fuse_tail || fx3) && l == L) continue;  // (in the fused last layer)
        if (upd2 && l <= 2) continue;                // (above)
        const int In = n->sizes[l - 1], Out = n->sizes[l];
        if (Out <= MAX_OUT) {
            UpdSmallArgs a;
            memset(&a, 0, sizeof a);
            a.d = n->del_ws[l]; a.d_z = (int64_t)B * Out;
            if (l == 1) { a.x = X; a.x_xrows = 1; a.x_ld = In; }
            else { a.x = n->act_ws[l - 1]; a.x_z = (int64_t)B * In; a.x_ld = In; }
            a.w = n->theta + n->off_w[l - 1]; a.w_z = ps;
            a.shadow = BF ? n->shadow + n->off_w[l - 1] : nullptr;
            a.bias = n->theta + n->off_b[l - 1]; a.bias_z = ps;
            a.H = In; a.O = Out; a.lr = n->cfg.lr;
            a.n_total = N; a.k_rep = K; a.r0 = r0; a.step_rows = B;
            dim3 grid((In + 255) / 256, 1, K);
            Launch lc(n, s, "upd_small");
            if (l == 1) upd_small_kernel<TH, float><<<grid, 256, 0, s>>>(a);
            else upd_small_kernel<TH, TH><<<grid, 256, 0, s>>>(a);
            TRY(lc.done());
        } else {
            GemmArgs g = gemm_base(n, Out, In, B, N, r0, B, 4);
            g.a = opnd(n->del_ws[l], (int64_t)B * Out, Out, 0);
            if (l == 1) g.b = opnd(X, 0, In, 1);
            else g.b = opnd(n->act_ws[l - 1], (int64_t)B * In, In, 0);
            g.c = n->theta + n->off_w[l - 1]; g.c_z = ps; g.c_ld = In;
            g.ubias = n->theta + n->off_b[l - 1]; g.bias_z = ps;
            g.lr = n->cfg.lr; g.scale_per_batch = 1;
            g.shadow = BF ? n->shadow + n->off_w[l - 1] : nullptr;
            if (fx3) {
                // A: the hidden activations; the errors are formed from the output errors
                g.a = opnd(n->act_ws[1], (int64_t)B * Out, Out, 0);
                g.dout = n->fx3_dout;
                g.w2 = n->theta + n->off_w[1]; g.b2 = n->theta + n->off_b[1]; g.w2_z = ps;
                g.o2 = n->sizes[2]; g.act2 = n->act[0];
                if (from_merged) {
                    g.rd_c = n->merged + n->off_w[0]; g.rd_w2 = n->merged + n->off_w[1];
                    g.rd_ub = n->merged + n->off_b[0]; g.rd_b2 = n->merged + n->off_b[1];
                }
            }
            if (l == 1) TRY((run_gemm<BF, TH, float, false, false, EPI_UPD, float>(n, s, g, K, "upd_gemm")));
            else TRY((run_gemm<BF, TH, TH, false, false, EPI_UPD, float>(n, s, g, K, "upd_gemm")));
        }
    }
    return PNN_OK;
}

// ---------------------------------------------------------------------------------------
// chunked per-sample plan

constexpr int PT = 64;            // chunk length of the persistent per-sample plan
constexpr long SPIN_LIMIT = 1L << 22;

// kernel instance: hidden neurons per lane of the live wave (1: <= 64, 2: <= 128) x
// activation specialisation x 16-row sub-tiles per tile workgroup (1, or 2 when more CNs must
// fit the chip)
template <int RT>
const void* persistent_fn_rt(const pnn_net* n) {
    const bool narrow = n->sizes[1] <= 64;
    if (n->pspecial)
        return narrow ? (const void*)psgd_persistent_kernel<PT, 1, ACT_SIGMOID, ACT_SIGMOID, LOSS_MSE, 10, RT>
                      : (const void*)psgd_persistent_kernel<PT, 2, ACT_SIGMOID, ACT_SIGMOID, LOSS_MSE, 10, RT>;
    return narrow ? (const void*)psgd_persistent_kernel<PT, 1, -1, -1, -1, 16, RT>
                  : (const void*)psgd_persistent_kernel<PT, 2, -1, -1, -1, 16, RT>;
}
const void* persistent_fn(const pnn_net* n) { return n->prt == 2 ? persistent_fn_rt<2>(n) : persistent_fn_rt<1>(n); }

// width of the live wave's neuron set (input-sum rows are padded to it)
int live_width(int H) { return H <= 64 ? 64 : 128; }

// after a persistent launch: its abort flag is read by the next call that consumes the CNs
pnn_status note_persistent_launch(pnn_net* n, hipStream_t s) {
    if (!n->abort_ev) HIP_TRY(n, hipEventCreateWithFlags(&n->abort_ev, hipEventDisableTiming));
    HIP_TRY(n, hipEventRecord(n->abort_ev, s));
    n->abort_pending = true;
    return PNN_OK;
}

pnn_status psgd_persistent_epoch(pnn_net* n, const float* X, const int32_t* Y, int64_t N, hipStream_t s) {
    const int K = n->cfg.replicas, H = n->sizes[1], In = n->sizes[0];
    const int64_t nmax = shard_len(N, K, 0);
    const int nch = (int)((nmax + PT - 1) / PT);
    auto grow = [&](float** buf, size_t* have, size_t need) -> pnn_status {
        if (need <= *have) return PNN_OK;
        if (*buf) (void)hipFree(*buf);
        *buf = nullptr;
        *have = 0;
        TRY(dev_alloc(n, buf, need));
        *have = need;
        return PNN_OK;
    };
    constexpr int GS = PT + 4;  // padded Gram row stride (matches the kernel's LDS layout)
    TRY(grow(&n->gram, &n->gram_elems, (size_t)K * nch * PT * GS));
    TRY(grow(&n->gramx, &n->gramx_elems, (size_t)K * std::max(nch - 1, 1) * PT * GS));
    {
        // G_c[t][s] = x_t . x_s within every chunk
        GemmArgs g = gemm_base(n, PT, PT, In, N, 0, PT, 3);
        g.a = opnd(X, 0, In, 1);
        g.b = opnd(X, 0, In, 1);
        g.zdiv = nch; g.r0_step = PT;
        g.c = n->gram; g.c_z = (int64_t)PT * GS; g.c_ld = GS;
        TRY((run_gemm<false, float, float, true, true, EPI_STORE, float>(n, s, g, K * nch, "psgd_gram")));
    }
    if (nch > 1) {
        // GX_c[t][s] = x_t . x_s, t in chunk c, s in chunk c-1 (always full), c >= 1
        GemmArgs g = gemm_base(n, PT, PT, In, N, PT, PT, 1);
        g.a = opnd(X, 0, In, 1);
        g.b = opnd(X, 0, In, 1, -PT);
        g.zdiv = nch - 1; g.r0_step = PT;
        g.c = n->gramx; g.c_z = (int64_t)PT * GS; g.c_ld = GS;
        TRY((run_gemm<false, float, float, true, true, EPI_STORE, float>(n, s, g, K * (nch - 1), "psgd_gram")));
    }
    {
        // (the abort slot flags[3K] is sticky: a launch after an abort ends at once)
        Launch l(n, s, "zero_flags");
        zero_ints_kernel<<<(3 * K + 255) / 256, 256, 0, s>>>(n->flags, 3 * K);
        TRY(l.done());
    }
    PsgdPArgs a;
    memset(&a, 0, sizeof a);
    a.theta = n->theta; a.pstride = n->pstride;
    a.off_w1 = n->off_w[0]; a.off_b1 = n->off_b[0]; a.off_w2 = n->off_w[1]; a.off_b2 = n->off_b[1];
    a.X = X; a.y = Y; a.n_total = N; a.k_rep = K;
    a.gram = n->gram; a.gramx = n->gramx; a.nch = nch;
    a.qbuf = n->qbuf; a.qstride = PT + 4; a.qslot = (int64_t)live_width(H) * (PT + 4);
    a.d1 = n->d1; a.flags = n->flags;
    a.H = H; a.O = n->sizes[2]; a.In = In; a.act1 = n->act[0]; a.act2 = n->act[1]; a.loss = n->cfg.loss;
    a.nrb = n->nrb;
    a.wait_skew = n->wait_skew;
    a.tile_delay = n->tile_delay;
    a.lr = n->cfg.lr;
    a.spin_limit = n->spin_limit;
    void* params[] = {&a};
    const void* fn = persistent_fn(n);
    // the CNs in groups of at most kgroup (balanced), one launch each
    const int G = (K + n->kgroup - 1) / n->kgroup;
    for (int gi = 0, c0 = 0; gi < G; ++gi) {
        const int kl = (K - c0) / (G - gi);
        a.cn0 = c0;
        a.k_launch = kl;
        const dim3 grid((unsigned)(kl * (1 + n->nrb)));
        Launch l(n, s, "psgd_persistent");
        hipError_t e = hipLaunchCooperativeKernel(fn, grid, dim3(256), params, (unsigned)n->psmem, s);
        if (e != hipSuccess) {
            (void)hipGetLastError();
            n->broken = true;
            return fail(n, PNN_EHIP, "cooperative launch of the per-sample kernel failed: %s", hipGetErrorString(e));
        }
        TRY(l.done());
        c0 += kl;
    }
    return note_persistent_launch(n, s);
}

// ---------------------------------------------------------------------------------------
// persistent mini-batch plan

const void* mbp_fn(int rt) { return rt == 2 ? (const void*)mbp_kernel<2> : (const void*)mbp_kernel<1>; }

pnn_status mbp_epoch(pnn_net* n, const float* X, const int32_t* Y, int64_t N, hipStream_t s) {
    const int K = n->cfg.replicas;
    const int64_t nsteps = (shard_len(N, K, 0) + n->cfg.batch - 1) / n->cfg.batch;
    if ((uint64_t)n->mbp_tag + (uint64_t)nsteps >= 0xFFFFFFFFull) {
        // the step tags would wrap: clear the shares (so that no stale tag can match) and restart
        const int ni = (int)(2 * n->zpart_elems);
        Launch l(n, s, "zero_flags");
        zero_ints_kernel<<<(ni + 255) / 256, 256, 0, s>>>((int*)n->zpart, ni);
        TRY(l.done());
        n->mbp_tag = 1;
    }
    {
        // (the abort slot flags[K] is sticky: a launch after an abort ends at once)
        Launch l(n, s, "zero_flags");
        zero_ints_kernel<<<(K + 255) / 256, 256, 0, s>>>(n->flags, K);
        TRY(l.done());
    }
    MbpArgs a;
    memset(&a, 0, sizeof a);
    a.theta = n->theta; a.pstride = n->pstride;
    a.off_w1 = n->off_w[0]; a.off_b1 = n->off_b[0]; a.off_w2 = n->off_w[1]; a.off_b2 = n->off_b[1];
    a.X = X; a.y = Y; a.n_total = N;
    a.zpart = n->zpart; a.flags = n->flags;
    a.k_rep = K; a.H = n->sizes[1]; a.O = n->sizes[2]; a.In = n->sizes[0];
    a.act1 = n->act[0]; a.act2 = n->act[1]; a.loss = n->cfg.loss;
    a.nrb = n->nrb; a.B = n->cfg.batch;
    a.tag0 = n->mbp_tag;
    a.tag_skew = n->tag_skew;
    n->mbp_tag += (unsigned)nsteps;
    a.lr = n->cfg.lr;
    a.spin_limit = n->spin_limit;
    void* params[] = {&a};
    // the CNs in groups of at most kgroup (balanced), one launch each (every CN has its own
    // share slots, so the groups' launches share the step tags)
    const int G = (K + n->kgroup - 1) / n->kgroup;
    for (int gi = 0, c0 = 0; gi < G; ++gi) {
        const int kl = (K - c0) / (G - gi);
        const int grid = kl * n->nrb;
        a.cn0 = c0;
        a.xcd_map = grid % 8 == 0;
        Launch l(n, s, "mb_persistent");
        hipError_t e = hipLaunchCooperativeKernel(mbp_fn(n->mrt), dim3((unsigned)grid), dim3(256), params,
                                                  (unsigned)n->psmem, s);
        if (e != hipSuccess) {
            (void)hipGetLastError();
            n->broken = true;
            return fail(n, PNN_EHIP, "cooperative launch of the mini-batch kernel failed: %s", hipGetErrorString(e));
        }
        TRY(l.done());
        c0 += kl;
    }
    return note_persistent_launch(n, s);
}

pnn_status psgd_epoch(pnn_net* n, const float* X, const int32_t* Y, int64_t N, hipStream_t s) {
    if (n->persistent) return psgd_persistent_epoch(n, X, Y, N, s);
    const int K = n->cfg.replicas, T = n->T, H = n->sizes[1], In = n->sizes[0];
    const int64_t nmax = shard_len(N, K, 0);
    const int nch = (int)((nmax + T - 1) / T);
    const size_t need = (size_t)K * nch * T * T;
    if (need > n->gram_elems) {
        if (n->gram) (void)hipFree(n->gram);
        n->gram = nullptr;
        n->gram_elems = 0;
        TRY(dev_alloc(n, &n->gram, need));
        n->gram_elems = need;
    }
    // Gram matrices of every chunk: G[t][s] = x_t . x_s
    {
        GemmArgs g = gemm_base(n, T, T, In, N, 0, T, 3);
        g.a = opnd(X, 0, In, 1);
        g.b = opnd(X, 0, In, 1);
        g.zdiv = nch; g.r0_step = T;
        g.c = n->gram; g.c_z = (int64_t)T * T; g.c_ld = T;
        TRY((run_gemm<false, float, float, true, true, EPI_STORE, float>(n, s, g, K * nch, "psgd_gram")));
    }
    auto run_p = [&](int c) -> pnn_status {
        GemmArgs g = gemm_base(n, T, H, In, N, (int64_t)c * T, T, 1);
        g.a = opnd(X, 0, In, 1);
        g.b = opnd(n->theta + n->off_w[0], n->pstride, In, 0);
        g.c = n->ppart; g.c_z = (int64_t)T * H; g.c_ld = H;
        g.ksplit = n->ksplit; g.kchunk = n->kchunk; g.c_split = (int64_t)K * T * H;
        return run_gemm<false, float, float, true, true, EPI_STORE, float>(n, s, g, K, "psgd_p");
    };
    TRY(run_p(0));
    const int threads = (int)round_up(H, 64);
    const size_t smem = (size_t)(2 * T * H + 2 * 16 * MAX_OUT) * sizeof(float);
    for (int c = 0; c < nch; ++c) {
        PsgdArgs a;
        memset(&a, 0, sizeof a);
        a.theta = n->theta; a.pstride = n->pstride;
        a.off_b1 = n->off_b[0]; a.off_w2 = n->off_w[1]; a.off_b2 = n->off_b[1];
        a.ppart = n->ppart; a.ksplit = n->ksplit; a.ppart_split = (int64_t)K * T * H;
        a.gram = n->gram; a.nch = nch; a.c = c;
        a.y = Y; a.d1 = n->d1;
        a.n_total = N; a.k_rep = K;
        a.H = H; a.O = n->sizes[2]; a.act1 = n->act[0]; a.act2 = n->act[1]; a.loss = n->cfg.loss;
        a.lr = n->cfg.lr;
        {
            Launch lc(n, s, "psgd_chunk");
            switch (T) {
            case 128: psgd_chunk_kernel<128><<<K, threads, smem, s>>>(a); break;
            case 64: psgd_chunk_kernel<64><<<K, threads, smem, s>>>(a); break;
            case 32: psgd_chunk_kernel<32><<<K, threads, smem, s>>>(a); break;
            default: psgd_chunk_kernel<16><<<K, threads, smem, s>>>(a); break;
            }
            TRY(lc.done());
        }
        // W1 -= eta * sum_t d1_t x_t^T  (the chunk's T rank-1 updates)
        {
            GemmArgs g = gemm_base(n, H, In, T, N, (int64_t)c * T, T, 4);
            g.a = opnd(n->d1, (int64_t)T * H, H, 0);
            g.b = opnd(X, 0, In, 1);
            g.c = n->theta + n->off_w[0]; g.c_z = n->pstride; g.c_ld = In;
            g.lr = n->cfg.lr; g.scale_per_batch = 0;
            TRY((run_gemm<false, float, float, false, false, EPI_UPD, float>(n, s, g, K, "psgd_upd")));
        }
        if (c + 1 < nch) TRY(run_p(c + 1));
    }
    return PNN_OK;
}

pnn_status refresh_shadows(pnn_net* n, hipStream_t s) {
    if (!n->bf16) return PNN_OK;
    const int64_t tot = (int64_t)n->cfg.replicas * n->pstride;
    {
        Launch l(n, s, "to_bf16");
        to_bf16_kernel<<<(unsigned)((tot + 255) / 256), 256, 0, s>>>(n->theta, n->shadow, tot);
        TRY(l.done());
    }
    Launch l(n, s, "to_bf16");
    to_bf16_kernel<<<(unsigned)((n->pstride + 255) / 256), 256, 0, s>>>(n->merged, n->mshadow, n->pstride);
    return l.done();
}

void pack(const pnn_net* n, const float* padded, float* flat) {
    int64_t o = 0;
    for (int l = 0; l < n->L; ++l) {
        const int64_t nw = (int64_t)n->sizes[l + 1] * n->sizes[l];
        memcpy(flat + o, padded + n->off_w[l], nw * sizeof(float));
        o += nw;
        memcpy(flat + o, padded + n->off_b[l], n->sizes[l + 1] * sizeof(float));
        o += n->sizes[l + 1];
    }
}
void unpack(const pnn_net* n, const float* flat, float* padded) {
    memset(padded, 0, n->pstride * sizeof(float));
    int64_t o = 0;
    for (int l = 0; l < n->L; ++l) {
        const int64_t nw = (int64_t)n->sizes[l + 1] * n->sizes[l];
        memcpy(padded + n->off_w[l], flat + o, nw * sizeof(float));
        o += nw;
        memcpy(padded + n->off_b[l], flat + o, n->sizes[l + 1] * sizeof(float));
        o += n->sizes[l + 1];
    }
}

void free_all(pnn_net* n) {
    auto f = [](void* p) { if (p) (void)hipFree(p); };
    f(n->theta); f(n->merged); f(n->shadow); f(n->mshadow);
    for (int l = 0; l < 9; ++l) { f(n->act_ws[l]); f(n->del_ws[l]); f(n->inf_ws[l]); }
    f(n->d_correct); f(n->d_cost); f(n->d_cost_sum); f(n->d_mw); f(n->ord_x); f(n->ord_y); f(n->ppart); f(n->d1); f(n->gram); f(n->flags); f(n->qbuf); f(n->gramx); f(n->zpart); f(n->fx3_zpart); f(n->fx3_dout);
    if (n->abort_ev) (void)hipEventDestroy(n->abort_ev);
    for (auto& r : n->pending) { (void)hipEventDestroy(r.a); (void)hipEventDestroy(r.b); }
    for (auto e : n->free_events) (void)hipEventDestroy(e);
}

// the kernels read input rows with 16-byte vector loads
bool aligned16(const void* p) { return ((uintptr_t)p & 15) == 0; }

// A persistent launch that gave up waiting leaves its (sticky) abort flag set and the CNs'
// parameters unspecified.  Every call that consumes the CNs reads the flag of the last such
// launch first: `wait` waits for that launch to end; without it the flag is read only if the
// launch has already ended (a later launch of the same kernel ends at once on a set flag).
pnn_status check_abort(pnn_net* n, bool wait) {
    if (!n->abort_pending) return PNN_OK;
    if (!wait) {
        const hipError_t q = hipEventQuery(n->abort_ev);
        if (q == hipErrorNotReady) return PNN_OK;
        if (q != hipSuccess) {
            n->broken = true;
            return fail(n, PNN_EHIP, "hipEventQuery failed: %s", hipGetErrorString(q));
        }
    } else {
        HIP_TRY(n, hipEventSynchronize(n->abort_ev));
    }
    int ab = 0;
    const int at = n->persistent ? 3 * n->cfg.replicas : n->cfg.replicas;
    HIP_TRY(n, hipMemcpy(&ab, n->flags + at, sizeof(int), hipMemcpyDeviceToHost));
    n->abort_pending = false;
    if (ab) {
        n->broken = true;
        return fail(n, PNN_EHIP, "the %s training kernel timed out waiting for a peer workgroup",
                    n->persistent ? "per-sample" : "mini-batch");
    }
    return PNN_OK;
}

pnn_status usable(pnn_net* n) {
    if (!n) return PNN_EINVAL;
    if (n->broken) return fail(n, PNN_ESTATE, "the handle is unusable after an earlier device failure");
    int dev = -1;
    (void)hipGetDevice(&dev);
    if (dev != n->device) HIP_TRY(n, hipSetDevice(n->device));
    return PNN_OK;
}

}  // namespace

// =======================================================================================
// C ABI

extern "C" {

pnn_status pnn_config_check(const pnn_config* cfg) { return check_config(cfg, nullptr); }

int64_t pnn_param_count(const pnn_config* cfg) {
    if (check_config(cfg, nullptr) != PNN_OK) return 0;
    return packed_count(cfg);
}

pnn_status pnn_shard(int64_t N, int32_t K, int32_t k, int64_t* start, int64_t* len) {
    if (!start || !len || K < 1 || k < 0 || k >= K || N < 0) return PNN_EINVAL;
    *start = shard_start(N, K, k);
    *len = shard_len(N, K, k);
    return PNN_OK;
}

pnn_status pnn_init(const pnn_config* cfg, const float* theta0_host, void* hip_stream, pnn_net** out) {
    if (!out) return fail(nullptr, PNN_EINVAL, "out is NULL");
    *out = nullptr;
    std::string why;
    if (check_config(cfg, &why) != PNN_OK) return fail(nullptr, PNN_EINVAL, "invalid config: %s", why.c_str());
    if (!theta0_host) return fail(nullptr, PNN_EINVAL, "theta0_host is NULL");
    pnn_net* n = new pnn_net();
    n->cfg = *cfg;
    n->L = cfg->n_layers;
    for (int l = 0; l <= n->L; ++l) n->sizes[l] = cfg->sizes[l];
    for (int l = 0; l < n->L; ++l) n->act[l] = cfg->act[l];
    n->P = packed_count(cfg);
    n->bf16 = cfg->precision == PNN_BF16_MIXED;
    int64_t o = 0;
    for (int l = 0; l < n->L; ++l) {
        n->off_w[l] = o;
        o = round_up(o + (int64_t)n->sizes[l + 1] * n->sizes[l], 64);
        n->off_b[l] = o;
        o = round_up(o + n->sizes[l + 1], 64);
    }
    n->pstride = o;
    hipStream_t s = (hipStream_t)hip_stream;
    auto bail = [&](pnn_status st) {
        g_init_error = n->err;
        free_all(n);
        delete n;
        return st;
    };
    if (hipGetDevice(&n->device) != hipSuccess) return bail(fail(n, PNN_EHIP, "no HIP device"));
    {
        // the device address of the fixed workspace, once per device (this device is current)
        if (n->device >= MAX_DEVICES) return bail(fail(n, PNN_EINVAL, "device %d: at most %d devices", n->device, MAX_DEVICES));
        std::lock_guard<std::mutex> g(g_scratch_mu);
        if (!g_scratch_addr[n->device]) {
            void* p = nullptr;
            const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
            if (e != hipSuccess || !p)
                return bail(fail(n, PNN_EHIP, "hipGetSymbolAddress of the workspace failed: %s", hipGetErrorString(e)));
            g_scratch_addr[n->device] = p;
        }
    }
    // failure-handling tests: PNN_SPIN_LIMIT bounds the persistent kernels' waits (polls);
    // PNN_TEST_STALL_WAITS=1 makes the persistent kernels' waits run into that bound
    if (const char* e = getenv("PNN_GEMM")) n->gemm_x3 = strcmp(e, "fp32") != 0;
    n->spin_limit = SPIN_LIMIT;
    if (const char* e = getenv("PNN_SPIN_LIMIT")) {
        const long v = strtol(e, nullptr, 10);
        if (v > 0) n->spin_limit = v;
    }
    if (const char* e = getenv("PNN_TEST_STALL_WAITS")) {
        const bool on = strcmp(e, "1") == 0;
        n->tag_skew = on ? 1u : 0u;
        n->wait_skew = on ? (1 << 29) : 0;  // (the tiles count up to nrb per chunk parity)
    }
    // PNN_TEST_TILE_DELAY=n: half of every CN's tile workgroups start n sleeps late (the
    // per-sample kernel's results must not change)
    if (const char* e = getenv("PNN_TEST_TILE_DELAY")) {
        const long v = strtol(e, nullptr, 10);
        n->tile_delay = v > 0 && v < (1 << 20) ? (int)v : 0;
    }
    const int K = cfg->replicas, B = cfg->batch;
    pnn_status st;
    if ((st = dev_alloc(n, &n->theta, (size_t)K * n->pstride)) != PNN_OK) return bail(st);
    if ((st = dev_alloc(n, &n->merged, (size_t)n->pstride)) != PNN_OK) return bail(st);
    if (n->bf16) {
        if ((st = dev_alloc(n, &n->shadow, (size_t)K * n->pstride)) != PNN_OK) return bail(st);
        if ((st = dev_alloc(n, &n->mshadow, (size_t)n->pstride)) != PNN_OK) return bail(st);
    }
    if ((st = dev_alloc(n, &n->d_correct, 1)) != PNN_OK) return bail(st);
    if ((st = dev_alloc(n, &n->d_cost_sum, 1)) != PNN_OK) return bail(st);
    if ((st = dev_alloc(n, &n->d_mw, (size_t)K)) != PNN_OK) return bail(st);

    n->psgd = (B == 1 && n->L == 2 && !n->bf16 && n->sizes[1] <= 1024 && n->sizes[2] <= MAX_OUT);
    if (n->psgd) {
        // persistent plan: every CN needs 1 + nrb co-resident workgroups
        int cus = 0;
        if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, n->device) != hipSuccess) cus = 0;
        const int H = n->sizes[1], In = n->sizes[0], O = n->sizes[2];
        const int HW = live_width(H);
        // tile workgroups of 16 rows of W1 (rt = 1) or 32 (rt = 2); the CNs go in groups whose
        // workgroups fit the CUs, one launch each.  Of the two, the one with the least estimated
        // time: launches x the relative time of a step (1 with 16-row tiles, 1.8 with 32-row
        // tiles, whose tiles do twice the work per chunk; 1.5 to 1.9 measured with 784-128-10
        // nets, growing with the CNs in flight)
        int rt = 1, kg = 0;
        double best = 1e30;
        for (int r = 1; r <= 2; ++r) {
            const int nb = (H + 16 * r - 1) / (16 * r);
            const int g = std::min(K, cus / (1 + nb));
            if (g < 1) continue;
            const double cost = (double)((K + g - 1) / g) * (r == 1 ? 1.0 : 1.8);
            if (cost < best) { best = cost; rt = r; kg = g; }
        }
        const int nrb = (H + 16 * rt - 1) / (16 * rt);
        n->prt = rt;
        // input sums [HW][T+4], errors [HW][T+4], Gram blocks 3 x [T][T+4], window
        // corrections [8][HW], labels [2][T], 12 counters
        const size_t rec_smem =
            (size_t)(2 * HW * (PT + 4) + 3 * PT * (PT + 4) + 8 * HW + 2 * PT + 12) * sizeof(float);
        const size_t tile_smem = (size_t)4 * (PT / 16) * rt * 64 * 4 * sizeof(float);
        n->psmem = std::max(rec_smem, tile_smem);
        n->pspecial = n->act[0] == PNN_SIGMOID && n->act[1] == PNN_SIGMOID && cfg->loss == PNN_LOSS_MSE && O == 10;
        const void* fn = persistent_fn(n);
        int per_cu = 0;
        bool fits = H <= 128 && In <= 4 * MAX_IB * 16 && kg >= 1;
        if (fits && hipFuncSetAttribute(fn, hipFuncAttributeMaxDynamicSharedMemorySize, (int)n->psmem) != hipSuccess)
            fits = false;
        if (fits && hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, fn, 256, n->psmem) != hipSuccess) fits = false;
        if (fits && (int64_t)per_cu * cus < (int64_t)kg * (1 + nrb)) fits = false;
        (void)hipGetLastError();
        if (fits) {
            n->persistent = true;
            n->nrb = nrb;
            n->kgroup = kg;
            const size_t qn = (size_t)2 * K * HW * (PT + 4);
            if ((st = dev_alloc(n, &n->qbuf, qn)) != PNN_OK) return bail(st);
            // padding neurons and rows of the input sums are never written by the kernel: zero them
            if (hipMemset(n->qbuf, 0, sizeof(float) * qn) != hipSuccess)
                return bail(fail(n, PNN_EHIP, "hipMemset of the input-sum buffer failed"));
            if ((st = dev_alloc(n, &n->d1, (size_t)2 * K * PT * H)) != PNN_OK) return bail(st);
            if ((st = dev_alloc(n, &n->flags, (size_t)(3 * K + 1))) != PNN_OK) return bail(st);
        }
    }
    if (n->psgd && !n->persistent) {
        const int H = n->sizes[1];
        int T = 128;
        while (T > 16 && (int64_t)T * H > 16384) T >>= 1;
        n->T = T;
        // split the 784-long contraction of P so that every CN's P uses several CUs
        n->kchunk = (int)round_up((n->sizes[0] + 7) / 8, 16);
        n->ksplit = (n->sizes[0] + n->kchunk - 1) / n->kchunk;
        if ((st = dev_alloc(n, &n->ppart, (size_t)n->ksplit * K * T * H)) != PNN_OK) return bail(st);
        if ((st = dev_alloc(n, &n->d1, (size_t)K * T * H)) != PNN_OK) return bail(st);
        const size_t smem = (size_t)(2 * T * H + 2 * 16 * MAX_OUT) * sizeof(float);
        hipError_t e = hipSuccess;
        switch (T) {
        case 128: e = hipFuncSetAttribute((const void*)psgd_chunk_kernel<128>, hipFuncAttributeMaxDynamicSharedMemorySize, (int)smem); break;
        case 64: e = hipFuncSetAttribute((const void*)psgd_chunk_kernel<64>, hipFuncAttributeMaxDynamicSharedMemorySize, (int)smem); break;
        case 32: e = hipFuncSetAttribute((const void*)psgd_chunk_kernel<32>, hipFuncAttributeMaxDynamicSharedMemorySize, (int)smem); break;
        default: e = hipFuncSetAttribute((const void*)psgd_chunk_kernel<16>, hipFuncAttributeMaxDynamicSharedMemorySize, (int)smem); break;
        }
        if (e != hipSuccess) return bail(fail(n, PNN_EHIP, "hipFuncSetAttribute: %s", hipGetErrorString(e)));
    } else if (!n->psgd) {
        const size_t el = n->bf16 ? 2 : 4;
        for (int l = 1; l <= n->L; ++l) {
            const size_t cnt = (size_t)K * B * n->sizes[l] * el;
            if (l < n->L && (st = dev_alloc(n, (char**)&n->act_ws[l], cnt)) != PNN_OK) return bail(st);
            if ((st = dev_alloc(n, (char**)&n->del_ws[l], cnt)) != PNN_OK) return bail(st);
        }
        // fp32, first layer with few output tiles (less than one workgroup per CU) and the
        // 784-long contraction: split the contraction into slices of 112
        if (!n->bf16 && n->L >= 2) {
            const int N1 = n->sizes[1], In = n->sizes[0];
            const int64_t wgs = (int64_t)((N1 + 63) / 64) * ((B + 63) / 64) * K;
            if (!(B >= 128 && N1 >= 128) && wgs < 256 && In >= 256) {
                n->kchunk = (int)round_up((In + 7) / 8, 16);
                n->ksplit = (In + n->kchunk - 1) / n->kchunk;
                if ((st = dev_alloc(n, &n->ppart, (size_t)n->ksplit * K * B * N1)) != PNN_OK) return bail(st);
            }
        }
        // persistent mini-batch plan: one hidden layer in fp32, batches of 2..32 rows, at most
        // 16 outputs, and every CN's ceil(H / 16 rt) tile workgroups co-resident (rt = 1, or 2
        // when 16-neuron tiles do not fit); PNN_MB_PLAN=launch selects the per-layer launches
        const char* plan = getenv("PNN_MB_PLAN");
        const bool forced_launch = plan && strcmp(plan, "launch") == 0;
        if (!forced_launch && !n->bf16 && n->L == 2 && B >= 2 && B <= MBP_TB && n->sizes[2] <= 16 &&
            n->sizes[0] % 16 == 0 && n->sizes[0] <= 4 * MAX_IB * 16) {
            int cus = 0;
            if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, n->device) != hipSuccess) cus = 0;
            const int H = n->sizes[1];
            // tile workgroups of 16 neurons (rt = 1) or 32 (rt = 2); the CNs in groups whose tiles
            // fit the CUs, one launch each; the one with the least estimated time (launches x the
            // relative time of a batch step: 1 with 16-neuron tiles, 1.45 with 32, as measured
            // with 784-256-10 nets)
            int rt = 0, kg = 0;
            double best = 1e30;
            for (int r = 1; r <= 2; ++r) {
                const int nb = (H + 16 * r - 1) / (16 * r);
                if (nb > MBP_NRB) continue;
                const int g = std::min(K, cus / nb);
                if (g < 1) continue;
                const double cost = (double)((K + g - 1) / g) * (r == 1 ? 1.0 : 1.45);
                if (cost < best) { best = cost; rt = r; kg = g; }
            }
            if (rt > 0) {
                const int nrb = (H + 16 * rt - 1) / (16 * rt);
                const size_t smem = (size_t)mbp_lds_floats(rt) * sizeof(float);
                const void* fn = mbp_fn(rt);
                int per_cu = 0;
                bool fits = hipFuncSetAttribute(fn, hipFuncAttributeMaxDynamicSharedMemorySize, (int)smem) == hipSuccess;
                if (fits && hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, fn, 256, smem) != hipSuccess) fits = false;
                if (fits && (int64_t)per_cu * cus < (int64_t)kg * nrb) fits = false;
                (void)hipGetLastError();
                if (fits) {
                    n->mbp = true;
                    n->mrt = rt;
                    n->nrb = nrb;
                    n->kgroup = kg;
                    n->psmem = smem;
                    n->zpart_elems = (size_t)2 * K * nrb * MBP_TB * 16;
                    // (zeroed: a share is valid only with its step's tag, which is >= 1)
                    if ((st = dev_alloc(n, &n->zpart, n->zpart_elems)) != PNN_OK) return bail(st);
                    if ((st = dev_alloc(n, &n->flags, (size_t)(K + 1))) != PNN_OK) return bail(st);
                }
            }
        }
        // the last layer fused into the split-bf16 products of one hidden layer (fp32, batches
        // of 128 rows, a hidden width of >= 256 neurons, <= 16 outputs): gemm256x3_kernel's
        // epilogue writes the output sums' partials, out_err_kernel the output errors and
        // upd128x3_kernel forms the hidden errors and updates W2 and b2 (no pass over the
        // hidden layer's activations and errors of its own); PNN_MB_PLAN=launch keeps the
        // separate last-layer kernel
        if (!forced_launch && !n->mbp && !n->bf16 && n->gemm_x3 && n->L == 2 && B == 128 && n->ksplit == 1 &&
            n->sizes[1] >= 256 && n->sizes[1] % 4 == 0 && n->sizes[2] <= MAX_OUT && n->sizes[0] >= 128 &&
            n->sizes[0] % 4 == 0 && n->off_w[1] % 4 == 0 && n->off_b[1] % 4 == 0 && n->pstride % 4 == 0) {
            const size_t ntile = (size_t)(n->sizes[1] + 255) / 256;
            if ((st = dev_alloc(n, &n->fx3_zpart, (size_t)K * ntile * B * 16)) != PNN_OK) return bail(st);
            if ((st = dev_alloc(n, &n->fx3_dout, (size_t)K * B * 16)) != PNN_OK) return bail(st);
            n->fx3 = true;
        }
        // the fused last layer may stage up to 160 KiB of LDS
        const void* tk[3] = {(const void*)tail_kernel<float, 1>, (const void*)tail_kernel<float, 2>,
                             (const void*)tail_kernel<float, 4>};
        const void* tkb[3] = {(const void*)tail_kernel<bf16_t, 1>, (const void*)tail_kernel<bf16_t, 2>,
                              (const void*)tail_kernel<bf16_t, 4>};
        for (int i = 0; i < 3; ++i) {
            hipError_t e = hipFuncSetAttribute(n->bf16 ? tkb[i] : tk[i], hipFuncAttributeMaxDynamicSharedMemorySize,
                                               160 * 1024);
            if (e != hipSuccess) return bail(fail(n, PNN_EHIP, "hipFuncSetAttribute: %s", hipGetErrorString(e)));
        }
    }
    // clone theta0 into every CN and the merged network
    std::vector<float> padded(n->pstride);
    unpack(n, theta0_host, padded.data());
    if (hipMemcpy(n->merged, padded.data(), n->pstride * sizeof(float), hipMemcpyHostToDevice) != hipSuccess)
        return bail(fail(n, PNN_EHIP, "copy of theta0 failed"));
    for (int k = 0; k < K; ++k)
        if (hipMemcpyAsync(n->theta + (size_t)k * n->pstride, n->merged, n->pstride * sizeof(float),
                           hipMemcpyDeviceToDevice, s) != hipSuccess)
            return bail(fail(n, PNN_EHIP, "clone of theta0 failed"));
    if ((st = refresh_shadows(n, s)) != PNN_OK) return bail(st);
    if (hipStreamSynchronize(s) != hipSuccess) return bail(fail(n, PNN_EHIP, "init synchronize failed"));
    *out = n;
    return PNN_OK;
}

// the copy of the merged network into the CNs that a merge deferred, if one is pending
static pnn_status settle(pnn_net* n, hipStream_t s) {
    if (!n->bcast_pending) return PNN_OK;
    const int64_t q = n->pstride / 4;
    Launch l(n, s, "broadcast");
    bcast_kernel<<<(unsigned)((q + 255) / 256), 256, 0, s>>>(n->theta, n->merged, n->pstride, n->cfg.replicas);
    TRY(l.done());
    n->bcast_pending = false;
    return PNN_OK;
}

pnn_status pnn_train_epoch(pnn_net* n, const float* x_dev, const int32_t* y_dev, int64_t N, void* hip_stream) {
    TRY(usable(n));
    if (!x_dev || !y_dev) return fail(n, PNN_EINVAL, "x_dev / y_dev is NULL");
    if (!aligned16(x_dev)) return fail(n, PNN_EINVAL, "x_dev is not 16-byte aligned");
    if (N < n->cfg.replicas) return fail(n, PNN_ESHAPE, "N = %lld < K = %d leaves a slice empty", (long long)N, n->cfg.replicas);
    TRY(check_abort(n, false));
    hipStream_t s = (hipStream_t)hip_stream;
    if (!n->fx3) TRY(settle(n, s));
    if (n->psgd) return psgd_epoch(n, x_dev, y_dev, N, s);
    if (n->mbp) return mbp_epoch(n, x_dev, y_dev, N, s);
    const int64_t nmax = shard_len(N, n->cfg.replicas, 0);
    for (int64_t r0 = 0; r0 < nmax; r0 += n->cfg.batch) {
        // (the first step writes every parameter of every CN: each CN has rows in it)
        const bool fm = r0 == 0 && n->bcast_pending;
        if (n->bf16) TRY(minibatch_step<true>(n, x_dev, y_dev, N, r0, s, fm));
        else TRY(minibatch_step<false>(n, x_dev, y_dev, N, r0, s, fm));
        if (fm) n->bcast_pending = false;
    }
    return PNN_OK;
}

pnn_status pnn_train_epoch_order(pnn_net* n, const float* x_dev, const int32_t* y_dev, int64_t N,
                                 const int32_t* order_dev, void* hip_stream) {
    TRY(usable(n));
    if (!x_dev || !y_dev || !order_dev) return fail(n, PNN_EINVAL, "x_dev / y_dev / order_dev is NULL");
    if (!aligned16(x_dev)) return fail(n, PNN_EINVAL, "x_dev is not 16-byte aligned");
    if (N < n->cfg.replicas) return fail(n, PNN_ESHAPE, "N = %lld < K = %d leaves a slice empty", (long long)N, n->cfg.replicas);
    if (N > INT32_MAX) return fail(n, PNN_ESHAPE, "N = %lld does not fit the int32 order", (long long)N);
    hipStream_t s = (hipStream_t)hip_stream;
    const int D = n->sizes[0];
    if (N > n->ord_rows) {
        HIP_TRY(n, hipStreamSynchronize(s));
        if (n->ord_x) (void)hipFree(n->ord_x);
        if (n->ord_y) (void)hipFree(n->ord_y);
        n->ord_x = nullptr; n->ord_y = nullptr; n->ord_rows = 0;
        TRY(dev_alloc(n, &n->ord_x, (size_t)N * D));
        TRY(dev_alloc(n, &n->ord_y, (size_t)N));
        n->ord_rows = N;
    }
    {
        Launch l(n, s, "gather_rows");
        gather_rows_kernel<<<(unsigned)N, 256, 0, s>>>(x_dev, y_dev, order_dev, N, D, n->ord_x, n->ord_y);
        TRY(l.done());
    }
    return pnn_train_epoch(n, n->ord_x, n->ord_y, N, hip_stream);
}

static pnn_status launch_merge(pnn_net* n, int32_t broadcast, const double* w_dev, double wsum, hipStream_t s) {
    TRY(settle(n, s));
    // with the fused last layer the broadcast is left to the next epoch's first step, which
    // reads the merged slot and writes every CN (saving a write of K copies and their reads)
    const bool defer = broadcast && n->fx3;
    MergeArgs a;
    a.theta = n->theta; a.merged = n->merged;
    a.shadow = n->bf16 ? n->shadow : nullptr;
    a.mshadow = n->bf16 ? n->mshadow : nullptr;
    a.pstride = n->pstride; a.K = n->cfg.replicas; a.broadcast = broadcast && !defer ? 1 : 0;
    a.w = w_dev; a.wsum = wsum;
    const int64_t q = n->pstride / 4;
    Launch l(n, s, "merge");
    merge_kernel<<<(unsigned)((q + 255) / 256), 256, 0, s>>>(a);
    TRY(l.done());
    n->bcast_pending = defer;
    return PNN_OK;
}

pnn_status pnn_merge(pnn_net* n, int32_t broadcast, void* hip_stream) {
    TRY(usable(n));
    TRY(check_abort(n, true));
    return launch_merge(n, broadcast, nullptr, (double)n->cfg.replicas, (hipStream_t)hip_stream);
}

pnn_status pnn_merge_weighted(pnn_net* n, const double* weights_host, int32_t broadcast, void* hip_stream) {
    TRY(usable(n));
    if (!weights_host) return fail(n, PNN_EINVAL, "weights_host is NULL");
    const int K = n->cfg.replicas;
    double ws = 0.0;
    for (int k = 0; k < K; ++k) {
        const double v = weights_host[k];
        if (!(v >= 0.0) || !std::isfinite(v)) return fail(n, PNN_EINVAL, "weight %d is %g (must be finite and >= 0)", k, v);
        ws += v;
    }
    if (!(ws > 0.0) || !std::isfinite(ws)) return fail(n, PNN_EINVAL, "the weights sum to %g (must be positive)", ws);
    TRY(check_abort(n, true));
    hipStream_t s = (hipStream_t)hip_stream;
    // the weights travel with the launch's stream order (the copy waits for earlier work)
    HIP_TRY(n, hipMemcpyAsync(n->d_mw, weights_host, sizeof(double) * K, hipMemcpyHostToDevice, s));
    HIP_TRY(n, hipStreamSynchronize(s));
    return launch_merge(n, broadcast, n->d_mw, ws, s);
}

// rows of one inference chunk
constexpr int INFER_CHUNK = 8192;

// workspace bytes of an allocation-free evaluation of nrows rows: counters, one chunk's hidden
// activations, per-row costs (when the cost is asked for)
static int64_t noalloc_eval_bytes(const pnn_net* n, int64_t nrows, bool cost) {
    const int rows = (int)std::min<int64_t>(nrows, INFER_CHUNK);
    const int64_t el = n->bf16 ? 2 : 4;
    int64_t b = 256;
    for (int l = 1; l < n->L; ++l) b += round_up((int64_t)rows * n->sizes[l] * el, 256);
    if (cost) b += nrows * (int64_t)sizeof(double);
    return b;
}

// the handle's inference workspace for min(nrows, INFER_CHUNK) rows (grown with hipMalloc)
static pnn_status grow_inference_ws(pnn_net* n, int64_t nrows, hipStream_t s) {
    const int L = n->L;
    const int rows = (int)std::min<int64_t>(nrows, INFER_CHUNK);
    if (L > 1 && rows > n->inf_rows) {
        HIP_TRY(n, hipStreamSynchronize(s));
        const size_t el = n->bf16 ? 2 : 4;
        for (int l = 1; l < L; ++l) {
            if (n->inf_ws[l]) (void)hipFree(n->inf_ws[l]);
            n->inf_ws[l] = nullptr;
            TRY(dev_alloc(n, (char**)&n->inf_ws[l], (size_t)rows * n->sizes[l] * el));
        }
        n->inf_rows = rows;
    }
    return PNN_OK;
}

// forward pass of one network over nrows data-set rows in chunks of INFER_CHUNK, then the
// output layer: predictions (pred, nullable), outputs (out, nullable), the correct count into
// *correct (count; zeroed first), per-row costs into cost (nullable; needs y).  ws[l] holds
// the activations of hidden layer l for a chunk.
static pnn_status run_inference(pnn_net* n, int32_t which, const float* x_dev, int64_t nrows, int32_t* pred_dev,
                                float* out_dev, bool count, const int32_t* y_dev, double* cost, void* const* ws,
                                unsigned long long* correct, hipStream_t s) {
    if (count) zero_ints_kernel<<<1, 256, 0, s>>>((int*)correct, 2);
    const int L = n->L;
    const int CH = INFER_CHUNK;
    const float* th = which < 0 ? n->merged : n->theta + (size_t)which * n->pstride;
    const bf16_t* sh = !n->bf16 ? nullptr : (which < 0 ? n->mshadow : n->shadow + (size_t)which * n->pstride);
    for (int64_t r0 = 0; r0 < nrows; r0 += CH) {
        // a single "CN" whose slice is the whole input: rows r0 .. r0+CH
        for (int l = 1; l <= L - 1; ++l) {
            GemmArgs g = gemm_base(n, CH, n->sizes[l], n->sizes[l - 1], nrows, r0, CH, 1);
            g.k_rep = 1;
            if (l == 1) g.a = opnd(x_dev, 0, n->sizes[0], 1);
            else g.a = opnd(ws[l - 1], 0, n->sizes[l - 1], 0);
            g.c = ws[l]; g.c_z = 0; g.c_ld = n->sizes[l];
            g.bias = th + n->off_b[l - 1]; g.bias_z = 0;
            g.act = n->act[l - 1];
            g.M = std::min<int64_t>(CH, nrows - r0);
            if (n->bf16) {
                g.b = opnd(sh + n->off_w[l - 1], 0, n->sizes[l - 1], 0);
                if (l == 1) TRY((run_gemm<true, float, bf16_t, true, true, EPI_FWD, bf16_t>(n, s, g, 1, "infer_fwd_gemm")));
                else TRY((run_gemm<true, bf16_t, bf16_t, true, true, EPI_FWD, bf16_t>(n, s, g, 1, "infer_fwd_gemm")));
            } else {
                g.b = opnd(th + n->off_w[l - 1], 0, n->sizes[l - 1], 0);
                if (l == 1) TRY((run_gemm<false, float, float, true, true, EPI_FWD, float>(n, s, g, 1, "infer_fwd_gemm")));
                else TRY((run_gemm<false, float, float, true, true, EPI_FWD, float>(n, s, g, 1, "infer_fwd_gemm")));
            }
        }
        RowArgs a;
        memset(&a, 0, sizeof a);
        if (L == 1) { a.x = x_dev; a.x_xrows = 1; a.x_ld = n->sizes[0]; }
        else { a.x = ws[L - 1]; a.x_z = 0; a.x_ld = n->sizes[L - 1]; }
        a.bias = th + n->off_b[L - 1];
        a.H = n->sizes[L - 1]; a.O = n->sizes[L]; a.act = n->act[L - 1]; a.loss = n->cfg.loss;
        a.n_total = nrows; a.k_rep = 1; a.r0 = r0; a.step_rows = CH;
        a.y = y_dev; a.out = out_dev; a.pred = pred_dev; a.correct = count ? correct : nullptr;
        a.cost = cost;
        const int rws = (int)std::min<int64_t>(CH, nrows - r0);
        dim3 grid((rws + 3) / 4, 1, 1);
        Launch lc(n, s, "infer_out");
        if (n->bf16) {
            a.w = sh + n->off_w[L - 1];
            if (L == 1) out_layer_kernel<float, bf16_t, float, false><<<grid, 256, 0, s>>>(a);
            else out_layer_kernel<bf16_t, bf16_t, float, false><<<grid, 256, 0, s>>>(a);
        } else {
            a.w = th + n->off_w[L - 1];
            out_layer_kernel<float, float, float, false><<<grid, 256, 0, s>>>(a);
        }
        TRY(lc.done());
    }
    return PNN_OK;
}

// the evaluation of pnn_eval on a given workspace: correct count into *correct, per-row costs
// into cost[nrows] summed in a fixed order into *cost_sum; waits for the device
static pnn_status eval_run(pnn_net* n, int32_t which, const float* x_dev, const int32_t* y_dev, int64_t nrows,
                           int64_t* correct_host, double* cost_host, void* const* ws, unsigned long long* correct,
                           double* cost, double* cost_sum, hipStream_t s) {
    TRY(run_inference(n, which, x_dev, nrows, nullptr, nullptr, correct_host != nullptr, y_dev,
                      cost_host ? cost : nullptr, ws, correct, s));
    if (cost_host) {
        Launch lc(n, s, "eval_cost_sum");
        sum_f64_kernel<<<1, 256, 0, s>>>(cost, nrows, cost_sum);
        TRY(lc.done());
    }
    unsigned long long c = 0;
    double cs = 0.0;
    if (correct_host) HIP_TRY(n, hipMemcpyAsync(&c, correct, sizeof c, hipMemcpyDeviceToHost, s));
    if (cost_host) HIP_TRY(n, hipMemcpyAsync(&cs, cost_sum, sizeof cs, hipMemcpyDeviceToHost, s));
    HIP_TRY(n, hipStreamSynchronize(s));
    if (correct_host) *correct_host = (int64_t)c;
    if (cost_host) *cost_host = cs / (double)nrows;
    return PNN_OK;
}

pnn_status pnn_infer(pnn_net* n, int32_t which, const float* x_dev, int64_t nrows, int32_t* pred_dev, float* out_dev,
                     int64_t* correct_host, const int32_t* y_dev, void* hip_stream) {
    TRY(usable(n));
    if (which < -1 || which >= n->cfg.replicas) return fail(n, PNN_EINVAL, "which = %d out of range", which);
    if (nrows < 0) return fail(n, PNN_ESHAPE, "n < 0");
    if (nrows == 0) {  // nothing to read or write
        if (correct_host) *correct_host = 0;
        return PNN_OK;
    }
    if (!x_dev || !pred_dev) return fail(n, PNN_EINVAL, "x_dev / pred_dev is NULL");
    if (!aligned16(x_dev)) return fail(n, PNN_EINVAL, "x_dev is not 16-byte aligned");
    TRY(check_abort(n, true));
    hipStream_t s = (hipStream_t)hip_stream;
    if (which >= 0) TRY(settle(n, s));
    const bool count = correct_host && y_dev;
    TRY(grow_inference_ws(n, nrows, s));
    TRY(run_inference(n, which, x_dev, nrows, pred_dev, out_dev, count, y_dev, nullptr, n->inf_ws, n->d_correct, s));
    if (count) {
        unsigned long long c = 0;
        HIP_TRY(n, hipMemcpyAsync(&c, n->d_correct, sizeof c, hipMemcpyDeviceToHost, s));
        HIP_TRY(n, hipStreamSynchronize(s));
        *correct_host = (int64_t)c;
    }
    return PNN_OK;
}

pnn_status pnn_eval(pnn_net* n, int32_t which, const float* x_dev, const int32_t* y_dev, int64_t nrows,
                    int64_t* correct_host, double* cost_host, void* hip_stream) {
    TRY(usable(n));
    if (which < -1 || which >= n->cfg.replicas) return fail(n, PNN_EINVAL, "which = %d out of range", which);
    if (nrows < 0) return fail(n, PNN_ESHAPE, "n < 0");
    if (nrows == 0) {
        if (correct_host) *correct_host = 0;
        if (cost_host) *cost_host = 0.0;
        return PNN_OK;
    }
    if (!x_dev || !y_dev) return fail(n, PNN_EINVAL, "x_dev / y_dev is NULL");
    if (!aligned16(x_dev)) return fail(n, PNN_EINVAL, "x_dev is not 16-byte aligned");
    TRY(check_abort(n, true));
    hipStream_t s = (hipStream_t)hip_stream;
    if (cost_host && nrows > n->cost_rows) {
        HIP_TRY(n, hipStreamSynchronize(s));
        if (n->d_cost) (void)hipFree(n->d_cost);
        n->d_cost = nullptr;
        n->cost_rows = 0;
        TRY(dev_alloc(n, &n->d_cost, (size_t)nrows));
        n->cost_rows = nrows;
    }
    TRY(grow_inference_ws(n, nrows, s));
    if (which >= 0) TRY(settle(n, s));
    return eval_run(n, which, x_dev, y_dev, nrows, correct_host, cost_host, n->inf_ws, n->d_correct, n->d_cost,
                    n->d_cost_sum, s);
}

pnn_status pnn_eval_noalloc(pnn_net* n, int32_t which, const float* x_dev, const int32_t* y_dev, int64_t nrows,
                            int64_t* correct_host, double* cost_host, void* hip_stream) {
    TRY(usable(n));
    if (which < -1 || which >= n->cfg.replicas) return fail(n, PNN_EINVAL, "which = %d out of range", which);
    if (nrows < 0) return fail(n, PNN_ESHAPE, "n < 0");
    if (nrows == 0) {
        if (correct_host) *correct_host = 0;
        if (cost_host) *cost_host = 0.0;
        return PNN_OK;
    }
    if (!x_dev || !y_dev) return fail(n, PNN_EINVAL, "x_dev / y_dev is NULL");
    if (!aligned16(x_dev)) return fail(n, PNN_EINVAL, "x_dev is not 16-byte aligned");
    char* base = (char*)scratch_ptr(n->device);
    if (!base) return fail(n, PNN_ESTATE, "no workspace address for device %d", n->device);
    // workspace layout: [correct count, cost sum] | hidden activations of a chunk, layer by
    // layer | per-row costs
    const int64_t need = noalloc_eval_bytes(n, nrows, cost_host != nullptr);
    if (need > (int64_t)SCRATCH_BYTES)
        return fail(n, PNN_ESHAPE, "evaluating %lld rows needs %lld bytes of workspace; the fixed workspace has %lld",
                    (long long)nrows, (long long)need, (long long)SCRATCH_BYTES);
    TRY(check_abort(n, true));
    hipStream_t s = (hipStream_t)hip_stream;
    unsigned long long* correct = (unsigned long long*)base;
    double* cost_sum = (double*)(base + 8);
    void* ws[9] = {nullptr};
    int64_t o = 256;
    const int rows = (int)std::min<int64_t>(nrows, INFER_CHUNK);
    const int64_t el = n->bf16 ? 2 : 4;
    for (int l = 1; l < n->L; ++l) {
        ws[l] = base + o;
        o += round_up((int64_t)rows * n->sizes[l] * el, 256);
    }
    double* cost = cost_host ? (double*)(base + o) : nullptr;
    if (which >= 0) TRY(settle(n, s));
    return eval_run(n, which, x_dev, y_dev, nrows, correct_host, cost_host, ws, correct, cost, cost_sum, s);
}

const char* pnn_plan(const pnn_net* n) {
    if (!n) return "";
    if (n->psgd) return n->persistent ? "per-sample persistent" : "per-sample chunked";
    return n->mbp ? "mini-batch persistent" : n->fx3 ? "mini-batch fused last layer" : "mini-batch";
}

pnn_status pnn_get_params(pnn_net* n, int32_t which, float* host_out) {
    TRY(usable(n));
    if (!host_out) return fail(n, PNN_EINVAL, "host_out is NULL");
    if (which < -1 || which >= n->cfg.replicas) return fail(n, PNN_EINVAL, "which = %d out of range", which);
    HIP_TRY(n, hipDeviceSynchronize());
    TRY(check_abort(n, true));
    if (which >= 0) {
        TRY(settle(n, nullptr));
        HIP_TRY(n, hipDeviceSynchronize());
    }
    std::vector<float> padded(n->pstride);
    const float* src = which < 0 ? n->merged : n->theta + (size_t)which * n->pstride;
    HIP_TRY(n, hipMemcpy(padded.data(), src, n->pstride * sizeof(float), hipMemcpyDeviceToHost));
    pack(n, padded.data(), host_out);
    return PNN_OK;
}

pnn_status pnn_set_params(pnn_net* n, int32_t which, const float* host_in) {
    TRY(usable(n));
    if (!host_in) return fail(n, PNN_EINVAL, "host_in is NULL");
    if (which < -2 || which >= n->cfg.replicas) return fail(n, PNN_EINVAL, "which = %d out of range", which);
    HIP_TRY(n, hipDeviceSynchronize());
    TRY(check_abort(n, true));
    TRY(settle(n, nullptr));
    std::vector<float> padded(n->pstride);
    unpack(n, host_in, padded.data());
    const size_t bytes = n->pstride * sizeof(float);
    if (which == -1 || which == -2) HIP_TRY(n, hipMemcpy(n->merged, padded.data(), bytes, hipMemcpyHostToDevice));
    if (which >= 0) HIP_TRY(n, hipMemcpy(n->theta + (size_t)which * n->pstride, padded.data(), bytes, hipMemcpyHostToDevice));
    if (which == -2)
        for (int k = 0; k < n->cfg.replicas; ++k)
            HIP_TRY(n, hipMemcpy(n->theta + (size_t)k * n->pstride, padded.data(), bytes, hipMemcpyHostToDevice));
    TRY(refresh_shadows(n, nullptr));
    HIP_TRY(n, hipDeviceSynchronize());
    return PNN_OK;
}

const char* pnn_last_error(const pnn_net* n) { return n ? n->err.c_str() : g_init_error.c_str(); }

pnn_status pnn_profile(pnn_net* n, int32_t enable) {
    if (!n) return PNN_EINVAL;
    prof_drain(n);
    n->prof_acc.clear();
    n->prof = enable != 0;
    return PNN_OK;
}

int32_t pnn_profile_read(pnn_net* n, const char** names, double* total_ms, int64_t* launches, int32_t cap) {
    if (!n) return 0;
    prof_drain(n);
    n->prof_names_store.clear();
    for (auto& kv : n->prof_acc) n->prof_names_store.push_back(kv.first);
    int32_t i = 0;
    for (auto& kv : n->prof_acc) {
        if (i >= cap) break;
        if (names) names[i] = n->prof_names_store[i].c_str();
        if (total_ms) total_ms[i] = kv.second.first;
        if (launches) launches[i] = kv.second.second;
        ++i;
    }
    return (int32_t)n->prof_acc.size();
}

void pnn_destroy(pnn_net* n) {
    if (!n) return;
    (void)hipDeviceSynchronize();
    free_all(n);
    delete n;
}

}  // extern "C"
