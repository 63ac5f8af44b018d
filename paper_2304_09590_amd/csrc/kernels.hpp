// kernels.hpp -- CDNA4 (gfx950) kernels of the PNN hot path.
//
// Every kernel is batched over the K child networks (CNs): blockIdx.z (or x) selects the
// CN, whose parameters sit at theta + z * pstride in the padded device layout, and whose
// data slice is the contiguous row range given by shard_start/shard_len below.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace pnn {

enum { ACT_SIGMOID = 0, ACT_TANH = 1, ACT_RELU = 2, ACT_LEAKY = 3, ACT_SOFTMAX = 4 };
enum { LOSS_MSE = 0, LOSS_XENT = 1 };

typedef uint16_t bf16_t;  // bfloat16 storage
typedef float f4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf8v __attribute__((ext_vector_type(8)));

constexpr int MAX_OUT = 16;  // widest output layer handled by the row kernels

// ------------------------------------------------------------------------------------
// slices of the data set (contiguous, the first N mod K slices one row longer)

__device__ __host__ inline int64_t shard_len(int64_t n, int k_total, int k) {
    return n / k_total + (k < n % k_total ? 1 : 0);
}
__device__ __host__ inline int64_t shard_start(int64_t n, int k_total, int k) {
    const int64_t q = n / k_total, r = n % k_total;
    return (int64_t)k * q + (k < r ? k : r);
}

// ------------------------------------------------------------------------------------
// bfloat16 conversion, round to nearest even

__device__ inline bf16_t f2bf(float f) {
    uint32_t u = __float_as_uint(f);
    if ((u & 0x7f800000u) == 0x7f800000u && (u & 0x007fffffu)) return (bf16_t)((u >> 16) | 0x40);  // quiet NaN
    u += 0x7fffu + ((u >> 16) & 1u);
    return (bf16_t)(u >> 16);
}
__device__ inline float bf2f(bf16_t b) { return __uint_as_float((uint32_t)b << 16); }

template <typename T> __device__ inline float to_f(T v);
template <> __device__ inline float to_f<float>(float v) { return v; }
template <> __device__ inline float to_f<bf16_t>(bf16_t v) { return bf2f(v); }
template <typename T> __device__ inline T from_f(float v);
template <> __device__ inline float from_f<float>(float v) { return v; }
template <> __device__ inline bf16_t from_f<bf16_t>(float v) { return f2bf(v); }

// ------------------------------------------------------------------------------------
// activations.  The rectifiers store z < 0 with its sign (a negative zero for ReLU), so
// that phi'(z) can be read back from the stored activation alone, with phi'(0) = 1.

__device__ inline float act_fn(int a, float z) {
    switch (a) {
    case ACT_SIGMOID: return 1.0f / (1.0f + expf(-z));
    case ACT_TANH: return tanhf(z);
    case ACT_RELU: return z >= 0.0f ? z + 0.0f : -0.0f;
    case ACT_LEAKY: return z >= 0.0f ? z + 0.0f : 0.01f * z;
    default: return z;
    }
}
// phi'(z) from x = phi(z)
__device__ inline float act_deriv(int a, float x) {
    switch (a) {
    case ACT_SIGMOID: return x * (1.0f - x);
    case ACT_TANH: return 1.0f - x * x;
    case ACT_RELU: return signbit(x) ? 0.0f : 1.0f;
    case ACT_LEAKY: return signbit(x) ? 0.01f : 1.0f;
    default: return 1.0f;
    }
}

__device__ inline float wave_sum(float v) {
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) v += __shfl_xor(v, off, 64);
    return v;
}

// ------------------------------------------------------------------------------------
// Batched GEMM on the matrix cores.
//
//   C[z](m, n) (op)= sum_k A[z](m, k) * B[z](k, n)
//
// An operand is a row-major matrix with leading dimension ld.  A_KC: A(m,k) = A[m*ld + k]
// (rows are m); otherwise A(m,k) = A[k*ld + m] (rows are k).  B_KC: B(k,n) = B[n*ld + k]
// (rows are n); otherwise B(k,n) = B[k*ld + n] (rows are k).  An operand flagged xrows
// addresses rows of the caller's data set: row r of CN z is data row
// shard_start(z) + r0(z) + r; otherwise row r is at ptr + z*zstride + r*ld.
//
// The batch index z covers CN and, for chunked launches, a chunk: cn = z / zdiv,
// r0 = r0_base + (z % zdiv) * r0_step.  Dimensions flagged in sample_dims (bit 0 = m,
// 1 = n, 2 = k) run over the rows of the current step and are cut to
// valid = clamp(shard_len(cn) - r0, 0, step_rows); others run to M, N, Kd.
//
// fp32: v_mfma_f32_16x16x4_f32.  bf16: v_mfma_f32_16x16x32_bf16, operands converted to
// bf16 (round to nearest even) while staged into LDS; accumulation is fp32 in both.

enum { EPI_STORE = 0, EPI_FWD = 1, EPI_BWD = 2, EPI_UPD = 3 };

struct Operand {
    const void* ptr;
    int64_t zstride;
    int64_t ld;
    int xrows;
    int64_t xshift;  // xrows only: row offset added to the step's first data row
};

struct GemmArgs {
    int M, N, Kd;
    Operand a, b;
    // output / in-place target
    void* c;
    int64_t c_z, c_ld;
    // batch -> (CN, step rows)
    int64_t n_total;
    int k_rep;
    int zdiv;
    int64_t r0_base, r0_step;
    int step_rows;
    int sample_dims;
    // split of the contraction: blockIdx.z = z * ksplit + slice; slice s covers
    // [s*kchunk, (s+1)*kchunk) and writes C + s * c_split (EPI_STORE only)
    int ksplit, kchunk;
    int64_t c_split;
    // epilogue
    const float* bias;      // EPI_FWD: bias[n] (+ z * bias_z)
    int64_t bias_z;
    float* ubias;           // EPI_UPD: bias[m] updated with the row sums of A (+ z * bias_z)
    int act;
    const void* aux;        // EPI_BWD: activation x^l, same layout as C
    float lr;
    int scale_per_batch;    // EPI_UPD: scale = lr / valid (1) or lr (0)
    bf16_t* shadow;         // EPI_UPD: bf16 copy of the updated target (+ z * c_z), nullable
};

template <bool BF> struct GemmTile;
template <> struct GemmTile<false> { static constexpr int BK = 16, LDK = 20; typedef float T; };
template <> struct GemmTile<true> { static constexpr int BK = 32, LDK = 40; typedef bf16_t T; };

__device__ inline void gemm_zinfo(const GemmArgs& g, int z, int& cn, int64_t& r0, int& valid) {
    cn = z / g.zdiv;
    r0 = g.r0_base + (int64_t)(z % g.zdiv) * g.r0_step;
    int64_t v = shard_len(g.n_total, g.k_rep, cn) - r0;
    valid = (int)(v < 0 ? 0 : (v > g.step_rows ? g.step_rows : v));
}

__device__ inline const char* operand_row(const Operand& o, int elem, int z, int cn, int64_t xbase, int64_t r) {
    const char* p = (const char*)o.ptr;
    if (o.xrows) return p + (size_t)((xbase + o.xshift + r) * o.ld) * elem;
    return p + (size_t)(z * o.zstride + r * o.ld) * elem;
}

// Stage a BR x BK tile (rows r0t.., k k0..) of an operand whose rows are the tile's
// non-contraction index ("KC" layout) into lds[row][k].
template <bool BF, typename TS>
__device__ inline void stage_kc(typename GemmTile<BF>::T* lds, const Operand& o, int z, int cn, int64_t xbase,
                                int row0, int rows_valid, int k0, int k_valid, int tid) {
    constexpr int BK = GemmTile<BF>::BK, LDK = GemmTile<BF>::LDK;
    if constexpr (!BF) {
        // 64 rows x 16 k fp32: one float4 per thread
        const int r = tid >> 2, kq = (tid & 3) * 4;
        float4 v = make_float4(0.f, 0.f, 0.f, 0.f);
        if (row0 + r < rows_valid && k0 + kq < k_valid)
            v = *(const float4*)(operand_row(o, 4, z, cn, xbase, row0 + r) + (size_t)(k0 + kq) * 4);
        *(float4*)(lds + r * LDK + kq) = v;
    } else if constexpr (sizeof(TS) == 4) {
        // 64 rows x 32 k from fp32: two float4 per thread, converted
#pragma unroll
        for (int h = 0; h < 2; ++h) {
            const int idx = tid + h * 256, r = idx >> 3, kq = (idx & 7) * 4;
            float4 v = make_float4(0.f, 0.f, 0.f, 0.f);
            if (row0 + r < rows_valid && k0 + kq < k_valid)
                v = *(const float4*)(operand_row(o, 4, z, cn, xbase, row0 + r) + (size_t)(k0 + kq) * 4);
            bf16_t* d = lds + r * LDK + kq;
            d[0] = f2bf(v.x); d[1] = f2bf(v.y); d[2] = f2bf(v.z); d[3] = f2bf(v.w);
        }
    } else {
        // 64 rows x 32 k from bf16: one 16-byte load per thread
        const int r = tid >> 2, kq = (tid & 3) * 8;
        uint4 v = make_uint4(0, 0, 0, 0);
        if (row0 + r < rows_valid && k0 + kq < k_valid)
            v = *(const uint4*)(operand_row(o, 2, z, cn, xbase, row0 + r) + (size_t)(k0 + kq) * 2);
        *(uint4*)(lds + r * LDK + kq) = v;
    }
    (void)BK;
}

// Stage a tile from an operand whose rows are the contraction index ("NC" layout):
// element (t, k) = row k, column t; stored transposed into lds[t][k].
template <bool BF, typename TS>
__device__ inline void stage_nc(typename GemmTile<BF>::T* lds, const Operand& o, int z, int cn, int64_t xbase,
                                int col0, int cols_valid, int k0, int k_valid, int tid) {
    constexpr int BK = GemmTile<BF>::BK, LDK = GemmTile<BF>::LDK;
    // BK rows (k) x 64 columns; 4 consecutive columns per access
#pragma unroll
    for (int h = 0; h < BK / 16; ++h) {
        const int idx = tid + h * 256, k = idx >> 4, cq = (idx & 15) * 4;
        float v[4] = {0.f, 0.f, 0.f, 0.f};
        if (k0 + k < k_valid && col0 + cq < cols_valid) {
            const char* row = operand_row(o, sizeof(TS), z, cn, xbase, k0 + k);
            if constexpr (sizeof(TS) == 4) {
                float4 q = *(const float4*)(row + (size_t)(col0 + cq) * 4);
                v[0] = q.x; v[1] = q.y; v[2] = q.z; v[3] = q.w;
            } else {
                uint2 q = *(const uint2*)(row + (size_t)(col0 + cq) * 2);
                v[0] = bf2f((bf16_t)(q.x & 0xffff)); v[1] = bf2f((bf16_t)(q.x >> 16));
                v[2] = bf2f((bf16_t)(q.y & 0xffff)); v[3] = bf2f((bf16_t)(q.y >> 16));
            }
        }
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            if constexpr (BF) lds[(cq + j) * LDK + k] = f2bf(v[j]);
            else lds[(cq + j) * LDK + k] = v[j];
        }
    }
}

template <bool BF, typename TA, typename TB, bool A_KC, bool B_KC, int EPI, typename TO>
__global__ __launch_bounds__(256) void gemm_kernel(GemmArgs g) {
    typedef typename GemmTile<BF>::T LT;
    constexpr int BK = GemmTile<BF>::BK, LDK = GemmTile<BF>::LDK;
    __shared__ __attribute__((aligned(16))) LT As[64 * LDK];
    __shared__ __attribute__((aligned(16))) LT Bs[64 * LDK];
    __shared__ float rowsum[64];

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int wm = wave >> 1, wn = wave & 1;
    const int zz = blockIdx.z / g.ksplit, slice = blockIdx.z % g.ksplit;
    int cn, valid;
    int64_t r0;
    gemm_zinfo(g, zz, cn, r0, valid);
    const int Mv = (g.sample_dims & 1) ? valid : g.M;
    const int Nv = (g.sample_dims & 2) ? valid : g.N;
    const int Kv = (g.sample_dims & 4) ? valid : g.Kd;
    const int m0 = blockIdx.y * 64, n0 = blockIdx.x * 64;
    if (m0 >= Mv || n0 >= Nv) return;
    const int kbeg = slice * g.kchunk;
    const int kend = min(Kv, kbeg + g.kchunk);
    const int64_t xbase = shard_start(g.n_total, g.k_rep, cn) + r0;
    const bool do_rowsum = (EPI == EPI_UPD) && g.ubias != nullptr && blockIdx.x == 0;
    if (do_rowsum && tid < 64) rowsum[tid] = 0.f;

    f4 acc[2][2];
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j) acc[i][j] = f4{0.f, 0.f, 0.f, 0.f};

    for (int k0 = kbeg; k0 < kend; k0 += BK) {
        if constexpr (A_KC) stage_kc<BF, TA>(As, g.a, zz, cn, xbase, m0, Mv, k0, kend, tid);
        else stage_nc<BF, TA>(As, g.a, zz, cn, xbase, m0, Mv, k0, kend, tid);
        if constexpr (B_KC) stage_kc<BF, TB>(Bs, g.b, zz, cn, xbase, n0, Nv, k0, kend, tid);
        else stage_nc<BF, TB>(Bs, g.b, zz, cn, xbase, n0, Nv, k0, kend, tid);
        __syncthreads();
        if (do_rowsum && tid < 64) {
            float s = 0.f;
#pragma unroll
            for (int k = 0; k < BK; ++k) s += (float)to_f<LT>(As[tid * LDK + k]);
            rowsum[tid] += s;
        }
        const int rl = lane & 15, kg = lane >> 4;
        if constexpr (!BF) {
            f4 av[2], bv[2];
#pragma unroll
            for (int i = 0; i < 2; ++i) av[i] = *(const f4*)(As + (wm * 32 + i * 16 + rl) * LDK + kg * 4);
#pragma unroll
            for (int j = 0; j < 2; ++j) bv[j] = *(const f4*)(Bs + (wn * 32 + j * 16 + rl) * LDK + kg * 4);
#pragma unroll
            for (int q = 0; q < 4; ++q)
#pragma unroll
                for (int i = 0; i < 2; ++i)
#pragma unroll
                    for (int j = 0; j < 2; ++j)
                        acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x4f32(av[i][q], bv[j][q], acc[i][j], 0, 0, 0);
        } else {
            bf8v av[2], bv[2];
#pragma unroll
            for (int i = 0; i < 2; ++i) av[i] = *(const bf8v*)(As + (wm * 32 + i * 16 + rl) * LDK + kg * 8);
#pragma unroll
            for (int j = 0; j < 2; ++j) bv[j] = *(const bf8v*)(Bs + (wn * 32 + j * 16 + rl) * LDK + kg * 8);
#pragma unroll
            for (int i = 0; i < 2; ++i)
#pragma unroll
                for (int j = 0; j < 2; ++j)
                    acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(av[i], bv[j], acc[i][j], 0, 0, 0);
        }
        __syncthreads();
    }

    // epilogue: lane holds C rows 4*(lane/16)+r, column lane%16 of each 16x16 block
    float scale = g.lr;
    if (EPI == EPI_UPD && g.scale_per_batch) scale = valid > 0 ? g.lr / (float)valid : 0.f;
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j)
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                const int m = m0 + wm * 32 + i * 16 + (lane >> 4) * 4 + r;
                const int n = n0 + wn * 32 + j * 16 + (lane & 15);
                if (m >= Mv || n >= Nv) continue;
                const float v = acc[i][j][r];
                const size_t ci = (size_t)zz * g.c_z + (size_t)m * g.c_ld + n;
                if constexpr (EPI == EPI_STORE) {
                    ((float*)g.c)[ci + (size_t)slice * g.c_split] = v;
                } else if constexpr (EPI == EPI_FWD) {
                    const float zv = v + g.bias[(size_t)cn * g.bias_z + n];
                    ((TO*)g.c)[ci] = from_f<TO>(act_fn(g.act, zv));
                } else if constexpr (EPI == EPI_BWD) {
                    const float x = to_f<TO>(((const TO*)g.aux)[ci]);
                    ((TO*)g.c)[ci] = from_f<TO>(v * act_deriv(g.act, x));
                } else {  // EPI_UPD: in-place W -= scale * acc (master fp32)
                    float* W = (float*)g.c;
                    const float w = W[ci] - scale * v;
                    W[ci] = w;
                    if (g.shadow) g.shadow[ci] = f2bf(w);
                }
            }
    if (do_rowsum && tid < 64 && m0 + tid < Mv) {
        float* b = g.ubias + (size_t)cn * g.bias_z;
        b[m0 + tid] -= scale * rowsum[tid];
    }
}

// ------------------------------------------------------------------------------------
// Output layer, one wavefront per sample row: z = W x + b over <= 16 outputs, the output
// activation (eq. (3), softmax eq. (5)), then either the output error (training, eq. (9)
// or (10)) or the predicted class and the correct count (inference).

struct RowArgs {
    const void* x;  // input activations: xrows (data set) or workspace [z][rows][ld]
    int x_xrows;
    int64_t x_z, x_ld;
    const void* w;  // W_L [O][H] (+ z * w_z): fp32 master or bf16 shadow
    int64_t w_z;
    const float* bias;  // b_L (+ z * bias_z)
    int64_t bias_z;
    int H, O, act, loss;
    int64_t n_total;
    int k_rep;
    int64_t r0;
    int step_rows;
    const int32_t* y;  // labels (data-set rows)
    void* delta;       // training: [z][rows][O] output error (TD)
    int64_t d_z;
    float* out;        // inference: [rows][O] outputs (nullable)
    int32_t* pred;     // inference: [rows] argmax
    unsigned long long* correct;  // inference: count of pred == y (nullable)
};

template <typename TX, typename TW, typename TD, bool TRAIN>
__global__ __launch_bounds__(256) void out_layer_kernel(RowArgs a) {
    const int lane = threadIdx.x & 63;
    const int row = blockIdx.x * 4 + (threadIdx.x >> 6);
    const int z = blockIdx.z;
    int64_t v = shard_len(a.n_total, a.k_rep, z) - a.r0;
    const int valid = (int)(v < 0 ? 0 : (v > a.step_rows ? a.step_rows : v));
    if (row >= valid) return;
    const int64_t drow = shard_start(a.n_total, a.k_rep, z) + a.r0 + row;  // data-set row
    const TX* x = a.x_xrows ? (const TX*)a.x + (size_t)drow * a.x_ld
                            : (const TX*)a.x + (size_t)z * a.x_z + (size_t)row * a.x_ld;
    const TW* W = (const TW*)a.w + (size_t)z * a.w_z;
    float acc[MAX_OUT];
#pragma unroll
    for (int o = 0; o < MAX_OUT; ++o) acc[o] = 0.f;
    for (int i = lane; i < a.H; i += 64) {
        float xi = to_f<TX>(x[i]);
        if constexpr (sizeof(TW) == 2 && sizeof(TX) == 4) xi = bf2f(f2bf(xi));  // bf16 operand
#pragma unroll
        for (int o = 0; o < MAX_OUT; ++o)
            if (o < a.O) acc[o] += to_f<TW>(W[(size_t)o * a.H + i]) * xi;
    }
    const float* b = a.bias + (size_t)z * a.bias_z;
    float zo[MAX_OUT], xo[MAX_OUT];
#pragma unroll
    for (int o = 0; o < MAX_OUT; ++o) zo[o] = (o < a.O) ? wave_sum(acc[o]) + b[o] : 0.f;
    if (a.act == ACT_SOFTMAX) {
        float m = zo[0];
#pragma unroll
        for (int o = 1; o < MAX_OUT; ++o) if (o < a.O) m = fmaxf(m, zo[o]);
        float s = 0.f;
#pragma unroll
        for (int o = 0; o < MAX_OUT; ++o) { xo[o] = (o < a.O) ? expf(zo[o] - m) : 0.f; s += xo[o]; }
        const float inv = 1.0f / s;
#pragma unroll
        for (int o = 0; o < MAX_OUT; ++o) xo[o] *= inv;
    } else {
#pragma unroll
        for (int o = 0; o < MAX_OUT; ++o) xo[o] = act_fn(a.act, zo[o]);
    }
    if constexpr (TRAIN) {
        const int label = a.y[drow];
        TD* d = (TD*)a.delta + (size_t)z * a.d_z + (size_t)row * a.O;
        if (lane < a.O) {
            float xv = 0.f;
#pragma unroll
            for (int o = 0; o < MAX_OUT; ++o) if (o == lane) xv = xo[o];
            const float e = (lane == label) ? 1.0f : 0.0f;
            const float dv = (a.loss == LOSS_XENT) ? (xv - e) : (xv - e) * act_deriv(a.act, xv);
            d[lane] = from_f<TD>(dv);
        }
    } else {
        int best = 0;
        float bv = xo[0];
#pragma unroll
        for (int o = 1; o < MAX_OUT; ++o) if (o < a.O && xo[o] > bv) { bv = xo[o]; best = o; }
        if (lane == 0) {
            a.pred[drow] = best;
            if (a.correct && a.y && a.y[drow] == best) atomicAdd(a.correct, 1ull);
        }
        if (a.out && lane < a.O) {
            float xv = 0.f;
#pragma unroll
            for (int o = 0; o < MAX_OUT; ++o) if (o == lane) xv = xo[o];
            a.out[(size_t)drow * a.O + lane] = xv;
        }
    }
}

// ------------------------------------------------------------------------------------
// Hidden error behind a narrow layer (eq. (11)): d_l[r][i] = (sum_o d_{l+1}[r][o] W[o][i])
// * phi'(x_l[r][i]), for a next layer of <= 16 neurons.  Thread per (row, i).

struct BwdSmallArgs {
    const void* dnext;  // [z][rows][O]
    int64_t dn_z;
    const void* w;      // W_{l+1} [O][H] (+ z * w_z)
    int64_t w_z;
    const void* x;      // x_l [z][rows][H]
    void* d;            // d_l [z][rows][H]
    int64_t xz;         // z stride of x and d
    int H, O, act;
    int64_t n_total;
    int k_rep;
    int64_t r0;
    int step_rows;
};

template <typename TD, typename TW>
__global__ __launch_bounds__(256) void bwd_small_kernel(BwdSmallArgs a) {
    const int i = blockIdx.x * 256 + threadIdx.x;
    const int row = blockIdx.y, z = blockIdx.z;
    int64_t v = shard_len(a.n_total, a.k_rep, z) - a.r0;
    const int valid = (int)(v < 0 ? 0 : (v > a.step_rows ? a.step_rows : v));
    if (row >= valid || i >= a.H) return;
    const TD* dn = (const TD*)a.dnext + (size_t)z * a.dn_z + (size_t)row * a.O;
    const TW* W = (const TW*)a.w + (size_t)z * a.w_z;
    float s = 0.f;
    for (int o = 0; o < a.O; ++o) s += to_f<TD>(dn[o]) * to_f<TW>(W[(size_t)o * a.H + i]);
    const size_t xi = (size_t)z * a.xz + (size_t)row * a.H + i;
    const float x = to_f<TD>(((const TD*)a.x)[xi]);
    ((TD*)a.d)[xi] = from_f<TD>(s * act_deriv(a.act, x));
}

// ------------------------------------------------------------------------------------
// Update of a narrow layer (<= 16 neurons), eq. (12)-(13) averaged over the batch:
// W[o][i] -= lr / B_t * sum_r d[r][o] x[r][i];  b[o] -= lr / B_t * sum_r d[r][o].
// Thread per input column i, all outputs in registers.

struct UpdSmallArgs {
    const void* d;  // [z][rows][O]
    int64_t d_z;
    const void* x;  // previous activations: xrows (data set) or [z][rows][H]
    int x_xrows;
    int64_t x_z, x_ld;
    float* w;       // W [O][H] (+ z * w_z), fp32 master
    bf16_t* shadow; // nullable, same indexing as w
    float* bias;    // b [O] (+ z * bias_z)
    int64_t w_z, bias_z;
    int H, O;
    float lr;
    int64_t n_total;
    int k_rep;
    int64_t r0;
    int step_rows;
};

template <typename TD, typename TX>
__global__ __launch_bounds__(256) void upd_small_kernel(UpdSmallArgs a) {
    const int i = blockIdx.x * 256 + threadIdx.x;
    const int z = blockIdx.z;
    int64_t v = shard_len(a.n_total, a.k_rep, z) - a.r0;
    const int valid = (int)(v < 0 ? 0 : (v > a.step_rows ? a.step_rows : v));
    if (valid == 0) return;
    const float scale = a.lr / (float)valid;
    const TD* d = (const TD*)a.d + (size_t)z * a.d_z;
    const int64_t xb = shard_start(a.n_total, a.k_rep, z) + a.r0;
    if (i < a.H) {
        float acc[MAX_OUT];
#pragma unroll
        for (int o = 0; o < MAX_OUT; ++o) acc[o] = 0.f;
        for (int r = 0; r < valid; ++r) {
            const TX* xr = a.x_xrows ? (const TX*)a.x + (size_t)(xb + r) * a.x_ld
                                     : (const TX*)a.x + (size_t)z * a.x_z + (size_t)r * a.x_ld;
            float xv = to_f<TX>(xr[i]);
            if constexpr (sizeof(TD) == 2 && sizeof(TX) == 4) xv = bf2f(f2bf(xv));  // bf16 operand
#pragma unroll
            for (int o = 0; o < MAX_OUT; ++o)
                if (o < a.O) acc[o] += to_f<TD>(d[(size_t)r * a.O + o]) * xv;
        }
        float* W = a.w + (size_t)z * a.w_z;
#pragma unroll
        for (int o = 0; o < MAX_OUT; ++o)
            if (o < a.O) {
                const size_t wi = (size_t)o * a.H + i;
                const float w = W[wi] - scale * acc[o];
                W[wi] = w;
                if (a.shadow) a.shadow[(size_t)z * a.w_z + wi] = f2bf(w);
            }
    }
    if (blockIdx.x == 0 && threadIdx.x < a.O) {
        const int o = threadIdx.x;
        float s = 0.f;
        for (int r = 0; r < valid; ++r) s += to_f<TD>(d[(size_t)r * a.O + o]);
        a.bias[(size_t)z * a.bias_z + o] -= scale * s;
    }
}

// ------------------------------------------------------------------------------------
// Combination by averaging: merged[p] = (sum_k theta_k[p]) / K with the sum in fp64 and k
// ascending; optionally broadcast back to every CN; bf16 shadows refreshed.  Four
// consecutive parameters per thread.

struct MergeArgs {
    float* theta;       // [K][pstride]
    float* merged;      // [pstride]
    bf16_t* shadow;     // [K][pstride] or null
    bf16_t* mshadow;    // [pstride] or null
    int64_t pstride;    // multiple of 4
    int K;
    int broadcast;
};

__global__ __launch_bounds__(256) void merge_kernel(MergeArgs a) {
    const int64_t p = ((int64_t)blockIdx.x * 256 + threadIdx.x) * 4;
    if (p >= a.pstride) return;
    double s0 = 0.0, s1 = 0.0, s2 = 0.0, s3 = 0.0;
    for (int k = 0; k < a.K; ++k) {
        const float4 v = *(const float4*)(a.theta + (size_t)k * a.pstride + p);
        s0 += (double)v.x; s1 += (double)v.y; s2 += (double)v.z; s3 += (double)v.w;
    }
    const double inv = (double)a.K;
    const float4 m = make_float4((float)(s0 / inv), (float)(s1 / inv), (float)(s2 / inv), (float)(s3 / inv));
    *(float4*)(a.merged + p) = m;
    if (a.mshadow) {
        a.mshadow[p] = f2bf(m.x); a.mshadow[p + 1] = f2bf(m.y); a.mshadow[p + 2] = f2bf(m.z); a.mshadow[p + 3] = f2bf(m.w);
    }
    if (a.broadcast) {
        for (int k = 0; k < a.K; ++k) {
            *(float4*)(a.theta + (size_t)k * a.pstride + p) = m;
            if (a.shadow) {
                bf16_t* s = a.shadow + (size_t)k * a.pstride + p;
                s[0] = f2bf(m.x); s[1] = f2bf(m.y); s[2] = f2bf(m.z); s[3] = f2bf(m.w);
            }
        }
    }
}

// fp32 -> bf16 copy of a whole parameter block (shadow refresh after init / set)
__global__ __launch_bounds__(256) void to_bf16_kernel(const float* src, bf16_t* dst, int64_t n) {
    const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (i < n) dst[i] = f2bf(src[i]);
}

// ------------------------------------------------------------------------------------
// Per-sample stochastic gradient descent of a one-hidden-layer network, chunked.
//
// Within a chunk of T consecutive samples t of one CN, the first-layer weights evolve as
// W1_t = W1_c - eta * sum_{s<t} d1_s x_s^T (W1_c: weights at the chunk start), so the
// first-layer input sum is exactly
//     z1_t = W1_t x_t + b1_t = P[t] + b1_t - eta * sum_{s<t} d1_s (x_s . x_t)
// with P[t] = W1_c x_t and the Gram matrix G[t][s] = x_s . x_t computed on the matrix
// cores beforehand.  This kernel runs the T sequential steps of one CN per workgroup:
// the small second layer (W2, b2) and b1 are updated in registers after every sample,
// exactly as eq. (12)-(13) prescribe, and the first-layer errors d1_t are written out so
// that the rank-T update of W1 (= the T rank-1 updates summed) is one more GEMM.
// Thread h owns hidden neuron h and column h of W2.

struct PsgdArgs {
    float* theta;         // [K][pstride]
    int64_t pstride, off_b1, off_w2, off_b2;
    const float* ppart;   // split partial sums of P: [ksplit][K][T][H]
    int ksplit;
    int64_t ppart_split;  // elements between splits
    const float* gram;    // [K][nch][T][T]
    int nch, c;           // number of chunks, this chunk
    const int32_t* y;     // data-set labels
    float* d1;            // out: [K][T][H]
    int64_t n_total;
    int k_rep;
    int H, O, act1, act2, loss;
    float lr;
};

template <int T>
__global__ __launch_bounds__(1024) void psgd_chunk_kernel(PsgdArgs a) {
    extern __shared__ float smem[];
    const int z = blockIdx.x;
    const int h = threadIdx.x, lane = h & 63, wave = h >> 6, nwaves = blockDim.x >> 6;
    const bool live = h < a.H;
    const int64_t nz = shard_len(a.n_total, a.k_rep, z);
    const int64_t r0 = (int64_t)a.c * T;
    const int tc = (int)(nz - r0 < 0 ? 0 : (nz - r0 > T ? T : nz - r0));
    if (tc == 0) return;
    const int H = a.H, O = a.O;
    float* Pl = smem;                       // [T][H]
    float* hist = smem + T * H;             // [T][H]
    float* red = smem + 2 * T * H;          // [2][16 waves][MAX_OUT]

    // sum the split partials of P = W1_c x_t
    for (int idx = threadIdx.x; idx < tc * H; idx += blockDim.x) {
        const int t = idx / H, hh = idx % H;
        float s = 0.f;
        for (int sp = 0; sp < a.ksplit; ++sp)
            s += a.ppart[(size_t)sp * a.ppart_split + ((size_t)z * T + t) * H + hh];
        Pl[t * H + hh] = s;
    }
    __syncthreads();

    float* th = a.theta + (size_t)z * a.pstride;
    float b1 = live ? th[a.off_b1 + h] : 0.f;
    float w2[MAX_OUT], b2[MAX_OUT];
#pragma unroll
    for (int o = 0; o < MAX_OUT; ++o) {
        w2[o] = (live && o < O) ? th[a.off_w2 + (size_t)o * H + h] : 0.f;
        b2[o] = (o < O) ? th[a.off_b2 + o] : 0.f;
    }
    const float* G = a.gram + ((size_t)z * a.nch + a.c) * T * T;
    const int32_t* y = a.y + shard_start(a.n_total, a.k_rep, z) + r0;
    float* dout = a.d1 + (size_t)z * T * H;
    const float lr = a.lr;

    for (int t = 0; t < tc; ++t) {
        float a1 = 0.f;
        if (live) {
            float corr = 0.f;
            const float* Gt = G + (size_t)t * T;
            for (int s = 0; s < t; ++s) corr += hist[s * H + h] * Gt[s];
            const float z1 = Pl[t * H + h] + b1 - lr * corr;
            a1 = act_fn(a.act1, z1);
        }
        float zo[MAX_OUT];
#pragma unroll
        for (int o = 0; o < MAX_OUT; ++o) zo[o] = wave_sum(w2[o] * a1);
        float* rb = red + (t & 1) * 16 * MAX_OUT;
        if (lane == 0) {
#pragma unroll
            for (int o = 0; o < MAX_OUT; ++o) rb[wave * MAX_OUT + o] = zo[o];
        }
        __syncthreads();
#pragma unroll
        for (int o = 0; o < MAX_OUT; ++o) {
            float s = 0.f;
            for (int w = 0; w < nwaves; ++w) s += rb[w * MAX_OUT + o];
            zo[o] = s + b2[o];
        }
        // output activation and error (eq. (3), (5), (9), (10))
        float xo[MAX_OUT];
        if (a.act2 == ACT_SOFTMAX) {
            float m = zo[0];
#pragma unroll
            for (int o = 1; o < MAX_OUT; ++o) if (o < O) m = fmaxf(m, zo[o]);
            float s = 0.f;
#pragma unroll
            for (int o = 0; o < MAX_OUT; ++o) { xo[o] = (o < O) ? expf(zo[o] - m) : 0.f; s += xo[o]; }
            const float inv = 1.0f / s;
#pragma unroll
            for (int o = 0; o < MAX_OUT; ++o) xo[o] *= inv;
        } else {
#pragma unroll
            for (int o = 0; o < MAX_OUT; ++o) xo[o] = act_fn(a.act2, zo[o]);
        }
        const int label = y[t];
        float d2[MAX_OUT];
#pragma unroll
        for (int o = 0; o < MAX_OUT; ++o) {
            const float e = (o == label) ? 1.0f : 0.0f;
            d2[o] = (o < O) ? ((a.loss == LOSS_XENT) ? (xo[o] - e) : (xo[o] - e) * act_deriv(a.act2, xo[o])) : 0.f;
        }
        // hidden error with the pre-update W2 (eq. (11)), then the updates (eq. (12)-(13))
        float back = 0.f;
#pragma unroll
        for (int o = 0; o < MAX_OUT; ++o) back += w2[o] * d2[o];
        const float d1 = live ? back * act_deriv(a.act1, a1) : 0.f;
#pragma unroll
        for (int o = 0; o < MAX_OUT; ++o) {
            w2[o] -= lr * d2[o] * a1;
            b2[o] -= lr * d2[o];
        }
        if (live) {
            b1 -= lr * d1;
            hist[t * H + h] = d1;
            dout[(size_t)t * H + h] = d1;
        }
    }
    if (live) {
        th[a.off_b1 + h] = b1;
        for (int o = 0; o < O; ++o) th[a.off_w2 + (size_t)o * H + h] = w2[o];
    }
    if (h == 0)
        for (int o = 0; o < O; ++o) th[a.off_b2 + o] = b2[o];
}

}  // namespace pnn

namespace pnn {

// ------------------------------------------------------------------------------------
// Cross-lane helpers (DPP, within rows of 16 lanes)

template <int CTRL>
__device__ inline float dpp(float v) {
    return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), CTRL, 0xf, 0xf, true));
}
constexpr int DPP_ROW_MIRROR = 0x140;       // lane i <-> 15 - i
constexpr int DPP_ROW_HALF_MIRROR = 0x141;  // lane i <-> 7 - i within each half row
constexpr int DPP_XOR2 = 0x4E;              // quad_perm [2,3,0,1]
constexpr int DPP_XOR1 = 0xB1;              // quad_perm [1,0,3,2]

// Reduce-scatter of 16 values over each row of 16 lanes: afterwards lane i of a row holds
// the row's sum of v[i & 15].  Four pairing rounds; every pair of partners agrees on the
// lane bits split so far and differs in the bit split now.
__device__ inline float row_reduce_scatter16(const float (&v)[16], int lane) {
    const bool b3 = lane & 8, b2 = lane & 4, b1 = lane & 2, b0 = lane & 1;
    float a[8], b[4], c[2];
#pragma unroll
    for (int j = 0; j < 8; ++j) {
        const float send = b3 ? v[j] : v[j + 8], keep = b3 ? v[j + 8] : v[j];
        a[j] = keep + dpp<DPP_ROW_MIRROR>(send);
    }
#pragma unroll
    for (int j = 0; j < 4; ++j) {
        const float send = b2 ? a[j] : a[j + 4], keep = b2 ? a[j + 4] : a[j];
        b[j] = keep + dpp<DPP_ROW_HALF_MIRROR>(send);
    }
#pragma unroll
    for (int j = 0; j < 2; ++j) {
        const float send = b1 ? b[j] : b[j + 2], keep = b1 ? b[j + 2] : b[j];
        c[j] = keep + dpp<DPP_XOR2>(send);
    }
    const float send = b0 ? c[0] : c[1], keep = b0 ? c[1] : c[0];
    return keep + dpp<DPP_XOR1>(send);
}
__device__ inline float row_allmax16(float v) {
    v = fmaxf(v, dpp<DPP_ROW_MIRROR>(v));
    v = fmaxf(v, dpp<DPP_ROW_HALF_MIRROR>(v));
    v = fmaxf(v, dpp<DPP_XOR2>(v));
    return fmaxf(v, dpp<DPP_XOR1>(v));
}
__device__ inline float row_allsum16(float v) {
    v += dpp<DPP_ROW_MIRROR>(v);
    v += dpp<DPP_ROW_HALF_MIRROR>(v);
    v += dpp<DPP_XOR2>(v);
    return v + dpp<DPP_XOR1>(v);
}
__device__ inline float readlane_f(float v, int l) { return __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), l)); }

// Activations of the sequential per-sample steps, on the hardware exp2 and reciprocal
// (about 1e-6 relative error for |z| < 10).
__device__ inline float act_fast(int a, float z) {
    switch (a) {
    case ACT_SIGMOID: return __builtin_amdgcn_rcpf(1.0f + __expf(-z));
    case ACT_TANH: return 1.0f - 2.0f * __builtin_amdgcn_rcpf(__expf(2.0f * z) + 1.0f);
    case ACT_RELU: return z >= 0.0f ? z + 0.0f : -0.0f;
    case ACT_LEAKY: return z >= 0.0f ? z + 0.0f : 0.01f * z;
    default: return z;
    }
}

// ------------------------------------------------------------------------------------
// Bounded cross-workgroup waits (device-scope release/acquire on a counter in global
// memory).  Thread 0 polls; on expiry of `limit` polls, or when another workgroup has
// raised the abort flag, every thread gets `false` and the caller leaves its loop, so the
// grid always drains.

__device__ inline bool wait_geq(int* flag, int target, int* abort, long limit) {
    __shared__ int ok;
    if (threadIdx.x == 0) {
        int good = 1;
        long it = 0;
        // relaxed polls (coherent loads, no cache maintenance); one acquire fence afterwards
        while (__hip_atomic_load(flag, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) < target) {
            if (__hip_atomic_load(abort, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT)) { good = 0; break; }
            if (++it > limit) {
                __hip_atomic_store(abort, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                good = 0;
                break;
            }
            __builtin_amdgcn_s_sleep(1);
        }
        ok = good;
    }
    __syncthreads();
    const bool r = __builtin_amdgcn_readfirstlane(ok) != 0;  // uniform: keeps later control flow scalar
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "agent");
    __syncthreads();
    return r;
}

// The workgroup barrier makes every wave's stores complete; thread 0's release fence then
// publishes them before the flag update.
__device__ inline void signal_add(int* flag, int v) {
    __syncthreads();
    if (threadIdx.x == 0) {
        __builtin_amdgcn_fence(__ATOMIC_RELEASE, "agent");
        __hip_atomic_fetch_add(flag, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
}
__device__ inline void signal_set(int* flag, int v) {
    __syncthreads();
    if (threadIdx.x == 0) {
        __builtin_amdgcn_fence(__ATOMIC_RELEASE, "agent");
        __hip_atomic_store(flag, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
}

// ------------------------------------------------------------------------------------
// Per-sample stochastic gradient descent of a one-hidden-layer fp32 network: one
// persistent launch per epoch.
//
// Chunked form of the sequential steps (see psgd_chunk_kernel).  With W1^(c) the
// first-layer weights before chunk c, the first-layer input sum of step t of chunk c is
//   z1_t = Q_c[t] + b1_t - eta * ( sum_{s in chunk c-1} d1_s GX_c[t][s]
//                                 + sum_{s < t in chunk c} d1_s G_c[t][s] )
// where Q_c[t] = W1^(c-1) x_t (for c = 0: W1^(0) x_t), G_c[t][s] = x_t . x_s within the
// chunk and GX_c[t][s] = x_t . x_s against the previous chunk.  Q_c therefore needs the
// first-layer errors only up to chunk c-2, and is computed while chunk c-1 runs.
//
// Grid (cooperative, all workgroups co-resident, 256 threads each):
//   blockIdx < K: the sequential workgroup of CN k.  Waves 0..HW/64-1 own one hidden
//     neuron per lane (W2 column and b1 in registers); the other "helper" waves compute,
//     one step ahead, the already-known part (s <= t-2) of the next step's in-chunk
//     correction.  At chunk start all four waves compute the previous-chunk correction on
//     the matrix cores.
//   blockIdx >= K: tile workgroups.  Tile (k, rb) keeps W1[16 rows][all inputs] of CN k in
//     registers for the epoch, laid out as the B operand of v_mfma_f32_16x16x4_f32 (lane l:
//     row 16 rb + l % 16, inputs 16 ib + 4 (l / 16) + q).  It publishes Q_0 and Q_1, then for
//     each later chunk waits for the previous chunk's errors, applies
//     W1 -= eta * sum_t d1_t x_t^T (a product whose accumulator layout equals the register
//     layout) and publishes the next Q.

struct PsgdPArgs {
    float* theta;
    int64_t pstride, off_w1, off_b1, off_w2, off_b2;
    const float* X;
    const int32_t* y;
    int64_t n_total;
    int k_rep;
    const float* gram;   // [K][nch][T][T]   within each chunk
    const float* gramx;  // [K][nch-1][T][T] chunk c (rows) against chunk c-1, c >= 1
    int nch;
    float* qbuf;         // [2][K][T][H]  by chunk parity
    float* d1;           // [2][K][H][T]  by chunk parity (transposed: one row per hidden neuron)
    int* flags;          // qready[K], dready[K], abort
    int H, O, In, act1, act2, loss, nrb;
    float lr;
    long spin_limit;
};

constexpr int MAX_IB = 13;  // input blocks of 16 per wave of a tile (4 waves x 13 x 16 >= 784)

// Wave-level bounded wait (no workgroup barrier inside): every lane polls the same flag.
__device__ inline bool wave_wait_geq(int* flag, int target, int* abort, long limit) {
    long it = 0;
    while (__hip_atomic_load(flag, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) < target) {
        if (__hip_atomic_load(abort, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT)) return false;
        if (++it > limit) {
            __hip_atomic_store(abort, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            return false;
        }
        __builtin_amdgcn_s_sleep(1);
    }
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "agent");
    return true;
}

typedef __attribute__((address_space(3))) void lds_void;

// One wave copies `bytes` (a multiple of 1 KiB) from global memory straight into LDS, in
// 1 KiB pieces piece0, piece0 + stride, ...; completion is tracked by the wave's vmcnt.
__device__ inline void wave_copy_to_lds(const void* src, float* dst_lds, int bytes, int piece0, int stride, int lane) {
    for (int pc = piece0; pc * 1024 < bytes; pc += stride)
        __builtin_amdgcn_global_load_lds((const char*)src + pc * 1024 + lane * 16,
                                         (lds_void*)((char*)dst_lds + pc * 1024), 16, 0, 0);
}
__device__ inline void wait_vm_all() { __builtin_amdgcn_s_waitcnt(0x0F70); }  // vmcnt(0)

template <int T, int HW, int A1, int A2, int LS, int OC>
__device__ __attribute__((always_inline)) inline void psgd_rec(const PsgdPArgs& a, int k, float* smem) {
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int H = a.H, K = a.k_rep;
    const int O = OC < 16 ? OC : a.O;
    const int act1 = A1 >= 0 ? A1 : a.act1;
    const int act2 = A2 >= 0 ? A2 : a.act2;
    const int loss = LS >= 0 ? LS : a.loss;
    constexpr int nlive = HW >> 6;
    constexpr int nhelp = 4 - nlive;  // helper waves
    const bool live = tid < HW;
    const int h = live ? tid : (tid - HW) % HW;
    const int part = live ? 0 : (tid - HW) / HW;
    const int hwave = wave - nlive;  // helper wave index (valid for helpers)
    const bool hv = h < H;
    constexpr int TS = T + 4;  // row stride of the transposed error history
    float* Pl = smem;                    // [T][HW]   input sums of the current chunk
    float* Qn = Pl + T * HW;             // [T][H]    next chunk's Q (prefetched)
    float* hist = Qn + T * HW;           // [HW][TS]  first-layer errors of the current chunk
    constexpr int GS = T + 4;            // Gram row stride: rows 4 banks apart (conflict-free MFMA operand reads)
    float* Gb = hist + HW * TS;          // [2][T][GS] Gram blocks by chunk parity
    float* GXn = Gb + 2 * T * GS;        // [T][GS]    next chunk against the current one
    float* red = GXn + T * GS;           // [2][16 outputs][16 rows]
    float* cpre = red + 2 * 256;         // [2][HW]
    int* yb = (int*)(cpre + 2 * HW);     // [2][T] labels by chunk parity

    const int64_t nz = shard_len(a.n_total, K, k), xs = shard_start(a.n_total, K, k);
    const int nchk = (int)((nz + T - 1) / T);
    float* th = a.theta + (size_t)k * a.pstride;
    float b1 = (live && hv) ? th[a.off_b1 + h] : 0.f;
    float w2[OC];
#pragma unroll
    for (int o = 0; o < OC; ++o) w2[o] = (live && hv && o < O) ? th[a.off_w2 + (size_t)o * H + h] : 0.f;
    const int ol = lane & 15;
    float b2v = (ol < O) ? th[a.off_b2 + ol] : 0.f;
    int* qready = a.flags + k;
    int* dready = a.flags + K + k;
    int* abort = a.flags + 2 * K;
    const float lr = a.lr;
    // padding neurons h >= H read zero errors and zero input sums
    for (int i = tid; i < HW * TS; i += 256) hist[i] = 0.f;
    for (int i = tid; i < T * HW; i += 256) Pl[i] = 0.f;

    // chunk 0: wait for Q_0 and stage it synchronously
    if (!wait_geq(qready, a.nrb, abort, a.spin_limit)) return;
    {
        const float* Q = a.qbuf + (size_t)k * T * H;
        const float* G = a.gram + (size_t)k * a.nch * T * GS;
        const int tc0 = (int)min<int64_t>(T, nz);
        for (int idx = tid; idx < tc0 * H; idx += 256) Pl[(idx / H) * HW + idx % H] = Q[idx];
        for (int idx = tid; idx < T * GS; idx += 256) Gb[idx] = G[idx];
        for (int idx = tid; idx < tc0; idx += 256) yb[idx] = a.y[xs + idx];
    }
    __syncthreads();

    // helper-side prefetch state for chunk c + 1
    bool issued = false;  // this helper wave issued its copies for the next chunk
    int qseen = 0;        // last value read from qready (a load in flight one step)
    for (int c = 0; c < nchk; ++c) {
        const int tc = __builtin_amdgcn_readfirstlane((int)min<int64_t>(T, nz - (int64_t)c * T));
        const float* Gl = Gb + (c & 1) * T * GS;
        const int* ylds = yb + (c & 1) * T;
        const bool has_next = c + 1 < nchk;
        const int tcn = has_next ? (int)min<int64_t>(T, nz - (int64_t)(c + 1) * T) : 0;
        // copies of chunk c + 1's inputs, issued by the helper waves as soon as the tiles
        // have published its Q (or synchronously at the chunk end)
        auto issue_next = [&]() {
            const float* Q = a.qbuf + ((size_t)((c + 1) & 1) * K + k) * T * H;
            const float* G = a.gram + ((size_t)k * a.nch + c + 1) * T * GS;
            const float* GX = a.gramx + ((size_t)k * (a.nch - 1) + c) * T * GS;
            wave_copy_to_lds(Q, Qn, T * H * 4, hwave, nhelp, lane);
            wave_copy_to_lds(G, Gb + ((c + 1) & 1) * T * GS, T * GS * 4, hwave, nhelp, lane);
            wave_copy_to_lds(GX, GXn, T * GS * 4, hwave, nhelp, lane);
            if (hwave == 0) {  // labels: one dword per lane, rows clamped into the slice
                const int r = min(lane, tcn - 1);
                __builtin_amdgcn_global_load_lds(a.y + xs + (int64_t)(c + 1) * T + r,
                                                 (lds_void*)(yb + ((c + 1) & 1) * T), 4, 0, 0);
            }
        };
        const int sig_step = min(4, tc - 1);  // step after which the previous chunk's errors are announced

        // Steps in blocks of 16.  At the start of block b the errors of block b-1 are folded
        // into the input sums of every later row of the chunk on the matrix cores, so a
        // step's in-chunk correction only needs the earlier steps of its own block.
        float corr = 0.f, dprev = 0.f;
        float pl_next = live ? Pl[h] : 0.f;
        for (int tt = 0; tt < tc; ++tt) {
            // the step index is read through readfirstlane so that it stays a scalar (the
            // live/helper branches below are divergent)
            const int t = __builtin_amdgcn_readfirstlane(tt);
            const int bs = t & ~15;  // first step of this block
            if (t > 0 && t == bs) {
                __syncthreads();  // errors of the finished block are in LDS
                const int sb = bs - 16;
                const int nmt = (T - bs) >> 4, ntl = nmt * (HW / 16);
                const int r16 = lane & 15, g = lane >> 4;
                for (int ti = wave; ti < ntl; ti += 4) {
                    const int mt = (bs >> 4) + ti % nmt, nt = ti / nmt;
                    const float4 av = *(const float4*)(Gl + (mt * 16 + r16) * GS + sb + 4 * g);
                    const float4 bv = *(const float4*)(hist + (nt * 16 + r16) * TS + sb + 4 * g);
                    f4 acc = {0.f, 0.f, 0.f, 0.f};
                    acc = __builtin_amdgcn_mfma_f32_16x16x4f32(av.x, bv.x, acc, 0, 0, 0);
                    acc = __builtin_amdgcn_mfma_f32_16x16x4f32(av.y, bv.y, acc, 0, 0, 0);
                    acc = __builtin_amdgcn_mfma_f32_16x16x4f32(av.z, bv.z, acc, 0, 0, 0);
                    acc = __builtin_amdgcn_mfma_f32_16x16x4f32(av.w, bv.w, acc, 0, 0, 0);
#pragma unroll
                    for (int r = 0; r < 4; ++r) Pl[(mt * 16 + 4 * g + r) * HW + nt * 16 + r16] -= lr * acc[r];
                }
                __syncthreads();
                pl_next = live ? Pl[t * HW + h] : 0.f;
            }
            float a1 = 0.f;
            if (live) {
                const float z1 = pl_next + b1 - lr * corr;
                pl_next = (t + 1 < tc) ? Pl[(t + 1) * HW + h] : 0.f;  // prefetch the next step's input sum
                a1 = hv ? act_fast(act1, z1) : 0.f;
                float p[16];
#pragma unroll
                for (int o = 0; o < 16; ++o) p[o] = o < OC ? w2[o < OC ? o : 0] * a1 : 0.f;
                const float v = row_reduce_scatter16(p, lane);
                red[(t & 1) * 256 + ol * 16 + wave * 4 + (lane >> 4)] = v;
            } else {
                if (part == 0 && hv) {
                    // in-block part of the next step's correction, sum over s in [bs1, t-2]
                    // of d1_s G[t+1][s] (at most 14 terms: four masked float4 groups)
                    const int t1 = t + 1, bs1 = t1 & ~15;
                    float sum = 0.f;
                    if (t1 < tc && t - 2 >= bs1) {
                        const float* g = Gl + t1 * GS + bs1;
                        const float* hr = hist + h * TS + bs1;
                        const int last = t - 2 - bs1;  // highest offset included
                        float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
#pragma unroll
                        for (int q = 0; q < 4; ++q) {
                            if (4 * q <= last) {
                                const float4 hv4 = *(const float4*)(hr + 4 * q), gv4 = *(const float4*)(g + 4 * q);
                                acc.x += hv4.x * gv4.x;
                                acc.y += (4 * q + 1 <= last) ? hv4.y * gv4.y : 0.f;
                                acc.z += (4 * q + 2 <= last) ? hv4.z * gv4.z : 0.f;
                                acc.w += (4 * q + 3 <= last) ? hv4.w * gv4.w : 0.f;
                            }
                        }
                        sum = (acc.x + acc.y) + (acc.z + acc.w);
                    }
                    cpre[((t + 1) & 1) * HW + h] = sum;
                }
                // prefetch of the next chunk: the flag value read last step decides
                if (has_next && !issued) {
                    if (__builtin_amdgcn_readfirstlane(qseen) >= a.nrb * (c + 2)) {
                        __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "agent");
                        issue_next();
                        issued = true;
                    } else {
                        qseen = __hip_atomic_load(qready, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                    }
                }
                // the previous chunk's errors (stored at the chunk start) are announced once
                // every helper wave's stores have completed
                if (c > 0 && t == sig_step) wait_vm_all();
            }
            __syncthreads();
            if (c > 0 && t == sig_step && tid == HW) {
                __builtin_amdgcn_fence(__ATOMIC_RELEASE, "agent");
                __hip_atomic_store(dready, c, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            }
            if (live) {
                // every operand of this phase is read up front
                const float4* rr = (const float4*)(red + (t & 1) * 256 + ol * 16);
                const float4 r0 = rr[0];
                const float4 r1 = nlive > 1 ? rr[1] : make_float4(0.f, 0.f, 0.f, 0.f);
                const int label = ylds[t];
                float cp = 0.f, g0 = 0.f, g1 = 0.f;
                const int bs1 = (t + 1) & ~15;
                if (t + 1 < tc) {
                    cp = cpre[((t + 1) & 1) * HW + h];
                    const float* g = Gl + (t + 1) * GS;
                    g1 = t >= bs1 ? g[t] : 0.f;
                    g0 = t - 1 >= bs1 ? g[t - 1] : 0.f;
                }
                const float z2 = b2v + ((r0.x + r0.y) + (r0.z + r0.w)) + ((r1.x + r1.y) + (r1.z + r1.w));
                float x2;
                if (act2 == ACT_SOFTMAX) {
                    const float m = row_allmax16(ol < O ? z2 : -INFINITY);
                    const float e = ol < O ? __expf(z2 - m) : 0.f;
                    x2 = e * __builtin_amdgcn_rcpf(row_allsum16(e));
                } else {
                    x2 = act_fast(act2, z2);
                }
                const float e = (ol == label) ? 1.0f : 0.0f;
                float d2 = (loss == LOSS_XENT) ? (x2 - e) : (x2 - e) * act_deriv(act2, x2);
                d2 = ol < O ? d2 : 0.f;
                b2v -= lr * d2;
                float bk[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
                for (int o = 0; o < OC; ++o) {
                    const float d2o = readlane_f(d2, o);
                    bk[o & 3] += w2[o] * d2o;
                    w2[o] -= (lr * d2o) * a1;
                }
                const float back = (bk[0] + bk[1]) + (bk[2] + bk[3]);
                const float d1 = hv ? back * act_deriv(act1, a1) : 0.f;
                b1 -= lr * d1;
                hist[h * TS + t] = d1;
                corr = cp + dprev * g0 + d1 * g1;
                dprev = d1;
            }
        }

        float* dout = a.d1 + ((size_t)(c & 1) * K + k) * T * H;
        if (has_next) {
            // chunk boundary: make sure the next chunk's inputs are in LDS
            if (!live) {
                if (!issued) {
                    if (wave_wait_geq(qready, a.nrb * (c + 2), abort, a.spin_limit)) issue_next();
                }
                wait_vm_all();
                issued = false;
                qseen = 0;
            }
            __syncthreads();
            // previous-chunk correction on the matrix cores, written with the prefetched Q:
            // Pl[t][h] = Q[t][h] - eta * sum_s GX[t][s] d1_s[h]; two output tiles per pass so
            // that two independent accumulation chains share the matrix core
            {
                constexpr int ntiles = (T / 16) * (HW / 16);
                const int r16 = lane & 15, g = lane >> 4;
                for (int ti = wave; ti < ntiles; ti += 8) {
                    const int tj = ti + 4;
                    const bool two = tj < ntiles;
                    const int mt0 = ti % (T / 16), nt0 = ti / (T / 16);
                    const int mt1 = tj % (T / 16), nt1 = (two ? tj : ti) / (T / 16);
                    f4 acc0 = {0.f, 0.f, 0.f, 0.f}, acc1 = {0.f, 0.f, 0.f, 0.f};
                    float4 av0[T / 16], bv0[T / 16], av1[T / 16], bv1[T / 16];
#pragma unroll
                    for (int sl = 0; sl < T / 16; ++sl) {
                        av0[sl] = *(const float4*)(GXn + (mt0 * 16 + r16) * GS + sl * 16 + 4 * g);
                        bv0[sl] = *(const float4*)(hist + (nt0 * 16 + r16) * TS + sl * 16 + 4 * g);
                        av1[sl] = *(const float4*)(GXn + ((two ? mt1 : mt0) * 16 + r16) * GS + sl * 16 + 4 * g);
                        bv1[sl] = *(const float4*)(hist + (nt1 * 16 + r16) * TS + sl * 16 + 4 * g);
                    }
#pragma unroll
                    for (int sl = 0; sl < T / 16; ++sl) {
                        acc0 = __builtin_amdgcn_mfma_f32_16x16x4f32(av0[sl].x, bv0[sl].x, acc0, 0, 0, 0);
                        acc1 = __builtin_amdgcn_mfma_f32_16x16x4f32(av1[sl].x, bv1[sl].x, acc1, 0, 0, 0);
                        acc0 = __builtin_amdgcn_mfma_f32_16x16x4f32(av0[sl].y, bv0[sl].y, acc0, 0, 0, 0);
                        acc1 = __builtin_amdgcn_mfma_f32_16x16x4f32(av1[sl].y, bv1[sl].y, acc1, 0, 0, 0);
                        acc0 = __builtin_amdgcn_mfma_f32_16x16x4f32(av0[sl].z, bv0[sl].z, acc0, 0, 0, 0);
                        acc1 = __builtin_amdgcn_mfma_f32_16x16x4f32(av1[sl].z, bv1[sl].z, acc1, 0, 0, 0);
                        acc0 = __builtin_amdgcn_mfma_f32_16x16x4f32(av0[sl].w, bv0[sl].w, acc0, 0, 0, 0);
                        acc1 = __builtin_amdgcn_mfma_f32_16x16x4f32(av1[sl].w, bv1[sl].w, acc1, 0, 0, 0);
                    }
#pragma unroll
                    for (int r = 0; r < 4; ++r) {
                        const int t0 = mt0 * 16 + 4 * g + r, h0 = nt0 * 16 + r16;
                        Pl[t0 * HW + h0] = (h0 < H && t0 < tcn ? Qn[t0 * H + h0] : 0.f) - lr * acc0[r];
                        if (two) {
                            const int t1 = mt1 * 16 + 4 * g + r, h1 = nt1 * 16 + r16;
                            Pl[t1 * HW + h1] = (h1 < H && t1 < tcn ? Qn[t1 * H + h1] : 0.f) - lr * acc1[r];
                        }
                    }
                }
            }
            // the helpers store this chunk's errors for the tiles (announced a few steps into
            // the next chunk, once the stores have completed)
            if (!live) {
                // errors published as [h][T] rows, the layout of the LDS history
                constexpr int NH = 256 - HW;
                for (int q = tid - HW; q < H * (T / 4); q += NH) {
                    const int hh = q / (T / 4), t4 = (q % (T / 4)) * 4;
                    *(float4*)(dout + (size_t)hh * T + t4) = *(const float4*)(hist + hh * TS + t4);
                }
            }
            __syncthreads();
        } else {
            // last chunk: publish synchronously
            __syncthreads();
            for (int q = tid; q < H * (T / 4); q += 256) {
                const int hh = q / (T / 4), t4 = (q % (T / 4)) * 4;
                *(float4*)(dout + (size_t)hh * T + t4) = *(const float4*)(hist + hh * TS + t4);
            }
            signal_set(dready, c + 1);
        }
    }
    if (live && hv) {
        th[a.off_b1 + h] = b1;
#pragma unroll
        for (int o = 0; o < OC; ++o)
            if (o < O) th[a.off_w2 + (size_t)o * H + h] = w2[o];
    }
    if (tid < O) th[a.off_b2 + tid] = b2v;
}

template <int T>
__device__ __attribute__((always_inline)) inline void psgd_tile(const PsgdPArgs& a, int k, int rb, float* smem) {
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int H = a.H, In = a.In, K = a.k_rep;
    const int h = rb * 16 + (lane & 15);
    const int g = lane >> 4;
    const int nib = (In + 15) / 16;  // input blocks of 16; wave w owns blocks w, w+4, ...
    float* th = a.theta + (size_t)k * a.pstride;
    float W[MAX_IB][4];
#pragma unroll
    for (int j = 0; j < MAX_IB; ++j)
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            const int ib = wave + 4 * j, i = ib * 16 + 4 * g + q;
            W[j][q] = (ib < nib && h < H && i < In) ? th[a.off_w1 + (size_t)h * In + i] : 0.f;
        }
    const int64_t nz = shard_len(a.n_total, K, k), xs = shard_start(a.n_total, K, k);
    const int nchk = (int)((nz + T - 1) / T);
    int* qready = a.flags + k;
    int* dready = a.flags + K + k;
    int* abort = a.flags + 2 * K;
    constexpr int NMT = T / 16;
    float* red4 = smem;  // [4 waves][NMT][64][4]

    // Q_c = W1 (current registers) x_t for the rows of chunk c, published to qbuf[c & 1].
    // Out-of-range rows and inputs are read from a clamped (valid) address and masked.
    auto publish_q = [&](int c) {
        const int tc = (int)min<int64_t>(T, nz - (int64_t)c * T);
        const int64_t xb = xs + (int64_t)c * T;
#pragma unroll
        for (int mt = 0; mt < NMT; ++mt) {
            const int row = mt * 16 + (lane & 15);
            const bool rok = row < tc;
            const float* xr = a.X + (size_t)(xb + (rok ? row : 0)) * In;
            float4 xv[MAX_IB];
#pragma unroll
            for (int j = 0; j < MAX_IB; ++j) {
                const int ib = wave + 4 * j, i = ib * 16 + 4 * g;
                const bool ok = rok && ib < nib && i < In;
                const float4 v = *(const float4*)(xr + (ok ? i : 0));
                xv[j] = ok ? v : make_float4(0.f, 0.f, 0.f, 0.f);
            }
            f4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int j = 0; j < MAX_IB; ++j) {
                acc = __builtin_amdgcn_mfma_f32_16x16x4f32(xv[j].x, W[j][0], acc, 0, 0, 0);
                acc = __builtin_amdgcn_mfma_f32_16x16x4f32(xv[j].y, W[j][1], acc, 0, 0, 0);
                acc = __builtin_amdgcn_mfma_f32_16x16x4f32(xv[j].z, W[j][2], acc, 0, 0, 0);
                acc = __builtin_amdgcn_mfma_f32_16x16x4f32(xv[j].w, W[j][3], acc, 0, 0, 0);
            }
            *(f4*)(red4 + ((size_t)(wave * NMT + mt) * 64 + lane) * 4) = acc;
        }
        __syncthreads();
        float* Q = a.qbuf + ((size_t)(c & 1) * K + k) * T * H;
        for (int e = tid; e < NMT * 256; e += 256) {
            const int mt = e >> 8, rem = e & 255, ln = rem >> 2, r = rem & 3;
            float sum = 0.f;
#pragma unroll
            for (int w = 0; w < 4; ++w) sum += red4[((size_t)(w * NMT + mt) * 64 + ln) * 4 + r];
            const int t = mt * 16 + 4 * (ln >> 4) + r, hh = rb * 16 + (ln & 15);
            if (t < tc && hh < H) Q[(size_t)t * H + hh] = sum;
        }
        signal_add(qready, 1);
    };
    // W1 tile -= eta * sum_t d1_t x_t^T over the rows of chunk c (errors stored [h][T])
    auto update = [&](int c) {
        const int tc = (int)min<int64_t>(T, nz - (int64_t)c * T);
        const int64_t xb = xs + (int64_t)c * T;
        const float* D = a.d1 + ((size_t)(c & 1) * K + k) * H * T + (size_t)(h < H ? h : 0) * T;
        float bv[T / 4];
#pragma unroll
        for (int sl = 0; sl < T / 16; ++sl) {
            const float4 d = *(const float4*)(D + sl * 16 + 4 * g);
            const int t0 = sl * 16 + 4 * g;
            bv[4 * sl + 0] = (h < H && t0 + 0 < tc) ? d.x : 0.f;
            bv[4 * sl + 1] = (h < H && t0 + 1 < tc) ? d.y : 0.f;
            bv[4 * sl + 2] = (h < H && t0 + 2 < tc) ? d.z : 0.f;
            bv[4 * sl + 3] = (h < H && t0 + 3 < tc) ? d.w : 0.f;
        }
        const float* xrow[T / 4];
#pragma unroll
        for (int u = 0; u < T / 4; ++u) {
            const int t = (u >> 2) * 16 + 4 * g + (u & 3);
            xrow[u] = a.X + (size_t)(xb + (t < tc ? t : 0)) * In;
        }
#pragma unroll
        for (int j = 0; j < MAX_IB; ++j) {
            const int ib = wave + 4 * j;
            if (ib >= nib) continue;
            const int icol = ib * 16 + (lane & 15);
            const int ic = icol < In ? icol : 0;
            float av[T / 4];
#pragma unroll
            for (int u = 0; u < T / 4; ++u) av[u] = xrow[u][ic];  // bv is zero where the row is out of range
            f4 dacc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int u = 0; u < T / 4; ++u) dacc = __builtin_amdgcn_mfma_f32_16x16x4f32(av[u], bv[u], dacc, 0, 0, 0);
#pragma unroll
            for (int r = 0; r < 4; ++r) W[j][r] -= a.lr * dacc[r];
        }
    };

    // Q_0 and Q_1 use the initial weights; afterwards chunk c's errors (c >= 0) are applied
    // before Q_{c+2} is computed.  One call site each keeps the code compact.
    bool ok = true;
    for (int step = 0; step <= nchk && ok; ++step) {
        // step 0: publish Q_0 (and Q_1); step s >= 1: apply the errors of chunk s-1, then
        // publish Q_{s+1}
        if (step >= 1) {
            if (!wait_geq(dready, step, abort, a.spin_limit)) { ok = false; break; }
            update(step - 1);
        }
        const int first = step == 0 ? 0 : step + 1;
        const int last = step == 0 ? min(1, nchk - 1) : step + 1;
        for (int cq = first; cq <= last; ++cq)
            if (cq < nchk) publish_q(cq);
    }
    if (!ok) return;
#pragma unroll
    for (int j = 0; j < MAX_IB; ++j)
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            const int ib = wave + 4 * j, i = ib * 16 + 4 * g + q;
            if (ib < nib && h < H && i < In) th[a.off_w1 + (size_t)h * In + i] = W[j][q];
        }
}

template <int T, int HW, int A1, int A2, int LS, int OC>
__global__ __launch_bounds__(256) void psgd_persistent_kernel(PsgdPArgs a) {
    extern __shared__ float smem[];
    const int b = blockIdx.x, K = a.k_rep;
    if (b < K) psgd_rec<T, HW, A1, A2, LS, OC>(a, b, smem);
    else {
        const int j = b - K;
        psgd_tile<T>(a, j / a.nrb, j % a.nrb, smem);
    }
}

__global__ void zero_ints_kernel(int* p, int n) {
    const int i = blockIdx.x * blockDim.x + threadIdx.x;
    if (i < n) p[i] = 0;
}

}  // namespace pnn
