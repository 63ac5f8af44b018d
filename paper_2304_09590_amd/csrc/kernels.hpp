// kernels.hpp -- CDNA4 (gfx950) kernels of the PNN hot path.
//
// Every kernel is batched over the K child networks (CNs): blockIdx.z (or x) selects the
// CN, whose parameters sit at theta + z * pstride in the padded device layout, and whose
// data slice is the contiguous row range given by shard_start/shard_len below.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>
#include <type_traits>

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

typedef __bf16 bf2v __attribute__((ext_vector_type(2)));
// two floats to packed bf16 (one v_cvt_pk_bf16_f32, round to nearest even), x in the low half
__device__ inline uint32_t cvt_pk_bf16(float x, float y) {
    const bf2v p = {(__bf16)x, (__bf16)y};
    return __builtin_bit_cast(uint32_t, p);
}

template <typename T> __device__ inline float to_f(T v);
template <> __device__ inline float to_f<float>(float v) { return v; }
template <> __device__ inline float to_f<bf16_t>(bf16_t v) { return bf2f(v); }
template <typename T> __device__ inline T from_f(float v);
template <> __device__ inline float from_f<float>(float v) { return v; }
template <> __device__ inline bf16_t from_f<bf16_t>(float v) { return f2bf(v); }

// four consecutive values of type T (16-byte aligned for fp32, 8-byte for bf16), as fp32
template <typename T>
__device__ inline float4 load4(const T* p) {
    if constexpr (sizeof(T) == 4) return *(const float4*)p;
    else {
        const uint2 q = *(const uint2*)p;
        return make_float4(bf2f((bf16_t)(q.x & 0xffff)), bf2f((bf16_t)(q.x >> 16)), bf2f((bf16_t)(q.y & 0xffff)),
                           bf2f((bf16_t)(q.y >> 16)));
    }
}
template <typename T>
__device__ inline void store4(T* p, float4 v) {
    if constexpr (sizeof(T) == 4) *(float4*)p = v;
    else {
        uint2 q;
        q.x = (uint32_t)f2bf(v.x) | ((uint32_t)f2bf(v.y) << 16);
        q.y = (uint32_t)f2bf(v.z) | ((uint32_t)f2bf(v.w) << 16);
        *(uint2*)p = q;
    }
}

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

// Activations of the sequential per-sample steps and of the split-bf16 forward's epilogue.
// The sigmoid runs on the hardware exp2 and
// reciprocal (relative error below |z| * 6e-8 + 2 ulp).  tanh takes the library function:
// written as 1 - 2 / (e^{2z} + 1) it would lose its relative accuracy near z = 0 (cancellation:
// about 1e-4 relative at z = 1e-3), which a cross-entropy output error then amplifies.
__device__ inline float act_fast(int a, float z) {
    switch (a) {
    case ACT_SIGMOID: return __builtin_amdgcn_rcpf(1.0f + __expf(-z));
    case ACT_TANH: return tanhf(z);
    case ACT_RELU: return z >= 0.0f ? z + 0.0f : -0.0f;
    case ACT_LEAKY: return z >= 0.0f ? z + 0.0f : 0.01f * z;
    default: return z;
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
    // a narrow last layer (O2 <= 16 neurons, fp32) fused around this hidden layer's products:
    //   forward (gemm256x3_kernel): partial output sums of each 256-column tile into zpart;
    //   update (upd128x3_kernel): A is the hidden activations, the hidden errors are formed
    //   from dout and the pre-update W2, and W2 / b2 take their own update.
    float* w2;              // W2 [O2][N or M] (+ z * w2_z), fp32 master; nullable (not fused)
    float* b2;              // b2 [O2] (+ z * bias_z)
    int64_t w2_z;
    float* zpart;           // [z][column tiles][M][16] partial sums of the last layer, nullable
    const float* dout;      // [z][step rows][16] output errors, nullable
    int o2;                 // O2
    int act2;               // update: activation of this hidden layer (its derivative)
    // update with the last layer fused, in the first step after a merge whose copy into the
    // CNs was deferred: W, W2, b and b2 are read from these (the merged network: one slot, no
    // CN stride) and the update is written to the CN's own (all nullable)
    const float* rd_c;
    const float* rd_w2;
    const float* rd_ub;
    const float* rd_b2;
};

template <bool BF> struct GemmTile;
template <> struct GemmTile<false> { static constexpr int BK = 16, LDK = 20; typedef float T; };
template <> struct GemmTile<true> { static constexpr int BK = 32, LDK = 40; typedef bf16_t T; };

// Tile of a GEMM workgroup.  Workgroups are handed to the 8 XCDs in turn by their linear id
// (x fastest); when the batch dimension z is a multiple of 8 and at least 64, the ids are
// renumbered so that all tiles of one z run on one XCD, one z after another, and share that
// XCD's L2 (the operand tiles of a CN are read by several tiles each).  (With fewer z per XCD
// the plain order measured faster.)
// (p: the workgroup's place in the dispatch order of a gx x gy x gz grid)
__device__ inline void gemm_tile_of(int p, int gx, int gy, int gz, int& bx, int& by, int& bz) {
    const int tpz = gx * gy;
    if (gz % 8 != 0 || gz < 64) {
        bz = p / tpz;
        const int t = p - bz * tpz;
        by = t / gx;
        bx = t - by * gx;
        return;
    }
    const int slot = p >> 3, zq = slot / tpz, t = slot - zq * tpz;
    bz = zq * 8 + (p & 7);
    by = t / gx;
    bx = t - by * gx;
}
__device__ inline void gemm_tile(int& bx, int& by, int& bz) {
    const int gx = gridDim.x, gy = gridDim.y;
    gemm_tile_of(blockIdx.x + gx * (blockIdx.y + gy * blockIdx.z), gx, gy, gridDim.z, bx, by, bz);
}

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

// Branch-free loads through a buffer descriptor: an element outside the tile's valid rows lies
// past the descriptor's range, one past the valid contraction gets an offset beyond it, and both
// read as zero, so the wait counters stay exact across the pipeline.  KC: the descriptor starts
// at the tile's first row (t0) and spans its valid rows; NC: it starts at the tile's first
// column (t0) of contraction row 0 and ends with the last valid contraction row.
struct B3Src {
    uint64_t base;  // first byte (the same in every lane)
    int nbytes;     // bytes in range
    uint32_t ld4;   // row stride in bytes
};

template <bool KC, int ES = 4>
__device__ inline B3Src b3_src(const Operand& o, int z, int cn, int64_t xbase, int t0, int t_valid, int k_valid) {
    B3Src r;
    r.ld4 = (uint32_t)(o.ld * ES);
    const int rows = KC ? t_valid - t0 : k_valid;
    const char* base = KC ? operand_row(o, ES, z, cn, xbase, t0) : operand_row(o, ES, z, cn, xbase, 0) + (size_t)t0 * ES;
    int64_t bytes = (int64_t)rows * o.ld * ES - (KC ? 0 : (int64_t)t0 * ES);
    if (rows <= 0 || bytes < 0) bytes = 0;
    if (bytes > 0x7fffffff) bytes = 0x7fffffff;
    r.base = (uint64_t)base;
    r.nbytes = (int)bytes;
    return r;
}

// the descriptor, built where it is used from values made scalar explicitly (they are the same
// in every lane; otherwise every buffer load would loop over the lanes' descriptors)
__device__ inline __amdgpu_buffer_rsrc_t b3_rsrc(const B3Src& src) {
    const uint64_t a = ((uint64_t)(uint32_t)__builtin_amdgcn_readfirstlane((int)(src.base >> 32)) << 32) |
                       (uint32_t)__builtin_amdgcn_readfirstlane((int)(uint32_t)src.base);
    return __builtin_amdgcn_make_buffer_rsrc((void*)a, (short)0, __builtin_amdgcn_readfirstlane(src.nbytes), 0x00020000);
}

// bf16 tiles, 64 rows or columns x 32 k, stored as lds[t][k] (row stride 40 bf16), loaded into
// registers first (up to 32 bytes per thread; fp32 sources are rounded to bf16 on the way in).
//   KC (rows = t): fp32 two float4 of 4 k, bf16 one 16-byte load of 8 k;
//   NC (rows = k): a 2 k x 4 t block per thread (lane bits 0-3 the k pair, so that the
//   transposing 4-byte stores of a wave fall on distinct banks).
struct BfRaw { uint4 r[2]; };

template <typename TS>
__device__ inline BfRaw bf_load_kc(const Operand& o, int z, int cn, int64_t xbase, int row0, int rows_valid, int k0,
                                   int k_valid, int tid) {
    BfRaw v;
    v.r[0] = v.r[1] = make_uint4(0, 0, 0, 0);
    if constexpr (sizeof(TS) == 4) {
#pragma unroll
        for (int h = 0; h < 2; ++h) {
            const int idx = tid + h * 256, r = idx >> 3, kq = (idx & 7) * 4;
            if (row0 + r < rows_valid && k0 + kq < k_valid)
                v.r[h] = *(const uint4*)(operand_row(o, 4, z, cn, xbase, row0 + r) + (size_t)(k0 + kq) * 4);
        }
    } else {
        const int r = tid >> 2, kq = (tid & 3) * 8;
        if (row0 + r < rows_valid && k0 + kq < k_valid)
            v.r[0] = *(const uint4*)(operand_row(o, 2, z, cn, xbase, row0 + r) + (size_t)(k0 + kq) * 2);
    }
    return v;
}
template <typename TS>
__device__ inline void bf_store_kc(bf16_t* lds, const BfRaw& v, int tid) {
    constexpr int LDK = GemmTile<true>::LDK;
    if constexpr (sizeof(TS) == 4) {
#pragma unroll
        for (int h = 0; h < 2; ++h) {
            const int idx = tid + h * 256, r = idx >> 3, kq = (idx & 7) * 4;
            const uint4 u = v.r[h];
            uint2 q;
            q.x = (uint32_t)f2bf(__uint_as_float(u.x)) | ((uint32_t)f2bf(__uint_as_float(u.y)) << 16);
            q.y = (uint32_t)f2bf(__uint_as_float(u.z)) | ((uint32_t)f2bf(__uint_as_float(u.w)) << 16);
            *(uint2*)(lds + r * LDK + kq) = q;
        }
    } else {
        *(uint4*)(lds + (tid >> 2) * LDK + (tid & 3) * 8) = v.r[0];
    }
}
template <typename TS>
__device__ inline BfRaw bf_load_nc(const Operand& o, int z, int cn, int64_t xbase, int col0, int cols_valid, int k0,
                                   int k_valid, int tid) {
    BfRaw v;
    v.r[0] = v.r[1] = make_uint4(0, 0, 0, 0);
    const int k = (tid & 15) * 2, cq = (tid >> 4) * 4;
#pragma unroll
    for (int h = 0; h < 2; ++h) {
        if (k0 + k + h < k_valid && col0 + cq < cols_valid) {
            const char* row = operand_row(o, sizeof(TS), z, cn, xbase, k0 + k + h);
            if constexpr (sizeof(TS) == 4) v.r[h] = *(const uint4*)(row + (size_t)(col0 + cq) * 4);
            else {
                const uint2 q = *(const uint2*)(row + (size_t)(col0 + cq) * 2);
                v.r[h].x = q.x; v.r[h].y = q.y;
            }
        }
    }
    return v;
}
template <typename TS>
__device__ inline void bf_store_nc(bf16_t* lds, const BfRaw& v, int tid) {
    constexpr int LDK = GemmTile<true>::LDK;
    const int k = (tid & 15) * 2, cq = (tid >> 4) * 4;
    uint32_t e[2][4];  // bf16 bits of (k + h, cq + j)
#pragma unroll
    for (int h = 0; h < 2; ++h) {
        if constexpr (sizeof(TS) == 4) {
            e[h][0] = f2bf(__uint_as_float(v.r[h].x)); e[h][1] = f2bf(__uint_as_float(v.r[h].y));
            e[h][2] = f2bf(__uint_as_float(v.r[h].z)); e[h][3] = f2bf(__uint_as_float(v.r[h].w));
        } else {
            e[h][0] = v.r[h].x & 0xffff; e[h][1] = v.r[h].x >> 16;
            e[h][2] = v.r[h].y & 0xffff; e[h][3] = v.r[h].y >> 16;
        }
    }
#pragma unroll
    for (int j = 0; j < 4; ++j) *(uint32_t*)(lds + (cq + j) * LDK + k) = e[0][j] | (e[1][j] << 16);
}

// The same tiles through a buffer descriptor (b3_src with the source's element size): rows
// past the tile's valid rows and contraction steps past k_valid read as zero, with no branch,
// so that several k-tiles can be in flight with exact wait counters.
template <typename TS, bool KC>
__device__ inline BfRaw bf_bload(const B3Src& src, int t_valid_rel, int k0, int k_valid, int tid) {
    constexpr uint32_t ES = sizeof(TS);
    BfRaw v;
    v.r[0] = v.r[1] = make_uint4(0, 0, 0, 0);
    if constexpr (KC) {
        if constexpr (ES == 4) {
#pragma unroll
            for (int h = 0; h < 2; ++h) {
                const int idx = tid + h * 256, r = idx >> 3, kq = (idx & 7) * 4;
                const uint32_t inv = (uint32_t)(k_valid - 1 - (k0 + kq)) >> 31;
                const uint32_t off = ((uint32_t)r * src.ld4 + (uint32_t)(k0 + kq) * ES) | (inv << 31);
                v.r[h] = __builtin_bit_cast(uint4, __builtin_amdgcn_raw_buffer_load_b128(b3_rsrc(src), off, 0, 0));
            }
        } else {
            const int r = tid >> 2, kq = (tid & 3) * 8;
            const uint32_t inv = (uint32_t)(k_valid - 1 - (k0 + kq)) >> 31;
            const uint32_t off = ((uint32_t)r * src.ld4 + (uint32_t)(k0 + kq) * ES) | (inv << 31);
            v.r[0] = __builtin_bit_cast(uint4, __builtin_amdgcn_raw_buffer_load_b128(b3_rsrc(src), off, 0, 0));
        }
    } else {
        const int k = (tid & 15) * 2, cq = (tid >> 4) * 4;
        const uint32_t inv = (uint32_t)(t_valid_rel - 1 - cq) >> 31;
#pragma unroll
        for (int h = 0; h < 2; ++h) {
            const uint32_t off = ((uint32_t)(k0 + k + h) * src.ld4 + (uint32_t)cq * ES) | (inv << 31);
            if constexpr (ES == 4) {
                v.r[h] = __builtin_bit_cast(uint4, __builtin_amdgcn_raw_buffer_load_b128(b3_rsrc(src), off, 0, 0));
            } else {
                typedef unsigned int u2v_t __attribute__((ext_vector_type(2)));
                const u2v_t q = __builtin_bit_cast(u2v_t, __builtin_amdgcn_raw_buffer_load_b64(b3_rsrc(src), off, 0, 0));
                v.r[h].x = q.x;
                v.r[h].y = q.y;
            }
        }
    }
    return v;
}

// fp32 tiles of an operand whose rows are the contraction index ("NC" layout) stay as they
// are in LDS, [k][t] with row stride GEMM_LDM: a lane then reads one value per instruction, and
// the 4 lane groups of a read (4 k apart) fall on disjoint banks.
constexpr int GEMM_LDM = 68;

// fp32 tiles, 64 rows or columns x 16 k, one float4 per thread, loaded into registers first
// (the next k-tile's loads are in flight during the current tile's matrix instructions)
__device__ inline float4 load_tile32(const Operand& o, bool kc, int z, int cn, int64_t xbase, int t0, int t_valid,
                                     int k0, int k_valid, int tid) {
    const int a = kc ? tid >> 2 : tid >> 4, b = kc ? (tid & 3) * 4 : (tid & 15) * 4;  // (row, k) or (k, column)
    const int t = kc ? a : b, k = kc ? b : a;
    if (t0 + t < t_valid && k0 + k < k_valid) {
        if (kc) return *(const float4*)(operand_row(o, 4, z, cn, xbase, t0 + t) + (size_t)(k0 + k) * 4);
        return *(const float4*)(operand_row(o, 4, z, cn, xbase, k0 + k) + (size_t)(t0 + t) * 4);
    }
    return make_float4(0.f, 0.f, 0.f, 0.f);
}
// KC: lds[row][k] (row stride 20); NC: lds[k][column] (row stride GEMM_LDM)
__device__ inline void store_tile32(float* lds, bool kc, const float4& v, int tid) {
    if (kc) *(float4*)(lds + (tid >> 2) * 20 + (tid & 3) * 4) = v;
    else *(float4*)(lds + (tid >> 4) * GEMM_LDM + (tid & 15) * 4) = v;
}

// WPRE (weight update with a short contraction): the update's targets are read before the
// contraction, their latency behind it (16 more registers per lane)
// the LDS of one workgroup: two buffers per operand (one barrier per k-tile) and the bias sums
template <bool BF, bool A_KC, bool B_KC>
struct GemmLds {
    typedef typename GemmTile<BF>::T LT;
    static constexpr int LDK = GemmTile<BF>::LDK;
    static constexpr int ASZ = (BF || A_KC) ? 64 * LDK : 16 * GEMM_LDM, BSZ = (BF || B_KC) ? 64 * LDK : 16 * GEMM_LDM;
    static constexpr int NBUF = 2;
    __attribute__((aligned(16))) LT As[NBUF * ASZ];
    __attribute__((aligned(16))) LT Bs[NBUF * BSZ];
    float rowsum[64];
};

template <bool BF, typename TA, typename TB, bool A_KC, bool B_KC, int EPI, typename TO, bool WPRE>
__device__ __attribute__((always_inline)) inline void gemm_body(const GemmArgs& g, int bx, int by, int bz,
                                                                GemmLds<BF, A_KC, B_KC>& lds) {
    typedef typename GemmTile<BF>::T LT;
    constexpr int BK = GemmTile<BF>::BK, LDK = GemmTile<BF>::LDK;
    constexpr int ASZ = GemmLds<BF, A_KC, B_KC>::ASZ, BSZ = GemmLds<BF, A_KC, B_KC>::BSZ;
    LT* As = lds.As;
    LT* Bs = lds.Bs;
    float* rowsum = lds.rowsum;

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int wm = wave >> 1, wn = wave & 1;
    const int zz = bz / g.ksplit, slice = bz % g.ksplit;
    int cn, valid;
    int64_t r0;
    gemm_zinfo(g, zz, cn, r0, valid);
    const int Mv = (g.sample_dims & 1) ? valid : g.M;
    const int Nv = (g.sample_dims & 2) ? valid : g.N;
    const int Kv = (g.sample_dims & 4) ? valid : g.Kd;
    const int m0 = by * 64, n0 = bx * 64;
    if (m0 >= Mv || n0 >= Nv) return;
    const int kbeg = slice * g.kchunk;
    const int kend = min(Kv, kbeg + g.kchunk);
    const int64_t xbase = shard_start(g.n_total, g.k_rep, cn) + r0;
    const bool do_rowsum = (EPI == EPI_UPD) && g.ubias != nullptr && bx == 0;
    if (do_rowsum && tid < 64) rowsum[tid] = 0.f;

    f4 acc[2][2];
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j) acc[i][j] = f4{0.f, 0.f, 0.f, 0.f};
    // SW: the operands enter the matrix instructions swapped (B as the first), so that a lane
    // holds C row m = m0 + 32 wm + 16 i + (lane & 15), columns n .. n+3 with
    // n = n0 + 32 wn + 16 j + 4 (lane >> 4), of each 16 x 16 block, and the epilogue reads and
    // writes 4 consecutive values at once where the target's strides allow.  Otherwise a lane
    // holds rows 4 (lane >> 4) + r, column lane & 15.  (The bf16 weight update, which also
    // writes the bf16 shadow, measured faster with the second layout.)
    constexpr bool SW = !(BF && EPI == EPI_UPD);
    const bool vec = SW && ((g.c_ld | g.c_z | g.c_split | g.bias_z) & 3) == 0;
    auto coord = [&](int i, int j, int r, int& m, int& n) {
        if (SW) { m = m0 + wm * 32 + i * 16 + (lane & 15); n = n0 + wn * 32 + j * 16 + (lane >> 4) * 4 + r; }
        else { m = m0 + wm * 32 + i * 16 + (lane >> 4) * 4 + r; n = n0 + wn * 32 + j * 16 + (lane & 15); }
    };
    float4 wpre[2][2];
    if constexpr (WPRE) {
#pragma unroll
        for (int i = 0; i < 2; ++i)
#pragma unroll
            for (int j = 0; j < 2; ++j) {
                int m, n;
                coord(i, j, 0, m, n);
                const float* W = (const float*)g.c + (size_t)zz * g.c_z;
                if (vec && m < Mv && n + 3 < Nv) {
                    wpre[i][j] = *(const float4*)(W + (size_t)m * g.c_ld + n);
                } else {
                    float t[4];
#pragma unroll
                    for (int r = 0; r < 4; ++r) {
                        coord(i, j, r, m, n);
                        t[r] = (m < Mv && n < Nv) ? W[(size_t)m * g.c_ld + n] : 0.f;
                    }
                    wpre[i][j] = make_float4(t[0], t[1], t[2], t[3]);
                }
            }
    }

    const int rl = lane & 15, kg = lane >> 4;
    if constexpr (!BF) {
        // fp32 NC operands are kept as [k][t]
        auto compute = [&](const float* A, const float* B) {
            if (do_rowsum && tid < 64) {
                float s = 0.f;
#pragma unroll
                for (int k = 0; k < BK; ++k) s += A_KC ? A[tid * LDK + k] : A[k * GEMM_LDM + tid];
                rowsum[tid] += s;
            }
            f4 av[2], bv[2];
            if constexpr (A_KC)
#pragma unroll
                for (int i = 0; i < 2; ++i) av[i] = *(const f4*)(A + (wm * 32 + i * 16 + rl) * LDK + kg * 4);
            if constexpr (B_KC)
#pragma unroll
                for (int j = 0; j < 2; ++j) bv[j] = *(const f4*)(B + (wn * 32 + j * 16 + rl) * LDK + kg * 4);
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                float aq[2], bq[2];
#pragma unroll
                for (int i = 0; i < 2; ++i)
                    aq[i] = A_KC ? av[i][q] : A[(kg * 4 + q) * GEMM_LDM + wm * 32 + i * 16 + rl];
#pragma unroll
                for (int j = 0; j < 2; ++j)
                    bq[j] = B_KC ? bv[j][q] : B[(kg * 4 + q) * GEMM_LDM + wn * 32 + j * 16 + rl];
#pragma unroll
                for (int i = 0; i < 2; ++i)
#pragma unroll
                    for (int j = 0; j < 2; ++j)
                        acc[i][j] = SW ? __builtin_amdgcn_mfma_f32_16x16x4f32(bq[j], aq[i], acc[i][j], 0, 0, 0)
                                       : __builtin_amdgcn_mfma_f32_16x16x4f32(aq[i], bq[j], acc[i][j], 0, 0, 0);
            }
        };
        float4 ra = make_float4(0.f, 0.f, 0.f, 0.f), rb = ra;
        if (kbeg < kend) {
            ra = load_tile32(g.a, A_KC, zz, cn, xbase, m0, Mv, kbeg, kend, tid);
            rb = load_tile32(g.b, B_KC, zz, cn, xbase, n0, Nv, kbeg, kend, tid);
            store_tile32((float*)As, A_KC, ra, tid);
            store_tile32((float*)Bs, B_KC, rb, tid);
        }
        __syncthreads();
        int buf = 0;
        for (int k0 = kbeg; k0 < kend; k0 += BK) {
            const bool more = k0 + BK < kend;
            if (more) {
                ra = load_tile32(g.a, A_KC, zz, cn, xbase, m0, Mv, k0 + BK, kend, tid);
                rb = load_tile32(g.b, B_KC, zz, cn, xbase, n0, Nv, k0 + BK, kend, tid);
            }
            compute((const float*)As + buf * ASZ, (const float*)Bs + buf * BSZ);
            if (more) {
                store_tile32((float*)As + (buf ^ 1) * ASZ, A_KC, ra, tid);
                store_tile32((float*)Bs + (buf ^ 1) * BSZ, B_KC, rb, tid);
            }
            __syncthreads();
            buf ^= 1;
        }
    } else {
        // the bf16 tiles of the contraction: the steps of the weight update (a short contraction
        // over the batch) as they come, one k-tile ahead; the others through the deeper pipeline
        // below
        auto compute_tile = [&](const LT* A, const LT* Bt) {
            if (do_rowsum && tid < 64) {
                float s = 0.f;
#pragma unroll
                for (int k = 0; k < BK; ++k) s += (float)to_f<LT>(A[tid * LDK + k]);
                rowsum[tid] += s;
            }
            bf8v av[2], bv[2];
#pragma unroll
            for (int i = 0; i < 2; ++i) av[i] = *(const bf8v*)(A + (wm * 32 + i * 16 + rl) * LDK + kg * 8);
#pragma unroll
            for (int j = 0; j < 2; ++j) bv[j] = *(const bf8v*)(Bt + (wn * 32 + j * 16 + rl) * LDK + kg * 8);
#pragma unroll
            for (int i = 0; i < 2; ++i)
#pragma unroll
                for (int j = 0; j < 2; ++j)
                    acc[i][j] = SW ? __builtin_amdgcn_mfma_f32_16x16x32_bf16(bv[j], av[i], acc[i][j], 0, 0, 0)
                                   : __builtin_amdgcn_mfma_f32_16x16x32_bf16(av[i], bv[j], acc[i][j], 0, 0, 0);
        };
        if constexpr (EPI == EPI_UPD) {
            BfRaw ra, rb;
            auto load = [&](int k0) {
                if constexpr (A_KC) ra = bf_load_kc<TA>(g.a, zz, cn, xbase, m0, Mv, k0, kend, tid);
                else ra = bf_load_nc<TA>(g.a, zz, cn, xbase, m0, Mv, k0, kend, tid);
                if constexpr (B_KC) rb = bf_load_kc<TB>(g.b, zz, cn, xbase, n0, Nv, k0, kend, tid);
                else rb = bf_load_nc<TB>(g.b, zz, cn, xbase, n0, Nv, k0, kend, tid);
            };
            auto store = [&](int buf) {
                if constexpr (A_KC) bf_store_kc<TA>(As + buf * ASZ, ra, tid);
                else bf_store_nc<TA>(As + buf * ASZ, ra, tid);
                if constexpr (B_KC) bf_store_kc<TB>(Bs + buf * BSZ, rb, tid);
                else bf_store_nc<TB>(Bs + buf * BSZ, rb, tid);
            };
            if (kbeg < kend) {
                load(kbeg);
                store(0);
            }
            __syncthreads();
            int buf = 0;
            for (int k0 = kbeg; k0 < kend; k0 += BK) {
                const bool more = k0 + BK < kend;
                if (more) load(k0 + BK);
                compute_tile(As + buf * ASZ, Bs + buf * BSZ);
                if (more) store(buf ^ 1);
                __syncthreads();
                buf ^= 1;
            }
        } else {
            // k-tile i is loaded into register set i % BF_PD, BF_PD tiles ahead of its use, through
            // buffer descriptors (no branch: exact wait counters); it goes to LDS buffer i & 1 one
            // tile ahead.  (The contraction of these layers is long and each tile's matrix work
            // short: the loop is bound by memory latency, which the tiles in flight cover.)
            constexpr int BF_PD = 2;
            BfRaw ra[BF_PD], rb[BF_PD];
            const B3Src sa = b3_src<A_KC, sizeof(TA)>(g.a, zz, cn, xbase, m0, Mv, kend);
            const B3Src sb = b3_src<B_KC, sizeof(TB)>(g.b, zz, cn, xbase, n0, Nv, kend);
            auto load = [&](BfRaw& xa, BfRaw& xb, int k0) {
                xa = bf_bload<TA, A_KC>(sa, Mv - m0, k0, kend, tid);
                xb = bf_bload<TB, B_KC>(sb, Nv - n0, k0, kend, tid);
            };
            auto store = [&](int buf, const BfRaw& xa, const BfRaw& xb) {
                if constexpr (A_KC) bf_store_kc<TA>(As + buf * ASZ, xa, tid);
                else bf_store_nc<TA>(As + buf * ASZ, xa, tid);
                if constexpr (B_KC) bf_store_kc<TB>(Bs + buf * BSZ, xb, tid);
                else bf_store_nc<TB>(Bs + buf * BSZ, xb, tid);
            };
            const int nk = kend > kbeg ? (kend - kbeg + BK - 1) / BK : 0;
#pragma unroll
            for (int p = 0; p < BF_PD; ++p)
                if (p < nk) load(ra[p], rb[p], kbeg + p * BK);
            // tile 0 to LDS; its register set takes tile BF_PD
            if (nk > 0) store(0, ra[0], rb[0]);
            if (BF_PD < nk) load(ra[0], rb[0], kbeg + BF_PD * BK);
            __syncthreads();
            // tile i = i0 + p (register set p); after its matrix instructions, tile i + 1 (set
            // (p + 1) % BF_PD) goes to the other buffer and that set takes tile i + 1 + BF_PD
            for (int i0 = 0; i0 < nk; i0 += BF_PD)
#pragma unroll
            for (int p = 0; p < BF_PD; ++p) {
                const int i = i0 + p;
                if (i >= nk) break;
                const int buf = i & 1;
                compute_tile(As + buf * ASZ, Bs + buf * BSZ);
                const int pn = (p + 1) % BF_PD;
                if (i + 1 < nk) store(buf ^ 1, ra[pn], rb[pn]);
                if (i + 1 + BF_PD < nk) load(ra[pn], rb[pn], kbeg + (i + 1 + BF_PD) * BK);
                __syncthreads();
            }
        }
    }

    // epilogue (layout above)
    float scale = g.lr;
    if (EPI == EPI_UPD && g.scale_per_batch) scale = valid > 0 ? g.lr / (float)valid : 0.f;
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j) {
            int m, n;
            coord(i, j, 0, m, n);
            const f4 v = acc[i][j];
            if (vec && m < Mv && n + 3 < Nv) {
                const size_t ci = (size_t)zz * g.c_z + (size_t)m * g.c_ld + n;
                const float4 c4 = make_float4(v[0], v[1], v[2], v[3]);
                if constexpr (EPI == EPI_STORE) {
                    *(float4*)((float*)g.c + ci + (size_t)slice * g.c_split) = c4;
                } else if constexpr (EPI == EPI_FWD) {
                    const float4 bb = *(const float4*)(g.bias + (size_t)cn * g.bias_z + n);
                    store4<TO>((TO*)g.c + ci, make_float4(act_fn(g.act, c4.x + bb.x), act_fn(g.act, c4.y + bb.y),
                                                          act_fn(g.act, c4.z + bb.z), act_fn(g.act, c4.w + bb.w)));
                } else if constexpr (EPI == EPI_BWD) {
                    const float4 x = load4<TO>((const TO*)g.aux + ci);
                    store4<TO>((TO*)g.c + ci, make_float4(c4.x * act_deriv(g.act, x.x), c4.y * act_deriv(g.act, x.y),
                                                          c4.z * act_deriv(g.act, x.z), c4.w * act_deriv(g.act, x.w)));
                } else {  // EPI_UPD: in-place W -= scale * acc (master fp32)
                    float* W = (float*)g.c + ci;
                    float4 w = WPRE ? wpre[i][j] : *(const float4*)W;
                    w.x -= scale * c4.x; w.y -= scale * c4.y; w.z -= scale * c4.z; w.w -= scale * c4.w;
                    *(float4*)W = w;
                    if (g.shadow) store4<bf16_t>(g.shadow + ci, w);
                }
            } else {
#pragma unroll
                for (int r = 0; r < 4; ++r) {
                    coord(i, j, r, m, n);
                    if (m >= Mv || n >= Nv) continue;
                    const size_t cr = (size_t)zz * g.c_z + (size_t)m * g.c_ld + n;
                    if constexpr (EPI == EPI_STORE) {
                        ((float*)g.c)[cr + (size_t)slice * g.c_split] = v[r];
                    } else if constexpr (EPI == EPI_FWD) {
                        const float zv = v[r] + g.bias[(size_t)cn * g.bias_z + n];
                        ((TO*)g.c)[cr] = from_f<TO>(act_fn(g.act, zv));
                    } else if constexpr (EPI == EPI_BWD) {
                        const float x = to_f<TO>(((const TO*)g.aux)[cr]);
                        ((TO*)g.c)[cr] = from_f<TO>(v[r] * act_deriv(g.act, x));
                    } else {
                        float* W = (float*)g.c;
                        const float wp[4] = {wpre[i][j].x, wpre[i][j].y, wpre[i][j].z, wpre[i][j].w};
                        const float w = (WPRE ? wp[r] : W[cr]) - scale * v[r];
                        W[cr] = w;
                        if (g.shadow) g.shadow[cr] = f2bf(w);
                    }
                }
            }
        }
    if (do_rowsum && tid < 64 && m0 + tid < Mv) {
        float* b = g.ubias + (size_t)cn * g.bias_z;
        b[m0 + tid] -= scale * rowsum[tid];
    }
}

template <bool BF, typename TA, typename TB, bool A_KC, bool B_KC, int EPI, typename TO, bool WPRE = false>
__global__ __launch_bounds__(256) void gemm_kernel(GemmArgs g) {
    __shared__ GemmLds<BF, A_KC, B_KC> lds;
    int bx, by, bz;
    gemm_tile(bx, by, bz);
    gemm_body<BF, TA, TB, A_KC, B_KC, EPI, TO, WPRE>(g, bx, by, bz, lds);
}

// Two independent weight updates of the bf16 mini-batch plan (two wide layers, samples along
// the contraction, the targets read before it) in one launch: the first grid's workgroups,
// then the second's, in one dispatch order (a one-dimensional grid of both counts; each part
// is mapped to its tiles as gemm_tile maps a grid of its own, and the first part's count is a
// multiple of 8, so that the XCD of a workgroup is as in a launch of its own).  The smaller
// update's last round of workgroups then shares the chip with the larger one instead of
// running alone, and one launch boundary goes.
template <typename TB1, typename TB2>
__global__ __launch_bounds__(256) void gemm_upd2_kernel(GemmArgs g1, GemmArgs g2, int gx1, int gy1, int gz1,
                                                       int gx2, int gy2, int gz2) {
    __shared__ GemmLds<true, false, false> lds;
    const int p = blockIdx.x, n1 = gx1 * gy1 * gz1;
    int bx, by, bz;
    if (p < n1) {
        gemm_tile_of(p, gx1, gy1, gz1, bx, by, bz);
        gemm_body<true, bf16_t, TB1, false, false, EPI_UPD, float, true>(g1, bx, by, bz, lds);
    } else {
        gemm_tile_of(p - n1, gx2, gy2, gz2, bx, by, bz);
        gemm_body<true, bf16_t, TB2, false, false, EPI_UPD, float, true>(g2, bx, by, bz, lds);
    }
}

// ------------------------------------------------------------------------------------
// bf16 forward product of at most 64 rows (one training step's batch) with both operands
// along k, C[64 x 64 tile] = A[64 x K] B[64 x K]^T with gemm_kernel's forward epilogue.  The
// four waves split the contraction (wave w takes the 32-deep steps w, w + 4, ...) and read
// their fragments straight from global memory in the matrix instruction's layout (A rows
// 16 i + lane % 16, B rows 16 j + lane % 16, k 8 (lane / 16) .. + 7 of the step; fp32 A rounded
// to bf16 on the way), KW_PD steps ahead through buffer descriptors (steps past K read zero):
// no LDS staging and no barrier in the loop, which in the staged kernel is bound by latency on
// these long, narrow contractions.  The partial tiles meet in LDS and are added in wave order;
// wave w then finishes rows 16 w .. 16 w + 15 of the tile.

constexpr int KW_PD = 2;

template <typename TA, typename TO>
__global__ __launch_bounds__(256) void gemm_kw_kernel(GemmArgs g) {
    __shared__ __attribute__((aligned(16))) float red[4 * 64 * 64];  // [wave][i][j][lane][4]
    constexpr int AV = sizeof(TA) / 2;  // 16-byte loads per A fragment
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6, rl = lane & 15, kg = lane >> 4;
    int bx, by, bz;
    gemm_tile(bx, by, bz);
    const int zz = bz;
    int cn, valid;
    int64_t r0;
    gemm_zinfo(g, zz, cn, r0, valid);
    const int Mv = (g.sample_dims & 1) ? valid : g.M;
    const int Nv = (g.sample_dims & 2) ? valid : g.N;
    const int Kv = g.Kd;
    const int m0 = by * 64, n0 = bx * 64;
    if (m0 >= Mv || n0 >= Nv) return;
    const int64_t xbase = shard_start(g.n_total, g.k_rep, cn) + r0;
    const B3Src sa = b3_src<true, sizeof(TA)>(g.a, zz, cn, xbase, m0, Mv, Kv);
    const B3Src sb = b3_src<true, 2>(g.b, zz, cn, xbase, n0, Nv, Kv);

    f4 acc[4][4];
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[i][j] = f4{0.f, 0.f, 0.f, 0.f};
    uint4 fa[KW_PD][4][AV], fb[KW_PD][4];
    auto load = [&](int p, int s) {
        const int k = 32 * s + 8 * kg;
        const uint32_t inv = (uint32_t)(Kv - 1 - k) >> 31;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const uint32_t o = ((uint32_t)(16 * i + rl) * sa.ld4 + (uint32_t)k * (uint32_t)sizeof(TA)) | (inv << 31);
#pragma unroll
            for (int v = 0; v < AV; ++v)
                fa[p][i][v] = __builtin_bit_cast(uint4, __builtin_amdgcn_raw_buffer_load_b128(b3_rsrc(sa), o + 16u * v, 0, 0));
        }
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const uint32_t o = ((uint32_t)(16 * j + rl) * sb.ld4 + (uint32_t)k * 2u) | (inv << 31);
            fb[p][j] = __builtin_bit_cast(uint4, __builtin_amdgcn_raw_buffer_load_b128(b3_rsrc(sb), o, 0, 0));
        }
    };
    auto mma = [&](int p) {
        bf8v av[4], bv[4];
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            if constexpr (AV == 2) {
                const uint4 x0 = fa[p][i][0], x1 = fa[p][i][1];
                const uint4 q = make_uint4(cvt_pk_bf16(__uint_as_float(x0.x), __uint_as_float(x0.y)),
                                           cvt_pk_bf16(__uint_as_float(x0.z), __uint_as_float(x0.w)),
                                           cvt_pk_bf16(__uint_as_float(x1.x), __uint_as_float(x1.y)),
                                           cvt_pk_bf16(__uint_as_float(x1.z), __uint_as_float(x1.w)));
                av[i] = __builtin_bit_cast(bf8v, q);
            } else {
                av[i] = __builtin_bit_cast(bf8v, fa[p][i][0]);
            }
        }
#pragma unroll
        for (int j = 0; j < 4; ++j) bv[j] = __builtin_bit_cast(bf8v, fb[p][j]);
#pragma unroll
        for (int i = 0; i < 4; ++i)
#pragma unroll
            for (int j = 0; j < 4; ++j) acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(bv[j], av[i], acc[i][j], 0, 0, 0);
    };
    // the wave's steps q = 0, 1, ... are the contraction steps wave + 4 q; register set q % KW_PD
    const int nsteps = (Kv + 31) / 32;
    const int nq = nsteps > wave ? (nsteps - wave + 3) / 4 : 0;
#pragma unroll
    for (int p = 0; p < KW_PD; ++p) load(p, wave + 4 * p);
    for (int q0 = 0; q0 < nq; q0 += KW_PD)
#pragma unroll
        for (int p = 0; p < KW_PD; ++p) {
            if (q0 + p >= nq) break;
            mma(p);
            load(p, wave + 4 * (q0 + p + KW_PD));  // (past the contraction: zeros, unused)
        }

    // the four partial tiles, added in wave order; wave w finishes block row i = w
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) *(f4*)(red + (((wave * 4 + i) * 4 + j) * 64 + lane) * 4) = acc[i][j];
    __syncthreads();
    const int i = wave;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
        f4 v = *(const f4*)(red + (((0 * 4 + i) * 4 + j) * 64 + lane) * 4);
#pragma unroll
        for (int w = 1; w < 4; ++w) v += *(const f4*)(red + (((w * 4 + i) * 4 + j) * 64 + lane) * 4);
        const int m = m0 + 16 * i + rl, n = n0 + 16 * j + 4 * kg;
        if (m >= Mv || n >= Nv) continue;
        const size_t ci = (size_t)zz * g.c_z + (size_t)m * g.c_ld + n;
        const float* bb = g.bias + (size_t)cn * g.bias_z + n;
        if (n + 3 < Nv && ((g.c_ld | g.c_z | g.bias_z) & 3) == 0) {
            const float4 b4 = *(const float4*)bb;
            store4<TO>((TO*)g.c + ci, make_float4(act_fn(g.act, v[0] + b4.x), act_fn(g.act, v[1] + b4.y),
                                                  act_fn(g.act, v[2] + b4.z), act_fn(g.act, v[3] + b4.w)));
        } else {
#pragma unroll
            for (int r = 0; r < 4; ++r)
                if (n + r < Nv) ((TO*)g.c)[ci + r] = from_f<TO>(act_fn(g.act, v[r] + bb[r]));
        }
    }
}

// ------------------------------------------------------------------------------------
// fp32 GEMM with 128 x 128 tiles for the large mini-batch shapes: four waves of 64 x 64
// (4 x 4 v_mfma_f32_16x16x4_f32 tiles each), two LDS buffers, the next k-tile's global
// loads issued before the current tile's matrix instructions and stored to the other buffer
// after them (one barrier per k-tile).  A KC operand (rows = the tile's non-contraction
// index) is kept as [row][k] (row stride 20 floats: a lane reads 4 consecutive k at once);
// an NC operand (rows = the contraction index) as [k][column] (row stride 144 floats: the
// 4 lane groups of a read hit disjoint banks), so neither is transposed on the way in.
// Instruction q of a 16-step k-tile contracts the steps {q, 4+q, 8+q, 12+q} on both
// operands.  Split of the contraction and epilogues as in gemm_kernel.

constexpr int G128_LDK = 20, G128_LDM = 144, G128_TL = 128 * 20;  // (16 * 144 <= 128 * 20)

// KC operand, 128 rows x 16 k: two float4 per thread
__device__ inline void load_kc128(float4 (&v)[2], const Operand& o, int z, int cn, int64_t xbase, int row0,
                                  int rows_valid, int k0, int k_valid, int tid) {
#pragma unroll
    for (int h = 0; h < 2; ++h) {
        const int idx = tid + h * 256, r = idx >> 2, kq = (idx & 3) * 4;
        v[h] = make_float4(0.f, 0.f, 0.f, 0.f);
        if (row0 + r < rows_valid && k0 + kq < k_valid)
            v[h] = *(const float4*)(operand_row(o, 4, z, cn, xbase, row0 + r) + (size_t)(k0 + kq) * 4);
    }
}
__device__ inline void store_kc128(float* lds, const float4 (&v)[2], int tid) {
#pragma unroll
    for (int h = 0; h < 2; ++h) {
        const int idx = tid + h * 256, r = idx >> 2, kq = (idx & 3) * 4;
        *(float4*)(lds + r * G128_LDK + kq) = v[h];
    }
}
// NC operand, 16 k x 128 columns: two float4 per thread
__device__ inline void load_nc128(float4 (&v)[2], const Operand& o, int z, int cn, int64_t xbase, int col0,
                                  int cols_valid, int k0, int k_valid, int tid) {
#pragma unroll
    for (int h = 0; h < 2; ++h) {
        const int idx = tid + h * 256, k = idx >> 5, cq = (idx & 31) * 4;
        v[h] = make_float4(0.f, 0.f, 0.f, 0.f);
        if (k0 + k < k_valid && col0 + cq < cols_valid)
            v[h] = *(const float4*)(operand_row(o, 4, z, cn, xbase, k0 + k) + (size_t)(col0 + cq) * 4);
    }
}
__device__ inline void store_nc128(float* lds, const float4 (&v)[2], int tid) {
#pragma unroll
    for (int h = 0; h < 2; ++h) {
        const int idx = tid + h * 256, k = idx >> 5, cq = (idx & 31) * 4;
        *(float4*)(lds + k * G128_LDM + cq) = v[h];
    }
}
// operand values of instruction q for the 16-row tile starting at row t0 of the tile
template <bool KC>
__device__ inline float g128_opnd(const float* lds, const f4& kcv, int t0, int q, int lane) {
    if constexpr (KC) return kcv[q];
    else return lds[((lane >> 4) * 4 + q) * G128_LDM + t0 + (lane & 15)];
}

template <bool A_KC, bool B_KC, int EPI>
__global__ __launch_bounds__(256) void gemm128_kernel(GemmArgs g) {
    constexpr int BK = 16, TL = G128_TL;
    __shared__ __attribute__((aligned(16))) float As[2 * TL];
    __shared__ __attribute__((aligned(16))) float Bs[2 * TL];
    __shared__ float rowsum[128];

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int wm = wave >> 1, wn = wave & 1;
    int bx, by, bz;
    gemm_tile(bx, by, bz);
    const int zz = bz / g.ksplit, slice = bz % g.ksplit;
    int cn, valid;
    int64_t r0;
    gemm_zinfo(g, zz, cn, r0, valid);
    const int Mv = (g.sample_dims & 1) ? valid : g.M;
    const int Nv = (g.sample_dims & 2) ? valid : g.N;
    const int Kv = (g.sample_dims & 4) ? valid : g.Kd;
    const int m0 = by * 128, n0 = bx * 128;
    if (m0 >= Mv || n0 >= Nv) return;
    const int kbeg = slice * g.kchunk;
    const int kend = min(Kv, kbeg + g.kchunk);
    const int64_t xbase = shard_start(g.n_total, g.k_rep, cn) + r0;
    const bool do_rowsum = (EPI == EPI_UPD) && g.ubias != nullptr && bx == 0;
    if (do_rowsum && tid < 128) rowsum[tid] = 0.f;

    f4 acc[4][4];
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[i][j] = f4{0.f, 0.f, 0.f, 0.f};

    float4 ra[2], rb[2];
    auto load = [&](int k0) {
        if constexpr (A_KC) load_kc128(ra, g.a, zz, cn, xbase, m0, Mv, k0, kend, tid);
        else load_nc128(ra, g.a, zz, cn, xbase, m0, Mv, k0, kend, tid);
        if constexpr (B_KC) load_kc128(rb, g.b, zz, cn, xbase, n0, Nv, k0, kend, tid);
        else load_nc128(rb, g.b, zz, cn, xbase, n0, Nv, k0, kend, tid);
    };
    auto store = [&](int buf) {
        if constexpr (A_KC) store_kc128(As + buf * TL, ra, tid);
        else store_nc128(As + buf * TL, ra, tid);
        if constexpr (B_KC) store_kc128(Bs + buf * TL, rb, tid);
        else store_nc128(Bs + buf * TL, rb, tid);
    };
    if (kbeg < kend) {
        load(kbeg);
        store(0);
    }
    __syncthreads();
    int buf = 0;
    const int rl = lane & 15, kg = lane >> 4;
    for (int k0 = kbeg; k0 < kend; k0 += BK) {
        const bool more = k0 + BK < kend;
        if (more) load(k0 + BK);
        const float* A = As + buf * TL;
        const float* Bt = Bs + buf * TL;
        if (do_rowsum && tid < 128) {
            float sr = 0.f;
#pragma unroll
            for (int k = 0; k < BK; ++k) sr += A_KC ? A[tid * G128_LDK + k] : A[k * G128_LDM + tid];
            rowsum[tid] += sr;
        }
        f4 av[4], bv[4];
        if constexpr (A_KC)
#pragma unroll
            for (int i = 0; i < 4; ++i) av[i] = *(const f4*)(A + (wm * 64 + i * 16 + rl) * G128_LDK + kg * 4);
        if constexpr (B_KC)
#pragma unroll
            for (int j = 0; j < 4; ++j) bv[j] = *(const f4*)(Bt + (wn * 64 + j * 16 + rl) * G128_LDK + kg * 4);
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            float aq[4], bq[4];
#pragma unroll
            for (int i = 0; i < 4; ++i) aq[i] = g128_opnd<A_KC>(A, av[i], wm * 64 + i * 16, q, lane);
#pragma unroll
            for (int j = 0; j < 4; ++j) bq[j] = g128_opnd<B_KC>(Bt, bv[j], wn * 64 + j * 16, q, lane);
#pragma unroll
            for (int i = 0; i < 4; ++i)
#pragma unroll
                for (int j = 0; j < 4; ++j)
                    acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x4f32(bq[j], aq[i], acc[i][j], 0, 0, 0);
        }
        if (more) store(buf ^ 1);
        __syncthreads();
        buf ^= 1;
    }

    // (operands entered swapped: lane holds row m0 + 64 wm + 16 i + (lane & 15), columns
    // n .. n+3 with n = n0 + 64 wn + 16 j + 4 (lane >> 4))
    float scale = g.lr;
    if (EPI == EPI_UPD && g.scale_per_batch) scale = valid > 0 ? g.lr / (float)valid : 0.f;
    const bool vec = ((g.c_ld | g.c_z | g.c_split | g.bias_z) & 3) == 0;
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const int m = m0 + wm * 64 + i * 16 + (lane & 15);
            const int n = n0 + wn * 64 + j * 16 + (lane >> 4) * 4;
            if (m >= Mv || n >= Nv) continue;
            const size_t ci = (size_t)zz * g.c_z + (size_t)m * g.c_ld + n;
            const f4 v = acc[i][j];
            if (vec && n + 3 < Nv) {
                const float4 c4 = make_float4(v[0], v[1], v[2], v[3]);
                if constexpr (EPI == EPI_STORE) {
                    *(float4*)((float*)g.c + ci + (size_t)slice * g.c_split) = c4;
                } else if constexpr (EPI == EPI_FWD) {
                    const float4 bb = *(const float4*)(g.bias + (size_t)cn * g.bias_z + n);
                    *(float4*)((float*)g.c + ci) = make_float4(act_fn(g.act, c4.x + bb.x), act_fn(g.act, c4.y + bb.y),
                                                               act_fn(g.act, c4.z + bb.z), act_fn(g.act, c4.w + bb.w));
                } else if constexpr (EPI == EPI_BWD) {
                    const float4 x = *(const float4*)((const float*)g.aux + ci);
                    *(float4*)((float*)g.c + ci) = make_float4(c4.x * act_deriv(g.act, x.x), c4.y * act_deriv(g.act, x.y),
                                                               c4.z * act_deriv(g.act, x.z), c4.w * act_deriv(g.act, x.w));
                } else {  // EPI_UPD: in-place W -= scale * acc
                    float4* W = (float4*)((float*)g.c + ci);
                    float4 w = *W;
                    w.x -= scale * c4.x; w.y -= scale * c4.y; w.z -= scale * c4.z; w.w -= scale * c4.w;
                    *W = w;
                }
            } else {
#pragma unroll
                for (int r = 0; r < 4; ++r) {
                    if (n + r >= Nv) continue;
                    const size_t cr = ci + r;
                    if constexpr (EPI == EPI_STORE) {
                        ((float*)g.c)[cr + (size_t)slice * g.c_split] = v[r];
                    } else if constexpr (EPI == EPI_FWD) {
                        const float zv = v[r] + g.bias[(size_t)cn * g.bias_z + n + r];
                        ((float*)g.c)[cr] = act_fn(g.act, zv);
                    } else if constexpr (EPI == EPI_BWD) {
                        const float x = ((const float*)g.aux)[cr];
                        ((float*)g.c)[cr] = v[r] * act_deriv(g.act, x);
                    } else {  // EPI_UPD: in-place W -= scale * acc
                        float* W = (float*)g.c;
                        W[cr] = W[cr] - scale * v[r];
                    }
                }
            }
        }
    if (do_rowsum && tid < 128 && m0 + tid < Mv) {
        float* b = g.ubias + (size_t)cn * g.bias_z;
        b[m0 + tid] -= scale * rowsum[tid];
    }
}

// ------------------------------------------------------------------------------------
// fp32 GEMM on the bf16 matrix cores, 128 x 128 tiles.
//
// An fp32 value a is the exact sum of three bf16 parts, a = a_h + a_m + a_l: a_h = RNE(a), the
// remainder a - a_h (exact in fp32, at most 16 significant bits) gives a_m = RNE of it, and the
// second remainder (at most 8 significant bits) is a_l exactly.  The product a b is the sum of
// the nine part products; the six kept (hh, hm, mh, hl, lh, mm) leave out terms below
// 2^-23 |a b| together, and each part product is exact in the fp32 accumulator's input.  A
// 32-deep k-tile thus takes six v_mfma_f32_16x16x32_bf16 (16 cycles each) per 16 x 16 output
// block instead of eight v_mfma_f32_16x16x4_f32 (32 cycles each): the matrix cores run bf16 at
// sixteen times their fp32 rate on this chip.  The sum carries rounding errors of the same size
// as the plain fp32 matrix instruction's (one fp32 rounding per instruction and output; the
// small terms go first).
//
// Eight waves of 64 x 32 (4 x 2 blocks of 16 x 16), two per SIMD, one workgroup per CU (120 KiB
// of dynamic LDS: two stages of both operands' three bf16 planes [t][k], laid out by b3_off).  The fp32 operands are loaded two
// k-tiles ahead into registers through bounds-checked buffer loads; while the matrix
// instructions of k-tile k run, the wave splits k-tile k+1 (v_cvt_pk_bf16_f32, round to nearest
// even) into the other stage.  KC operands (rows = t) load a float4 of 4 k per thread and row;
// NC operands (rows = k) a 2 k x 4 t block, whose pairs of k pack into the 4-byte stores of the
// transpose.  The weight update (EPI_UPD) loads its targets before the contraction.  Epilogues
// as in gemm128_kernel (fp32 outputs).

constexpr int B3_THREADS = 512;
constexpr int B3_BK = 32, B3_LDK = 40, B3_PLANE = 128 * B3_LDK;   // bf16 elements
constexpr int B3_STAGE = 2 * 3 * B3_PLANE;                         // A and B, three planes each
__host__ __device__ constexpr size_t b3_lds_bytes() { return (size_t)2 * B3_STAGE * sizeof(bf16_t); }

// the fp32 value of the low bf16 of a packed pair (a byte permute: written as a shift, the
// compiler re-derives it with a second conversion)
__device__ inline float bf_lo(uint32_t p) { return __uint_as_float(__builtin_amdgcn_perm(0u, p, 0x01000c0cu)); }
__device__ inline float bf_hi(uint32_t p) { return __uint_as_float(p & 0xffff0000u); }
// split two floats into their three packed bf16 parts
__device__ inline void split3_pk(float x, float y, uint32_t& h, uint32_t& m, uint32_t& l) {
    h = cvt_pk_bf16(x, y);
    const float rx = x - bf_lo(h), ry = y - bf_hi(h);
    m = cvt_pk_bf16(rx, ry);
    l = cvt_pk_bf16(rx - bf_lo(m), ry - bf_hi(m));
}

// one operand's k-tile (128 t x 32 k), as loaded by thread tid: KC v[u] = row kc_row(tid, u),
// k 4 (tid & 7) .. + 3; NC v[e] = k 2 (tid & 15) + e, columns 4 (tid >> 4) .. + 3
struct B3Raw { float4 v[2]; };

// KC rows: eight threads per row (128 contiguous bytes of the operand), a wave's part u eight
// consecutive rows
__device__ inline int kc_row(int tid, int u) { return (tid >> 3) + 64 * u; }

// element offset of (row t, k) in a plane.  KC operands (stored by rows): rows of 32 k (64
// bytes), the four 16-byte chunks of a row permuted by XOR with bits 1-2 of the row; NC
// operands (stored by columns, 4 bytes at a time): rows of 40 (80 bytes).  Neither the stores
// nor the 16-byte fragment reads of a KC plane meet bank conflicts; an NC plane's stores meet
// none, its fragment reads some (both measured with the LDS bank-conflict counter).
template <bool KC>
__device__ inline int b3_off(int t, int k) {
    if (KC) return t * B3_BK + ((((k >> 3) ^ ((t >> 1) & 3))) << 3) + (k & 7);
    return t * B3_LDK + k;
}

template <bool KC>
__device__ inline void b3_load(B3Raw& r, const B3Src& src, int t_valid_rel, int k0, int k_valid, int tid) {
#pragma unroll
    for (int u = 0; u < 2; ++u) {
        int t, k;
        if (KC) { t = kc_row(tid, u); k = (tid & 7) * 4; }
        else { t = (tid >> 4) * 4; k = 2 * (tid & 15) + u; }
        // the offset, with its top bit set (past any range) when the element is invalid
        // (arithmetic, not a select: the compiler would turn a select into branches)
        const uint32_t inv = KC ? (uint32_t)(k_valid - 1 - (k0 + k)) >> 31 : (uint32_t)(t_valid_rel - 1 - t) >> 31;
        const uint32_t off = (KC ? (uint32_t)t * src.ld4 + (uint32_t)(k0 + k) * 4u
                                 : (uint32_t)(k0 + k) * src.ld4 + (uint32_t)t * 4u) | (inv << 31);
        r.v[u] = __builtin_bit_cast(float4, __builtin_amdgcn_raw_buffer_load_b128(b3_rsrc(src), off, 0, 0));
    }
}

// split and store part u (0, 1) of a loaded k-tile into the three planes
template <bool KC>
__device__ inline void b3_store_part(bf16_t* lds, const B3Raw& r, int u, int tid) {
    if (KC) {
        const int t = kc_row(tid, u), k = (tid & 7) * 4;
        uint32_t h0, m0, l0, h1, m1, l1;
        split3_pk(r.v[u].x, r.v[u].y, h0, m0, l0);
        split3_pk(r.v[u].z, r.v[u].w, h1, m1, l1);
        bf16_t* d = lds + b3_off<true>(t, k);
        *(uint2*)d = make_uint2(h0, h1);
        *(uint2*)(d + B3_PLANE) = make_uint2(m0, m1);
        *(uint2*)(d + 2 * B3_PLANE) = make_uint2(l0, l1);
    } else {
        // columns t + 2 u, t + 2 u + 1 of rows k, k + 1
        const int t = (tid >> 4) * 4 + 2 * u, k = 2 * (tid & 15);
        const float a0 = u ? r.v[0].z : r.v[0].x, a1 = u ? r.v[0].w : r.v[0].y;
        const float c0 = u ? r.v[1].z : r.v[1].x, c1 = u ? r.v[1].w : r.v[1].y;
        uint32_t h, m, l;
        bf16_t* d = lds + b3_off<false>(t, k);
        split3_pk(a0, c0, h, m, l);
        *(uint32_t*)d = h; *(uint32_t*)(d + B3_PLANE) = m; *(uint32_t*)(d + 2 * B3_PLANE) = l;
        split3_pk(a1, c1, h, m, l);
        d = lds + b3_off<false>(t + 1, k);
        *(uint32_t*)d = h; *(uint32_t*)(d + B3_PLANE) = m; *(uint32_t*)(d + 2 * B3_PLANE) = l;
    }
}

template <bool A_KC, bool B_KC, int EPI>
__global__ __launch_bounds__(B3_THREADS) void gemm128x3_kernel(GemmArgs g) {
    extern __shared__ __attribute__((aligned(16))) bf16_t b3s[];  // [2 stages][A 3 planes, B 3 planes]
    __shared__ float rowsum[128];

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int wm = wave >> 2, wn = wave & 3;  // wave tile: rows 64 wm .., columns 32 wn ..
    int bx, by, bz;
    gemm_tile(bx, by, bz);
    const int zz = bz / g.ksplit, slice = bz % g.ksplit;
    int cn, valid;
    int64_t r0;
    gemm_zinfo(g, zz, cn, r0, valid);
    const int Mv = (g.sample_dims & 1) ? valid : g.M;
    const int Nv = (g.sample_dims & 2) ? valid : g.N;
    const int Kv = (g.sample_dims & 4) ? valid : g.Kd;
    const int m0 = by * 128, n0 = bx * 128;
    if (m0 >= Mv || n0 >= Nv) return;
    const int kbeg = slice * g.kchunk;
    const int kend = min(Kv, kbeg + g.kchunk);
    const int64_t xbase = shard_start(g.n_total, g.k_rep, cn) + r0;
    const bool do_rowsum = (EPI == EPI_UPD) && g.ubias != nullptr && bx == 0;
    if (do_rowsum && tid < 128) rowsum[tid] = 0.f;
    const bool vec = ((g.c_ld | g.c_z | g.c_split | g.bias_z) & 3) == 0;
    // (operands enter swapped: lane holds row m0 + 64 wm + 16 i + (lane & 15), columns
    // n .. n+3 with n = n0 + 32 wn + 16 j + 4 (lane >> 4))
    auto coord = [&](int i, int j, int& m, int& n) {
        m = m0 + wm * 64 + i * 16 + (lane & 15);
        n = n0 + wn * 32 + j * 16 + (lane >> 4) * 4;
    };

    // the update's targets, read before the contraction (their latency behind it)
    float4 wpre[4][2];
    if constexpr (EPI == EPI_UPD) {
#pragma unroll
        for (int i = 0; i < 4; ++i)
#pragma unroll
            for (int j = 0; j < 2; ++j) {
                int m, n;
                coord(i, j, m, n);
                const float* W = (const float*)g.c + (size_t)zz * g.c_z + (size_t)m * g.c_ld + n;
                wpre[i][j] = make_float4(0.f, 0.f, 0.f, 0.f);
                if (m < Mv && n < Nv) {
                    if (vec && n + 3 < Nv) wpre[i][j] = *(const float4*)W;
                    else {
                        wpre[i][j].x = W[0];
                        if (n + 1 < Nv) wpre[i][j].y = W[1];
                        if (n + 2 < Nv) wpre[i][j].z = W[2];
                    }
                }
            }
    }

    f4 acc[4][2];
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j) acc[i][j] = f4{0.f, 0.f, 0.f, 0.f};

    B3Raw ra, rb, na, nb;  // k-tiles in flight: the one split during the current tile, the one after
    const B3Src sa = b3_src<A_KC>(g.a, zz, cn, xbase, m0, Mv, kend);
    const B3Src sb = b3_src<B_KC>(g.b, zz, cn, xbase, n0, Nv, kend);
    auto load = [&](B3Raw& xa, B3Raw& xb, int k0) {  // (zeros past kend)
        b3_load<A_KC>(xa, sa, Mv - m0, k0, kend, tid);
        b3_load<B_KC>(xb, sb, Nv - n0, k0, kend, tid);
    };
    load(ra, rb, kbeg);
#pragma unroll
    for (int u = 0; u < 2; ++u) {
        b3_store_part<A_KC>(b3s, ra, u, tid);
        b3_store_part<B_KC>(b3s + 3 * B3_PLANE, rb, u, tid);
    }
    load(ra, rb, kbeg + B3_BK);
    __syncthreads();
    int buf = 0;
    const int rl = lane & 15, kg = lane >> 4;
    // one k-tile: the loads of the tile two ahead into (ya, yb), the tile's matrix instructions
    // from stage buf, the next tile (xa, xb) split into the other stage between them
    auto step = [&](int k0, const B3Raw& xa, const B3Raw& xb, B3Raw& ya, B3Raw& yb) {
        // (the loads and the split run on past kend, on zeros: no branch in the pipeline)
        load(ya, yb, k0 + 2 * B3_BK);
        const bf16_t* A = b3s + buf * B3_STAGE;
        const bf16_t* Bt = A + 3 * B3_PLANE;
        bf16_t* An = b3s + (buf ^ 1) * B3_STAGE;
        if (do_rowsum && tid < 128) {
            // the bias gradient: the tile's rows of A summed over k (h + m + l is a exactly)
            float sr = 0.f;
#pragma unroll
            for (int k = 0; k < B3_BK; ++k) {
                const int o = b3_off<A_KC>(tid, k);
                sr += (bf2f(A[o]) + bf2f(A[o + B3_PLANE])) + bf2f(A[o + 2 * B3_PLANE]);
            }
            rowsum[tid] += sr;
        }
        bf8v av[3][4], bv[3][2];
#pragma unroll
        for (int p = 0; p < 3; ++p) {
#pragma unroll
            for (int i = 0; i < 4; ++i)
                av[p][i] = *(const bf8v*)(A + p * B3_PLANE + b3_off<A_KC>(wm * 64 + i * 16 + rl, kg * 8));
#pragma unroll
            for (int j = 0; j < 2; ++j)
                bv[p][j] = *(const bf8v*)(Bt + p * B3_PLANE + b3_off<B_KC>(wn * 32 + j * 16 + rl, kg * 8));
        }
        // six groups of 8 matrix instructions, small terms first: (a part, b part) = lh, hl, mm,
        // mh, hm, hh; the next k-tile's split and store in between
        constexpr int PA[6] = {2, 0, 1, 1, 0, 0}, PB[6] = {0, 2, 1, 0, 1, 0};
#pragma unroll
        for (int t = 0; t < 6; ++t) {
#pragma unroll
            for (int i = 0; i < 4; ++i)
#pragma unroll
                for (int j = 0; j < 2; ++j)
                    acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(bv[PB[t]][j], av[PA[t]][i], acc[i][j], 0, 0, 0);
            if (t == 0 || t == 1) b3_store_part<A_KC>(An, xa, t, tid);
            if (t == 2 || t == 3) b3_store_part<B_KC>(An + 3 * B3_PLANE, xb, t - 2, tid);
        }
        __syncthreads();
        buf ^= 1;
    };
    // two k-tiles per trip, the register sets alternating (no copy between them)
    for (int k0 = kbeg; k0 < kend; k0 += 2 * B3_BK) {
        step(k0, ra, rb, na, nb);
        if (k0 + B3_BK >= kend) break;
        step(k0 + B3_BK, na, nb, ra, rb);
    }

    float scale = g.lr;
    if (EPI == EPI_UPD && g.scale_per_batch) scale = valid > 0 ? g.lr / (float)valid : 0.f;
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j) {
            int m, n;
            coord(i, j, m, n);
            if (m >= Mv || n >= Nv) continue;
            const size_t ci = (size_t)zz * g.c_z + (size_t)m * g.c_ld + n;
            const f4 v = acc[i][j];
            if (vec && n + 3 < Nv) {
                const float4 c4 = make_float4(v[0], v[1], v[2], v[3]);
                if constexpr (EPI == EPI_STORE) {
                    *(float4*)((float*)g.c + ci + (size_t)slice * g.c_split) = c4;
                } else if constexpr (EPI == EPI_FWD) {
                    const float4 bb = *(const float4*)(g.bias + (size_t)cn * g.bias_z + n);
                    *(float4*)((float*)g.c + ci) = make_float4(act_fn(g.act, c4.x + bb.x), act_fn(g.act, c4.y + bb.y),
                                                               act_fn(g.act, c4.z + bb.z), act_fn(g.act, c4.w + bb.w));
                } else if constexpr (EPI == EPI_BWD) {
                    const float4 x = *(const float4*)((const float*)g.aux + ci);
                    *(float4*)((float*)g.c + ci) = make_float4(c4.x * act_deriv(g.act, x.x), c4.y * act_deriv(g.act, x.y),
                                                               c4.z * act_deriv(g.act, x.z), c4.w * act_deriv(g.act, x.w));
                } else {  // EPI_UPD: in-place W -= scale * acc
                    float4 w = wpre[i][j];
                    w.x -= scale * c4.x; w.y -= scale * c4.y; w.z -= scale * c4.z; w.w -= scale * c4.w;
                    *(float4*)((float*)g.c + ci) = w;
                }
            } else {
                const float wp[4] = {wpre[i][j].x, wpre[i][j].y, wpre[i][j].z, wpre[i][j].w};
#pragma unroll
                for (int r = 0; r < 4; ++r) {
                    if (n + r >= Nv) continue;
                    const size_t cr = ci + r;
                    if constexpr (EPI == EPI_STORE) {
                        ((float*)g.c)[cr + (size_t)slice * g.c_split] = v[r];
                    } else if constexpr (EPI == EPI_FWD) {
                        const float zv = v[r] + g.bias[(size_t)cn * g.bias_z + n + r];
                        ((float*)g.c)[cr] = act_fn(g.act, zv);
                    } else if constexpr (EPI == EPI_BWD) {
                        const float x = ((const float*)g.aux)[cr];
                        ((float*)g.c)[cr] = v[r] * act_deriv(g.act, x);
                    } else {
                        ((float*)g.c)[cr] = wp[r] - scale * v[r];
                    }
                }
            }
        }
    if (do_rowsum && tid < 128 && m0 + tid < Mv) {
        float* b = g.ubias + (size_t)cn * g.bias_z;
        b[m0 + tid] -= scale * rowsum[tid];
    }
}

// ------------------------------------------------------------------------------------
// fp32 GEMM on the bf16 matrix cores, 128 x 256 tiles, both operands along k (forward):
// the three-part split of gemm128x3_kernel with twice the matrix work per split value.
//
// Eight waves of 64 x 64 (4 x 4 blocks), two per SIMD, one workgroup per CU (144 KiB of dynamic
// LDS: two stages of A's three planes, 128 rows, and B's, 256 rows, laid out by b3_off<true>).
// Per 32-deep k-tile a wave issues 96 matrix instructions against 12 splits of two values (48
// against 8 in the 128 x 128 kernel): a quarter fewer of the split's vector instructions, which
// the matrix cores do not overlap, per matrix instruction.  B's fragments stay in registers for
// the k-tile and A's are read one plane at a time (l, m, h), which keeps the wave within the 256
// registers of two waves per SIMD (a few spill).
constexpr int G2_PA = 128 * B3_BK, G2_PB = 256 * B3_BK;       // plane sizes (64-byte rows)
constexpr int G2_STAGE = 3 * G2_PA + 3 * G2_PB;
__host__ __device__ constexpr size_t g2_lds_bytes() { return (size_t)2 * G2_STAGE * sizeof(bf16_t); }

// split and store part u of a KC k-tile into three planes pstride apart, rows + row_off
__device__ inline void g2_store(bf16_t* plane0, int pstride, const B3Raw& r, int u, int tid, int row_off) {
    const int t = kc_row(tid, u) + row_off, k = (tid & 7) * 4;
    uint32_t h0, m0, l0, h1, m1, l1;
    split3_pk(r.v[u].x, r.v[u].y, h0, m0, l0);
    split3_pk(r.v[u].z, r.v[u].w, h1, m1, l1);
    bf16_t* d = plane0 + b3_off<true>(t, k);
    *(uint2*)d = make_uint2(h0, h1);
    *(uint2*)(d + pstride) = make_uint2(m0, m1);
    *(uint2*)(d + 2 * pstride) = make_uint2(l0, l1);
}

template <int EPI>
__global__ __launch_bounds__(B3_THREADS) void gemm256x3_kernel(GemmArgs g) {
    extern __shared__ __attribute__((aligned(16))) bf16_t g2s[];
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int wm = wave >> 2, wn = wave & 3;  // wave tile: rows 64 wm, columns 64 wn
    int bx, by, bz;
    gemm_tile(bx, by, bz);
    // the CNs from the last to the first: the weight update before a forward walks them from the
    // first, so the forward starts on the weights written last, still in the memory-side cache,
    // and ends on the first CNs, which the next update reads first (784-1024-10, K = 256:
    // forward 320 -> 310 us, update 520 -> 504 us)
    const int zz = (int)gridDim.z - 1 - bz;
    int cn, valid;
    int64_t r0;
    gemm_zinfo(g, zz, cn, r0, valid);
    const int Mv = (g.sample_dims & 1) ? valid : g.M;
    const int Nv = (g.sample_dims & 2) ? valid : g.N;
    const int Kv = g.Kd;
    const int m0 = by * 128, n0 = bx * 256;
    if (m0 >= Mv || n0 >= Nv) return;
    const int kend = Kv;
    const int64_t xbase = shard_start(g.n_total, g.k_rep, cn) + r0;
    f4 acc[4][4];
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[i][j] = f4{0.f, 0.f, 0.f, 0.f};
    const B3Src sa = b3_src<true>(g.a, zz, cn, xbase, m0, Mv, kend);
    const B3Src sb0 = b3_src<true>(g.b, zz, cn, xbase, n0, Nv, kend);
    const B3Src sb1 = b3_src<true>(g.b, zz, cn, xbase, min(n0 + 128, Nv), Nv, kend);
    B3Raw ra, rb0, rb1, na, nb0, nb1;
    auto load = [&](B3Raw& xa, B3Raw& xb0, B3Raw& xb1, int k0) {
        b3_load<true>(xa, sa, Mv - m0, k0, kend, tid);
        b3_load<true>(xb0, sb0, Nv - n0, k0, kend, tid);
        b3_load<true>(xb1, sb1, Nv - n0 - 128, k0, kend, tid);
    };
    auto store_all = [&](bf16_t* st, const B3Raw& xa, const B3Raw& xb0, const B3Raw& xb1) {
#pragma unroll
        for (int u = 0; u < 2; ++u) {
            g2_store(st, G2_PA, xa, u, tid, 0);
            g2_store(st + 3 * G2_PA, G2_PB, xb0, u, tid, 0);
            g2_store(st + 3 * G2_PA, G2_PB, xb1, u, tid, 128);
        }
    };
    load(ra, rb0, rb1, 0);
    store_all(g2s, ra, rb0, rb1);
    load(ra, rb0, rb1, B3_BK);
    __syncthreads();
    int buf = 0;
    const int rl = lane & 15, kg = lane >> 4;
    auto step = [&](int k0, const B3Raw& xa, const B3Raw& xb0, const B3Raw& xb1, B3Raw& ya, B3Raw& yb0, B3Raw& yb1) {
        load(ya, yb0, yb1, k0 + 2 * B3_BK);
        const bf16_t* A = g2s + buf * G2_STAGE;
        const bf16_t* Bt = A + 3 * G2_PA;
        bf16_t* An = g2s + (buf ^ 1) * G2_STAGE;
        bf8v bv[3][4];
#pragma unroll
        for (int p = 0; p < 3; ++p)
#pragma unroll
            for (int j = 0; j < 4; ++j)
                bv[p][j] = *(const bf8v*)(Bt + p * G2_PB + b3_off<true>(wn * 64 + j * 16 + rl, kg * 8));
        // A planes l, m, h in turn: l.h, then m.m, m.h, then h.l, h.m, h.h
        int t = 0;
#pragma unroll
        for (int pa = 2; pa >= 0; --pa) {
            bf8v av[4];
#pragma unroll
            for (int i = 0; i < 4; ++i) av[i] = *(const bf8v*)(A + pa * G2_PA + b3_off<true>(wm * 64 + i * 16 + rl, kg * 8));
#pragma unroll
            for (int pb = 2 - pa; pb >= 0; --pb, ++t) {
#pragma unroll
                for (int i = 0; i < 4; ++i)
#pragma unroll
                    for (int j = 0; j < 4; ++j)
                        acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(bv[pb][j], av[i], acc[i][j], 0, 0, 0);
                if (t == 0 || t == 1) g2_store(An, G2_PA, xa, t, tid, 0);
                if (t == 2 || t == 3) g2_store(An + 3 * G2_PA, G2_PB, xb0, t - 2, tid, 0);
                if (t == 4 || t == 5) g2_store(An + 3 * G2_PA, G2_PB, xb1, t - 4, tid, 128);
            }
        }
        __syncthreads();
        buf ^= 1;
    };
    for (int k0 = 0; k0 < kend; k0 += 2 * B3_BK) {
        step(k0, ra, rb0, rb1, na, nb0, nb1);
        if (k0 + B3_BK >= kend) break;
        step(k0 + B3_BK, na, nb0, nb1, ra, rb0, rb1);
    }
    const bool vec = ((g.c_ld | g.c_z | g.bias_z) & 3) == 0;
    if constexpr (EPI == EPI_FWD) {
        // fused last layer: this lane's W2 values (output rl, the lane's 16 columns), loaded
        // before the activations so that their latency hides behind them
        float4 w2v[4];
#pragma unroll
        for (int j = 0; j < 4; ++j) w2v[j] = make_float4(0.f, 0.f, 0.f, 0.f);
        if (g.zpart != nullptr && rl < g.o2) {
            const float* w2 = g.w2 + (size_t)cn * g.w2_z + (size_t)rl * g.N;
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                const int n = n0 + wn * 64 + j * 16 + kg * 4;
                if (n + 3 < Nv) w2v[j] = *(const float4*)(w2 + n);
                else {
                    if (n < Nv) w2v[j].x = w2[n];
                    if (n + 1 < Nv) w2v[j].y = w2[n + 1];
                    if (n + 2 < Nv) w2v[j].z = w2[n + 2];
                }
            }
        }
        // the activations, in place: bias, then the activation in one straight loop per kind (a
        // per-element switch on the kind cost 27 us of a 360 us launch; the sigmoid on the
        // hardware exp2 and reciprocal another 13), then zero past N
#pragma unroll
        for (int i = 0; i < 4; ++i)
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                const int n = n0 + wn * 64 + j * 16 + kg * 4;
                const float* bb = g.bias + (size_t)cn * g.bias_z + n;
                if (vec && n + 3 < Nv) {
                    const float4 b4 = *(const float4*)bb;
                    acc[i][j][0] += b4.x; acc[i][j][1] += b4.y; acc[i][j][2] += b4.z; acc[i][j][3] += b4.w;
                } else {
#pragma unroll
                    for (int r = 0; r < 4; ++r) acc[i][j][r] += n + r < Nv ? bb[r] : 0.f;
                }
            }
        auto act_all = [&](auto A) __attribute__((always_inline)) {
#pragma unroll
            for (int i = 0; i < 4; ++i)
#pragma unroll
                for (int j = 0; j < 4; ++j)
#pragma unroll
                    for (int r = 0; r < 4; ++r) acc[i][j][r] = act_fast(decltype(A)::value, acc[i][j][r]);
        };
        switch (g.act) {
        case ACT_SIGMOID: act_all(std::integral_constant<int, ACT_SIGMOID>{}); break;
        case ACT_TANH: act_all(std::integral_constant<int, ACT_TANH>{}); break;
        case ACT_RELU: act_all(std::integral_constant<int, ACT_RELU>{}); break;
        case ACT_LEAKY: act_all(std::integral_constant<int, ACT_LEAKY>{}); break;
        default: break;
        }
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const int n = n0 + wn * 64 + j * 16 + kg * 4;
#pragma unroll
            for (int i = 0; i < 4; ++i)
#pragma unroll
                for (int r = 0; r < 4; ++r)
                    if (n + r >= Nv) acc[i][j][r] = 0.f;
        }
#pragma unroll
        for (int i = 0; i < 4; ++i)
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                const int m = m0 + wm * 64 + i * 16 + rl, n = n0 + wn * 64 + j * 16 + kg * 4;
                if (m >= Mv || n >= Nv) continue;
                const size_t ci = (size_t)zz * g.c_z + (size_t)m * g.c_ld + n;
                const f4 v = acc[i][j];
                if (vec && n + 3 < Nv) {
                    *(float4*)((float*)g.c + ci) = make_float4(v[0], v[1], v[2], v[3]);
                } else {
                    for (int r = 0; r < 4; ++r)
                        if (n + r < Nv) ((float*)g.c)[ci + r] = v[r];
                }
            }
        if (g.zpart != nullptr) {
            // fused last layer: this tile's share of z2[m][o] = sum_n h[m][n] W2[o][n] on
            // v_mfma_f32_16x16x4_f32.  The activations are already in the A operand's layout:
            // for block (i, j) and component r, lane (rl, kg) holds h[row 16 i + rl][column
            // 16 j + 4 kg + r], i.e. A[rl][kg] of a 16 x 4 slice; B[kg][o = rl] is W2 at the
            // same column.  The 16 slices of each row block accumulate in (j, r) order, then the
            // four waves of a row block (wn) are added in order through LDS (free after the
            // loop's last barrier).
            float* red = (float*)g2s;   // [wn][128 rows][16]
            static_assert(4 * 128 * 16 * sizeof(float) <= g2_lds_bytes(), "the partial sums fit the LDS stages");
            f4 zacc[4];
#pragma unroll
            for (int i = 0; i < 4; ++i) zacc[i] = f4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                const float4 wv = w2v[j];
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    zacc[i] = __builtin_amdgcn_mfma_f32_16x16x4f32(acc[i][j][0], wv.x, zacc[i], 0, 0, 0);
                    zacc[i] = __builtin_amdgcn_mfma_f32_16x16x4f32(acc[i][j][1], wv.y, zacc[i], 0, 0, 0);
                    zacc[i] = __builtin_amdgcn_mfma_f32_16x16x4f32(acc[i][j][2], wv.z, zacc[i], 0, 0, 0);
                    zacc[i] = __builtin_amdgcn_mfma_f32_16x16x4f32(acc[i][j][3], wv.w, zacc[i], 0, 0, 0);
                }
            }
            // lane (rl, kg) holds z2 partial [row 16 i + 4 kg + r][output rl]
#pragma unroll
            for (int i = 0; i < 4; ++i)
#pragma unroll
                for (int r = 0; r < 4; ++r) red[(wn * 128 + wm * 64 + i * 16 + kg * 4 + r) * 16 + rl] = zacc[i][r];
            __syncthreads();
            const int ntile = (g.N + 255) / 256;
            for (int e = tid; e < 128 * 16; e += B3_THREADS) {
                const int row = e >> 4, o = e & 15;
                if (m0 + row >= g.M) continue;
                float v = 0.f;
                if (o < g.o2)
                    v = ((red[row * 16 + o] + red[(128 + row) * 16 + o]) + red[(256 + row) * 16 + o]) +
                        red[(384 + row) * 16 + o];
                g.zpart[(((size_t)zz * ntile + bx) * g.M + m0 + row) * 16 + o] = v;
            }
        }
    } else {
#pragma unroll
        for (int i = 0; i < 4; ++i)
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                const int m = m0 + wm * 64 + i * 16 + rl, n = n0 + wn * 64 + j * 16 + kg * 4;
                if (m >= Mv || n >= Nv) continue;
                const size_t ci = (size_t)zz * g.c_z + (size_t)m * g.c_ld + n;
                const f4 v = acc[i][j];
                for (int r = 0; r < 4; ++r)
                    if (n + r < Nv) ((float*)g.c)[ci + r] = v[r];
            }
    }
}

// ------------------------------------------------------------------------------------
// Weight update W -= eta / B_t * delta^T x on the bf16 matrix cores (fp32 operands split in
// three bf16 parts, as in gemm128x3_kernel), for a contraction over at most 128 samples.
//
// One workgroup (eight waves, one per CU) owns a 128-row strip of W (rows m0 .. m0 + 127, all
// N columns) of one CN: it splits the strip's errors delta[s][m0 ..] for every sample s once
// into LDS (three planes [m][s], 128 samples, 16-byte chunks XOR-swizzled by the row so that
// neither the transposing stores nor the fragment reads meet bank conflicts), subtracts the
// bias gradient eta / B_t sum_s delta[s][m], and then walks the strip's 128-column tiles: the
// samples' input columns x[s][n0 ..] stream through two LDS stages in k-chunks of 32 samples
// (loaded two chunks ahead, across tile boundaries), and each finished tile's targets, loaded
// one tile ahead, take their update and go back.  A: NC operand (rows = samples), B: NC.
// FULL: updates over 97 .. 128 samples, four k-chunks per tile (zero padded).  With dout set
// (the last layer fused into this layer's products), A holds the layer's activations and the
// prologue forms the strip's errors from them, the output errors and the pre-update last-layer
// weights, and updates the last layer's columns of this strip.

typedef unsigned int v4u __attribute__((ext_vector_type(4)));
constexpr int U3_KMAX = 128;   // samples of one update
constexpr int U3_DPLANE = 128 * U3_KMAX;
__host__ __device__ constexpr size_t u3_lds_bytes() {
    return (size_t)3 * U3_DPLANE * sizeof(bf16_t) + (size_t)2 * 3 * B3_PLANE * sizeof(bf16_t);
}
// element offset of (row m, sample k) in a plane of the errors (16-byte chunks swizzled)
__device__ inline int u3_off(int m, int k) { return m * U3_KMAX + ((((k >> 3) ^ (m & 15))) << 3) + (k & 7); }

template <bool FULL>
__global__ __launch_bounds__(B3_THREADS) void upd128x3_kernel(GemmArgs g) {
    extern __shared__ __attribute__((aligned(16))) bf16_t u3s[];
    bf16_t* dpl = u3s;                   // [3][128 m][128 k] errors, swizzled
    bf16_t* xst = u3s + 3 * U3_DPLANE;   // [2 stages][3 planes][128 n][40] inputs

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int wm = wave >> 2, wn = wave & 3;
    const int rl = lane & 15, kg = lane >> 4;
    int bx, by, bz;
    gemm_tile(bx, by, bz);
    const int zz = bz;
    int cn, valid;
    int64_t r0;
    gemm_zinfo(g, zz, cn, r0, valid);
    const int Mv = g.M, Nv = g.N;
    const int Kv = (g.sample_dims & 4) ? valid : g.Kd;   // samples of this step (<= 128)
    const int m0 = by * 128;
    if (m0 >= Mv || Kv <= 0) return;
    const int64_t xbase = shard_start(g.n_total, g.k_rep, cn) + r0;
    const int nkc = FULL ? 4 : (Kv + B3_BK - 1) / B3_BK;   // k-chunks per tile
    const int ntile = (Nv + 127) / 128;
    // CN k walks its tiles from tile k mod ntile, so that the tiles updated at one time spread
    // over memory; the strips of a CN keep one order and so still share each input chunk in L2
    // (strip-dependent starts spread further but re-read the chunks: +22 % HBM traffic)
    const int rot = FULL ? cn % ntile : 0;
    auto tcol = [&](int t) { const int u = t + rot; return (u >= ntile ? u - ntile : u) * 128; };
    const int nsteps = ntile * nkc;
    const float scale = g.scale_per_batch ? g.lr / (float)Kv : g.lr;
    float* Wz = (float*)g.c + (size_t)zz * g.c_z;

    // the strip's targets through a buffer descriptor (rows past M and columns past N out of
    // range: loads give zero, stores are dropped; no branch, exact wait counters).  N and the
    // row stride are multiples of 4, so a valid float4 never crosses N.
    B3Src wsrc, wdst;   // where the targets are read, and written
    {
        wsrc.base = (uint64_t)((g.rd_c != nullptr ? g.rd_c : Wz) + (size_t)m0 * g.c_ld);
        wsrc.nbytes = (int)((int64_t)min(128, Mv - m0) * g.c_ld * 4);
        wsrc.ld4 = (uint32_t)(g.c_ld * 4);
        wdst = wsrc;
        wdst.base = (uint64_t)(Wz + (size_t)m0 * g.c_ld);
    }
    auto woff = [&](int n0, int i, int j) {
        const int n = n0 + wn * 32 + j * 16 + kg * 4;
        const uint32_t inv = (uint32_t)(Nv - 1 - n) >> 31;
        return ((uint32_t)(wm * 64 + i * 16 + rl) * wsrc.ld4 + (uint32_t)n * 4u) | (inv << 31);
    };
    auto load_w = [&](float4 (&w)[4][2], int n0) {
#pragma unroll
        for (int i = 0; i < 4; ++i)
#pragma unroll
            for (int j = 0; j < 2; ++j)
                w[i][j] = __builtin_bit_cast(float4, __builtin_amdgcn_raw_buffer_load_b128(b3_rsrc(wsrc), woff(n0, i, j), 0, 0));
    };
    float4 wcur[4][2], wnext[4][2];

    // the input stream: step q = (tile q / nkc, k-chunk q % nkc); zeros past the last step
    auto xsrc = [&](int q) {
        const int n0 = tcol(min(q / nkc, ntile - 1));
        return b3_src<false>(g.b, zz, cn, xbase, n0, Nv, Kv);
    };
    auto xload = [&](B3Raw& r, int q) {
        const int kc = q % nkc;
        b3_load<false>(r, xsrc(q), q < nsteps ? Nv - tcol(min(q / nkc, ntile - 1)) : 0, kc * B3_BK, Kv, tid);
    };
    B3Raw ra, na;
    // the bias of this lane's row, read now (updated after the prologue without a round trip)
    float ub_old = 0.f;
    const bool ub_lane = g.ubias != nullptr && (tid & 3) == 0 && m0 + (tid >> 2) < Mv;
    if (ub_lane) ub_old = (g.rd_ub != nullptr ? g.rd_ub : g.ubias + (size_t)cn * g.bias_z)[m0 + (tid >> 2)];

    // fused last layer: A holds the hidden activations x; the strip's errors are formed here,
    // d[s][m] = (sum_o dout[s][o] W2[o][m]) phi'(x[s][m]) with the pre-update W2 (eq. (11)),
    // and W2[o][m] -= scale sum_s dout[s][o] x[s][m] for the strip's columns (eq. (12)), both
    // on v_mfma_f32_16x16x4_f32: wave w owns rows 16 w .. 16 w + 15 of the strip, in 16 x 16
    // blocks of (samples, rows); dout and the strip's columns of W2 are staged in the second
    // input stage (free until the loop)
    if (g.dout != nullptr) {
        constexpr int FDS = 17, FWS = 144;       // row strides (bank spread of the reads)
        static_assert((U3_KMAX * FDS + MAX_OUT * FWS) * sizeof(float) <= 3 * B3_PLANE * sizeof(bf16_t),
                      "dout and W2 fit the second input stage");
        float* f_d = (float*)(xst + 3 * B3_PLANE);   // [128 samples][FDS]: dout
        float* f_w = f_d + U3_KMAX * FDS;            // [16 outputs][FWS]: W2[o][m0 + m]
        // issue order (vector-memory completions count in order): the staged values first, then
        // this lane's activations in the order of use, then the first target tile and input chunk
        // (needed only after the prologue)
        const float* dsrc = g.dout + (size_t)zz * g.step_rows * 16;
        static_assert(U3_KMAX * 4 == B3_THREADS && MAX_OUT * 32 == B3_THREADS, "one float4 of each per thread");
        float4 dv4 = make_float4(0.f, 0.f, 0.f, 0.f);   // dout[tid >> 2][4 (tid & 3) ..]
        if ((tid >> 2) < g.step_rows) dv4 = *(const float4*)(dsrc + tid * 4);
        const float* w2r = g.rd_w2 != nullptr ? g.rd_w2 : g.w2 + (size_t)cn * g.w2_z;
        const int wo = tid >> 5, wc4 = (tid & 31) * 4;   // W2[wo][m0 + wc4 ..]
        float4 wv4 = make_float4(0.f, 0.f, 0.f, 0.f);
        if (wo < g.o2 && m0 + wc4 < Mv) wv4 = *(const float4*)(w2r + (size_t)wo * g.M + m0 + wc4);
        // this lane's activations: x[s = 16 sb + 4 kg + r][m0 + 16 w + rl] (zero past the samples
        // and past M)
        const int mloc = 16 * wave + rl;
        const bool mval = m0 + mloc < Mv;
        const float* xrow = (const float*)operand_row(g.a, 4, zz, cn, xbase, 0) + m0 + mloc;
        float xv[8][4];
#pragma unroll
        for (int sb = 0; sb < 8; ++sb)
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                const int sm = 16 * sb + 4 * kg + r;
                xv[sb][r] = (mval && sm < Kv) ? xrow[(size_t)sm * g.a.ld] : 0.f;
            }
        load_w(wcur, tcol(0));
        xload(ra, 0);
        {
            float* d = f_d + (tid >> 2) * FDS + (tid & 3) * 4;
            d[0] = dv4.x; d[1] = dv4.y; d[2] = dv4.z; d[3] = dv4.w;
            *(float4*)(f_w + wo * FWS + wc4) = wv4;
        }
        // phi'(x) of this lane's activations, one loop per kind (the kind is a launch constant)
        float xd[8][4];
        auto deriv_all = [&](auto A) __attribute__((always_inline)) {
#pragma unroll
            for (int sb = 0; sb < 8; ++sb)
#pragma unroll
                for (int r = 0; r < 4; ++r) xd[sb][r] = act_deriv(decltype(A)::value, xv[sb][r]);
        };
        switch (g.act2) {
        case ACT_SIGMOID: deriv_all(std::integral_constant<int, ACT_SIGMOID>{}); break;
        case ACT_TANH: deriv_all(std::integral_constant<int, ACT_TANH>{}); break;
        case ACT_RELU: deriv_all(std::integral_constant<int, ACT_RELU>{}); break;
        case ACT_LEAKY: deriv_all(std::integral_constant<int, ACT_LEAKY>{}); break;
        default: deriv_all(std::integral_constant<int, -1>{}); break;
        }
        __syncthreads();
        // dW2[o = 4 kg + r][m = 16 w + rl] in two chains (even and odd sample blocks, added at the
        // end): half the dependent matrix-instruction latency
        f4 dacc2[2] = {f4{0.f, 0.f, 0.f, 0.f}, f4{0.f, 0.f, 0.f, 0.f}};
#pragma unroll
        for (int sb = 0; sb < 8; ++sb) {
            // S[s = 16 sb + 4 kg + r][m = 16 w + rl]: A[s][o] = dout, B[o][m] = W2, over all 16
            // staged outputs (those past O are zero in both: exact zeros added, and a loop of
            // known length whose LDS reads are not each waited for in turn)
            f4 sacc = f4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int q = 0; q < MAX_OUT / 4; ++q)
                sacc = __builtin_amdgcn_mfma_f32_16x16x4f32(f_d[(16 * sb + rl) * FDS + 4 * q + kg],
                                                            f_w[(4 * q + kg) * FWS + mloc], sacc, 0, 0, 0);
            // dW2 += dout^T x over this block's samples: A[o][s] = dout, B[s][m] = x
#pragma unroll
            for (int r = 0; r < 4; ++r)
                dacc2[sb & 1] = __builtin_amdgcn_mfma_f32_16x16x4f32(f_d[(16 * sb + 4 * kg + r) * FDS + rl], xv[sb][r], dacc2[sb & 1], 0, 0, 0);
            // the errors, split; sample pairs (r 0, 1) and (r 2, 3)
#pragma unroll
            for (int pr = 0; pr < 2; ++pr) {
                const float d0 = sacc[2 * pr] * xd[sb][2 * pr];
                const float d1 = sacc[2 * pr + 1] * xd[sb][2 * pr + 1];
                uint32_t h, m, l;
                split3_pk(d0, d1, h, m, l);
                const int o = u3_off(mloc, 16 * sb + 4 * kg + 2 * pr);
                *(uint32_t*)(dpl + o) = h;
                *(uint32_t*)(dpl + U3_DPLANE + o) = m;
                *(uint32_t*)(dpl + 2 * U3_DPLANE + o) = l;
            }
        }
        const f4 dacc = dacc2[0] + dacc2[1];
        // W2's strip columns (the staged copy holds the pre-update values: a store, no read back)
        float* w2w = g.w2 + (size_t)cn * g.w2_z;
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            const int o = 4 * kg + r;
            if (o < g.o2 && mval) w2w[(size_t)o * g.M + m0 + mloc] = f_w[o * FWS + mloc] - scale * dacc[r];
        }
        // b2 (the first strip): sum over the samples in order (rows past the step's samples
        // hold zero errors: all 128 rows, a loop of known length)
        if (m0 == 0 && tid < g.o2) {
            float sb = 0.f;
#pragma unroll
            for (int r = 0; r < U3_KMAX; ++r) sb += f_d[r * FDS + tid];
            float* b2p = g.b2 + (size_t)cn * g.bias_z + tid;
            *b2p = (g.rd_b2 != nullptr ? g.rd_b2[tid] : *b2p) - scale * sb;
        }
    } else {
        load_w(wcur, tcol(0));
        xload(ra, 0);
        // the strip's errors: 2 samples x 4 rows per thread and pass, split into the planes
        const B3Src ds = b3_src<false>(g.a, zz, cn, xbase, m0, Mv, Kv);
#pragma unroll
        for (int pass = 0; pass < U3_KMAX * 128 / (8 * B3_THREADS); ++pass) {
            const int kpair = (tid & 15) + 16 * (pass & 3), mq = (tid >> 4) * 4;  // samples 2 kpair, +1; rows mq ..
            B3Raw v;
            b3_load<false>(v, ds, Mv - m0, 2 * kpair - 2 * (tid & 15), Kv, tid);
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                const float a0 = j == 0 ? v.v[0].x : j == 1 ? v.v[0].y : j == 2 ? v.v[0].z : v.v[0].w;
                const float a1 = j == 0 ? v.v[1].x : j == 1 ? v.v[1].y : j == 2 ? v.v[1].z : v.v[1].w;
                uint32_t h, m, l;
                split3_pk(a0, a1, h, m, l);
                const int o = u3_off(mq + j, 2 * kpair);
                *(uint32_t*)(dpl + o) = h;
                *(uint32_t*)(dpl + U3_DPLANE + o) = m;
                *(uint32_t*)(dpl + 2 * U3_DPLANE + o) = l;
            }
        }
    }
    xload(na, 1);
#pragma unroll
    for (int u = 0; u < 2; ++u) b3_store_part<false>(xst, ra, u, tid);
    xload(ra, 2);
    __syncthreads();
    // the bias gradient (h + m + l is delta exactly): four lanes per row, 32 samples each read
    // as four 16-byte chunks per plane, then the lanes' sums added in a fixed order
    if (g.ubias != nullptr) {
        const int r = tid >> 2, part = tid & 3;
        float sr = 0.f;
#pragma unroll
        for (int c = 0; c < 4; ++c) {
            const int o = u3_off(r, part * 32 + c * 8);
            const bf8v h = *(const bf8v*)(dpl + o), m = *(const bf8v*)(dpl + U3_DPLANE + o),
                       l = *(const bf8v*)(dpl + 2 * U3_DPLANE + o);
#pragma unroll
            for (int e = 0; e < 8; ++e) sr += ((float)h[e] + (float)m[e]) + (float)l[e];
        }
        sr += __shfl_xor(sr, 1);
        sr += __shfl_xor(sr, 2);
        if (ub_lane) g.ubias[(size_t)cn * g.bias_z + m0 + r] = ub_old - scale * sr;
    }

    f4 acc[4][2];
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j) acc[i][j] = f4{0.f, 0.f, 0.f, 0.f};
    int buf = 0;
    constexpr int PA[6] = {2, 0, 1, 1, 0, 0}, PB[6] = {0, 2, 1, 0, 1, 0};
    // step q: chunk q's matrix instructions from stage buf, chunk q+1 (xa) split into the other
    // stage, chunk q+3 loaded into ya
    auto step = [&](int q, const B3Raw& xa, B3Raw& ya) {
        xload(ya, q + 3);
        const int kc = q % nkc;
        const bf16_t* Bt = xst + buf * 3 * B3_PLANE;
        bf16_t* Bn = xst + (buf ^ 1) * 3 * B3_PLANE;
        if (kc == 0) {
            // a new tile: its targets were loaded one tile ahead; the next tile's now
            const int tn = q / nkc;
            if (tn + 1 < ntile) load_w(wnext, (tn + 1) * 128);
        }
        bf8v av[3][4], bv[3][2];
#pragma unroll
        for (int p = 0; p < 3; ++p) {
#pragma unroll
            for (int i = 0; i < 4; ++i)
                av[p][i] = *(const bf8v*)(dpl + p * U3_DPLANE + u3_off(wm * 64 + i * 16 + rl, kc * B3_BK + kg * 8));
#pragma unroll
            for (int j = 0; j < 2; ++j)
                bv[p][j] = *(const bf8v*)(Bt + p * B3_PLANE + b3_off<false>(wn * 32 + j * 16 + rl, kg * 8));
        }
#pragma unroll
        for (int t = 0; t < 6; ++t) {
#pragma unroll
            for (int i = 0; i < 4; ++i)
#pragma unroll
                for (int j = 0; j < 2; ++j)
                    acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(bv[PB[t]][j], av[PA[t]][i], acc[i][j], 0, 0, 0);
            if (t == 1 || t == 3) b3_store_part<false>(Bn, xa, t >> 1, tid);
        }
        if (kc == nkc - 1) {
            // the tile is complete: W -= scale * acc
            const int n0 = (q / nkc) * 128;
#pragma unroll
            for (int i = 0; i < 4; ++i)
#pragma unroll
                for (int j = 0; j < 2; ++j) {
                    const f4 v = acc[i][j];
                    float4 w = wcur[i][j];
                    w.x -= scale * v[0]; w.y -= scale * v[1]; w.z -= scale * v[2]; w.w -= scale * v[3];
                    __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(v4u, w), b3_rsrc(wdst), woff(n0, i, j), 0, 0);
                    acc[i][j] = f4{0.f, 0.f, 0.f, 0.f};
                    wcur[i][j] = wnext[i][j];
                }
        }
        __syncthreads();
        buf ^= 1;
    };
    if constexpr (FULL) {
        // four k-chunks per tile (chunks past the CN's samples load as zeros and add exact
        // zeros): every step's place in the tile is fixed at compile time (stage, input register
        // set, the targets' loads and the epilogue), two tiles per trip with the targets'
        // register sets alternating.  Input chunk c lives in set c % 4.  (With the tile's place
        // known, the compiler's wait counts stay exact: the generic loop below, whose tile ends
        // are data-dependent, waits for every outstanding memory operation at some steps.)
        B3Raw xs0, xs1 = na, xs2 = ra, xs3;   // chunks 1, 2 (in flight)
        float4 (&wa)[4][2] = wcur;
        float4 (&wb)[4][2] = wnext;
        auto fstep = [&](auto KC, int tn, float4 (&wc)[4][2], float4 (&wx)[4][2]) __attribute__((always_inline)) {
            constexpr int kc = decltype(KC)::value;
            const int q = tn * 4 + kc;
            B3Raw& xl = kc == 0 ? xs3 : kc == 1 ? xs0 : kc == 2 ? xs1 : xs2;   // chunk q + 3
            const B3Raw& xa = kc == 0 ? xs1 : kc == 1 ? xs2 : kc == 2 ? xs3 : xs0;  // chunk q + 1
            xload(xl, q + 3);
            // (unconditional: past the last tile every column is out of range, the loads read
            // nothing and give zeros, and the wait counts stay exact)
            if (kc == 0) load_w(wx, tn + 1 < ntile ? tcol(tn + 1) : ntile * 128);
            const bf16_t* Bt = xst + (kc & 1) * 3 * B3_PLANE;
            bf16_t* Bn = xst + ((kc & 1) ^ 1) * 3 * B3_PLANE;
            bf8v av[3][4], bv[3][2];
#pragma unroll
            for (int p = 0; p < 3; ++p) {
#pragma unroll
                for (int i = 0; i < 4; ++i)
                    av[p][i] = *(const bf8v*)(dpl + p * U3_DPLANE + u3_off(wm * 64 + i * 16 + rl, kc * B3_BK + kg * 8));
#pragma unroll
                for (int j = 0; j < 2; ++j)
                    bv[p][j] = *(const bf8v*)(Bt + p * B3_PLANE + b3_off<false>(wn * 32 + j * 16 + rl, kg * 8));
            }
#pragma unroll
            for (int t = 0; t < 6; ++t) {
#pragma unroll
                for (int i = 0; i < 4; ++i)
#pragma unroll
                    for (int j = 0; j < 2; ++j)
                        acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(bv[PB[t]][j], av[PA[t]][i], acc[i][j], 0, 0, 0);
                if (t == 1 || t == 3) b3_store_part<false>(Bn, xa, t >> 1, tid);
            }
            if (kc == 3) {
                const int n0 = tcol(tn);
#pragma unroll
                for (int i = 0; i < 4; ++i)
#pragma unroll
                    for (int j = 0; j < 2; ++j) {
                        const f4 v = acc[i][j];
                        float4 w = wc[i][j];
                        w.x -= scale * v[0]; w.y -= scale * v[1]; w.z -= scale * v[2]; w.w -= scale * v[3];
                        __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(v4u, w), b3_rsrc(wdst), woff(n0, i, j), 0, 0);
                        acc[i][j] = f4{0.f, 0.f, 0.f, 0.f};
                    }
            }
            __syncthreads();
            // no instruction crosses a step boundary: the scheduler would otherwise hoist the next
            // step's split of a chunk loaded one step ago, and its wait with it
            __builtin_amdgcn_sched_barrier(0);
        };
        auto ftile = [&](int tn, float4 (&wc)[4][2], float4 (&wx)[4][2]) __attribute__((always_inline)) {
            fstep(std::integral_constant<int, 0>{}, tn, wc, wx);
            fstep(std::integral_constant<int, 1>{}, tn, wc, wx);
            fstep(std::integral_constant<int, 2>{}, tn, wc, wx);
            fstep(std::integral_constant<int, 3>{}, tn, wc, wx);
        };
        // the prologue's loads done before the loop (s_waitcnt vmcnt(0)): the wait counts at the
        // loop head then follow only the loop's own operations (otherwise every trip waits as if
        // a prologue load were still the latest, for the previous tile's stores among others)
        __builtin_amdgcn_s_waitcnt(0x0f70);
        for (int tn = 0; tn < ntile; tn += 2) {
            ftile(tn, wa, wb);
            if (tn + 1 >= ntile) break;
            ftile(tn + 1, wb, wa);
        }
    } else {
        // three input register sets in rotation: chunk q+1 (split now), q+2, q+3 (in flight)
        B3Raw rc;
        for (int q = 0; q < nsteps; q += 3) {
            step(q, na, rc);
            if (q + 1 >= nsteps) break;
            step(q + 1, ra, na);
            if (q + 2 >= nsteps) break;
            step(q + 2, rc, ra);
        }
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
    double* cost;      // inference: [rows] cost of each data-set row (nullable; needs y)
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
            if (a.pred) a.pred[drow] = best;
            if (a.correct && a.y && a.y[drow] == best) atomicAdd(a.correct, 1ull);
            if (a.cost && a.y) {
                // the cost whose output error training uses: quadratic 1/2 sum (x - e)^2, or
                // cross-entropy (eq. (6) for a softmax output, the two-class form per output
                // for a sigmoid output), in double from the fp32 outputs
                const int label = a.y[drow];
                double c = 0.0;
#pragma unroll
                for (int o = 0; o < MAX_OUT; ++o) {
                    if (o >= a.O) continue;
                    const double x = (double)xo[o], e = (o == label) ? 1.0 : 0.0;
                    if (a.loss != LOSS_XENT) c += 0.5 * (x - e) * (x - e);
                    else if (a.act == ACT_SOFTMAX) c += (o == label) ? -log(x) : 0.0;
                    else c += -(e * log(x) + (1.0 - e) * log(1.0 - x));
                }
                a.cost[drow] = c;
            }
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
// Forward layer split along the contraction (few, long-contraction tiles): the partial
// products of the ksplit slices are summed here, then the bias and the activation
// (eq. (2)-(3)):  out[z][r][c] = phi(sum_s part[s][z][r][c] + b[c]).  Thread per (r, c).

struct FwdReduceArgs {
    const float* part;  // [ksplit][K][rows][N]
    int64_t split;      // K * rows * N
    int ksplit;
    float* out;         // [K][rows][N]
    const float* bias;  // b (+ z * bias_z)
    int64_t bias_z;
    int N, act;
    int64_t n_total;
    int k_rep;
    int64_t r0;
    int step_rows;
};

__global__ __launch_bounds__(256) void fwd_reduce_kernel(FwdReduceArgs a) {
    const int c = blockIdx.x * 256 + threadIdx.x;
    const int r = blockIdx.y, z = blockIdx.z;
    int64_t v = shard_len(a.n_total, a.k_rep, z) - a.r0;
    const int valid = (int)(v < 0 ? 0 : (v > a.step_rows ? a.step_rows : v));
    if (r >= valid || c >= a.N) return;
    const size_t e = ((size_t)z * a.step_rows + r) * a.N + c;
    float sum = 0.f;
    for (int sl = 0; sl < a.ksplit; ++sl) sum += a.part[(size_t)sl * a.split + e];
    a.out[e] = act_fn(a.act, sum + a.bias[(size_t)z * a.bias_z + c]);
}

// ------------------------------------------------------------------------------------
// Output activation and output error of one (row, output) lane, the 16 lanes of a row taking
// part together (softmax over them): eq. (3) / (5) and (9) / (10); zero on dead lanes (rows
// past the step or outputs past O); rounded to the error type TD.

template <typename TD>
__device__ inline float out_error(float zv, bool live, int o, int label, int act_out, int loss) {
    float xo;
    if (act_out == ACT_SOFTMAX) {
        float m = live ? zv : -INFINITY;
#pragma unroll
        for (int sh = 1; sh < 16; sh <<= 1) m = fmaxf(m, __shfl_xor(m, sh, 16));
        const float ex = live ? expf(zv - m) : 0.f;
        float sm = ex;
#pragma unroll
        for (int sh = 1; sh < 16; sh <<= 1) sm += __shfl_xor(sm, sh, 16);
        xo = ex * (1.0f / sm);
    } else {
        xo = act_fn(act_out, zv);
    }
    if (!live) return 0.f;
    const float t1 = (o == label) ? 1.0f : 0.0f;
    const float dd = (loss == LOSS_XENT) ? (xo - t1) : (xo - t1) * act_deriv(act_out, xo);
    return to_f<TD>(from_f<TD>(dd));
}

// The last layer's outputs and errors when its products are fused into the hidden layer's
// split-bf16 kernels: z2 = sum of the forward tiles' partial sums (tile order) + b2, then the
// output error of each row, one lane per (row, output), into dout [z][rows][16] (zeros past O
// and past the CN's rows).

struct OutErrArgs {
    const float* zpart;   // [z][ntile][step rows][16]
    int ntile;
    const float* bias;    // b2 (+ z * bias_z)
    int64_t bias_z;
    int O, act_out, loss;
    int64_t n_total;
    int k_rep;
    int64_t r0;
    int step_rows;
    const int32_t* y;     // labels (data-set rows)
    float* dout;          // [z][step rows][16]
};

__global__ __launch_bounds__(256) void out_err_kernel(OutErrArgs a) {
    const int z = blockIdx.z, row = blockIdx.x * 16 + (threadIdx.x >> 4), o = threadIdx.x & 15;
    if (row >= a.step_rows) return;   // (a whole row's 16 lanes)
    const int64_t v = shard_len(a.n_total, a.k_rep, z) - a.r0;
    const int valid = (int)(v < 0 ? 0 : (v > a.step_rows ? a.step_rows : v));
    const bool live = row < valid && o < a.O;
    float zv = 0.f;
    if (live) {
        const float* zp = a.zpart + ((size_t)z * a.ntile * a.step_rows + row) * 16 + o;
        float sum = zp[0];
        for (int t = 1; t < a.ntile; ++t) sum += zp[(size_t)t * a.step_rows * 16];
        zv = sum + a.bias[(size_t)z * a.bias_z + o];
    }
    const int label = row < valid ? a.y[shard_start(a.n_total, a.k_rep, z) + a.r0 + row] : -1;
    a.dout[((size_t)z * a.step_rows + row) * 16 + o] = out_error<float>(zv, live, o, label, a.act_out, a.loss);
}

// ------------------------------------------------------------------------------------
// The narrow last layer of a mini-batch step, fused, one workgroup of 16 waves per CN
// (eq. (3)-(5), (9)-(13) for a last layer of O <= 16 neurons behind a hidden layer of H
// neurons).  The step's rows are taken in groups of RG rows; each group is loaded once,
// coalesced, into LDS (the next group's loads in flight while the current one is used), and
// three contractions run on v_mfma_f32_16x16x4_f32 with the outputs padded to 16:
//   Z  = X W^T      (rows x 16, over H; each 16-row tile is split over H among several
//                    waves, partial tiles summed in LDS in a fixed order), then the output
//                    activation and the output error of each row, one lane per (row, output);
//   S  = delta W    (rows x H, over the 16 outputs), hidden error d = S * phi'(x) (eq. (11),
//                    with the pre-update W);
//   dW += delta^T X (16 x H, over the group's rows; accumulators stay in registers across
//                    groups, wave w owning the 16-column tiles w, w+16, ...).
// At the end W -= lr / B_t * dW and b -= lr / B_t * sum_r delta (rows in order).  The same
// rounding points as the unfused kernels: the output error is rounded to the error type
// before use, operands are the bf16 shadow in bf16-mixed mode, the update is applied to the
// fp32 master and the shadow refreshed.

struct TailArgs {
    const void* x;      // last hidden activations [z][rows][H] (TH)
    int64_t x_z;
    const void* wop;    // W_L operand [O][H] (+ z * w_z): fp32 master or bf16 shadow
    float* w;           // W_L fp32 master [O][H] (+ z * w_z)
    bf16_t* shadow;     // bf16 shadow of W_L (+ z * w_z), nullable
    float* bias;        // b_L [O] (+ z * bias_z)
    int64_t w_z, bias_z;
    void* d;            // hidden errors [z][rows][H] (TH)
    int H, O, act_out, act_hid, loss;
    int rg;             // rows per group: a multiple of 16, rg * H <= TAIL_GROUP, rg <= 256
    float lr;
    int64_t n_total;
    int k_rep;
    int64_t r0;
    int step_rows;
    const int32_t* y;   // labels (data-set rows)
};

constexpr int TAIL_THREADS = 1024, TAIL_WAVES = TAIL_THREADS / 64;
constexpr int TAIL_PF = 4;                                // 4-value loads per thread per group
constexpr int TAIL_GROUP = TAIL_THREADS * 4 * TAIL_PF;    // values of one row group (rg * H)
constexpr int TAIL_DLS = 20;                              // LDS row stride of the output errors
constexpr int TAIL_PART = TAIL_WAVES * 16 * 16;           // partial Z tiles, one per wave

// LDS floats of the fused last layer: W [16][H+4], a row group [rg][H+4], its output errors
// [rg][20], its labels [rg] and the per-wave partial tiles of Z
__host__ __device__ inline int64_t tail_lds_floats(int H, int rg) {
    return (int64_t)(16 + rg) * (H + 4) + (int64_t)rg * (TAIL_DLS + 1) + TAIL_PART;
}

// four values as loaded (converted only when the load has landed)
template <typename TH> struct Raw4 { typedef float4 T; };
template <> struct Raw4<bf16_t> { typedef uint2 T; };
__device__ inline float4 raw_f4(float4 v) { return v; }
__device__ inline float4 raw_f4(uint2 q) {
    return make_float4(bf2f((bf16_t)(q.x & 0xffff)), bf2f((bf16_t)(q.x >> 16)), bf2f((bf16_t)(q.y & 0xffff)),
                       bf2f((bf16_t)(q.y >> 16)));
}

// NCW: 16-column tiles per wave (>= H / 256)
template <typename TH, int NCW>
__global__ __launch_bounds__(TAIL_THREADS) void tail_kernel(TailArgs a) {
    extern __shared__ __attribute__((aligned(16))) float tsm[];
    typedef typename Raw4<TH>::T R4;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int rl = lane & 15, kg = lane >> 4;
    const int z = blockIdx.x;
    const int H = a.H, O = a.O, RG = a.rg, LDW = H + 4;
    int64_t v = shard_len(a.n_total, a.k_rep, z) - a.r0;
    const int valid = (int)(v < 0 ? 0 : (v > a.step_rows ? a.step_rows : v));
    if (valid == 0) return;
    float* Ws = tsm;                       // [16][LDW] operand weights (fp32 values), rows >= O zero
    float* xs = Ws + 16 * LDW;             // [RG][LDW] the row group, rows past the data zero
    float* dl = xs + RG * LDW;             // [RG][TAIL_DLS] output errors (rounded), zero padded
    int* yl = (int*)(dl + RG * TAIL_DLS);  // [RG] labels of the group
    float* part = (float*)(yl + RG);       // [k-part][rows][16] partial sums of Z
    const int h4 = H / 4, nct = H / 16;
    {
        const TH* wop = (const TH*)a.wop + (size_t)z * a.w_z;
#pragma unroll 4
        for (int e = tid; e < 16 * h4; e += TAIL_THREADS) {
            const int o = e / h4, c = (e - o * h4) * 4;
            *(float4*)(Ws + o * LDW + c) = o < O ? load4(wop + (size_t)o * H + c) : make_float4(0.f, 0.f, 0.f, 0.f);
        }
    }
    const TH* x = (const TH*)a.x + (size_t)z * a.x_z;
    TH* d = (TH*)a.d + (size_t)z * a.x_z;
    const int64_t drow0 = shard_start(a.n_total, a.k_rep, z) + a.r0;
    const int ngrp = (valid + RG - 1) / RG;
    const int eo = tid & 15;  // output of this lane in the per-row work
    const float bo = eo < O ? a.bias[(size_t)z * a.bias_z + eo] : 0.f;

    R4 pf[TAIL_PF];
    int ypf = 0;
    auto load_group = [&](int g) {  // the group's rows are contiguous: value 4e is load e
        const int rows = min(RG, valid - g * RG), n4 = rows * h4;
        const TH* xg = x + (size_t)g * RG * H;
#pragma unroll
        for (int u = 0; u < TAIL_PF; ++u) {
            const int e = tid + TAIL_THREADS * u;
            if (e < n4) pf[u] = *(const R4*)(xg + (size_t)e * 4);
        }
        if (tid < rows) ypf = a.y[drow0 + g * RG + tid];
    };
    auto store_group = [&](int g) {
        const int rows = min(RG, valid - g * RG), n4 = rows * h4;
#pragma unroll
        for (int u = 0; u < TAIL_PF; ++u) {
            const int e = tid + TAIL_THREADS * u;
            if (e < RG * h4) {
                const int r = e / h4, c = (e - r * h4) * 4;
                *(float4*)(xs + r * LDW + c) = e < n4 ? raw_f4(pf[u]) : make_float4(0.f, 0.f, 0.f, 0.f);
            }
        }
        if (tid < RG) yl[tid] = ypf;
    };

    f4 dacc[NCW];
#pragma unroll
    for (int j = 0; j < NCW; ++j) dacc[j] = f4{0.f, 0.f, 0.f, 0.f};
    float sb = 0.f;  // bias sum of output tid (tid < O)
    load_group(0);
    for (int g = 0; g < ngrp; ++g) {
        const int g0 = g * RG, rows = min(RG, valid - g0);
        const int nt = (rows + 15) >> 4;
        __syncthreads();  // (the previous group's readers are done; W staged)
        store_group(g);
        if (g + 1 < ngrp) load_group(g + 1);
        __syncthreads();
        // Z = X W^T: row tile t is split over H into KP parts (16-column tiles kp, kp+KP, ...)
        const int KP = TAIL_WAVES / nt;
        if (wave < KP * nt) {
            const int t = wave / KP, kp = wave - t * KP;
            f4 acc = f4{0.f, 0.f, 0.f, 0.f};
            for (int kt = kp; kt < nct; kt += KP) {
                const f4 xv = *(const f4*)(xs + (t * 16 + rl) * LDW + kt * 16 + kg * 4);
                const f4 wv = *(const f4*)(Ws + rl * LDW + kt * 16 + kg * 4);
#pragma unroll
                for (int q = 0; q < 4; ++q) acc = __builtin_amdgcn_mfma_f32_16x16x4f32(xv[q], wv[q], acc, 0, 0, 0);
            }
#pragma unroll
            for (int r = 0; r < 4; ++r) part[(kp * nt * 16 + t * 16 + kg * 4 + r) * 16 + rl] = acc[r];
        }
        __syncthreads();
        // output activation and output error: lane (row, output) = (e / 16, e % 16)
        for (int e = tid; e < RG * 16; e += TAIL_THREADS) {
            const int r = e >> 4;
            const bool live = r < rows && eo < O;
            float zv = 0.f;
            if (r < rows) {
                float s = part[r * 16 + eo];
                for (int kp = 1; kp < KP; ++kp) s += part[(kp * nt * 16 + r) * 16 + eo];
                zv = s + bo;
            }
            dl[r * TAIL_DLS + eo] = out_error<TH>(zv, live, eo, live ? yl[r] : -1, a.act_out, a.loss);
        }
        __syncthreads();
        if (tid < O)
            for (int r = 0; r < rows; ++r) sb += dl[r * TAIL_DLS + tid];
#pragma unroll
        for (int j = 0; j < NCW; ++j) {
            const int ct = wave + TAIL_WAVES * j;
            __builtin_amdgcn_sched_barrier(0);  // (one tile at a time: keeps the live registers down)
            if (ct < nct) {
                const int col = ct * 16 + rl;
                float wq[4];
#pragma unroll
                for (int q = 0; q < 4; ++q) wq[q] = Ws[(kg * 4 + q) * LDW + col];
                // S = delta W for the tile's columns, then the hidden errors
                for (int t = 0; t < nt; ++t) {
                    const f4 dv = *(const f4*)(dl + (t * 16 + rl) * TAIL_DLS + kg * 4);
                    f4 s = f4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
                    for (int q = 0; q < 4; ++q) s = __builtin_amdgcn_mfma_f32_16x16x4f32(dv[q], wq[q], s, 0, 0, 0);
#pragma unroll
                    for (int r = 0; r < 4; ++r) {
                        const int row = t * 16 + kg * 4 + r;
                        if (row < rows)
                            d[(size_t)(g0 + row) * H + col] = from_f<TH>(s[r] * act_deriv(a.act_hid, xs[row * LDW + col]));
                    }
                }
                // dW += delta^T X over the group's rows, four rows per instruction
                for (int m = 0; m < rows; m += 4) {
                    const int row = m + kg;
                    dacc[j] = __builtin_amdgcn_mfma_f32_16x16x4f32(dl[row * TAIL_DLS + rl], xs[row * LDW + col], dacc[j], 0, 0, 0);
                }
            }
        }
    }
    // the update: lane holds dW[4 kg + r][16 ct + rl]; in fp32 the staged operand weights are
    // the master values
    const float scale = a.lr / (float)valid;
    float* wm = a.w + (size_t)z * a.w_z;
    const bool staged_master = (const void*)wm == (const void*)((const TH*)a.wop + (size_t)z * a.w_z);
#pragma unroll
    for (int j = 0; j < NCW; ++j) {
        const int ct = wave + TAIL_WAVES * j;
        if (ct < nct) {
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                const int o = kg * 4 + r;
                if (o < O) {
                    const size_t i = (size_t)o * H + ct * 16 + rl;
                    const float w = (staged_master ? Ws[o * LDW + ct * 16 + rl] : wm[i]) - scale * dacc[j][r];
                    wm[i] = w;
                    if (a.shadow) a.shadow[(size_t)z * a.w_z + i] = f2bf(w);
                }
            }
        }
    }
    if (tid < O) a.bias[(size_t)z * a.bias_z + tid] -= scale * sb;
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
    const double* w;    // nullable: weights of the CNs (weighted combination)
    double wsum;        // sum of the weights (K without weights)
};

__global__ __launch_bounds__(256) void merge_kernel(MergeArgs a) {
    const int64_t p = ((int64_t)blockIdx.x * 256 + threadIdx.x) * 4;
    if (p >= a.pstride) return;
    double s0 = 0.0, s1 = 0.0, s2 = 0.0, s3 = 0.0;
    if (a.w == nullptr) {
        for (int k = 0; k < a.K; ++k) {
            const float4 v = *(const float4*)(a.theta + (size_t)k * a.pstride + p);
            s0 += (double)v.x; s1 += (double)v.y; s2 += (double)v.z; s3 += (double)v.w;
        }
    } else {
        for (int k = 0; k < a.K; ++k) {
            const float4 v = *(const float4*)(a.theta + (size_t)k * a.pstride + p);
            const double wk = a.w[k];
            s0 += wk * (double)v.x; s1 += wk * (double)v.y; s2 += wk * (double)v.z; s3 += wk * (double)v.w;
        }
    }
    const double inv = a.wsum;
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

// the merged network copied into every CN (a broadcast that a merge deferred), fp32 only
__global__ __launch_bounds__(256) void bcast_kernel(float* theta, const float* merged, int64_t pstride, int K) {
    const int64_t p = ((int64_t)blockIdx.x * 256 + threadIdx.x) * 4;
    if (p >= pstride) return;
    const float4 m = *(const float4*)(merged + p);
    for (int k = 0; k < K; ++k) *(float4*)(theta + (size_t)k * pstride + p) = m;
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
// Bounded wait of a single wave on a global counter, then an acquire fence.
__device__ inline bool wait_geq_wave(int* flag, int target, int* abort, long limit) {
    long it = 0;
    while (__builtin_amdgcn_readfirstlane(__hip_atomic_load(flag, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT)) < target) {
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
// (One launch trains CNs cn0 .. cn0 + KL - 1; where all K CNs' workgroups do not fit the CUs
// at once, the CNs go in groups, one launch each.)
//   blockIdx < KL: the sequential workgroup of CN cn0 + blockIdx.  Waves 0..HW/64-1 own one hidden
//     neuron per lane (W2 column and b1 in registers); the other "helper" waves compute,
//     one step ahead, the already-known part (s <= t-2) of the next step's in-chunk
//     correction.  At chunk start all four waves compute the previous-chunk correction on
//     the matrix cores.
//   blockIdx >= KL: tile workgroups.  Tile (k, rb) keeps W1[16 rows][all inputs] of CN k in
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
    float* qbuf;         // [2][K] slots of qslot floats by chunk parity: Q transposed, [neuron][row]
    int qstride;         // row stride (per neuron) within a slot
    int64_t qslot;
    float* d1;           // [2][K][H][T]  by chunk parity (transposed: one row per hidden neuron)
    int* flags;          // qready[2][K] by chunk parity, dready[K], abort (sticky: cleared only at allocation)
    int H, O, In, act1, act2, loss, nrb;
    int cn0, k_launch;   // this launch trains CNs cn0 .. cn0 + k_launch - 1 (all K share the flags)
    int wait_skew;       // 0; a large value makes the first wait of every sequential workgroup
                         // wait for more tile signals than ever come (failure-handling test:
                         // the bound is reached)
    int tile_delay;      // 0; n > 0 holds the upper half of every CN's tile workgroups back for
                         // n sleeps before their first publish (ordering test: the CN must wait
                         // for every tile's Q_0 however far the others run ahead)
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

// Workgroup barrier for exchanges through LDS only: waits for the wave's own LDS accesses
// (lgkmcnt) but not for its global loads, so copies and polls in flight stay in flight.
// (__syncthreads also waits for every outstanding global access of every wave.)
__device__ inline void lds_barrier() { asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory"); }

// ------------------------------------------------------------------------------------
// Cross-lane building blocks of the sequential per-sample steps (one wavefront).

// Reduction of 10 per-lane values over the whole wavefront.  Afterwards, in every row of
// 16 lanes, lanes 0, 1, 2, 4, 6, 8, 9, 10, 12, 14 hold the wave totals of values 0..9
// (own10 below); the other lanes hold no total.  Rounds 1 and 2 are reduce-scatters with
// bank-masked DPP (row mirror, half-row mirror), so each pairing costs one instruction per
// kept value; rounds 3 and 4 pair lanes within quads; the four rows are then summed with
// the permlane swaps.
__device__ inline float reduce10(const float (&p)[10], int lane) {
    float a0, a1, a2, a3, a4, b0, b1, b2;
    asm volatile(
        "s_nop 1\n\t"
        // lanes 0-7 keep values 0-4, lanes 8-15 keep values 5-9 (partner: lane 15 - i)
        "v_add_f32_dpp %0, %8, %8 row_mirror row_mask:0xf bank_mask:0x3\n\t"
        "v_add_f32_dpp %1, %9, %9 row_mirror row_mask:0xf bank_mask:0x3\n\t"
        "v_add_f32_dpp %2, %10, %10 row_mirror row_mask:0xf bank_mask:0x3\n\t"
        "v_add_f32_dpp %3, %11, %11 row_mirror row_mask:0xf bank_mask:0x3\n\t"
        "v_add_f32_dpp %4, %12, %12 row_mirror row_mask:0xf bank_mask:0x3\n\t"
        "v_add_f32_dpp %0, %13, %13 row_mirror row_mask:0xf bank_mask:0xc\n\t"
        "v_add_f32_dpp %1, %14, %14 row_mirror row_mask:0xf bank_mask:0xc\n\t"
        "v_add_f32_dpp %2, %15, %15 row_mirror row_mask:0xf bank_mask:0xc\n\t"
        "v_add_f32_dpp %3, %16, %16 row_mirror row_mask:0xf bank_mask:0xc\n\t"
        "v_add_f32_dpp %4, %17, %17 row_mirror row_mask:0xf bank_mask:0xc\n\t"
        // lanes of banks 0 and 2 keep their first three, banks 1 and 3 their last two
        // (in b0 and b2) (partner: lane 7 - i within each half row)
        "v_add_f32_dpp %5, %0, %0 row_half_mirror row_mask:0xf bank_mask:0x5\n\t"
        "v_add_f32_dpp %6, %1, %1 row_half_mirror row_mask:0xf bank_mask:0x5\n\t"
        "v_add_f32_dpp %7, %2, %2 row_half_mirror row_mask:0xf bank_mask:0x5\n\t"
        "v_add_f32_dpp %5, %3, %3 row_half_mirror row_mask:0xf bank_mask:0xa\n\t"
        "v_add_f32_dpp %7, %4, %4 row_half_mirror row_mask:0xf bank_mask:0xa"
        : "=&v"(a0), "=&v"(a1), "=&v"(a2), "=&v"(a3), "=&v"(a4), "=&v"(b0), "=&v"(b1), "=&v"(b2)
        : "v"(p[0]), "v"(p[1]), "v"(p[2]), "v"(p[3]), "v"(p[4]), "v"(p[5]), "v"(p[6]), "v"(p[7]), "v"(p[8]),
          "v"(p[9]));
    // quads: lanes with bit 1 set keep b2, the others b0 and b1; then bit 0 splits b0 / b1
    const bool q1 = lane & 2, q0 = lane & 1;
    const float k3 = q1 ? b2 : b0, s3 = q1 ? b0 : b2;
    const float c0 = k3 + dpp<DPP_XOR2>(s3);
    const float c1 = b1 + dpp<DPP_XOR2>(b1);
    const float k4 = q0 ? c1 : c0, s4 = q0 ? c0 : c1;
    float d = k4 + dpp<DPP_XOR1>(s4);
    // sum of the four rows
    auto r16 = __builtin_amdgcn_permlane16_swap(__float_as_uint(d), __float_as_uint(d), false, false);
    d = __uint_as_float(r16[0]) + __uint_as_float(r16[1]);
    auto r32 = __builtin_amdgcn_permlane32_swap(__float_as_uint(d), __float_as_uint(d), false, false);
    return __uint_as_float(r32[0]) + __uint_as_float(r32[1]);
}
// value index held by lane l (mod 16) after reduce10, -1 for none:
// 0 1 2 - 3 - 4 - | 5 6 7 - 8 - 9 -
__device__ inline int own10(int l16) {
    const int base = (l16 >> 3) * 5, r = l16 & 7;
    return r < 3 ? base + r : (r == 4 ? base + 3 : (r == 6 ? base + 4 : -1));
}
constexpr int SRC10[10] = {0, 1, 2, 4, 6, 8, 9, 10, 12, 14};  // lane of each total within a row

// Reduction of 16 per-lane values over the wavefront; afterwards lane l holds the total of
// value l & 15 (all rounds are reduce-scatters, bank-masked where the pairing allows).
__device__ inline float reduce16(const float (&p)[16], int lane) {
    float a[8], b[4];
    asm volatile(
        "s_nop 1\n\t"
        "v_add_f32_dpp %0, %12, %12 row_mirror row_mask:0xf bank_mask:0x3\n\t"
        "v_add_f32_dpp %1, %13, %13 row_mirror row_mask:0xf bank_mask:0x3\n\t"
        "v_add_f32_dpp %2, %14, %14 row_mirror row_mask:0xf bank_mask:0x3\n\t"
        "v_add_f32_dpp %3, %15, %15 row_mirror row_mask:0xf bank_mask:0x3\n\t"
        "v_add_f32_dpp %4, %16, %16 row_mirror row_mask:0xf bank_mask:0x3\n\t"
        "v_add_f32_dpp %5, %17, %17 row_mirror row_mask:0xf bank_mask:0x3\n\t"
        "v_add_f32_dpp %6, %18, %18 row_mirror row_mask:0xf bank_mask:0x3\n\t"
        "v_add_f32_dpp %7, %19, %19 row_mirror row_mask:0xf bank_mask:0x3\n\t"
        "v_add_f32_dpp %0, %20, %20 row_mirror row_mask:0xf bank_mask:0xc\n\t"
        "v_add_f32_dpp %1, %21, %21 row_mirror row_mask:0xf bank_mask:0xc\n\t"
        "v_add_f32_dpp %2, %22, %22 row_mirror row_mask:0xf bank_mask:0xc\n\t"
        "v_add_f32_dpp %3, %23, %23 row_mirror row_mask:0xf bank_mask:0xc\n\t"
        "v_add_f32_dpp %4, %24, %24 row_mirror row_mask:0xf bank_mask:0xc\n\t"
        "v_add_f32_dpp %5, %25, %25 row_mirror row_mask:0xf bank_mask:0xc\n\t"
        "v_add_f32_dpp %6, %26, %26 row_mirror row_mask:0xf bank_mask:0xc\n\t"
        "v_add_f32_dpp %7, %27, %27 row_mirror row_mask:0xf bank_mask:0xc\n\t"
        "v_add_f32_dpp %8, %0, %0 row_half_mirror row_mask:0xf bank_mask:0x5\n\t"
        "v_add_f32_dpp %9, %1, %1 row_half_mirror row_mask:0xf bank_mask:0x5\n\t"
        "v_add_f32_dpp %10, %2, %2 row_half_mirror row_mask:0xf bank_mask:0x5\n\t"
        "v_add_f32_dpp %11, %3, %3 row_half_mirror row_mask:0xf bank_mask:0x5\n\t"
        "v_add_f32_dpp %8, %4, %4 row_half_mirror row_mask:0xf bank_mask:0xa\n\t"
        "v_add_f32_dpp %9, %5, %5 row_half_mirror row_mask:0xf bank_mask:0xa\n\t"
        "v_add_f32_dpp %10, %6, %6 row_half_mirror row_mask:0xf bank_mask:0xa\n\t"
        "v_add_f32_dpp %11, %7, %7 row_half_mirror row_mask:0xf bank_mask:0xa"
        : "=&v"(a[0]), "=&v"(a[1]), "=&v"(a[2]), "=&v"(a[3]), "=&v"(a[4]), "=&v"(a[5]), "=&v"(a[6]), "=&v"(a[7]),
          "=&v"(b[0]), "=&v"(b[1]), "=&v"(b[2]), "=&v"(b[3])
        : "v"(p[0]), "v"(p[1]), "v"(p[2]), "v"(p[3]), "v"(p[4]), "v"(p[5]), "v"(p[6]), "v"(p[7]), "v"(p[8]),
          "v"(p[9]), "v"(p[10]), "v"(p[11]), "v"(p[12]), "v"(p[13]), "v"(p[14]), "v"(p[15]));
    const bool q1 = lane & 2, q0 = lane & 1;
    float c[2];
#pragma unroll
    for (int j = 0; j < 2; ++j) {
        const float kk = q1 ? b[j + 2] : b[j], ss = q1 ? b[j] : b[j + 2];
        c[j] = kk + dpp<DPP_XOR2>(ss);
    }
    const float kk = q0 ? c[1] : c[0], ss = q0 ? c[0] : c[1];
    float d = kk + dpp<DPP_XOR1>(ss);
    auto r16 = __builtin_amdgcn_permlane16_swap(__float_as_uint(d), __float_as_uint(d), false, false);
    d = __uint_as_float(r16[0]) + __uint_as_float(r16[1]);
    auto r32 = __builtin_amdgcn_permlane32_swap(__float_as_uint(d), __float_as_uint(d), false, false);
    return __uint_as_float(r32[0]) + __uint_as_float(r32[1]);
}

// back += bcast(d2 from lane SRC of the row) * w;  w += bcast(d2) * na  (one output, one
// neuron per lane; na = -eta * a1).  FIRST adds the two wait states a DPP read needs after a
// VALU write of its source; they sit in the same statement as the reads of d2, so the
// compiler cannot separate them from the write.
#define PNN_BCAST_UPD(SRC)                                                                                   \
    template <bool FIRST>                                                                                    \
    __device__ inline void bcast_upd_##SRC(float& back, float& w, float d2, float na) {                     \
        if (FIRST)                                                                                           \
            asm volatile("s_nop 1\n\t"                                                                      \
                         "v_fmac_f32_dpp %0, %2, %1 row_newbcast:" #SRC " row_mask:0xf bank_mask:0xf\n\t"  \
                         "v_fmac_f32_dpp %1, %2, %3 row_newbcast:" #SRC " row_mask:0xf bank_mask:0xf"      \
                         : "+v"(back), "+v"(w)                                                               \
                         : "v"(d2), "v"(na));                                                                \
        else                                                                                                 \
            asm volatile("v_fmac_f32_dpp %0, %2, %1 row_newbcast:" #SRC " row_mask:0xf bank_mask:0xf\n\t"  \
                         "v_fmac_f32_dpp %1, %2, %3 row_newbcast:" #SRC " row_mask:0xf bank_mask:0xf"      \
                         : "+v"(back), "+v"(w)                                                               \
                         : "v"(d2), "v"(na));                                                                \
    }
PNN_BCAST_UPD(0) PNN_BCAST_UPD(1) PNN_BCAST_UPD(2) PNN_BCAST_UPD(3) PNN_BCAST_UPD(4) PNN_BCAST_UPD(5)
PNN_BCAST_UPD(6) PNN_BCAST_UPD(7) PNN_BCAST_UPD(8) PNN_BCAST_UPD(9) PNN_BCAST_UPD(10) PNN_BCAST_UPD(11)
PNN_BCAST_UPD(12) PNN_BCAST_UPD(13) PNN_BCAST_UPD(14) PNN_BCAST_UPD(15)
#undef PNN_BCAST_UPD

template <int SRC, bool FIRST>
__device__ inline void bcast_upd(float& back, float& w, float d2, float na) {
    if constexpr (SRC == 0) bcast_upd_0<FIRST>(back, w, d2, na);
    else if constexpr (SRC == 1) bcast_upd_1<FIRST>(back, w, d2, na);
    else if constexpr (SRC == 2) bcast_upd_2<FIRST>(back, w, d2, na);
    else if constexpr (SRC == 3) bcast_upd_3<FIRST>(back, w, d2, na);
    else if constexpr (SRC == 4) bcast_upd_4<FIRST>(back, w, d2, na);
    else if constexpr (SRC == 5) bcast_upd_5<FIRST>(back, w, d2, na);
    else if constexpr (SRC == 6) bcast_upd_6<FIRST>(back, w, d2, na);
    else if constexpr (SRC == 7) bcast_upd_7<FIRST>(back, w, d2, na);
    else if constexpr (SRC == 8) bcast_upd_8<FIRST>(back, w, d2, na);
    else if constexpr (SRC == 9) bcast_upd_9<FIRST>(back, w, d2, na);
    else if constexpr (SRC == 10) bcast_upd_10<FIRST>(back, w, d2, na);
    else if constexpr (SRC == 11) bcast_upd_11<FIRST>(back, w, d2, na);
    else if constexpr (SRC == 12) bcast_upd_12<FIRST>(back, w, d2, na);
    else if constexpr (SRC == 13) bcast_upd_13<FIRST>(back, w, d2, na);
    else if constexpr (SRC == 14) bcast_upd_14<FIRST>(back, w, d2, na);
    else bcast_upd_15<FIRST>(back, w, d2, na);
}

// Output error broadcast and second-layer update for every output o (compile-time loop):
// back_j += W2[o][h_j] * d2_o (pre-update weights, eq. (11)); W2[o][h_j] -= eta d2_o a1_j.
template <int OC, int NH, int O>
__device__ inline void backprop_outputs(float (&back)[NH], float (&w2)[NH][OC], float d2, const float (&na)[NH]) {
    if constexpr (O < OC) {
        constexpr int src = OC == 10 ? SRC10[O] : O;
#pragma unroll
        for (int j = 0; j < NH; ++j) {
            if (j == 0) bcast_upd<src, O == 0>(back[j], w2[j][O], d2, na[j]);
            else bcast_upd<src, false>(back[j], w2[j][O], d2, na[j]);
        }
        backprop_outputs<OC, NH, O + 1>(back, w2, d2, na);
    }
}

// ------------------------------------------------------------------------------------
// Fold of one finished block of BS = 8 steps into a chunk's input-sum accumulator held in
// registers, on the matrix cores:
//   acc[t][h] += scale * sum_{s in block} G[t][s] * D[h][s]      (scale = -eta)
// for the row tiles mt >= mt0 (16 rows each) and the NT neuron tiles starting at nt0 (16
// neurons each).  G rows have stride GS; D rows (one per neuron) have stride TS.
// v_mfma_f32_16x16x4_f32 contracts 4 steps per instruction; lane group g = lane / 16
// supplies the steps s0 + 2g + q of instruction q (the same permutation of the steps on both
// operands).  A lane's accumulator acc[mt][nt] holds rows mt*16 + 4g .. +3 of neuron
// (nt0 + nt)*16 + lane % 16.  Rows of tile mt0 before the first row that needs the block
// also receive it; they are final already and never written again.
template <int GS, int TS, int MT, int NT>
__device__ __attribute__((always_inline)) inline void fold_acc(f4 (&acc)[MT][NT], const float* G, const float* D,
                                                               int mt0, int s0, float scale, int nt0, int lane) {
    typedef float v2 __attribute__((ext_vector_type(2)));
    const int r16 = lane & 15, g = lane >> 4;
    v2 av[MT], bv[NT];
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) av[mt] = *(const v2*)(G + (mt * 16 + r16) * GS + s0 + 2 * g);
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) bv[nt] = *(const v2*)(D + ((nt0 + nt) * 16 + r16) * TS + s0 + 2 * g) * scale;
#pragma unroll
    for (int mt = 0; mt < MT; ++mt)
        if (mt >= mt0)  // wave-uniform
#pragma unroll
            for (int nt = 0; nt < NT; ++nt) {
                acc[mt][nt] = __builtin_amdgcn_mfma_f32_16x16x4f32(av[mt][0], bv[nt][0], acc[mt][nt], 0, 0, 0);
                acc[mt][nt] = __builtin_amdgcn_mfma_f32_16x16x4f32(av[mt][1], bv[nt][1], acc[mt][nt], 0, 0, 0);
            }
}
// acc[t][h] += Q[h][t] for every row of the chunk and this wave's neurons (Q in global
// memory, [neuron][row] with row stride TS): the tiles' W1 x term of the input sums.
template <int TS, int MT, int NT>
__device__ __attribute__((always_inline)) inline void add_q(f4 (&acc)[MT][NT], const float* Q, int nt0, int lane) {
    const int r16 = lane & 15, g = lane >> 4;
    float4 q[MT][NT];
#pragma unroll
    for (int mt = 0; mt < MT; ++mt)
#pragma unroll
        for (int nt = 0; nt < NT; ++nt) q[mt][nt] = *(const float4*)(Q + ((nt0 + nt) * 16 + r16) * TS + mt * 16 + 4 * g);
#pragma unroll
    for (int mt = 0; mt < MT; ++mt)
#pragma unroll
        for (int nt = 0; nt < NT; ++nt) {
            acc[mt][nt][0] += q[mt][nt].x;
            acc[mt][nt][1] += q[mt][nt].y;
            acc[mt][nt][2] += q[mt][nt].z;
            acc[mt][nt][3] += q[mt][nt].w;
        }
}
// The eight rows of block B of a chunk are final: PlT[h][t] = acc[t][h] for those rows and
// this wave's neurons (PlT [neuron][row], row stride TS).  The rows are half of row tile
// B / 2: lane groups 2 (B & 1) and 2 (B & 1) + 1.
template <int TS, int MT, int NT>
__device__ __attribute__((always_inline)) inline void write_rows(const f4 (&acc)[MT][NT], float* PlT, int B, int nt0,
                                                                 int lane) {
    const int r16 = lane & 15, g = lane >> 4;
    const int mtw = B >> 1;  // wave-uniform
    const bool mine = (g >> 1) == (B & 1);
#pragma unroll
    for (int mt = 0; mt < MT; ++mt)
        if (mt == mtw && mine) {
#pragma unroll
            for (int nt = 0; nt < NT; ++nt) {
                const int idx = ((nt0 + nt) * 16 + r16) * TS + mt * 16 + 4 * g;
                *(float4*)(PlT + idx) = make_float4(acc[mt][nt][0], acc[mt][nt][1], acc[mt][nt][2], acc[mt][nt][3]);
            }
        }
}

// Bounded wait on a counter in LDS written by another wave of the workgroup.  The LDS
// abort flag (or the spin limit, which raises it together with the grid-wide abort flag)
// ends every wait, so the workgroup always drains.
__device__ inline bool lds_wait_geq(const int* f, int target, int* lab, int* gabort, long limit, bool sleep) {
    long it = 0;
    while (__hip_atomic_load(f, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP) < target) {
        if (__hip_atomic_load(lab, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP)) return false;
        if (++it > limit) {
            __hip_atomic_store(lab, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
            __hip_atomic_store(gabort, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            // (cold path) complete the stores here, so that the compiler need not protect
            // their operand registers with a wait on the hot path after the call
            __builtin_amdgcn_s_waitcnt(0x0070);
            return false;
        }
        if (sleep) __builtin_amdgcn_s_sleep(1);
    }
    asm volatile("" ::: "memory");  // later LDS reads stay after the counter read
    return true;
}
// Three counters at once: a single LDS round trip when all have reached their targets.
__device__ inline void lds_wait3(const int* f0, int t0, const int* f1, int t1, const int* f2, int t2, int* lab,
                                 int* gabort, long limit) {
    const int v0 = __hip_atomic_load(f0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
    const int v1 = __hip_atomic_load(f1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
    const int v2 = __hip_atomic_load(f2, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
    __builtin_amdgcn_s_waitcnt(0xC07F);  // lgkmcnt(0): no path leaves one of the reads in flight
    if (__builtin_amdgcn_readfirstlane(v0) < t0 || __builtin_amdgcn_readfirstlane(v1) < t1 ||
        __builtin_amdgcn_readfirstlane(v2) < t2) {
        lds_wait_geq(f0, t0, lab, gabort, limit, false);
        lds_wait_geq(f1, t1, lab, gabort, limit, false);
        lds_wait_geq(f2, t2, lab, gabort, limit, false);
    }
    asm volatile("" ::: "memory");  // later LDS reads stay after the counter reads
}
__device__ inline int lds_read(const int* f) {
    const int v = __hip_atomic_load(f, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
    asm volatile("" ::: "memory");
    return __builtin_amdgcn_readfirstlane(v);
}
// Counter update after LDS stores: a wave's LDS accesses complete in issue order, so a
// reader that sees the counter (and reads the data after it) sees the data.  The compiler
// barrier keeps the stores before the counter.
__device__ inline void lds_publish(int* f, int v) {
    asm volatile("" ::: "memory");
    __hip_atomic_store(f, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
}

// ------------------------------------------------------------------------------------
// The sequential workgroup of one CN (per-sample SGD, one persistent launch per epoch).
//
// Notation: steps are numbered over the CN's slice (global step r); chunk c holds steps
// [cT, cT + T), block B holds steps [BS B, BS B + BS) (BS = 8: eight blocks per chunk).  With W1^(c)
// the first-layer weights before chunk c, the first-layer input sum of step r in chunk c is
//   z1_r = Q_c[r] + b1_r - eta * sum_{s in [T(c-1), r)} d1_s (x_s . x_r)
// where Q_c[r] = W1^(c-1) x_r is published by the tile workgroups.  The dot products come
// from the Gram blocks G_c (within chunk c) and GX_c (chunk c against chunk c-1).
//
// Who adds which term d1_s (x_s . x_r) of row r (block B):
//   s < BS(B-1):        folded into the stored input sums Pl of row r in the background, on
//                       the matrix cores, a whole block at a time;
//   s in [BS(B-1), r-6]: the window correction cpre[r] (at most 2 BS - 6 terms), computed by
//                       wave 1 while the live wave runs steps r-5 to r-1;
//   s = r-5 .. r-1:     the live wave, with its own fresh errors (NLIVE = 5 terms).
//
// Waves (256 threads), each in its own loop, coordinated through counters in LDS:
//   wave 0, live:  the steps.  Lane l owns hidden neurons l and l + 64 (NH = 2) or l
//                  (NH = 1): their b1 and W2 columns stay in registers.
//   wave 1:        the window corrections, one row ahead of the live wave.
//   waves 2, 3:    the folds, each for half of the neurons.  A wave keeps the sums
//                  sum_s d1_s (x_s . x_t) of the current chunk's rows (accC) and of the next
//                  chunk's rows (accN) in registers, as MFMA accumulator tiles holding
//                  Q - eta sum (Q, the tiles' W1 x, is added once it is published).  A
//                  finished block B' is added to the rows of blocks >= B'+2 of accC, after
//                  which the rows of block B'+2 are final and are written once to the input-
//                  sum array Pl; and, once the next chunk's Gram blocks are in LDS, to all
//                  rows of accN (block NB-2 completes the next chunk's block 0, block NB-1 its
//                  block 1: both are written then, and accN becomes accC).
//                  Wave 2 also publishes each finished block's d1 for the tile workgroups
//                  and announces finished chunks to them; wave 3 early in each chunk loads
//                  the next chunk's Gram blocks and labels into LDS.
// Counters (LDS): d1done (steps whose d1 is in hist), cdone (rows whose cpre is ready),
// rdy (per folding wave: leading blocks whose rows of Pl are final), gready (chunks whose
// Gram blocks and labels are in LDS), pubd (blocks whose d1 has been copied out of hist),
// abort.
template <int T, int NH, int A1, int A2, int LS, int OC>
__device__ __attribute__((always_inline)) inline void psgd_rec(const PsgdPArgs& a, int k, float* smem) {
    constexpr int HW = 64 * NH;     // neurons covered by the live wave
    constexpr int TS = T + 4;       // row stride of the error history ([neuron][step in chunk])
    constexpr int GS = T + 4;       // row stride of the Gram blocks (conflict-free MFMA operand reads)
    constexpr int BS = 8;           // steps per fold block
    constexpr int NLIVE = 5;        // latest errors whose terms the live wave adds itself (<= BS; the
                                    // live step below is written out for five)
    constexpr int NB = T / BS;      // blocks per chunk
    static_assert(T == 64, "chunks of 64 steps");
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int H = a.H, K = a.k_rep;
    const float lr = a.lr;

    float* Pl = smem;                   // [HW][TS]   input sums (transposed: [neuron][row in chunk])
    float* hist = Pl + HW * TS;         // [HW][TS]   first-layer errors by step mod T
    float* Gin = hist + HW * TS;        // [2][T][GS] Gram blocks within a chunk, by parity
    float* GX = Gin + 2 * T * GS;       // [T][GS]    a chunk (rows) against the previous one
    float* cpre = GX + T * GS;          // [8][HW]    window corrections by row mod 8
    int* yb = (int*)(cpre + 8 * HW);    // [2][T]     labels by chunk parity
    int* lf = yb + 2 * T;
    int* d1done = lf;
    int* cdone = lf + 1;
    int* rdy = lf + 2;     // [2]: one counter per folding wave
    int* gready = lf + 6;
    int* lab = lf + 7;
    int* pubd = lf + 8;

    const int64_t nz = shard_len(a.n_total, K, k), xs = shard_start(a.n_total, K, k);
    const int nsteps = (int)nz;
    const int nchk = (nsteps + T - 1) / T;
    const int nblk = (nsteps + BS - 1) / BS;
    float* th = a.theta + (size_t)k * a.pstride;
    // Q_c is complete when the counter of parity c & 1 reaches nrb (c / 2 + 1): no tile can
    // publish Q_{c+2} before chunk c's errors exist, which take Q_c, so a tile's count on that
    // parity reaches c / 2 + 1 only by publishing Q_c.  (A single counter for both parities
    // could reach nrb (c + 1) with some tiles at Q_{c+1} and others still short of Q_c.)
    auto qready = [&](int c) { return a.flags + (c & 1) * K + k; };
    auto qtarget = [&](int c) { return a.nrb * (c / 2 + 1); };
    int* dready = a.flags + 2 * K + k;
    int* gabort = a.flags + 3 * K;

    // padding neurons h >= H read zero errors and zero input sums
    for (int i = tid; i < HW * TS; i += 256) hist[i] = 0.f;
    for (int i = tid; i < HW * TS; i += 256) Pl[i] = 0.f;
    if (tid < 12) lf[tid] = 0;

    // chunk 0: wait for Q_0 and stage it with the Gram block and labels
    if (!wait_geq(qready(0), qtarget(0) + a.wait_skew, gabort, a.spin_limit)) return;
    {
        const float* Q = a.qbuf + (size_t)k * HW * TS;
        const float* G = a.gram + (size_t)k * a.nch * T * GS;
        const int tc0 = min(T, nsteps);
        for (int idx = tid; idx < HW * TS; idx += 256) Pl[idx] = Q[idx];
        for (int idx = tid; idx < T * GS; idx += 256) Gin[idx] = G[idx];
        for (int idx = tid; idx < tc0; idx += 256) yb[idx] = a.y[xs + idx];
        if (tid == 0) { gready[0] = 1; rdy[0] = 2; rdy[1] = 2; }
    }
    __syncthreads();

    auto chunk_len = [&](int c) { return min(T, nsteps - c * T); };
    // Gram block of chunk c against itself
    auto grow_in = [&](int c) { return Gin + (c & 1) * T * GS; };

    if (wave == 0) {
        // ================= live wave
        const int O = OC < 16 ? OC : a.O;
        const int act1 = A1 >= 0 ? A1 : a.act1;
        const int act2 = A2 >= 0 ? A2 : a.act2;
        const int loss = LS >= 0 ? LS : a.loss;
        float w2[NH][OC], b1[NH], corr[NH], dprev[NH], dprev2[NH], dprev3[NH], dprev4[NH], pln[NH];
        const int ol = lane & 15;
        const int own = OC == 10 ? own10(ol) : ol;  // output whose total this lane holds
        const bool owner = own >= 0 && own < O;
#pragma unroll
        for (int j = 0; j < NH; ++j) {
            const int h = lane + 64 * j;
            b1[j] = h < H ? th[a.off_b1 + h] : 0.f;
#pragma unroll
            for (int o = 0; o < OC; ++o) w2[j][o] = (h < H && o < O) ? th[a.off_w2 + (size_t)o * H + h] : 0.f;
            corr[j] = 0.f;
            dprev[j] = 0.f;
            dprev2[j] = 0.f;
            dprev3[j] = 0.f;
            dprev4[j] = 0.f;
            pln[j] = Pl[h * TS];
        }
        float b2v = owner ? th[a.off_b2 + own] : 0.f;
        int label = yb[0];  // label of the current row; the next row's is read a step ahead
        __builtin_amdgcn_s_waitcnt(0x0070);  // vmcnt(0) lgkmcnt(0), visible to the compiler's wait placement

        // One block of BS steps per outer iteration, unrolled: the block-boundary logic and
        // the in-block offsets are compile-time, and the rotation of the recent errors is a
        // register renaming.
        for (int r0 = 0; r0 < nsteps; r0 += BS) {
            const int c = r0 >> 6, t0 = r0 & (T - 1);
            const int tc = chunk_len(c);
#pragma unroll
        for (int i = 0; i < BS; ++i) {
            const int r = r0 + i;
            if (r >= nsteps) break;  // (last block of a ragged slice)
            const int t = t0 + i;
            // the row after this step: same chunk, or the next chunk's first row
            const bool more = r + 1 < nsteps;
            const bool cross = more && t + 1 == tc;
            if (more && i == BS - 1) {
                // the next row opens block Bn: its input sums must be final in Pl (both
                // folding waves; at a chunk's first row this also means the chunk's Gram
                // blocks and labels are in LDS), and the hist columns it will overwrite must
                // have been copied out (block Bn - NB)
                const int Bn = (r + 1) / BS;
                lds_wait3(rdy, Bn + 1, rdy + 1, Bn + 1, pubd, Bn - NB + 1, lab, gabort, a.spin_limit);
            }
            // operands of the step's end, read up front (unconditional loads from valid
            // addresses, so every path leaves the same LDS reads in flight)
            const int rn = more ? r + 1 : r;
            const int cn = rn >> 6, tn = rn & (T - 1);
            float cp[NH], pnx[NH];
#pragma unroll
            for (int j = 0; j < NH; ++j) pnx[j] = Pl[(lane + 64 * j) * TS + tn];
            // Gram entries of the next row against steps r .. r-4 (NLIVE): within the next row's chunk
            // from its G block, against the chunk before it from GX (which holds the next
            // row's chunk against the previous one whenever the next row needs it)
            const float* gin = grow_in(cn) + tn * GS;
            const float* gx = GX + tn * GS;
            const float g1v = cross ? gx[t] : gin[t];
            const int tp = (t + T - 1) & (T - 1);      // position of step r-1 in its chunk
            const float g0v = (cross || t < 1) ? gx[tp] : gin[tp];
            const int tp2 = (t + T - 2) & (T - 1);     // position of step r-2 in its chunk
            const float g2v = (cross || t < 2) ? gx[tp2] : gin[tp2];
            const int tp3 = (t + T - 3) & (T - 1);     // position of step r-3 in its chunk
            const float g3v = (cross || t < 3) ? gx[tp3] : gin[tp3];
            const int tp4 = (t + T - 4) & (T - 1);     // position of step r-4 in its chunk
            const float g4v = (cross || t < 4) ? gx[tp4] : gin[tp4];
            const int labn = yb[(cn & 1) * T + tn];

            float a1[NH], na[NH];
#pragma unroll
            for (int j = 0; j < NH; ++j) {
                const float z1 = pln[j] + b1[j] - lr * corr[j];
                a1[j] = (lane + 64 * j < H) ? act_fast(act1, z1) : 0.f;
                na[j] = -lr * a1[j];
            }
            float z2;
            if constexpr (OC == 10) {
                float p[10];
#pragma unroll
                for (int o = 0; o < 10; ++o) {
                    p[o] = w2[0][o] * a1[0];
#pragma unroll
                    for (int j = 1; j < NH; ++j) p[o] = __builtin_fmaf(w2[j][o], a1[j], p[o]);
                }
                z2 = reduce10(p, lane) + b2v;
            } else {
                float p[16];
#pragma unroll
                for (int o = 0; o < 16; ++o) {
                    p[o] = w2[0][o] * a1[0];
#pragma unroll
                    for (int j = 1; j < NH; ++j) p[o] = __builtin_fmaf(w2[j][o], a1[j], p[o]);
                }
                z2 = reduce16(p, lane) + b2v;
            }
            // the window correction of the next row (wave 1 has normally finished it)
            const int cd = __hip_atomic_load(cdone, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
            asm volatile("" ::: "memory");
#pragma unroll
            for (int j = 0; j < NH; ++j) cp[j] = cpre[(rn & 7) * HW + lane + 64 * j];
            float x2;
            if (act2 == ACT_SOFTMAX) {
                const float m = row_allmax16(owner ? z2 : -INFINITY);
                const float e = owner ? __expf(z2 - m) : 0.f;
                x2 = e * __builtin_amdgcn_rcpf(row_allsum16(e));
            } else {
                x2 = act_fast(act2, z2);
            }
            const float e = (own == label) ? 1.0f : 0.0f;
            const float dv = (loss == LOSS_XENT) ? (x2 - e) : (x2 - e) * act_deriv(act2, x2);
            const float d2 = owner ? dv : 0.f;
            b2v -= lr * d2;
            float back[NH];
#pragma unroll
            for (int j = 0; j < NH; ++j) back[j] = 0.f;
            backprop_outputs<OC, NH, 0>(back, w2, d2, na);
            // Every LDS read of this step has long returned: an explicit wait (seen by the
            // compiler's wait placement) leaves only stores in flight at the loop head, so the
            // next step starts without waiting for this step's stores to complete.
            __builtin_amdgcn_s_waitcnt(0xC07F);  // lgkmcnt(0)
            float d1[NH];
#pragma unroll
            for (int j = 0; j < NH; ++j) {
                d1[j] = (lane + 64 * j < H) ? back[j] * act_deriv(act1, a1[j]) : 0.f;
                b1[j] -= lr * d1[j];
                hist[(lane + 64 * j) * TS + t] = d1[j];
            }
            if (more && __builtin_amdgcn_readfirstlane(cd) < r + 2) {
                lds_wait_geq(cdone, r + 2, lab, gabort, a.spin_limit, false);
#pragma unroll
                for (int j = 0; j < NH; ++j) cp[j] = cpre[(rn & 7) * HW + lane + 64 * j];
                __builtin_amdgcn_s_waitcnt(0xC07F);  // (slow path) lgkmcnt(0) here, not after the join
            }
            // terms of steps r .. r-4, the NLIVE latest (all lie in the next row's two-block
            // window, not yet folded: they are at most five steps back).  Also done after the last step
            // (unused then): every path consumes the loads it issued, so none is still in
            // flight into a register at the loop head.
            {
                const float g1 = g1v, g0 = r >= 1 ? g0v : 0.f, g2 = r >= 2 ? g2v : 0.f, g3 = r >= 3 ? g3v : 0.f;
                const float g4 = r >= 4 ? g4v : 0.f;
#pragma unroll
                for (int j = 0; j < NH; ++j) {
                    corr[j] = cp[j] + dprev4[j] * g4 + dprev3[j] * g3 + dprev2[j] * g2 + dprev[j] * g0 + d1[j] * g1;
                    dprev4[j] = dprev3[j];
                    dprev3[j] = dprev2[j];
                    dprev2[j] = dprev[j];
                    dprev[j] = d1[j];
                    pln[j] = pnx[j];
                }
                label = labn;
            }
            // d1 of this step is in hist, and this step's reads of the correction slot are
            // done: wave 1 may refill it
            lds_publish(d1done, r + 1);
        }
        }
#pragma unroll
        for (int j = 0; j < NH; ++j) {
            const int h = lane + 64 * j;
            if (h < H) {
                th[a.off_b1 + h] = b1[j];
#pragma unroll
                for (int o = 0; o < OC; ++o)
                    if (o < O) th[a.off_w2 + (size_t)o * H + h] = w2[j][o];
            }
        }
        if (lane < 16 && owner) th[a.off_b2 + own] = b2v;
    } else if (wave == 1) {
        // ================= window corrections: for row q = r + 1 (block B = q / BS),
        // cpre[q] = sum over s in [BS(B-1), q-1-NLIVE] of d1_s (x_s . x_q)
        for (int r = 0; r + 1 < nsteps; ++r) {
            const int q = r + 1;
            const int cq = q >> 6, tq = q & (T - 1), B = q / BS;
            // the live wave has finished step q-1-NLIVE: d1 up to there is in hist.  The slot
            // (q & 7) last held the correction of row q-8, read in step q-9: free.
            lds_wait_geq(d1done, r + 1 - NLIVE, lab, gabort, a.spin_limit, false);
            // a chunk's first rows read its Gram blocks (and GX) before the live wave enters it
            if (tq < BS && cq >= 1) lds_wait_geq(gready, cq + 1, lab, gabort, a.spin_limit, true);
            float sum[NH];
#pragma unroll
            for (int j = 0; j < NH; ++j) sum[j] = 0.f;
            const int lo = max(0, BS * (B - 1)), hi = q - 1 - NLIVE;  // inclusive range
            // two aligned groups of BS steps: the previous block and the row's own block
#pragma unroll
            for (int part = 0; part < 2; ++part) {
                const int sb = BS * (B - 1 + part);  // first step of the group
                if (sb < lo || sb > hi) continue;
                const int cs = sb >> 6, ts = sb & (T - 1);
                // Gram row of q against the group's steps: same chunk -> G_cq, else GX_cq
                const float* gq = (cs == cq ? grow_in(cq) : GX) + tq * GS + ts;
                const int last = hi - sb;  // highest offset included (>= 0)
#pragma unroll
                for (int u = 0; u < BS / 4; ++u) {
                    if (4 * u > last) break;
                    float4 gv = *(const float4*)(gq + 4 * u);
                    gv.y = (4 * u + 1 <= last) ? gv.y : 0.f;
                    gv.z = (4 * u + 2 <= last) ? gv.z : 0.f;
                    gv.w = (4 * u + 3 <= last) ? gv.w : 0.f;
#pragma unroll
                    for (int j = 0; j < NH; ++j) {
                        const float4 hv = *(const float4*)(hist + (lane + 64 * j) * TS + ts + 4 * u);
                        sum[j] = __builtin_fmaf(hv.x, gv.x, sum[j]);
                        sum[j] = __builtin_fmaf(hv.y, gv.y, sum[j]);
                        sum[j] = __builtin_fmaf(hv.z, gv.z, sum[j]);
                        sum[j] = __builtin_fmaf(hv.w, gv.w, sum[j]);
                    }
                }
            }
#pragma unroll
            for (int j = 0; j < NH; ++j) cpre[(q & 7) * HW + lane + 64 * j] = sum[j];
            lds_publish(cdone, q + 1);
        }
    } else {
        // ================= waves 2 and 3: the folds, each wave for half of the neuron tiles;
        // wave 2 also publishes the finished blocks' d1, wave 3 loads the next chunk's data
        constexpr int NNT = HW / 16;
        constexpr int NT = NNT / 2;  // neuron tiles of this wave
        constexpr int MT = T / 16;   // row tiles of a chunk
        const int w2i = wave - 2;
        const bool pw = wave == 2;  // publishes the errors
        const bool lw = wave == 3;  // loads the next chunk's Gram blocks and labels
        const int nt0 = w2i * NT;
        int* rd = rdy + w2i;
        f4 accC[MT][NT], accN[MT][NT];  // sums of the current and of the next chunk's rows
#pragma unroll
        for (int mt = 0; mt < MT; ++mt)
#pragma unroll
            for (int nt = 0; nt < NT; ++nt) {
                accC[mt][nt] = f4{0.f, 0.f, 0.f, 0.f};
                accN[mt][nt] = f4{0.f, 0.f, 0.f, 0.f};
            }
        auto qrows = [&](int c) { return a.qbuf + ((size_t)(c & 1) * K + k) * HW * TS; };  // Q_c, [HW][TS]
        add_q<TS, MT, NT>(accC, qrows(0), nt0, lane);  // (Q_0 was acquired before the roles split)
        bool qn = false;  // Q of accN's chunk added
        int fc = 0;      // next block to fold into its own chunk's rows
        int fn = 0;      // next block to fold into the next chunk's rows
        int pub = 0;     // (wave 2) next block to publish
        int loaded = 1;  // (wave 3) chunks whose Gram blocks and labels are in LDS
        long idle = 0;
        while (fc < nblk || fn < nblk || (pw && pub < nblk) || (lw && loaded < nchk)) {
            bool progress = false;
            const int dd = lds_read(d1done);
            if (pw && pub < nblk && dd >= min(BS * (pub + 1), nsteps)) {
                // ---- publish block `pub` for the tile workgroups
                const int c = pub / NB, b = pub % NB, tc = chunk_len(c);
                float* dout = a.d1 + ((size_t)(c & 1) * K + k) * T * H;  // [h][T] errors of chunk c
                const int s0 = BS * b;
                // all of the lane's LDS reads first, then the stores (HW * BS / 4 float4 per block)
                constexpr int NQ = HW * (BS / 4) / 64;
                float4 dv[NQ];
#pragma unroll
                for (int i = 0; i < NQ; ++i) {
                    const int q = lane + 64 * i, hh = q / (BS / 4), s4 = s0 + (q % (BS / 4)) * 4;
                    dv[i] = *(const float4*)(hist + hh * TS + s4);
                }
#pragma unroll
                for (int i = 0; i < NQ; ++i) {
                    const int q = lane + 64 * i, hh = q / (BS / 4), s4 = s0 + (q % (BS / 4)) * 4;
                    if (hh < H) *(float4*)(dout + (size_t)hh * T + s4) = dv[i];
                }
                ++pub;
                lds_publish(pubd, pub);  // (the hist reads completed: the stores consumed them)
                if (BS * (b + 1) >= tc) {
                    // every error of chunk c is stored: announce it to the tiles
                    wait_vm_all();
                    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "agent");
                    if (lane == 0) __hip_atomic_store(dready, c + 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                }
                progress = true;
            } else if (fc < nblk && dd >= min(BS * (fc + 1), nsteps) && fn >= NB * (fc / NB)) {
                // ---- block fc into the later rows of its own chunk (accC is that chunk's:
                // every fold of the previous chunk into it is done); rows of block b+2 final
                const int c = fc / NB, b = fc % NB;
                if (BS * (b + 2) < chunk_len(c)) {
                    fold_acc<GS, TS, MT, NT>(accC, grow_in(c), hist, (b + 2) >> 1, BS * b, -lr, nt0, lane);
                    write_rows<TS, MT, NT>(accC, Pl, b + 2, nt0, lane);
                    lds_publish(rd, fc + 3);
                } else if (c + 1 >= nchk) {
                    lds_publish(rd, fc + 3);  // no rows left to complete
                }
                ++fc;
                progress = true;
            } else if (lw && loaded < nchk) {
                // ---- load chunk `loaded`'s Gram blocks and labels into the buffers of parity
                // loaded & 1 once the current chunk no longer needs the cross Gram block: the
                // first block's window corrections are done and both waves have completed
                // the chunk's rows of blocks 0 and 1 (the folds that read it).  The buffers of
                // that parity last served the chunk before the current one.
                const int c = loaded - 1;  // chunk the live wave is in (or before)
                // (The live wave reads the cross block for the chunk's rows tn < NLIVE, in steps up
                // to T c + NLIVE - 2.)
                const bool gx_free = (c == 0) || (lds_read(cdone) >= min(T * c + BS + 1, nsteps) &&
                                                  lds_read(d1done) >= min(T * c + NLIVE, nsteps) &&
                                                  lds_read(rdy) >= NB * c + 2 && lds_read(rdy + 1) >= NB * c + 2);
                if (gx_free) {
                    const int cn = loaded, tcn = chunk_len(cn);
                    const float* G = a.gram + ((size_t)k * a.nch + cn) * T * GS;
                    const float* GXg = a.gramx + ((size_t)k * (a.nch - 1) + cn - 1) * T * GS;
                    wave_copy_to_lds(G, Gin + (cn & 1) * T * GS, T * GS * 4, 0, 1, lane);
                    wave_copy_to_lds(GXg, GX, T * GS * 4, 0, 1, lane);
                    {
                        const int rr = min(lane, tcn - 1);
                        __builtin_amdgcn_global_load_lds(a.y + xs + (int64_t)cn * T + rr,
                                                         (lds_void*)(yb + (cn & 1) * T), 4, 0, 0);
                    }
                    wait_vm_all();
                    ++loaded;
                    lds_publish(gready, loaded);
                    progress = true;
                }
            }
            if (!progress && fn < fc) {
                // ---- block fn into every row of the next chunk, once its Gram blocks are in
                // LDS; blocks NB-2 and NB-1 complete the next chunk's blocks 0 and 1 (Q of
                // the next chunk needed: the tiles publish it one chunk ahead)
                const int c = fn / NB, b = fn % NB;
                if (c + 1 >= nchk) {
                    ++fn;  // nothing of this block goes into a next chunk
                    progress = true;
                } else if (lds_read(gready) >= c + 2) {
                    fold_acc<GS, TS, MT, NT>(accN, GX, hist, 0, BS * b, -lr, nt0, lane);
                    if (b >= NB - 2) {
                        if (!qn) {
                            if (!wait_geq_wave(qready(c + 1), qtarget(c + 1), gabort, a.spin_limit)) {
                                lds_publish(lab, 1);
                                break;
                            }
                            add_q<TS, MT, NT>(accN, qrows(c + 1), nt0, lane);
                            qn = true;
                        }
                        write_rows<TS, MT, NT>(accN, Pl, b - (NB - 2), nt0, lane);
                        lds_publish(rd, NB * (c + 1) + b - (NB - 2) + 1);
                        if (b == NB - 1) {
#pragma unroll
                            for (int mt = 0; mt < MT; ++mt)
#pragma unroll
                                for (int nt = 0; nt < NT; ++nt) {
                                    accC[mt][nt] = accN[mt][nt];
                                    accN[mt][nt] = f4{0.f, 0.f, 0.f, 0.f};
                                }
                            qn = false;
                        }
                    }
                    ++fn;
                    progress = true;
                }
            }
            if (!progress && !qn && fn / NB + 1 < nchk && (idle & 7) == 0) {
                // ---- Q of accN's chunk, as soon as the tiles have published it
                const int cq = fn / NB + 1;
                const int qv = __builtin_amdgcn_readfirstlane(
                    __hip_atomic_load(qready(cq), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT));
                if (qv >= qtarget(cq)) {
                    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "agent");
                    add_q<TS, MT, NT>(accN, qrows(cq), nt0, lane);
                    qn = true;
                    progress = true;
                }
            }
            if (!progress) {
                if (lds_read(lab)) break;
                if (++idle > a.spin_limit) {
                    lds_publish(lab, 1);
                    __hip_atomic_store(gabort, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                    break;
                }
                __builtin_amdgcn_s_sleep(1);
            } else {
                idle = 0;
            }
        }
    }
}

// A tile workgroup owns RT x 16 neurons (RT sub-tiles of 16 rows of W1) of one CN: more CNs
// fit the chip with RT = 2, and the input rows each sub-tile needs are loaded once for all.
template <int T, int RT>
__device__ __attribute__((always_inline)) inline void psgd_tile(const PsgdPArgs& a, int k, int rb, float* smem) {
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int H = a.H, In = a.In, K = a.k_rep;
    const int hb = rb * RT * 16;  // first neuron of the tile
    const int g = lane >> 4;
    const int nib = (In + 15) / 16;  // input blocks of 16; wave w owns blocks w, w+4, ...
    float* th = a.theta + (size_t)k * a.pstride;
    float W[RT][MAX_IB][4];
#pragma unroll
    for (int r = 0; r < RT; ++r) {
        const int h = hb + r * 16 + (lane & 15);
#pragma unroll
        for (int j = 0; j < MAX_IB; ++j)
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                const int ib = wave + 4 * j, i = ib * 16 + 4 * g + q;
                W[r][j][q] = (ib < nib && h < H && i < In) ? th[a.off_w1 + (size_t)h * In + i] : 0.f;
            }
    }
    const int64_t nz = shard_len(a.n_total, K, k), xs = shard_start(a.n_total, K, k);
    const int nchk = (int)((nz + T - 1) / T);
    int* dready = a.flags + 2 * K + k;
    int* abort = a.flags + 3 * K;
    constexpr int NMT = T / 16;
    float* red4 = smem;  // [4 waves][NMT][RT][64][4]

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
#pragma unroll
            for (int r = 0; r < RT; ++r) {
                f4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
                for (int j = 0; j < MAX_IB; ++j) {
                    acc = __builtin_amdgcn_mfma_f32_16x16x4f32(xv[j].x, W[r][j][0], acc, 0, 0, 0);
                    acc = __builtin_amdgcn_mfma_f32_16x16x4f32(xv[j].y, W[r][j][1], acc, 0, 0, 0);
                    acc = __builtin_amdgcn_mfma_f32_16x16x4f32(xv[j].z, W[r][j][2], acc, 0, 0, 0);
                    acc = __builtin_amdgcn_mfma_f32_16x16x4f32(xv[j].w, W[r][j][3], acc, 0, 0, 0);
                }
                *(f4*)(red4 + (((size_t)(wave * NMT + mt) * RT + r) * 64 + lane) * 4) = acc;
            }
        }
        __syncthreads();
        float* Q = a.qbuf + ((size_t)(c & 1) * K + k) * a.qslot;
        for (int e = tid; e < NMT * RT * 256; e += 256) {
            const int mr = e >> 8, rem = e & 255, ln = rem >> 2, rr = rem & 3;  // mr = mt * RT + r
            const int mt = mr / RT, r = mr - mt * RT;
            float sum = 0.f;
#pragma unroll
            for (int w = 0; w < 4; ++w) sum += red4[(((size_t)(w * NMT + mt) * RT + r) * 64 + ln) * 4 + rr];
            const int t = mt * 16 + 4 * (ln >> 4) + rr, hh = hb + r * 16 + (ln & 15);
            if (t < tc && hh < H) Q[(size_t)hh * a.qstride + t] = sum;
        }
        signal_add(a.flags + (c & 1) * K + k, 1);  // one counter per chunk parity
    };
    // W1 tile -= eta * sum_t d1_t x_t^T over the rows of chunk c (errors stored [h][T])
    auto update = [&](int c) {
        const int tc = (int)min<int64_t>(T, nz - (int64_t)c * T);
        const int64_t xb = xs + (int64_t)c * T;
        float bv[RT][T / 4];
#pragma unroll
        for (int r = 0; r < RT; ++r) {
            const int h = hb + r * 16 + (lane & 15);
            const float* D = a.d1 + ((size_t)(c & 1) * K + k) * H * T + (size_t)(h < H ? h : 0) * T;
#pragma unroll
            for (int sl = 0; sl < T / 16; ++sl) {
                const float4 d = *(const float4*)(D + sl * 16 + 4 * g);
                const int t0 = sl * 16 + 4 * g;
                bv[r][4 * sl + 0] = (h < H && t0 + 0 < tc) ? d.x : 0.f;
                bv[r][4 * sl + 1] = (h < H && t0 + 1 < tc) ? d.y : 0.f;
                bv[r][4 * sl + 2] = (h < H && t0 + 2 < tc) ? d.z : 0.f;
                bv[r][4 * sl + 3] = (h < H && t0 + 3 < tc) ? d.w : 0.f;
            }
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
#pragma unroll
            for (int r = 0; r < RT; ++r) {
                f4 dacc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
                for (int u = 0; u < T / 4; ++u) dacc = __builtin_amdgcn_mfma_f32_16x16x4f32(av[u], bv[r][u], dacc, 0, 0, 0);
#pragma unroll
                for (int q = 0; q < 4; ++q) W[r][j][q] -= a.lr * dacc[q];
            }
        }
    };

    // Q_0 and Q_1 use the initial weights; afterwards chunk c's errors (c >= 0) are applied
    // before Q_{c+2} is computed.  One call site each keeps the code compact.
    bool ok = true;
    if (a.tile_delay > 0 && 2 * rb >= a.nrb)
        for (int i = 0; i < a.tile_delay; ++i) __builtin_amdgcn_s_sleep(127);
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
    for (int r = 0; r < RT; ++r) {
        const int h = hb + r * 16 + (lane & 15);
#pragma unroll
        for (int j = 0; j < MAX_IB; ++j)
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                const int ib = wave + 4 * j, i = ib * 16 + 4 * g + q;
                if (ib < nib && h < H && i < In) th[a.off_w1 + (size_t)h * In + i] = W[r][j][q];
            }
    }
}

template <int T, int NH, int A1, int A2, int LS, int OC, int RT>
__global__ __launch_bounds__(256) void psgd_persistent_kernel(PsgdPArgs a) {
    extern __shared__ float smem[];
    const int b = blockIdx.x, K = a.k_rep, KL = a.k_launch;
    // an earlier launch gave up waiting: the parameters are unspecified, train no further
    if (__hip_atomic_load(a.flags + 3 * K, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT)) return;
    if (b < KL) psgd_rec<T, NH, A1, A2, LS, OC>(a, a.cn0 + b, smem);
    else {
        const int j = b - KL;
        psgd_tile<T, RT>(a, a.cn0 + j / a.nrb, j % a.nrb, smem);
    }
}

// ------------------------------------------------------------------------------------
// Mini-batch gradient descent of a one-hidden-layer fp32 network with batches of at most
// 32 rows: one persistent launch per epoch (forward eq. (2)-(3), output error eq. (9)-(10),
// hidden error eq. (11), updates eq. (12)-(13) with the gradients averaged over each batch).
//
// Tile workgroup (k, rb) owns, for CN k, the hidden neurons j in [16 RT rb, 16 RT (rb + 1)):
// their rows of W1 in registers (laid out as in psgd_tile), their biases b1 and their
// columns of W2 in LDS, and a private copy of b2.  Batch step c (rows of the step t < B_c):
//   1. a1[t][j] = phi(W1[j] . x_t + b1[j]) for the tile's neurons; the batch's rows (loaded
//      during the previous step's update) are staged in LDS on the way;
//   2. the tile's share of the output sums, Z2_rb[t][o] = sum_j W2[o][j] a1[t][j], goes to
//      global memory;
//   3. every tile reads the nrb shares of its CN, adds them in the same order, adds b2 and
//      forms the output error delta2 (the same values in every tile of the CN);
//   4. d1[t][j] = phi'(a1[t][j]) sum_o W2[o][j] delta2[t][o] with the pre-update W2; then W2
//      (tile columns), b2, b1 and W1 (tile rows) -= eta / B_c * their gradients summed over
//      the batch (every tile updates its copy of b2 identically).
// Each share value is one 64-bit word written and read with agent-scope relaxed atomics:
// the float in the low half and the step's tag (tag0 + c, increasing across launches) in
// the high half, so a reader polls each value until it carries the step's tag and needs no
// cache-wide release or acquire.  Shares are double buffered by step parity: a tile writes
// step c+2's share only after it has read every share of step c+1, and every tile computed
// its step c+1 share from the step c shares it had read.

constexpr int MBP_TB = 32;    // most rows of a batch step
constexpr int MBP_NRB = 16;   // most tile workgroups per CN

struct MbpArgs {
    float* theta;
    int64_t pstride, off_w1, off_b1, off_w2, off_b2;
    const float* X;
    const int32_t* y;
    int64_t n_total;
    unsigned long long* zpart;  // [2][K][nrb][MBP_TB][16] tagged output-sum shares
    int* flags;                 // [K + 1]; flags[K]: abort (sticky: cleared only at allocation)
    int k_rep, H, O, In, act1, act2, loss, nrb, B;
    int cn0;                    // this launch trains CNs cn0 .. cn0 + gridDim.x / nrb - 1
    int xcd_map;                // 1: the tiles of a CN run on one XCD (grid a multiple of 8)
    unsigned tag0;              // tag of step 0 (>= 1)
    unsigned tag_skew;          // 0; > 0 makes the readers wait for tags never written (abort test)
    float lr;
    long spin_limit;
};

// LDS floats: the batch's rows transposed [64 MAX_IB][36] (every input block of the four
// waves, zero past the inputs), partial input sums of the 4 waves, activations
// [32][16 RT + 1], W2 columns [16][16 RT + 1], output errors [32][17], hidden errors
// [16 RT][36], b1 [16 RT], b2 [16]
__host__ __device__ constexpr int mbp_lds_floats(int rt) {
    return 64 * MAX_IB * (MBP_TB + 4) + 4 * (MBP_TB / 16) * rt * 256 + MBP_TB * (16 * rt + 1) +
           16 * (16 * rt + 1) + MBP_TB * 17 + 16 * rt * (MBP_TB + 4) + 16 * rt + 16;
}

template <int RT>
__global__ __launch_bounds__(256) void mbp_kernel(MbpArgs a) {
    extern __shared__ __attribute__((aligned(16))) float smem[];
    constexpr int NR = 16 * RT, NMT = MBP_TB / 16, LA = NR + 1, LD1 = MBP_TB + 4, ZS = MBP_TB * 16;
    constexpr int XT = MBP_TB + 4;  // row stride of the transposed batch rows
    const int tid = threadIdx.x, lane = tid & 63, g = lane >> 4, l16 = lane & 15;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);  // (uniform: keeps the block tests scalar)
    const int H = a.H, O = a.O, In = a.In, K = a.k_rep, nrb = a.nrb;
    // an earlier launch gave up waiting: the parameters are unspecified, train no further
    if (__hip_atomic_load(a.flags + K, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT)) return;
    // workgroups go to the 8 XCDs in turn by id: with xcd_map, ids x, x + 8, x + 16, ... hold
    // consecutive tiles, so that a CN's tiles share one L2
    int lin = blockIdx.x;
    if (a.xcd_map) lin = (blockIdx.x & 7) * (gridDim.x >> 3) + (blockIdx.x >> 3);
    const int k = a.cn0 + lin / nrb, rb = lin % nrb;
    const int hb = rb * NR;
    const int nib = (In + 15) / 16;
    float* xsm = smem;                       // [64 MAX_IB][XT] the batch's rows transposed: [input][row]
    float* red4 = xsm + 64 * MAX_IB * XT;    // [4 waves][NMT][RT][64][4]
    float* a1s = red4 + 4 * NMT * RT * 256;  // [MBP_TB][LA]
    float* w2s = a1s + MBP_TB * LA;          // [16][LA], rows o >= O and columns past H zero
    float* dls = w2s + 16 * LA;              // [MBP_TB][17]
    float* d1s = dls + MBP_TB * 17;          // [NR][LD1]
    float* b1s = d1s + NR * LD1;             // [NR]
    float* b2s = b1s + NR;                   // [16]
    float* th = a.theta + (size_t)k * a.pstride;

    float W[RT][MAX_IB][4];
#pragma unroll
    for (int r = 0; r < RT; ++r) {
        const int h = hb + r * 16 + l16;
#pragma unroll
        for (int j = 0; j < MAX_IB; ++j)
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                const int ib = wave + 4 * j, i = ib * 16 + 4 * g + q;
                W[r][j][q] = (ib < nib && h < H && i < In) ? th[a.off_w1 + (size_t)h * In + i] : 0.f;
            }
    }
    for (int e = tid; e < 16 * NR; e += 256) {
        const int o = e / NR, j = e - o * NR;
        w2s[o * LA + j] = (o < O && hb + j < H) ? th[a.off_w2 + (size_t)o * H + hb + j] : 0.f;
    }
    if (tid < NR) b1s[tid] = hb + tid < H ? th[a.off_b1 + hb + tid] : 0.f;
    if (tid < 16) b2s[tid] = tid < O ? th[a.off_b2 + tid] : 0.f;

    const int64_t nz = shard_len(a.n_total, K, k), xs = shard_start(a.n_total, K, k);
    const int nsteps = (int)((nz + a.B - 1) / a.B);
    int* abort = a.flags + K;
    // the batch's rows as operands of the input sums (lane: row mt * 16 + l16, inputs
    // 16 ib + 4 g .. + 3 of the blocks ib = wave + 4 j), zero past the batch and past In;
    // loaded one step ahead
    float4 xn[NMT][MAX_IB];
    int yn[ZS / 256];  // labels of the rows (tid + 256 u) / 16
    // (bounds-checked buffer loads over the step's rows: rows past the step read as zero;
    // blocks past In (In is a multiple of 16) read the next row, or zero after the last, and
    // meet zero weights in the input sums and a zero mask in the weight update)
    // rows_rsrc(c): descriptor of step c's rows; load_row_block(rs, idx): operand idx = mt * MAX_IB
    // + j of buffer xn (issued one by one so that they can be spread over other work)
    auto rows_rsrc = [&](int c) {
        const int tcn = (int)min<int64_t>(a.B, nz - (int64_t)c * a.B);
        const int64_t xbn = xs + (int64_t)c * a.B;
        return __builtin_amdgcn_make_buffer_rsrc((void*)(a.X + (size_t)xbn * In), (short)0, tcn * In * 4, 0x00020000);
    };
    auto load_row_block = [&](__amdgpu_buffer_rsrc_t rs, int idx) {
        const int mt = idx / MAX_IB, j = idx - mt * MAX_IB;
        const unsigned vo = (unsigned)((mt * 16 + l16) * In + wave * 16 + 4 * g) * 4u;
        xn[mt][j] = __builtin_bit_cast(float4, __builtin_amdgcn_raw_buffer_load_b128(rs, vo + 256u * j, 0, 0));
    };
    auto load_labels = [&](int c) {
        const int tcn = (int)min<int64_t>(a.B, nz - (int64_t)c * a.B);
        const int64_t xbn = xs + (int64_t)c * a.B;
#pragma unroll
        for (int u = 0; u < ZS / 256; ++u) {
            const int t = (tid + 256 * u) >> 4;
            yn[u] = a.y[xbn + (t < tcn ? t : 0)];
        }
    };
    if (nsteps > 0) {
        const __amdgpu_buffer_rsrc_t rs0 = rows_rsrc(0);
#pragma unroll
        for (int idx = 0; idx < NMT * MAX_IB; ++idx) load_row_block(rs0, idx);
        load_labels(0);
    }
    __syncthreads();
    bool ok = true;
    for (int c = 0; c < nsteps; ++c) {
        const int tc = (int)min<int64_t>(a.B, nz - (int64_t)c * a.B);
        const float scale = a.lr / (float)tc;
        const unsigned long long tag = (unsigned long long)(a.tag0 + (unsigned)c) << 32;
        int yc[ZS / 256];
#pragma unroll
        for (int u = 0; u < ZS / 256; ++u) yc[u] = yn[u];
        // 1. input sums of the tile's neurons (wave w adds the input blocks w, w + 4, ...),
        //    then the activations; rows past the batch and neurons past H are zero.  The rows
        //    are staged transposed for the weight update.
#pragma unroll
        for (int mt = 0; mt < NMT; ++mt) {
            const int row = mt * 16 + l16;
            f4 acc[RT];
#pragma unroll
            for (int r = 0; r < RT; ++r) acc[r] = f4{0.f, 0.f, 0.f, 0.f};
            // (each block's staging stores follow its matrix instructions, which run meanwhile)
#pragma unroll
            for (int j = 0; j < MAX_IB; ++j) {
#pragma unroll
                for (int r = 0; r < RT; ++r) {
                    acc[r] = __builtin_amdgcn_mfma_f32_16x16x4f32(xn[mt][j].x, W[r][j][0], acc[r], 0, 0, 0);
                    acc[r] = __builtin_amdgcn_mfma_f32_16x16x4f32(xn[mt][j].y, W[r][j][1], acc[r], 0, 0, 0);
                    acc[r] = __builtin_amdgcn_mfma_f32_16x16x4f32(xn[mt][j].z, W[r][j][2], acc[r], 0, 0, 0);
                    acc[r] = __builtin_amdgcn_mfma_f32_16x16x4f32(xn[mt][j].w, W[r][j][3], acc[r], 0, 0, 0);
                }
                float* xt = xsm + ((wave + 4 * j) * 16 + 4 * g) * XT + row;
                xt[0] = xn[mt][j].x;
                xt[XT] = xn[mt][j].y;
                xt[2 * XT] = xn[mt][j].z;
                xt[3 * XT] = xn[mt][j].w;
            }
#pragma unroll
            for (int r = 0; r < RT; ++r)
                *(f4*)(red4 + (((size_t)(wave * NMT + mt) * RT + r) * 64 + lane) * 4) = acc[r];
        }
        __syncthreads();
        for (int e = tid; e < NMT * RT * 256; e += 256) {
            const int mr = e >> 8, rem = e & 255, ln = rem >> 2, rr = rem & 3;  // mr = mt * RT + r
            const int mt = mr / RT, r = mr - mt * RT;
            float sum = 0.f;
#pragma unroll
            for (int w = 0; w < 4; ++w) sum += red4[(((size_t)(w * NMT + mt) * RT + r) * 64 + ln) * 4 + rr];
            const int t = mt * 16 + 4 * (ln >> 4) + rr, jj = r * 16 + (ln & 15);
            a1s[t * LA + jj] = (t < tc && hb + jj < H) ? act_fn(a.act1, sum + b1s[jj]) : 0.f;
        }
        __syncthreads();
        // 2. the tile's share of the output sums, Z2_rb = a1 W2_rb^T: wave mt takes rows
        //    16 mt .. 16 mt + 15 (lane: rows 16 mt + 4 g + i, output l16)
        unsigned long long* zp = a.zpart + (size_t)((c & 1) * K + k) * nrb * ZS;
        if (wave < NMT) {
            f4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int r = 0; r < RT; ++r)
#pragma unroll
                for (int ks = 0; ks < 4; ++ks) {
                    const int jj = r * 16 + 4 * ks + g;
                    acc = __builtin_amdgcn_mfma_f32_16x16x4f32(a1s[(wave * 16 + l16) * LA + jj], w2s[l16 * LA + jj], acc,
                                                               0, 0, 0);
                }
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const int t = wave * 16 + 4 * g + i;
                if (t < tc && l16 < O)
                    __hip_atomic_store(zp + (size_t)rb * ZS + t * 16 + l16, tag | __float_as_uint(acc[i]), __ATOMIC_RELAXED,
                                       __HIP_MEMORY_SCOPE_AGENT);
            }
        }
        // 3. every share of the CN, polled until it carries this step's tag (bounded: on
        //    expiry, or when another workgroup gave up, the abort flag ends every workgroup)
        float sv[ZS / 256][MBP_NRB];
        {
            unsigned need = 0;
#pragma unroll
            for (int u = 0; u < ZS / 256; ++u) {
                const int e = tid + 256 * u, t = e >> 4, o = e & 15;
#pragma unroll
                for (int q = 0; q < MBP_NRB; ++q)
                    if (q < nrb && t < tc && o < O) need |= 1u << (u * MBP_NRB + q);
            }
            long it = 0;
            bool good = true;
            while (need) {
                unsigned long long v[ZS / 256][MBP_NRB];
#pragma unroll
                for (int u = 0; u < ZS / 256; ++u)
#pragma unroll
                    for (int q = 0; q < MBP_NRB; ++q)
                        if (need & (1u << (u * MBP_NRB + q)))
                            v[u][q] = __hip_atomic_load(zp + (size_t)q * ZS + tid + 256 * u, __ATOMIC_RELAXED,
                                                        __HIP_MEMORY_SCOPE_AGENT);
#pragma unroll
                for (int u = 0; u < ZS / 256; ++u)
#pragma unroll
                    for (int q = 0; q < MBP_NRB; ++q)
                        if ((need & (1u << (u * MBP_NRB + q))) && (v[u][q] >> 32) == (tag >> 32) + a.tag_skew) {
                            sv[u][q] = __uint_as_float((unsigned)v[u][q]);
                            need &= ~(1u << (u * MBP_NRB + q));
                        }
                if (!need) break;
                if (__hip_atomic_load(abort, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT)) { good = false; break; }
                if (++it > a.spin_limit) {
                    __hip_atomic_store(abort, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                    good = false;
                    break;
                }
                __builtin_amdgcn_s_sleep(1);
            }
            if (__syncthreads_or(!good)) { ok = false; break; }
        }
        // output sums, output activation and output error; the 16 outputs of a row are 16
        // adjacent lanes
#pragma unroll
        for (int u = 0; u < ZS / 256; ++u) {
            const int e = tid + 256 * u, t = e >> 4, o = e & 15;
            const bool live = t < tc && o < O;
            float zv = 0.f;
            if (live) {
                float s = 0.f;
#pragma unroll
                for (int q = 0; q < MBP_NRB; ++q)
                    if (q < nrb) s += sv[u][q];
                zv = s + b2s[o];
            }
            float xo;
            if (a.act2 == ACT_SOFTMAX) {
                float m = live ? zv : -INFINITY;
#pragma unroll
                for (int sh = 1; sh < 16; sh <<= 1) m = fmaxf(m, __shfl_xor(m, sh, 16));
                const float ex = live ? expf(zv - m) : 0.f;
                float sm = ex;
#pragma unroll
                for (int sh = 1; sh < 16; sh <<= 1) sm += __shfl_xor(sm, sh, 16);
                xo = ex * (1.0f / sm);
            } else {
                xo = act_fn(a.act2, zv);
            }
            float dv = 0.f;
            if (live) {
                const float t1 = (o == yc[u]) ? 1.0f : 0.0f;
                dv = (a.loss == LOSS_XENT) ? (xo - t1) : (xo - t1) * act_deriv(a.act2, xo);
            }
            dls[t * 17 + o] = dv;
        }
        __syncthreads();
        // 4. hidden errors of the tile's neurons with the pre-update W2, S = delta2 W2_rb:
        //    wave mt takes rows 16 mt .. 16 mt + 15 (lane: rows 16 mt + 4 g + i, neuron l16)
        if (wave < NMT) {
#pragma unroll
            for (int r = 0; r < RT; ++r) {
                f4 sacc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
                for (int ks = 0; ks < 4; ++ks)
                    sacc = __builtin_amdgcn_mfma_f32_16x16x4f32(dls[(wave * 16 + l16) * 17 + 4 * ks + g],
                                                                w2s[(4 * ks + g) * LA + r * 16 + l16], sacc, 0, 0, 0);
                const int t0 = wave * 16 + 4 * g, jj = r * 16 + l16;
                float4 d;
                d.x = sacc[0] * act_deriv(a.act1, a1s[(t0 + 0) * LA + jj]);
                d.y = sacc[1] * act_deriv(a.act1, a1s[(t0 + 1) * LA + jj]);
                d.z = sacc[2] * act_deriv(a.act1, a1s[(t0 + 2) * LA + jj]);
                d.w = sacc[3] * act_deriv(a.act1, a1s[(t0 + 3) * LA + jj]);
                *(float4*)(d1s + jj * LD1 + t0) = d;
            }
        }
        __syncthreads();
        // W2 columns (wave 2: dW2 = delta2^T a1 over the batch, lane: outputs 4 g + i, neuron
        // l16), b2 (wave 1) and b1 (wave 3); their readers in the next step follow a barrier.
        // Rows past the batch are zero in delta2, a1 and d1.
        if (wave == 2) {
            float da[MBP_TB / 4];
#pragma unroll
            for (int ks = 0; ks < MBP_TB / 4; ++ks) da[ks] = dls[(4 * ks + g) * 17 + l16];
#pragma unroll
            for (int r = 0; r < RT; ++r) {
                float xa[MBP_TB / 4];
#pragma unroll
                for (int ks = 0; ks < MBP_TB / 4; ++ks) xa[ks] = a1s[(4 * ks + g) * LA + r * 16 + l16];
                f4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
                for (int ks = 0; ks < MBP_TB / 4; ++ks) acc = __builtin_amdgcn_mfma_f32_16x16x4f32(da[ks], xa[ks], acc, 0, 0, 0);
                const int jj = r * 16 + l16;
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    const int o = 4 * g + i;
                    if (o < O && hb + jj < H) w2s[o * LA + jj] -= scale * acc[i];
                }
            }
        } else if (wave == 1) {
            // lane: output l16, rows 8 g .. 8 g + 7; the four partial sums added in lane order
            float p = 0.f;
#pragma unroll
            for (int t = 0; t < 8; ++t) p += dls[(8 * g + t) * 17 + l16];
            const float s = __shfl(p, l16) + __shfl(p, l16 + 16) + __shfl(p, l16 + 32) + __shfl(p, l16 + 48);
            if (lane < O) b2s[lane] -= scale * s;
        } else if (wave == 3) {
            if (lane < NR && hb + lane < H) {
                float s = 0.f;
#pragma unroll
                for (int t4 = 0; t4 < MBP_TB / 4; ++t4) {
                    const float4 d = *(const float4*)(d1s + lane * LD1 + 4 * t4);
                    s += d.x;
                    s += d.y;
                    s += d.z;
                    s += d.w;
                }
                b1s[lane] -= scale * s;
            }
        }
        // W1 rows of the tile -= eta / B_c sum_t d1_t x_t^T (a product whose accumulator layout
        // equals the register layout); the next step's rows are loaded meanwhile, a few loads
        // per pair of blocks
        // (with 32-neuron tiles all of them at once: spreading them costs registers that tile
        // does not have)
        const bool more = c + 1 < nsteps;
        const __amdgpu_buffer_rsrc_t rsn = rows_rsrc(more ? c + 1 : c);
        if (more) load_labels(c + 1);
        if (RT > 1 && more) {
#pragma unroll
            for (int idx = 0; idx < NMT * MAX_IB; ++idx) load_row_block(rsn, idx);
        }
        {
            float bv[RT][MBP_TB / 4];
#pragma unroll
            for (int r = 0; r < RT; ++r) {
                const float* D = d1s + (r * 16 + l16) * LD1;
#pragma unroll
                for (int sl = 0; sl < MBP_TB / 16; ++sl) {
                    const float4 d = *(const float4*)(D + sl * 16 + 4 * g);
                    bv[r][4 * sl + 0] = d.x;
                    bv[r][4 * sl + 1] = d.y;
                    bv[r][4 * sl + 2] = d.z;
                    bv[r][4 * sl + 3] = d.w;
                }
            }
            // Blocks in pairs: two independent accumulation chains interleaved, and the next
            // pair's staged rows read before this pair's matrix instructions (blocks past the
            // inputs hold zero rows and weights: one branch-free sequence).
            // rows (u >> 2) * 16 + 4 g + (u & 3) of input (wave + 4 j) * 16 + l16; blocks past In
            // stay zero
            auto read_block = [&](int j, float (&av)[MBP_TB / 4]) {
                const bool jok = wave + 4 * j < nib;
                const float* xt = xsm + ((wave + 4 * j) * 16 + l16) * XT + 4 * g;
                const float4 x0 = *(const float4*)xt, x1 = *(const float4*)(xt + 16);
                av[0] = jok ? x0.x : 0.f; av[1] = jok ? x0.y : 0.f; av[2] = jok ? x0.z : 0.f; av[3] = jok ? x0.w : 0.f;
                av[4] = jok ? x1.x : 0.f; av[5] = jok ? x1.y : 0.f; av[6] = jok ? x1.z : 0.f; av[7] = jok ? x1.w : 0.f;
            };
            float avA[MBP_TB / 4], avB[MBP_TB / 4];
            read_block(0, avA);
            if (1 < MAX_IB) read_block(1, avB);
            constexpr int LPP = (NMT * MAX_IB + (MAX_IB + 1) / 2 - 1) / ((MAX_IB + 1) / 2);  // loads per pair
#pragma unroll
            for (int j = 0; j < MAX_IB; j += 2) {
                const bool two = j + 1 < MAX_IB;
                if (RT == 1 && more) {
#pragma unroll
                    for (int i = 0; i < LPP; ++i)
                        if ((j / 2) * LPP + i < NMT * MAX_IB) load_row_block(rsn, (j / 2) * LPP + i);
                }
                float nA[MBP_TB / 4], nB[MBP_TB / 4];
                if (j + 2 < MAX_IB) read_block(j + 2, nA);
                if (j + 3 < MAX_IB) read_block(j + 3, nB);
#pragma unroll
                for (int r = 0; r < RT; ++r) {
                    f4 dA = {0.f, 0.f, 0.f, 0.f}, dB = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
                    for (int u = 0; u < MBP_TB / 4; ++u) {
                        dA = __builtin_amdgcn_mfma_f32_16x16x4f32(avA[u], bv[r][u], dA, 0, 0, 0);
                        if (two) dB = __builtin_amdgcn_mfma_f32_16x16x4f32(avB[u], bv[r][u], dB, 0, 0, 0);
                    }
#pragma unroll
                    for (int q = 0; q < 4; ++q) {
                        W[r][j][q] -= scale * dA[q];
                        if (two) W[r][j + 1][q] -= scale * dB[q];
                    }
                }
#pragma unroll
                for (int u = 0; u < MBP_TB / 4; ++u) {
                    if (j + 2 < MAX_IB) avA[u] = nA[u];
                    if (j + 3 < MAX_IB) avB[u] = nB[u];
                }
            }
        }
        // (the next step's forward overwrites the staged rows; LDS only, so the barrier does not
        // wait for the next step's row loads, which the forward waits for itself)
        lds_barrier();
    }
    if (!ok) return;
#pragma unroll
    for (int r = 0; r < RT; ++r) {
        const int h = hb + r * 16 + l16;
#pragma unroll
        for (int j = 0; j < MAX_IB; ++j)
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                const int ib = wave + 4 * j, i = ib * 16 + 4 * g + q;
                if (ib < nib && h < H && i < In) th[a.off_w1 + (size_t)h * In + i] = W[r][j][q];
            }
    }
    for (int e = tid; e < 16 * NR; e += 256) {
        const int o = e / NR, j = e - o * NR;
        if (o < O && hb + j < H) th[a.off_w2 + (size_t)o * H + hb + j] = w2s[o * LA + j];
    }
    if (tid < NR && hb + tid < H) th[a.off_b1 + hb + tid] = b1s[tid];
    if (rb == 0 && tid < O) th[a.off_b2 + tid] = b2s[tid];
}

// Rows of an epoch in a given order: row r of (xo, yo) is data-set row order[r] (entries
// outside [0, N) select row 0).  One workgroup per row.
__global__ __launch_bounds__(256) void gather_rows_kernel(const float* x, const int32_t* y, const int32_t* order,
                                                          int64_t N, int D, float* xo, int32_t* yo) {
    const int64_t r = blockIdx.x;
    int64_t src = order[r];
    if (src < 0 || src >= N) src = 0;
    const float* xs = x + (size_t)src * D;
    float* xd = xo + (size_t)r * D;
    if ((D & 3) == 0) {
        for (int c = threadIdx.x; c < D / 4; c += 256) ((float4*)xd)[c] = ((const float4*)xs)[c];
    } else {
        for (int c = threadIdx.x; c < D; c += 256) xd[c] = xs[c];
    }
    if (threadIdx.x == 0) yo[r] = y[src];
}

// sum of n doubles in a fixed order (thread t takes t, t + 256, ...; then a fixed tree)
__global__ __launch_bounds__(256) void sum_f64_kernel(const double* v, int64_t n, double* out) {
    __shared__ double part[256];
    const int t = threadIdx.x;
    double s = 0.0;
    for (int64_t i = t; i < n; i += 256) s += v[i];
    part[t] = s;
    __syncthreads();
    for (int h = 128; h > 0; h >>= 1) {
        if (t < h) part[t] += part[t + h];
        __syncthreads();
    }
    if (t == 0) *out = part[0];
}

__global__ void zero_ints_kernel(int* p, int n) {
    const int i = blockIdx.x * blockDim.x + threadIdx.x;
    if (i < n) p[i] = 0;
}

}  // namespace pnn
