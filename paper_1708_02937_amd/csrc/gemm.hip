// Dense-W comparison arm: Z^T = W^T Y^T on matrix cores with the bias and activation fused.
//
// This is the layer product with every zero of W_k stored explicitly, the dense-linear-algebra version
// the paper measures its sparse library against (Sec. V.A, V.B).  C (M x N) = A (M x K) B (K x N) with
// A = W_k^T (n_out x n_in), B = Y^T (n_in x batch, fp32), C = Y_{k+1}^T.  A is kept as W_k itself
// (n_in x n_out, row-major, fp64), i.e. k-major, so both operands are copied into LDS without a
// transpose.
//
// Arithmetic: the fp32 operands are widened to fp64 (exactly) and multiplied on the fp64 matrix cores
// (v_mfma_f64_16x16x4_f64), so every product is exact and partial sums carry fp64 rounding only, the
// same arithmetic as the sparse paths; the epilogue adds b_j in fp64, applies h and rounds once to fp32.
//
// Tiling for CDNA4: a 256-thread workgroup computes a 128 x 64 tile of C; each of its four wave64s owns a
// 64 x 32 quadrant as 4 x 2 blocks of 16 x 16 MFMAs (32 fp64 accumulators per lane).  Two workgroups share a
// CU (56 KiB of LDS and at most 256 registers per lane each), so one's barrier and LDS waits are covered by
// the other's MFMAs: measured on MI355X at n = 4096, batch 1024, 0.53 ms per layer (82% of the fp64 matrix
// peak) against 0.70 ms for 128 x 128 tiles at one workgroup per CU.  K advances 16
// at a time through double-buffered LDS (one barrier per step): the next slab is loaded into registers
// while the current one is multiplied and stored into the other buffer afterwards.  Rows of the LDS
// slabs are padded by 16 doubles so the four k-rows an MFMA operand reads land on different banks.
//
// Small batches give few tiles (n = 4096, batch 64: 32 workgroups for 256 CUs), so K is then split over
// blockIdx.z: each split writes its fp64 partial tile, and a second kernel adds the splits in a fixed
// order, then the bias, h and the rounding.
#include "common.h"

namespace sdnn {

namespace {

typedef double doublex4 __attribute__((ext_vector_type(4)));

constexpr int BM = 128, BN = 64, BK = 16;
constexpr int kPad = 16;

// kFast: every tile is interior and aligned (M % 128 == 0, N % 64 == 0, K % 16 == 0, 16-byte rows), so
// loads need no guards and no branch depends on the thread; otherwise every element is guarded.
template <bool kFast>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(2, 2))) void gemm_dense_layer_kernel(int64_t M, int64_t N, int64_t K,
                                                               int64_t ld, int64_t kc, const double *__restrict__ Wk,
                                                               const float *__restrict__ B,
                                                               const float *__restrict__ bias, double ymax,
                                                               float *__restrict__ C, double *__restrict__ partial) {
    __shared__ __align__(16) double As[2][BK][BM + kPad];
    __shared__ __align__(16) double Bs[2][BK][BN + kPad];
    constexpr int kNB = BN / 32;  // 16-column MFMA blocks per wave, and 32-column staging groups of B

    const int tid = threadIdx.x;
    const int lane = tid & 63, wave = tid >> 6;
    const int wm = wave >> 1, wn = wave & 1;
    // blockIdx.x walks M: consecutive workgroups (dealt round-robin to the XCDs) take different column
    // blocks of W, and the batch blocks of one of them land on one XCD and share it in its L2.
    const int64_t m0 = (int64_t)blockIdx.x * BM;
    const int64_t n0 = (int64_t)blockIdx.y * BN;
    const int64_t kb = (int64_t)blockIdx.z * kc;             // this split's K range [kb, ke)
    const int64_t ke = kb + kc < K ? kb + kc : K;

    // global -> register staging: thread -> k row tid / 16, column pairs (tid % 16) * 2 + 32 q (q = 0..3 for
    // A, q = 0..1 for B), so the 16 threads of a k row store one contiguous 256-byte run per q (no LDS bank
    // conflicts)
    const int s_k = tid >> 4, s_c = (tid & 15) * 2;
    double ra[8];
    float rb[2 * kNB];
    auto load_tiles = [&](int64_t k0) {
        const int64_t gk = k0 + s_k;
        if constexpr (kFast) {
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                const double2 v = *reinterpret_cast<const double2 *>(Wk + gk * M + m0 + s_c + 32 * q);
                ra[2 * q] = v.x;
                ra[2 * q + 1] = v.y;
            }
#pragma unroll
            for (int q = 0; q < kNB; ++q) {
                const float2 u = *reinterpret_cast<const float2 *>(B + gk * ld + n0 + s_c + 32 * q);
                rb[2 * q] = u.x;
                rb[2 * q + 1] = u.y;
            }
        } else {
#pragma unroll
            for (int q = 0; q < 4; ++q)
#pragma unroll
                for (int h = 0; h < 2; ++h) {
                    const int64_t gm = m0 + s_c + 32 * q + h;
                    ra[2 * q + h] = (gk < ke && gm < M) ? Wk[gk * M + gm] : 0.0;
                }
#pragma unroll
            for (int q = 0; q < kNB; ++q)
#pragma unroll
                for (int h = 0; h < 2; ++h) {
                    const int64_t gc = n0 + s_c + 32 * q + h;
                    rb[2 * q + h] = (gk < ke && gc < N) ? B[gk * ld + gc] : 0.0f;
                }
        }
    };
    auto store_tiles = [&](int buf) {
#pragma unroll
        for (int q = 0; q < 4; ++q)
            *reinterpret_cast<double2 *>(&As[buf][s_k][s_c + 32 * q]) = make_double2(ra[2 * q], ra[2 * q + 1]);
#pragma unroll
        for (int q = 0; q < kNB; ++q)
            *reinterpret_cast<double2 *>(&Bs[buf][s_k][s_c + 32 * q]) =
                make_double2((double)rb[2 * q], (double)rb[2 * q + 1]);
    };

    doublex4 acc[4][kNB];
#pragma unroll
    for (int mi = 0; mi < 4; ++mi)
#pragma unroll
        for (int ni = 0; ni < kNB; ++ni) acc[mi][ni] = doublex4{0.0, 0.0, 0.0, 0.0};

    const int rc = lane & 15, kq = lane >> 4;  // operand row/column within a 16-block, k within a step of 4
    auto compute = [&](int cur) {
#pragma unroll
        for (int kk = 0; kk < BK; kk += 4) {
            double a[4], b[kNB];
#pragma unroll
            for (int mi = 0; mi < 4; ++mi) a[mi] = As[cur][kk + kq][wm * 64 + mi * 16 + rc];
#pragma unroll
            for (int ni = 0; ni < kNB; ++ni) b[ni] = Bs[cur][kk + kq][wn * (BN / 2) + ni * 16 + rc];
#pragma unroll
            for (int mi = 0; mi < 4; ++mi)
#pragma unroll
                for (int ni = 0; ni < kNB; ++ni)
                    acc[mi][ni] = __builtin_amdgcn_mfma_f64_16x16x4f64(a[mi], b[ni], acc[mi][ni], 0, 0, 0);
        }
    };

    const int64_t ktiles = (ke - kb + BK - 1) / BK;  // >= 1: the launcher gives every split some of K
    load_tiles(kb);
    store_tiles(0);
    __syncthreads();
    // steady state: the next slab is loaded while this one is multiplied, then stored into the other
    // buffer (last read one step earlier, before the barrier); the final step is peeled off
    for (int64_t kt = 0; kt + 1 < ktiles; ++kt) {
        const int cur = (int)(kt & 1);
        load_tiles(kb + (kt + 1) * BK);
        compute(cur);
        store_tiles(cur ^ 1);
        __syncthreads();
    }
    compute((int)((ktiles - 1) & 1));

    // Output layout of the 16x16 f64 MFMA: lane l holds column l % 16 and, in element v, row l / 16 + 4 * v.
#pragma unroll
    for (int mi = 0; mi < 4; ++mi)
#pragma unroll
        for (int ni = 0; ni < kNB; ++ni)
#pragma unroll
            for (int v = 0; v < 4; ++v) {
                const int64_t m = m0 + wm * 64 + mi * 16 + kq + 4 * v;
                const int64_t col = n0 + wn * (BN / 2) + ni * 16 + rc;
                if (kFast || (m < M && col < N)) {
                    if (partial)
                        partial[((int64_t)blockIdx.z * M + m) * N + col] = acc[mi][ni][v];
                    else
                        C[m * ld + col] = activate(acc[mi][ni][v] + (double)bias[m], ymax);
                }
            }
}

// Sum of the K splits in split order, then the bias, h and one rounding.
__global__ void gemm_split_reduce_kernel(int64_t M, int64_t N, int64_t ld, int splits, const double *__restrict__ partial,
                                         const float *__restrict__ bias, double ymax, float *__restrict__ C) {
    const int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (e >= M * N) return;
    double z = 0.0;
    for (int sp = 0; sp < splits; ++sp) z += partial[(int64_t)sp * M * N + e];
    C[(e / N) * ld + e % N] = activate(z + (double)bias[e / N], ymax);
}

// Dense W_k (n_in x n_out, row-major, fp64) with explicit zeros: row i holds the fan-out of input i.
__global__ void dense_from_fanin_kernel(int64_t n, const int64_t *__restrict__ fan_ptr, const Edge *__restrict__ fan,
                                        double *__restrict__ wk) {
    const int64_t j = blockIdx.x;
    for (int64_t e = fan_ptr[j] + threadIdx.x; e < fan_ptr[j + 1]; e += blockDim.x) {
        const Edge ed = fan[e];
        wk[(int64_t)ed.idx * n + j] = (double)ed.w;
    }
}

// ---------------------------------------------------------------------------- fp32 matrix-core arm
// The same product with fp32 operands and fp32 accumulation on v_mfma_f32_16x16x4_f32, the arithmetic of a
// single-precision BLAS sgemm (the dense library of the paper's comparison, Sec. V.A).  Same 128 x 64 tiles,
// four waves of 64 x 32 (4 x 2 blocks of 16 x 16), double-buffered LDS with K steps of 16 and the
// split-K scheme for small batches (fp32 partials, summed in split order).  Output layout of the 16 x 16
// f32 MFMA: lane l holds column l % 16 and, in element v, row 4 * (l / 16) + v.
typedef float floatx4 __attribute__((ext_vector_type(4)));
constexpr int kPad32 = 4;

template <bool kFast>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(2, 2))) void gemm32_dense_layer_kernel(
    int64_t M, int64_t N, int64_t K, int64_t ld, int64_t kc, const float *__restrict__ Wk, const float *__restrict__ B,
    const float *__restrict__ bias, double ymax, float *__restrict__ C, float *__restrict__ partial) {
    __shared__ __align__(16) float As[2][BK][BM + kPad32];
    __shared__ __align__(16) float Bs[2][BK][BN + kPad32];
    constexpr int kNB = BN / 32;

    const int tid = threadIdx.x;
    const int lane = tid & 63, wave = tid >> 6;
    const int wm = wave >> 1, wn = wave & 1;
    const int64_t m0 = (int64_t)blockIdx.x * BM;
    const int64_t n0 = (int64_t)blockIdx.y * BN;
    const int64_t kb = (int64_t)blockIdx.z * kc;
    const int64_t ke = kb + kc < K ? kb + kc : K;

    // staging: thread -> k row tid / 16, A columns (tid % 16) * 8 .. + 7, B columns (tid % 16) * 4 .. + 3
    const int s_k = tid >> 4, s_a = (tid & 15) * 8, s_b = (tid & 15) * 4;
    float ra[8], rb[4];
    auto load_tiles = [&](int64_t k0) {
        const int64_t gk = k0 + s_k;
        if constexpr (kFast) {
            const float4 v0 = *reinterpret_cast<const float4 *>(Wk + gk * M + m0 + s_a);
            const float4 v1 = *reinterpret_cast<const float4 *>(Wk + gk * M + m0 + s_a + 4);
            ra[0] = v0.x; ra[1] = v0.y; ra[2] = v0.z; ra[3] = v0.w;
            ra[4] = v1.x; ra[5] = v1.y; ra[6] = v1.z; ra[7] = v1.w;
            const float4 u = *reinterpret_cast<const float4 *>(B + gk * ld + n0 + s_b);
            rb[0] = u.x; rb[1] = u.y; rb[2] = u.z; rb[3] = u.w;
        } else {
#pragma unroll
            for (int h = 0; h < 8; ++h) {
                const int64_t gm = m0 + s_a + h;
                ra[h] = (gk < ke && gm < M) ? Wk[gk * M + gm] : 0.0f;
            }
#pragma unroll
            for (int h = 0; h < 4; ++h) {
                const int64_t gc = n0 + s_b + h;
                rb[h] = (gk < ke && gc < N) ? B[gk * ld + gc] : 0.0f;
            }
        }
    };
    auto store_tiles = [&](int buf) {
        *reinterpret_cast<float4 *>(&As[buf][s_k][s_a]) = make_float4(ra[0], ra[1], ra[2], ra[3]);
        *reinterpret_cast<float4 *>(&As[buf][s_k][s_a + 4]) = make_float4(ra[4], ra[5], ra[6], ra[7]);
        *reinterpret_cast<float4 *>(&Bs[buf][s_k][s_b]) = make_float4(rb[0], rb[1], rb[2], rb[3]);
    };

    floatx4 acc[4][kNB];
#pragma unroll
    for (int mi = 0; mi < 4; ++mi)
#pragma unroll
        for (int ni = 0; ni < kNB; ++ni) acc[mi][ni] = floatx4{0.0f, 0.0f, 0.0f, 0.0f};

    const int rc = lane & 15, kq = lane >> 4;
    auto compute = [&](int cur) {
#pragma unroll
        for (int kk = 0; kk < BK; kk += 4) {
            float a[4], b[kNB];
#pragma unroll
            for (int mi = 0; mi < 4; ++mi) a[mi] = As[cur][kk + kq][wm * 64 + mi * 16 + rc];
#pragma unroll
            for (int ni = 0; ni < kNB; ++ni) b[ni] = Bs[cur][kk + kq][wn * (BN / 2) + ni * 16 + rc];
#pragma unroll
            for (int mi = 0; mi < 4; ++mi)
#pragma unroll
                for (int ni = 0; ni < kNB; ++ni)
                    acc[mi][ni] = __builtin_amdgcn_mfma_f32_16x16x4f32(a[mi], b[ni], acc[mi][ni], 0, 0, 0);
        }
    };

    const int64_t ktiles = (ke - kb + BK - 1) / BK;
    load_tiles(kb);
    store_tiles(0);
    __syncthreads();
    for (int64_t kt = 0; kt + 1 < ktiles; ++kt) {
        const int cur = (int)(kt & 1);
        load_tiles(kb + (kt + 1) * BK);
        compute(cur);
        store_tiles(cur ^ 1);
        __syncthreads();
    }
    compute((int)((ktiles - 1) & 1));

#pragma unroll
    for (int mi = 0; mi < 4; ++mi)
#pragma unroll
        for (int ni = 0; ni < kNB; ++ni)
#pragma unroll
            for (int v = 0; v < 4; ++v) {
                const int64_t m = m0 + wm * 64 + mi * 16 + 4 * kq + v;
                const int64_t col = n0 + wn * (BN / 2) + ni * 16 + rc;
                if (kFast || (m < M && col < N)) {
                    if (partial)
                        partial[((int64_t)blockIdx.z * M + m) * N + col] = acc[mi][ni][v];
                    else
                        C[m * ld + col] = activate((double)(acc[mi][ni][v] + bias[m]), ymax);
                }
            }
}

__global__ void gemm32_split_reduce_kernel(int64_t M, int64_t N, int64_t ld, int splits, const float *__restrict__ partial,
                                           const float *__restrict__ bias, double ymax, float *__restrict__ C) {
    const int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (e >= M * N) return;
    float z = 0.0f;
    for (int sp = 0; sp < splits; ++sp) z += partial[(int64_t)sp * M * N + e];
    C[(e / N) * ld + e % N] = activate((double)(z + bias[e / N]), ymax);
}

__global__ void dense32_from_fanin_kernel(int64_t n, const int64_t *__restrict__ fan_ptr, const Edge *__restrict__ fan,
                                          float *__restrict__ wk) {
    const int64_t j = blockIdx.x;
    for (int64_t e = fan_ptr[j] + threadIdx.x; e < fan_ptr[j + 1]; e += blockDim.x) {
        const Edge ed = fan[e];
        wk[(int64_t)ed.idx * n + j] = ed.w;
    }
}

}  // namespace

hipError_t launch_dense32_from_fanin(int64_t n, const int64_t *fan_ptr, const Edge *fan, float *wt, hipStream_t s) {
    hipError_t err = hipMemsetAsync(wt, 0, (size_t)n * (size_t)n * sizeof(float), s);
    if (err != hipSuccess) return err;
    dense32_from_fanin_kernel<<<(unsigned)n, 256, 0, s>>>(n, fan_ptr, fan, wt);
    return hipGetLastError();
}

hipError_t launch_gemm32_dense_layer(int64_t n, int64_t batch, int64_t ld, const float *wt, const float *bias,
                                     double ymax, const float *yt, float *zt, float *partial, int num_cu, hipStream_t s) {
    if (n == 0 || batch == 0) return hipSuccess;
    const int64_t gx = (n + BM - 1) / BM, gy = (batch + BN - 1) / BN;
    if (gx > 0x7fffffffLL || gy > 65535) return hipErrorInvalidValue;
    int sp = gemm_splits(n, batch, num_cu);
    const int64_t steps = (n + BK - 1) / BK;
    const int64_t kc = ((steps + sp - 1) / sp) * BK;
    sp = (int)((n + kc - 1) / kc);
    float *part = sp > 1 ? partial : nullptr;
    const bool fast = n % BM == 0 && batch % BN == 0 && n % BK == 0 && ld % 4 == 0;
    const dim3 grid((unsigned)gx, (unsigned)gy, (unsigned)sp);
    if (fast)
        gemm32_dense_layer_kernel<true><<<grid, 256, 0, s>>>(n, batch, n, ld, kc, wt, yt, bias, ymax, zt, part);
    else
        gemm32_dense_layer_kernel<false><<<grid, 256, 0, s>>>(n, batch, n, ld, kc, wt, yt, bias, ymax, zt, part);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess || sp == 1) return e;
    gemm32_split_reduce_kernel<<<(unsigned)((n * batch + 255) / 256), 256, 0, s>>>(n, batch, ld, sp, partial, bias,
                                                                                  ymax, zt);
    return hipGetLastError();
}

hipError_t launch_dense_from_fanin(int64_t n, const int64_t *fan_ptr, const Edge *fan, double *wt, hipStream_t s) {
    hipError_t err = hipMemsetAsync(wt, 0, (size_t)n * (size_t)n * sizeof(double), s);
    if (err != hipSuccess) return err;
    dense_from_fanin_kernel<<<(unsigned)n, 256, 0, s>>>(n, fan_ptr, fan, wt);
    return hipGetLastError();
}

// K splits for an n x n layer on `batch` samples: enough workgroups for two per CU, at least 8 K steps each.
int gemm_splits(int64_t n, int64_t batch, int num_cu) {
    const int64_t tiles = ((n + BM - 1) / BM) * ((batch + BN - 1) / BN);
    if (tiles == 0 || tiles >= 2 * (int64_t)num_cu) return 1;
    int64_t sp = (2 * (int64_t)num_cu + tiles - 1) / tiles;
    const int64_t most = n / (8 * BK);
    if (sp > most) sp = most;
    if (sp > 64) sp = 64;
    return sp < 1 ? 1 : (int)sp;
}

size_t gemm_partial_bytes(int64_t n, int64_t batch, int num_cu) {
    const int sp = gemm_splits(n, batch, num_cu);
    return sp > 1 ? (size_t)sp * (size_t)n * (size_t)batch * sizeof(double) : 0;
}

hipError_t launch_gemm_dense_layer(int64_t n, int64_t batch, int64_t ld, const double *wt, const float *bias, double ymax,
                                   const float *yt, float *zt, double *partial, int num_cu, hipStream_t s) {
    if (n == 0 || batch == 0) return hipSuccess;
    const int64_t gx = (n + BM - 1) / BM, gy = (batch + BN - 1) / BN;
    if (gx > 0x7fffffffLL || gy > 65535) return hipErrorInvalidValue;
    int sp = gemm_splits(n, batch, num_cu);
    // split length in whole K steps; the last split may be shorter, none is empty
    const int64_t steps = (n + BK - 1) / BK;
    const int64_t kc = ((steps + sp - 1) / sp) * BK;
    sp = (int)((n + kc - 1) / kc);
    double *part = sp > 1 ? partial : nullptr;
    const bool fast = n % BM == 0 && batch % BN == 0 && n % BK == 0 && ld % 4 == 0;
    const dim3 grid((unsigned)gx, (unsigned)gy, (unsigned)sp);
    if (fast)
        gemm_dense_layer_kernel<true><<<grid, 256, 0, s>>>(n, batch, n, ld, kc, wt, yt, bias, ymax, zt, part);
    else
        gemm_dense_layer_kernel<false><<<grid, 256, 0, s>>>(n, batch, n, ld, kc, wt, yt, bias, ymax, zt, part);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess || sp == 1) return e;
    gemm_split_reduce_kernel<<<(unsigned)((n * batch + 255) / 256), 256, 0, s>>>(n, batch, ld, sp, partial, bias, ymax,
                                                                                zt);
    return hipGetLastError();
}

}  // namespace sdnn
