// Dense-W comparison arm: Z^T = W^T Y^T on matrix cores with the bias and activation fused.
//
// This is the layer product with every zero of W_k stored explicitly, the dense-linear-algebra version
// the paper measures its sparse library against (Sec. V.A, V.B).  C (M x N) = A (M x K) B (K x N) with
// A = W_k^T (n_out x n_in, row-major, held in fp64), B = Y^T (n_in x batch, fp32), C = Y_{k+1}^T.
//
// Arithmetic: the fp32 operands are widened to fp64 (exactly) and multiplied on the fp64 matrix cores
// (v_mfma_f64_16x16x4_f64), so every product is exact and partial sums carry fp64 rounding only, the
// same arithmetic as the sparse paths; the epilogue adds b_j in fp64, applies h and rounds once to fp32.
//
// Tiling for CDNA4: a 256-thread workgroup computes a 128 x 128 tile of C; each of its four wave64s owns
// a 64 x 64 quadrant as 4 x 4 blocks of 16 x 16 MFMAs (64 fp64 accumulators per lane).  K advances 16 at
// a time through LDS, both operands stored k-major so the 16 rows or columns an MFMA operand needs are
// contiguous; the next K slab is prefetched into registers while the current one is multiplied.
#include "common.h"

namespace sdnn {

namespace {

typedef double doublex4 __attribute__((ext_vector_type(4)));

constexpr int BM = 128, BN = 128, BK = 16;
constexpr int kPad = 2;

__global__ __launch_bounds__(256) void gemm_dense_layer_kernel(int64_t M, int64_t N, int64_t K,
                                                               const double *__restrict__ A,
                                                               const float *__restrict__ B,
                                                               const float *__restrict__ bias, double ymax,
                                                               float *__restrict__ C) {
    __shared__ double As[BK][BM + kPad];
    __shared__ double Bs[BK][BN + kPad];

    const int tid = threadIdx.x;
    const int lane = tid & 63, wave = tid >> 6;
    const int wm = wave >> 1, wn = wave & 1;
    // blockIdx.x walks M: consecutive workgroups (dealt round-robin to the XCDs) take different row
    // blocks of A, and the column blocks of one row block land on one XCD and share A in its L2.
    const int64_t m0 = (int64_t)blockIdx.x * BM;
    const int64_t n0 = (int64_t)blockIdx.y * BN;

    // global -> register staging.  A: 128 rows x 16 k, thread -> row tid/2, k (tid%2)*8 .. +8.
    const int a_row = tid >> 1, a_k = (tid & 1) * 8;
    // B: 16 k x 128 columns, thread -> k tid/16, columns (tid%16)*8 .. +8.
    const int b_k = tid >> 4, b_c = (tid & 15) * 8;

    double ra[8];
    float rb[8];
    auto load_tiles = [&](int64_t k0) {
        const int64_t gr = m0 + a_row;
#pragma unroll
        for (int q = 0; q < 8; ++q) {
            const int64_t gk = k0 + a_k + q;
            ra[q] = (gr < M && gk < K) ? A[gr * K + gk] : 0.0;
        }
        const int64_t gk = k0 + b_k;
#pragma unroll
        for (int q = 0; q < 8; ++q) {
            const int64_t gc = n0 + b_c + q;
            rb[q] = (gk < K && gc < N) ? B[gk * N + gc] : 0.0f;
        }
    };
    auto store_tiles = [&]() {
#pragma unroll
        for (int q = 0; q < 8; ++q) As[a_k + q][a_row] = ra[q];
#pragma unroll
        for (int q = 0; q < 8; ++q) Bs[b_k][b_c + q] = (double)rb[q];
    };

    doublex4 acc[4][4];
#pragma unroll
    for (int mi = 0; mi < 4; ++mi)
#pragma unroll
        for (int ni = 0; ni < 4; ++ni) acc[mi][ni] = doublex4{0.0, 0.0, 0.0, 0.0};

    const int rc = lane & 15, kq = lane >> 4;  // operand row/column within a 16-block, k within a step of 4
    const int64_t ktiles = (K + BK - 1) / BK;
    load_tiles(0);
    store_tiles();
    __syncthreads();
    for (int64_t kt = 0; kt < ktiles; ++kt) {
        if (kt + 1 < ktiles) load_tiles((kt + 1) * BK);
#pragma unroll
        for (int kk = 0; kk < BK; kk += 4) {
            double a[4], b[4];
#pragma unroll
            for (int mi = 0; mi < 4; ++mi) a[mi] = As[kk + kq][wm * 64 + mi * 16 + rc];
#pragma unroll
            for (int ni = 0; ni < 4; ++ni) b[ni] = Bs[kk + kq][wn * 64 + ni * 16 + rc];
#pragma unroll
            for (int mi = 0; mi < 4; ++mi)
#pragma unroll
                for (int ni = 0; ni < 4; ++ni)
                    acc[mi][ni] = __builtin_amdgcn_mfma_f64_16x16x4f64(a[mi], b[ni], acc[mi][ni], 0, 0, 0);
        }
        __syncthreads();
        if (kt + 1 < ktiles) {
            store_tiles();
            __syncthreads();
        }
    }

    // Output layout of the 16x16 f64 MFMA: lane l holds column l % 16 and, in element v, row l / 16 + 4 * v.
#pragma unroll
    for (int mi = 0; mi < 4; ++mi)
#pragma unroll
        for (int ni = 0; ni < 4; ++ni)
#pragma unroll
            for (int v = 0; v < 4; ++v) {
                const int64_t m = m0 + wm * 64 + mi * 16 + kq + 4 * v;
                const int64_t col = n0 + wn * 64 + ni * 16 + rc;
                if (m < M && col < N) C[m * N + col] = activate(acc[mi][ni][v] + (double)bias[m], ymax);
            }
}

// Dense W_k^T (n_out x n_in, row-major, fp64): row j holds the fan-in of output j, zeros elsewhere.
__global__ void dense_from_fanin_kernel(int64_t n, const int64_t *__restrict__ fan_ptr, const Edge *__restrict__ fan,
                                        double *__restrict__ wt) {
    const int64_t j = blockIdx.x;
    for (int64_t e = fan_ptr[j] + threadIdx.x; e < fan_ptr[j + 1]; e += blockDim.x) {
        const Edge ed = fan[e];
        wt[j * n + ed.idx] = (double)ed.w;
    }
}

}  // namespace

hipError_t launch_dense_from_fanin(int64_t n, const int64_t *fan_ptr, const Edge *fan, double *wt, hipStream_t s) {
    hipError_t err = hipMemsetAsync(wt, 0, (size_t)n * (size_t)n * sizeof(double), s);
    if (err != hipSuccess) return err;
    dense_from_fanin_kernel<<<(unsigned)n, 256, 0, s>>>(n, fan_ptr, fan, wt);
    return hipGetLastError();
}

hipError_t launch_gemm_dense_layer(int64_t n, int64_t batch, const double *wt, const float *bias, double ymax,
                                   const float *yt, float *zt, hipStream_t s) {
    if (n == 0 || batch == 0) return hipSuccess;
    const int64_t gx = (n + BM - 1) / BM, gy = (batch + BN - 1) / BN;
    if (gx > 0x7fffffffLL || gy > 65535) return hipErrorInvalidValue;
    gemm_dense_layer_kernel<<<dim3((unsigned)gx, (unsigned)gy), 256, 0, s>>>(n, batch, n, wt, yt, bias, ymax, zt);
    return hipGetLastError();
}

}  // namespace sdnn
