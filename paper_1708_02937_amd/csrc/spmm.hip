// Dense-Y layer product on CSR weights, with the bias and activation fused (Sec. III, Sec. IV loop body).
//
// Activations are kept neuron-major (Y^T, n x batch: the paper's own m x n layout of Y, Sec. IV), so
// the batch entries of one neuron are contiguous.  One 64-lane wavefront owns one output neuron j and a
// chunk of 64*V batch columns: it walks the fan-in list of j (input i, weight W(i, j)), loads the list 64
// entries at a time with one coalesced 8-byte load per lane, broadcasts each entry to the whole wave
// (readlane, so the row address is scalar), and every lane does V fused multiply-adds into fp64
// accumulators from a coalesced load of row i of Y^T.  The epilogue adds b_j, applies h and rounds once
// to fp32 (the element-wise max.+ steps of Fig. 4, fused so Y_k W_k never reaches memory).
//
// XCD-aware launch: workgroups are dealt round-robin to the 8 XCDs, so the batch chunk is taken from
// blockIdx % chunks; with 8 chunks every XCD touches only its own n x 64V slice of Y^T, which stays in
// that XCD's L2 while all output neurons gather from it.
#include "common.h"

namespace sdnn {

namespace {

template <int V>
struct VecF;
template <>
struct VecF<1> {
    using T = float;
};
template <>
struct VecF<2> {
    using T = float2;
};
template <>
struct VecF<4> {
    using T = float4;
};

template <int V>
__device__ __forceinline__ void load_v(const float *p, float (&y)[V]) {
    if constexpr (V == 1) {
        y[0] = *p;
    } else if constexpr (V == 2) {
        const float2 t = *reinterpret_cast<const float2 *>(p);
        y[0] = t.x;
        y[1] = t.y;
    } else {
        const float4 t = *reinterpret_cast<const float4 *>(p);
        y[0] = t.x;
        y[1] = t.y;
        y[2] = t.z;
        y[3] = t.w;
    }
}

template <int V>
__device__ __forceinline__ void store_v(float *p, const float (&y)[V]) {
    if constexpr (V == 1) {
        *p = y[0];
    } else if constexpr (V == 2) {
        *reinterpret_cast<float2 *>(p) = make_float2(y[0], y[1]);
    } else {
        *reinterpret_cast<float4 *>(p) = make_float4(y[0], y[1], y[2], y[3]);
    }
}

__device__ __forceinline__ int32_t bcast_i(int32_t v, int lane) { return __builtin_amdgcn_readlane(v, lane); }
__device__ __forceinline__ float bcast_f(float v, int lane) {
    return __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), lane));
}

constexpr int kUnroll = 8;

template <int V>
__global__ __launch_bounds__(256) void spmm_fanin_kernel(int64_t n, int64_t batch, int chunks,
                                                         const int64_t *__restrict__ fan_ptr,
                                                         const Edge *__restrict__ fan, const float *__restrict__ bias,
                                                         double ymax, const float *__restrict__ yt,
                                                         float *__restrict__ zt) {
    const int lane = threadIdx.x & 63;
    const int wave = threadIdx.x >> 6;
    const int64_t c = blockIdx.x % chunks;
    const int64_t j = (int64_t)(blockIdx.x / chunks) * 4 + wave;
    if (j >= n) return;
    const int64_t col = c * (64 * V) + (int64_t)lane * V;
    const bool active = col < batch;       // batch is a multiple of V, so col < batch => col + V <= batch
    const int64_t colc = active ? col : 0; // inactive lanes read a valid address and discard it

    double acc[V];
#pragma unroll
    for (int v = 0; v < V; ++v) acc[v] = 0.0;

    const int64_t e_beg = fan_ptr[j], e_end = fan_ptr[j + 1];
    for (int64_t e0 = e_beg; e0 < e_end; e0 += 64) {
        const int cnt = (int)((e_end - e0) < 64 ? (e_end - e0) : 64);
        Edge mine;
        mine.idx = 0;
        mine.w = 0.0f;
        if (lane < cnt) mine = fan[e0 + lane];
        int t = 0;
        for (; t + kUnroll <= cnt; t += kUnroll) {
            float y[kUnroll][V];
            float w[kUnroll];
#pragma unroll
            for (int u = 0; u < kUnroll; ++u) {
                const int32_t i = bcast_i(mine.idx, t + u);
                w[u] = bcast_f(mine.w, t + u);
                load_v<V>(yt + (int64_t)i * batch + colc, y[u]);
            }
#pragma unroll
            for (int u = 0; u < kUnroll; ++u) {
                const double wd = (double)w[u];
#pragma unroll
                for (int v = 0; v < V; ++v) acc[v] = __builtin_fma((double)y[u][v], wd, acc[v]);
            }
        }
        for (; t < cnt; ++t) {
            float y[V];
            const int32_t i = bcast_i(mine.idx, t);
            const double wd = (double)bcast_f(mine.w, t);
            load_v<V>(yt + (int64_t)i * batch + colc, y);
#pragma unroll
            for (int v = 0; v < V; ++v) acc[v] = __builtin_fma((double)y[v], wd, acc[v]);
        }
    }
    if (!active) return;
    const double bj = (double)bias[j];
    float out[V];
#pragma unroll
    for (int v = 0; v < V; ++v) out[v] = activate(acc[v] + bj, ymax);
    store_v<V>(zt + j * batch + col, out);
}

// 64 x 64 tile transpose through LDS (padded against bank conflicts): out (cols x rows) = in^T.
__global__ __launch_bounds__(256) void transpose_kernel(const float *__restrict__ in, float *__restrict__ out,
                                                        int64_t rows, int64_t cols) {
    __shared__ float tile[64][65];
    const int64_t r0 = (int64_t)blockIdx.y * 64, c0 = (int64_t)blockIdx.x * 64;
    const int tx = threadIdx.x & 63, ty = threadIdx.x >> 6;
    for (int rr = ty; rr < 64; rr += 4) {
        const int64_t r = r0 + rr, c = c0 + tx;
        if (r < rows && c < cols) tile[rr][tx] = in[r * cols + c];
    }
    __syncthreads();
    for (int cc = ty; cc < 64; cc += 4) {
        const int64_t c = c0 + cc, r = r0 + tx;
        if (r < rows && c < cols) out[c * rows + r] = tile[tx][cc];
    }
}

}  // namespace

hipError_t launch_transpose(const float *in, float *out, int64_t rows, int64_t cols, hipStream_t s) {
    if (rows == 0 || cols == 0) return hipSuccess;
    const int64_t gx = (cols + 63) / 64, gy = (rows + 63) / 64;
    if (gy > 65535) return hipErrorInvalidValue;
    transpose_kernel<<<dim3((unsigned)gx, (unsigned)gy), 256, 0, s>>>(in, out, rows, cols);
    return hipGetLastError();
}

hipError_t launch_spmm_fanin(int64_t n, int64_t batch, const int64_t *fan_ptr, const Edge *fan, const float *bias,
                             double ymax, const float *yt, float *zt, hipStream_t s) {
    if (n == 0 || batch == 0) return hipSuccess;
    // Columns per lane: wide enough to keep 8 independent loads in flight, and a multiple that divides batch.
    int V = 1;
    if (batch % 4 == 0 && batch >= 2048) V = 4;
    else if (batch % 2 == 0 && batch >= 128) V = 2;
    const int64_t chunks = (batch + 64 * V - 1) / (64 * V);
    const int64_t groups = (n + 3) / 4;
    const int64_t blocks = groups * chunks;
    if (blocks > 0x7fffffffLL) return hipErrorInvalidValue;
    switch (V) {
        case 4:
            spmm_fanin_kernel<4><<<(unsigned)blocks, 256, 0, s>>>(n, batch, (int)chunks, fan_ptr, fan, bias, ymax, yt, zt);
            break;
        case 2:
            spmm_fanin_kernel<2><<<(unsigned)blocks, 256, 0, s>>>(n, batch, (int)chunks, fan_ptr, fan, bias, ymax, yt, zt);
            break;
        default:
            spmm_fanin_kernel<1><<<(unsigned)blocks, 256, 0, s>>>(n, batch, (int)chunks, fan_ptr, fan, bias, ymax, yt, zt);
    }
    return hipGetLastError();
}

}  // namespace sdnn
