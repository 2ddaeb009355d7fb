// Matrix multiply over the semirings of Sec. II on the dense-Y gather skeleton.
//
// Z = Y (+).(x) W_k with Z(r, j) = (+) over the stored entries W_k(i, j) of Y(r, i) (x) W_k(i, j), starting
// from the semiring's 0-element (Sec. II.D matrix multiply; Sec. II.E 0-element).  Activations are
// neuron-major (Y^T, n x batch) as in the forward pass; one wave64 owns an output neuron and 64 * V batch
// columns and walks the neuron's fan-in list (sorted by input index, so every output is reduced in
// ascending input order), broadcasting each entry with readlane.  Values are carried in fp64 and rounded
// once to fp32: +.x multiplies exactly and sums in fp64 as the forward pass does; max.+ adds in fp64 and
// max.min, min.max and xor.and only select or compare, so those four are exact.
#include "common.h"

namespace sdnn {

namespace {

struct PlusTimes {
    static __device__ double zero() { return 0.0; }
    static __device__ double add(double a, double b) { return a + b; }
    static __device__ double mul(double y, double w) { return y * w; }  // exact for fp32 operands
};
struct MaxPlus {
    static __device__ double zero() { return -__builtin_huge_val(); }
    static __device__ double add(double a, double b) { return a > b ? a : b; }
    static __device__ double mul(double y, double w) { return y + w; }
};
struct MaxMin {
    static __device__ double zero() { return -__builtin_huge_val(); }
    static __device__ double add(double a, double b) { return a > b ? a : b; }
    static __device__ double mul(double y, double w) { return y < w ? y : w; }
};
struct MinMax {
    static __device__ double zero() { return __builtin_huge_val(); }
    static __device__ double add(double a, double b) { return a < b ? a : b; }
    static __device__ double mul(double y, double w) { return y > w ? y : w; }
};
struct XorAnd {  // GF(2): a value counts as 1 when it is nonzero
    static __device__ double zero() { return 0.0; }
    static __device__ double add(double a, double b) { return (double)((a != 0.0) != (b != 0.0)); }
    static __device__ double mul(double y, double w) { return (double)(y != 0.0 && w != 0.0); }
};

constexpr int kSrUnroll = 8;

template <int V, class SR>
__global__ __launch_bounds__(256) void semiring_gather_kernel(int64_t n, int64_t batch, int64_t ld, int chunks,
                                                              int64_t block_base,
                                                              const int64_t *__restrict__ fan_ptr,
                                                              const Edge *__restrict__ fan,
                                                              const float *__restrict__ yt, float *__restrict__ zt) {
    const int lane = threadIdx.x & 63;
    const int wave = threadIdx.x >> 6;
    const int64_t b = block_base + blockIdx.x;  // large grids are launched in segments
    const int64_t c = b % chunks;
    const int64_t j = (b / chunks) * 4 + wave;
    if (j >= n) return;
    const int64_t col = c * (64 * V) + (int64_t)lane * V;
    const bool active = col < batch;        // batch is a multiple of V
    const int64_t colc = active ? col : 0;  // inactive lanes read a valid address and discard it
    double acc[V];
#pragma unroll
    for (int v = 0; v < V; ++v) acc[v] = SR::zero();
    const int64_t e_beg = fan_ptr[j], e_end = fan_ptr[j + 1];
    for (int64_t e0 = e_beg; e0 < e_end; e0 += 64) {
        const int cnt = (int)((e_end - e0) < 64 ? (e_end - e0) : 64);
        Edge mine;
        mine.idx = 0;
        mine.w = 0.0f;
        if (lane < cnt) mine = fan[e0 + lane];
        for (int t = 0; t < cnt; t += kSrUnroll) {
            float y[kSrUnroll][V];
            float w[kSrUnroll];
#pragma unroll
            for (int u = 0; u < kSrUnroll; ++u) {
                const int src = t + u < cnt ? t + u : t;  // past the list end: repeat a valid entry, unused
                const int32_t i = __builtin_amdgcn_readlane(mine.idx, src);
                w[u] = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(mine.w), src));
                const float *p = yt + (int64_t)i * ld + colc;
#pragma unroll
                for (int v = 0; v < V; ++v) y[u][v] = p[v];
            }
#pragma unroll
            for (int u = 0; u < kSrUnroll; ++u) {
                if (t + u < cnt) {
#pragma unroll
                    for (int v = 0; v < V; ++v) acc[v] = SR::add(acc[v], SR::mul((double)y[u][v], (double)w[u]));
                }
            }
        }
    }
    if (!active) return;
#pragma unroll
    for (int v = 0; v < V; ++v) zt[j * ld + col + v] = (float)acc[v];
}

// Y^T (n x batch, row pitch ld) filled with `fill`, then the stored entries of CSR rows scattered into it.
__global__ void semiring_fill_kernel(int64_t count, float fill, float *__restrict__ yt) {
    const int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (e < count) yt[e] = fill;
}

__global__ __launch_bounds__(256) void semiring_scatter_kernel(int64_t n, int64_t batch, int64_t ld,
                                                               const int64_t *__restrict__ row_ptr,
                                                               const int32_t *__restrict__ col,
                                                               const float *__restrict__ val, float *__restrict__ yt,
                                                               uint32_t *err) {
    const int64_t r = blockIdx.x;
    const int64_t nnz = (col && val) ? row_ptr[batch] : 0;
    const int64_t b = row_ptr[r], len = row_ptr[r + 1] - b;
    if (b < 0 || len < 0 || len > n || b + len > nnz) {
        if (threadIdx.x == 0) atomicOr(err, 1u);
        return;
    }
    for (int64_t t = threadIdx.x; t < len; t += blockDim.x) {
        const int32_t i = col[b + t];
        if (i < 0 || i >= n) {
            atomicOr(err, 1u);
            continue;
        }
        yt[(int64_t)i * ld + r] = val[b + t];
    }
}

template <class SR>
hipError_t launch_sr(int64_t n, int64_t batch, int64_t ld, const int64_t *fan_ptr, const Edge *fan, const float *yt, float *zt,
                     hipStream_t s) {
    int V = 1;
    if (batch % 4 == 0 && batch >= 256) V = 4;
    else if (batch % 2 == 0 && batch >= 128) V = 2;
    const int64_t chunks = (batch + 64 * V - 1) / (64 * V);
    const int64_t blocks = ((n + 3) / 4) * chunks;
    constexpr int64_t kSeg = 1ll << 23;  // at most 2^32 - 1 work-items per launch
    for (int64_t base = 0; base < blocks; base += kSeg) {
        const unsigned nb = (unsigned)(blocks - base < kSeg ? blocks - base : kSeg);
        if (V == 4)
            semiring_gather_kernel<4, SR><<<nb, 256, 0, s>>>(n, batch, ld, (int)chunks, base, fan_ptr, fan, yt, zt);
        else if (V == 2)
            semiring_gather_kernel<2, SR><<<nb, 256, 0, s>>>(n, batch, ld, (int)chunks, base, fan_ptr, fan, yt, zt);
        else
            semiring_gather_kernel<1, SR><<<nb, 256, 0, s>>>(n, batch, ld, (int)chunks, base, fan_ptr, fan, yt, zt);
        hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    return hipGetLastError();
}

}  // namespace

float semiring_zero(int semiring) {
    switch (semiring) {
        case kSemiringMaxPlus:
        case kSemiringMaxMin: return -__builtin_huge_valf();
        case kSemiringMinMax: return __builtin_huge_valf();
        default: return 0.0f;
    }
}

hipError_t launch_semiring_mxm(int semiring, int64_t n, int64_t batch, int64_t ld, const int64_t *fan_ptr, const Edge *fan,
                               const float *yt, float *zt, hipStream_t s) {
    if (n == 0 || batch == 0) return hipSuccess;
    switch (semiring) {
        case kSemiringPlusTimes: return launch_sr<PlusTimes>(n, batch, ld, fan_ptr, fan, yt, zt, s);
        case kSemiringMaxPlus: return launch_sr<MaxPlus>(n, batch, ld, fan_ptr, fan, yt, zt, s);
        case kSemiringMaxMin: return launch_sr<MaxMin>(n, batch, ld, fan_ptr, fan, yt, zt, s);
        case kSemiringMinMax: return launch_sr<MinMax>(n, batch, ld, fan_ptr, fan, yt, zt, s);
        case kSemiringXorAnd: return launch_sr<XorAnd>(n, batch, ld, fan_ptr, fan, yt, zt, s);
        default: return hipErrorInvalidValue;
    }
}

hipError_t launch_semiring_densify(int64_t n, int64_t batch, int64_t ld, float fill, const int64_t *row_ptr, const int32_t *col,
                                   const float *val, float *yt, uint32_t *err, hipStream_t s) {
    if (n == 0 || batch == 0) return hipSuccess;
    const int64_t count = n * ld;
    semiring_fill_kernel<<<(unsigned)((count + 255) / 256), 256, 0, s>>>(count, fill, yt);
    semiring_scatter_kernel<<<(unsigned)batch, 256, 0, s>>>(n, batch, ld, row_ptr, col, val, yt, err);
    return hipGetLastError();
}

}  // namespace sdnn
