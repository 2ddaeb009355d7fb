// Matrix multiply over the semirings of Sec. II on the dense-Y gather skeleton.
//
// Z = Y (+).(x) W_k with Z(r, j) = (+) over the stored entries W_k(i, j) of Y(r, i) (x) W_k(i, j), starting
// from the semiring's 0-element (Sec. II.D matrix multiply; Sec. II.E 0-element).  Activations are
// neuron-major (Y^T, n x batch) as in the forward pass; one wave64 owns an output neuron and 64 * V batch
// columns and walks the neuron's fan-in list (sorted by input index, so every output is reduced in
// ascending input order), broadcasting each entry with readlane.  Values are carried in fp64 and rounded
// once to fp32: +.x multiplies exactly and sums in fp64 as the forward pass does; max.+ adds in fp64 and
// max.min, min.max and xor.and only select or compare, so those four are exact.
#include <type_traits>

#include "common.h"

namespace sdnn {

namespace {

// Each semiring also says how a product is folded into an LDS accumulator slot (an atomic (+) on fp64,
// or for GF(2) an exclusive or on the slot's low word) for the row-wise product on CSR input.
struct PlusTimes {
    static __device__ double zero() { return 0.0; }
    static __device__ double add(double a, double b) { return a + b; }
    static __device__ double mul(double y, double w) { return y * w; }  // exact for fp32 operands
    static __device__ void fold(double *slot, double p) { atomicAdd(slot, p); }
};
struct MaxPlus {
    static __device__ double zero() { return -__builtin_huge_val(); }
    static __device__ double add(double a, double b) { return a > b ? a : b; }
    static __device__ double mul(double y, double w) { return y + w; }
    static __device__ void fold(double *slot, double p) {
        __hip_atomic_fetch_max(slot, p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
    }
};
struct MaxMin {
    static __device__ double zero() { return -__builtin_huge_val(); }
    static __device__ double add(double a, double b) { return a > b ? a : b; }
    static __device__ double mul(double y, double w) { return y < w ? y : w; }
    static __device__ void fold(double *slot, double p) {
        __hip_atomic_fetch_max(slot, p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
    }
};
struct MinMax {
    static __device__ double zero() { return __builtin_huge_val(); }
    static __device__ double add(double a, double b) { return a < b ? a : b; }
    static __device__ double mul(double y, double w) { return y > w ? y : w; }
    static __device__ void fold(double *slot, double p) {
        __hip_atomic_fetch_min(slot, p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
    }
};
struct XorAnd {  // GF(2): a value counts as 1 when it is nonzero
    static __device__ double zero() { return 0.0; }
    static __device__ double add(double a, double b) { return (double)((a != 0.0) != (b != 0.0)); }
    static __device__ double mul(double y, double w) { return (double)(y != 0.0 && w != 0.0); }
    // the slot holds a parity counter in its low 32 bits (the accumulator is read back through value())
    static __device__ void fold(double *slot, double p) {
        if (p != 0.0) atomicXor(reinterpret_cast<unsigned *>(slot), 1u);
    }
};

// The accumulator slot's value for the result: GF(2) reads its parity word, the others the fp64 value.
template <class SR>
__device__ __forceinline__ double slot_value(const double *slot) {
    if constexpr (std::is_same<SR, XorAnd>::value) return (double)(*reinterpret_cast<const unsigned *>(slot) & 1u);
    else return *slot;
}
template <class SR>
__device__ __forceinline__ void slot_init(double *slot) {
    if constexpr (std::is_same<SR, XorAnd>::value) *slot = 0.0;  // parity word 0
    else *slot = SR::zero();
}

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

// Row-wise product on CSR input (the SpGEMM skeleton of the forward pass, Sec. II.D computed row by row):
// one workgroup per sample keeps a window of kSrWin output columns in LDS, initialised to the 0-element;
// each wave takes one stored entry (i, y) of the sample at a time and its lanes walk the window's part of
// W_k's fan-out row i (rows are sorted by column, so the part is found by binary search), folding y (x) w
// into the column's slot with an LDS atomic ((+) is an fp64 add, max, min or, for GF(2), an exclusive or).
// Unstored entries are the 0-element, which changes nothing, so only stored ones are visited; the window
// is written to Z's row (batch-major) as fp32.  +.x sums exact products in fp64 in the order the atomics
// land and rounds once; the other semirings only select, compare or count, so they are exact.  Row extents
// and columns are checked as in the forward pass (flagged, offending rows or entries skipped).
constexpr int kSrWin = 16384;
constexpr int kSrThreads = 512;

template <class SR>
__global__ __launch_bounds__(kSrThreads) void semiring_rows_kernel(int64_t n, int64_t batch,
                                                                   const int64_t *__restrict__ row_ptr,
                                                                   const int32_t *__restrict__ col,
                                                                   const float *__restrict__ val,
                                                                   const int64_t *__restrict__ w_ptr,
                                                                   const Edge *__restrict__ w, float *__restrict__ z,
                                                                   uint32_t *err) {
    __shared__ double acc[kSrWin];
    const int64_t r = blockIdx.x;
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    constexpr int kW = kSrThreads / 64;
    const int64_t nnz = (col && val) ? row_ptr[batch] : 0;
    int64_t b = row_ptr[r], len = row_ptr[r + 1] - b;
    if (b < 0 || len < 0 || len > n || b + len > nnz) {
        if (threadIdx.x == 0) atomicOr(err, 1u);
        len = 0;
    }
    for (int64_t w0 = 0; w0 < n; w0 += kSrWin) {
        const int64_t wn = n - w0 < kSrWin ? n - w0 : kSrWin;
        for (int64_t c = threadIdx.x; c < wn; c += kSrThreads) slot_init<SR>(&acc[c]);
        __syncthreads();
        for (int64_t t = wave; t < len; t += kW) {
            const int32_t i = col[b + t];
            if (i < 0 || i >= n) {
                if (lane == 0 && w0 == 0) atomicOr(err, 1u);
                continue;
            }
            const double y = (double)val[b + t];
            int64_t lo = w_ptr[i], hi = w_ptr[(int64_t)i + 1];
            if (w0 > 0 || wn < n) {  // the window's part of the sorted row: [first col >= w0, first col >= w0 + wn)
                int64_t a = lo, e = hi;
                while (a < e) {
                    const int64_t m = (a + e) >> 1;
                    if (w[m].idx < w0) a = m + 1;
                    else e = m;
                }
                int64_t a2 = a, e2 = hi;
                while (a2 < e2) {
                    const int64_t m = (a2 + e2) >> 1;
                    if (w[m].idx < w0 + wn) a2 = m + 1;
                    else e2 = m;
                }
                lo = a;
                hi = a2;
            }
            for (int64_t q = lo + lane; q < hi; q += 64) {
                const Edge ed = w[q];
                SR::fold(&acc[ed.idx - w0], SR::mul(y, (double)ed.w));
            }
        }
        __syncthreads();
        float *zr = z + r * n + w0;
        for (int64_t c = threadIdx.x; c < wn; c += kSrThreads) zr[c] = (float)slot_value<SR>(&acc[c]);
        __syncthreads();
    }
}

template <class SR>
hipError_t launch_sr_rows(int64_t n, int64_t batch, const int64_t *row_ptr, const int32_t *col, const float *val,
                          const int64_t *w_ptr, const Edge *w, float *z, uint32_t *err, hipStream_t s) {
    if (batch > 0x7fffffffLL) return hipErrorInvalidValue;
    semiring_rows_kernel<SR><<<(unsigned)batch, kSrThreads, 0, s>>>(n, batch, row_ptr, col, val, w_ptr, w, z, err);
    return hipGetLastError();
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

hipError_t launch_semiring_rows(int semiring, int64_t n, int64_t batch, const int64_t *row_ptr, const int32_t *col,
                                const float *val, const int64_t *w_ptr, const Edge *w, float *z, uint32_t *err,
                                hipStream_t s) {
    if (n == 0 || batch == 0) return hipSuccess;
    switch (semiring) {
        case kSemiringPlusTimes: return launch_sr_rows<PlusTimes>(n, batch, row_ptr, col, val, w_ptr, w, z, err, s);
        case kSemiringMaxPlus: return launch_sr_rows<MaxPlus>(n, batch, row_ptr, col, val, w_ptr, w, z, err, s);
        case kSemiringMaxMin: return launch_sr_rows<MaxMin>(n, batch, row_ptr, col, val, w_ptr, w, z, err, s);
        case kSemiringMinMax: return launch_sr_rows<MinMax>(n, batch, row_ptr, col, val, w_ptr, w, z, err, s);
        case kSemiringXorAnd: return launch_sr_rows<XorAnd>(n, batch, row_ptr, col, val, w_ptr, w, z, err, s);
        default: return hipErrorInvalidValue;
    }
}

}  // namespace sdnn
