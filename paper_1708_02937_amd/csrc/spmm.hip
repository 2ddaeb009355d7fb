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
// XCD-aware launch: workgroups are dealt round-robin to the 8 XCDs, so the batch chunk follows from
// blockIdx % 8.  Each XCD owns every eighth chunk and works through its chunks one at a time, so the
// rows of Y^T that its current output neurons gather stay in that XCD's L2.
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
    int64_t c, g;
    if (chunks % 8 == 0) {
        // chunk-major per XCD: XCD x works through chunks x, x+8, ... one at a time, every neuron group
        // of a chunk before the next, so the input rows its current neurons gather stay in its L2
        const int64_t groups = (n + 3) / 4;
        const int64_t local = blockIdx.x / 8;
        c = (blockIdx.x % 8) + 8 * (local / groups);
        g = local % groups;
    } else {
        c = blockIdx.x % chunks;
        g = blockIdx.x / chunks;
    }
    const int64_t j = g * 4 + wave;
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

// High fan-in variant: the same product with the gathered rows of Y^T served from LDS.
//
// A workgroup (4 wave64s) owns 32 output neurons (8 per wave) and a chunk of 256 batch columns.  Input
// neurons are walked in tiles of 16 rows.  For every tile the workgroup stages the 16 x 256 slab of Y^T
// in LDS, widened to fp64 once at staging (32 KiB), the tile's segment of each of its 32 fan-in lists
// (tile_ptr says where each list crosses each tile boundary) and the segment lengths.  Everything is
// double-buffered: the global loads for tile t+1 are issued before tile t is multiplied and written to
// the other buffer afterwards, so the multiply reads only LDS.  Each list entry is read by the whole
// wave from one LDS address (a broadcast).  Lane l owns batch columns {2l, 2l+1} and {128+2l, 128+2l+1}
// of the chunk, so each of its two ds_read_b128 per entry is one contiguous 1 KiB across the wave (no
// bank conflicts) and feeds the fp64 FMAs directly, with no conversion per product.  A slab row is loaded
// from memory once per 32 neurons instead of once per list entry; two workgroups share a CU.
constexpr int kTileRows = 16;           // input neurons per LDS tile (<= 64: a tile segment fits one load)
constexpr int kTiledCB = 256;           // batch columns per workgroup (4 per lane)
constexpr int kTiledThreads = 256;
constexpr int kTiledNPW = 8;            // output neurons per wave
constexpr int kTiledNJ = (kTiledThreads / 64) * kTiledNPW;
constexpr int kRowF4 = kTiledCB / 4;                          // float4 per slab row (global side)
constexpr int kRowD2 = kTiledCB / 2;                          // double2 per slab row (LDS side)
constexpr int kStageF4 = kTileRows * kRowF4 / kTiledThreads;  // float4 staged per thread per tile

__global__ __launch_bounds__(kTiledThreads, 2) void spmm_tiled_kernel(
    int64_t n, int64_t batch, int chunks, int ntiles, const int32_t *__restrict__ tile_ptr,
    const Edge *__restrict__ fan, const float *__restrict__ bias, double ymax, const float *__restrict__ yt,
    float *__restrict__ zt) {
    __shared__ double2 slab[2][kTileRows * kRowD2];
    __shared__ Edge ents[2][kTiledNJ][kTileRows];
    __shared__ int32_t cnts[2][kTiledNJ];
    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);  // wave-uniform: keeps list addresses scalar
    const int64_t c = blockIdx.x % chunks;
    const int64_t jw = (int64_t)(blockIdx.x / chunks) * kTiledNJ + wave * kTiledNPW;  // first neuron of the wave
    const int64_t col0 = c * kTiledCB;

    double acc[kTiledNPW][4];  // columns 2l, 2l+1, 128+2l, 128+2l+1 of the chunk
#pragma unroll
    for (int q = 0; q < kTiledNPW; ++q)
#pragma unroll
        for (int v = 0; v < 4; ++v) acc[q][v] = 0.0;

    float4 st[kStageF4];
    Edge eg[kTiledNPW];
    auto load_slab = [&](int t) {
        const int64_t i0 = (int64_t)t * kTileRows;
#pragma unroll
        for (int s = 0; s < kStageF4; ++s) {
            const int q = s * kTiledThreads + tid;
            const int64_t gi = i0 + q / kRowF4, gc = col0 + (int64_t)(q % kRowF4) * 4;
            st[s] = (gi < n && gc < batch) ? *reinterpret_cast<const float4 *>(yt + gi * batch + gc)
                                           : make_float4(0.f, 0.f, 0.f, 0.f);
        }
    };
    // segment [b[q], e[q]) of neuron jw + q for one tile; uniform per wave, so these are scalar loads
    auto load_bounds = [&](int t, int32_t (&b)[kTiledNPW], int32_t (&e)[kTiledNPW]) {
        const int32_t *tp0 = tile_ptr + (int64_t)t * n + jw;
        const int32_t *tp1 = tp0 + n;
#pragma unroll
        for (int q = 0; q < kTiledNPW; ++q) {
            const bool ok = jw + q < n;
            b[q] = ok ? tp0[q] : 0;
            e[q] = ok ? tp1[q] : 0;
        }
    };
    auto load_entries = [&](const int32_t (&b)[kTiledNPW], const int32_t (&e)[kTiledNPW]) {
#pragma unroll
        for (int q = 0; q < kTiledNPW; ++q) {
            eg[q].idx = 0;
            eg[q].w = 0.0f;
            if (lane < e[q] - b[q]) eg[q] = fan[b[q] + lane];
        }
    };
    auto stage = [&](int buf, const int32_t (&b)[kTiledNPW], const int32_t (&e)[kTiledNPW]) {
#pragma unroll
        for (int s = 0; s < kStageF4; ++s) {
            const int q = s * kTiledThreads + tid;  // row q / kRowF4, columns 4 (q % kRowF4) .. +3
            slab[buf][2 * q] = make_double2((double)st[s].x, (double)st[s].y);
            slab[buf][2 * q + 1] = make_double2((double)st[s].z, (double)st[s].w);
        }
        if (lane < kTileRows) {
#pragma unroll
            for (int q = 0; q < kTiledNPW; ++q) ents[buf][wave * kTiledNPW + q][lane] = eg[q];
        }
        if (lane == 0) {
#pragma unroll
            for (int q = 0; q < kTiledNPW; ++q) cnts[buf][wave * kTiledNPW + q] = e[q] - b[q];
        }
    };

    int32_t b_nxt[kTiledNPW], e_nxt[kTiledNPW], b_nn[kTiledNPW], e_nn[kTiledNPW];
    load_bounds(0, b_nxt, e_nxt);
    load_slab(0);
    load_entries(b_nxt, e_nxt);
    stage(0, b_nxt, e_nxt);
    if (ntiles > 1) load_bounds(1, b_nxt, e_nxt);
    __syncthreads();

    for (int t = 0; t < ntiles; ++t) {
        const int cur = t & 1;
        const bool more = t + 1 < ntiles;
        if (more) {
            load_slab(t + 1);
            load_entries(b_nxt, e_nxt);
            if (t + 2 < ntiles) load_bounds(t + 2, b_nn, e_nn);
        }
        const int32_t i0 = t * kTileRows;
        const double2 *sl = slab[cur] + lane;
#pragma unroll
        for (int q = 0; q < kTiledNPW; ++q) {
            // entries are read from LDS at a wave-uniform address (a broadcast), straight into VGPRs
            const int nq = wave * kTiledNPW + q;
            const int cnt = cnts[cur][nq];
            const Edge *el = ents[cur][nq];
            int u = 0;
            for (; u + 4 <= cnt; u += 4) {
                double2 ya[4], yb[4];
                double w[4];
#pragma unroll
                for (int k = 0; k < 4; ++k) {
                    const Edge ed = el[u + k];
                    const int r = (ed.idx - i0) * kRowD2;
                    w[k] = (double)ed.w;
                    ya[k] = sl[r];
                    yb[k] = sl[r + 64];
                }
#pragma unroll
                for (int k = 0; k < 4; ++k) {
                    acc[q][0] = __builtin_fma(ya[k].x, w[k], acc[q][0]);
                    acc[q][1] = __builtin_fma(ya[k].y, w[k], acc[q][1]);
                    acc[q][2] = __builtin_fma(yb[k].x, w[k], acc[q][2]);
                    acc[q][3] = __builtin_fma(yb[k].y, w[k], acc[q][3]);
                }
            }
            for (; u < cnt; ++u) {
                const Edge ed = el[u];
                const int r = (ed.idx - i0) * kRowD2;
                const double w = (double)ed.w;
                const double2 ya = sl[r], yb = sl[r + 64];
                acc[q][0] = __builtin_fma(ya.x, w, acc[q][0]);
                acc[q][1] = __builtin_fma(ya.y, w, acc[q][1]);
                acc[q][2] = __builtin_fma(yb.x, w, acc[q][2]);
                acc[q][3] = __builtin_fma(yb.y, w, acc[q][3]);
            }
        }
        if (more) {
            stage(cur ^ 1, b_nxt, e_nxt);  // that buffer was last read in tile t-1, which ended with a barrier
#pragma unroll
            for (int q = 0; q < kTiledNPW; ++q) {
                b_nxt[q] = b_nn[q];
                e_nxt[q] = e_nn[q];
            }
        }
        __syncthreads();
    }
    const int64_t ca = col0 + 2 * lane, cb = ca + 128;  // batch is a multiple of 4, so pairs never straddle it
#pragma unroll
    for (int q = 0; q < kTiledNPW; ++q) {
        const int64_t j = jw + q;
        if (j >= n) break;
        const double bj = (double)bias[j];
        if (ca < batch)
            *reinterpret_cast<float2 *>(zt + j * batch + ca) =
                make_float2(activate(acc[q][0] + bj, ymax), activate(acc[q][1] + bj, ymax));
        if (cb < batch)
            *reinterpret_cast<float2 *>(zt + j * batch + cb) =
                make_float2(activate(acc[q][2] + bj, ymax), activate(acc[q][3] + bj, ymax));
    }
}

// tile_ptr[t * n + j] = first position of fan-in list j whose input index is >= t * kTileRows.
__global__ void tile_ptr_kernel(int64_t n, int ntiles, const int64_t *__restrict__ fan_ptr,
                                const Edge *__restrict__ fan, int32_t *__restrict__ tile_ptr) {
    const int64_t j = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (j >= n) return;
    int64_t e = fan_ptr[j];
    const int64_t end = fan_ptr[j + 1];
    for (int t = 0; t <= ntiles; ++t) {
        const int64_t bound = (int64_t)t * kTileRows;
        while (e < end && fan[e].idx < bound) ++e;
        tile_ptr[(int64_t)t * n + j] = (int32_t)e;
    }
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

int spmm_tile_count(int64_t n) { return (int)((n + kTileRows - 1) / kTileRows); }

// Measured on MI355X (n = 4096, batch = 1024): the LDS-tiled product wins at 50% density (1.34 vs 1.85 ms
// per layer), the L2 gather wins at 10% (0.38 vs 0.78 ms); switch at an average fan-in of 1024.
bool spmm_wants_tiles(int64_t n, int64_t nnz) { return n <= 65536 && nnz >= 1024 * n; }

hipError_t launch_spmm_tile_ptr(int64_t n, const int64_t *fan_ptr, const Edge *fan, int32_t *tile_ptr, hipStream_t s) {
    tile_ptr_kernel<<<(unsigned)((n + 255) / 256), 256, 0, s>>>(n, spmm_tile_count(n), fan_ptr, fan, tile_ptr);
    return hipGetLastError();
}

hipError_t launch_spmm_fanin(int64_t n, int64_t batch, const int64_t *fan_ptr, const Edge *fan,
                             const int32_t *tile_ptr, const float *bias, double ymax, const float *yt, float *zt,
                             hipStream_t s) {
    if (n == 0 || batch == 0) return hipSuccess;
    if (tile_ptr && batch % 4 == 0 && batch >= 128) {
        const int64_t chunks = (batch + kTiledCB - 1) / kTiledCB;
        const int64_t blocks = ((n + kTiledNJ - 1) / kTiledNJ) * chunks;
        spmm_tiled_kernel<<<(unsigned)blocks, kTiledThreads, 0, s>>>(n, batch, (int)chunks, spmm_tile_count(n),
                                                                     tile_ptr, fan, bias, ymax, yt, zt);
        return hipGetLastError();
    }
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
