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

template <int V, bool kPattern>
__global__ __launch_bounds__(256) void spmm_fanin_kernel(int64_t n, int64_t batch, int64_t ld, int chunks,
                                                         int64_t block_base,
                                                         const int64_t *__restrict__ fan_ptr,
                                                         const Edge *__restrict__ fan, const float *__restrict__ bias,
                                                         double ymax, const float *__restrict__ yt,
                                                         float *__restrict__ zt) {
    const int lane = threadIdx.x & 63;
    const int wave = threadIdx.x >> 6;
    const int64_t b = block_base + blockIdx.x;  // large grids are launched in segments (see the launcher)
    int64_t c, g;
    if (chunks % 8 == 0) {
        // chunk-major per XCD: XCD x works through chunks x, x+8, ... one at a time, every neuron group
        // of a chunk before the next, so the input rows its current neurons gather stay in its L2
        const int64_t groups = (n + 3) / 4;
        const int64_t local = b / 8;
        c = (b % 8) + 8 * (local / groups);
        g = local % groups;
    } else if (8 % chunks == 0) {
        // 1, 2 or 4 chunks: XCD x keeps to chunk x % chunks and takes every (8 / chunks)-th neuron group of
        // it, so its L2 holds one chunk's slice of Y^T rather than all of Y^T
        const int64_t xcd = b % 8;
        c = xcd % chunks;
        g = (b / 8) * (8 / chunks) + xcd / chunks;
    } else {
        c = b % chunks;
        g = b / chunks;
    }
    const int64_t j = g * 4 + wave;
    if (j >= n) return;
    const int64_t col = c * (64 * V) + (int64_t)lane * V;
    const bool active = col < batch;       // batch is a multiple of V, so col < batch => col + V <= batch
    const int64_t colc = active ? col : 0; // inactive lanes read a valid address and discard it

    double acc[V];
    uint32_t hit[V];  // pattern mode: OR of the input bits; nonzero magnitude bits = a structural product
#pragma unroll
    for (int v = 0; v < V; ++v) {
        acc[v] = 0.0;
        hit[v] = 0u;
    }

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
                load_v<V>(yt + (int64_t)i * ld + colc, y[u]);
            }
#pragma unroll
            for (int u = 0; u < kUnroll; ++u) {
                const double wd = (double)w[u];
#pragma unroll
                for (int v = 0; v < V; ++v) {
                    acc[v] = __builtin_fma((double)y[u][v], wd, acc[v]);
                    if constexpr (kPattern) hit[v] |= __float_as_uint(y[u][v]);
                }
            }
        }
        for (; t < cnt; ++t) {
            float y[V];
            const int32_t i = bcast_i(mine.idx, t);
            const double wd = (double)bcast_f(mine.w, t);
            load_v<V>(yt + (int64_t)i * ld + colc, y);
#pragma unroll
            for (int v = 0; v < V; ++v) {
                acc[v] = __builtin_fma((double)y[v], wd, acc[v]);
                if constexpr (kPattern) hit[v] |= __float_as_uint(y[v]);
            }
        }
    }
    if (!active) return;
    const double bj = (double)bias[j];
    float out[V];
#pragma unroll
    for (int v = 0; v < V; ++v)
        out[v] = (kPattern && (hit[v] & 0x7fffffffu) == 0u) ? 0.0f : activate(acc[v] + bj, ymax);
    store_v<V>(zt + j * ld + col, out);
}

// Narrow-chunk variant for wide layers.  A chunk of the kernel above is 256 batch columns, so its slice of
// Y^T is n KiB: beyond n = 4096 it no longer fits an XCD's 4 MiB L2, and every one of a row segment's ~32
// consumers fetches it from memory again.  Here each 16-lane row of a wave owns one output neuron and 64
// columns (4 per lane), so a chunk's slice is n x 256 bytes (4 MiB at n = 16384), which the L2 keeps when
// the rows sit at a padded pitch (act_ld).  All XCDs work on the same chunk at a time, XCD x on its own
// contiguous eighth of the neurons (a layer whose lists stay near the diagonal keeps its rows local; a ragged
// last chunk still spreads over every XCD).  A row loads 16 list entries at once (lane k holds entry k) and
// broadcasts entry t to its 16 lanes with a DPP row broadcast; the four rows of a wave walk their lists in
// step, the shortest list's length unpredicated and the rest with a per-row guard.  Each output is still
// summed in list (ascending input) order, as in the kernel above.
constexpr int kNarrowP = 16;  // lanes per output neuron: one DPP row

template <int T>
__device__ __forceinline__ int32_t bcast_row(int32_t v) {
    return __builtin_amdgcn_mov_dpp(v, 0x150 + T, 0xf, 0xf, false);  // row_newbcast: lane T of each 16-lane row
}

constexpr int kNarrowUnroll = 8;

// f(integral_constant<int, U>) for U = B .. E - 1 (a DPP lane select must be a compile-time constant)
template <int B, int E, typename F>
__device__ __forceinline__ void static_for(F &&f) {
    if constexpr (B < E) {
        f(std::integral_constant<int, B>{});
        static_for<B + 1, E>(f);
    }
}

// row i of Y^T at this lane's columns: i < 2^24 and the row pitch in bytes < 2^24 (the launcher checks)
__device__ __forceinline__ const float *narrow_row(const char *yl, int32_t i, uint32_t pitch) {
    return reinterpret_cast<const float *>(yl + (uint64_t)((uint32_t)i & 0xffffffu) * (uint64_t)(pitch & 0xffffffu));
}

// list slots T0 .. T0 + kNarrowUnroll - 1 of the 16 a row holds: unpredicated while every row of the wave has
// them (full), else with each row's loads guarded by its own length
template <int V, bool kPattern, int T0>
__device__ __forceinline__ void narrow_batch(const Edge &mine, int full, int base, int cnt, const char *yl,
                                             uint32_t pitch, double (&acc)[V], uint32_t (&hit)[V]) {
    float y[kNarrowUnroll][V];
    float w[kNarrowUnroll];
    int32_t idx[kNarrowUnroll];
    static_for<0, kNarrowUnroll>([&](auto u) {
        idx[u] = bcast_row<T0 + u>(mine.idx);
        w[u] = __int_as_float(bcast_row<T0 + u>(__float_as_int(mine.w)));
    });
#pragma unroll
    for (int u = 0; u < kNarrowUnroll; ++u) load_v<V>(narrow_row(yl, idx[u], pitch), y[u]);
    if (T0 + kNarrowUnroll <= full) {
#pragma unroll
        for (int u = 0; u < kNarrowUnroll; ++u) {
            const double wd = (double)w[u];
#pragma unroll
            for (int v = 0; v < V; ++v) {
                acc[v] = __builtin_fma((double)y[u][v], wd, acc[v]);
                if constexpr (kPattern) hit[v] |= __float_as_uint(y[u][v]);
            }
        }
    } else {
        // a row whose list has ended read row 0 of Y^T (the zero index its lanes hold past the end: a line the
        // chunk keeps hot) and adds the product of a zeroed input and the zero weight held there: +0 leaves an
        // accumulator unchanged (one that starts at +0 never becomes -0)
#pragma unroll
        for (int u = 0; u < kNarrowUnroll; ++u) {
            const bool ok = base + T0 + u < cnt;
            const double wd = (double)w[u];
#pragma unroll
            for (int v = 0; v < V; ++v) {
                asm volatile("" : "+v"(y[u][v]));  // keeps the load whole and unconditional
                const float yv = ok ? y[u][v] : 0.0f;
                acc[v] = __builtin_fma((double)yv, wd, acc[v]);
                if constexpr (kPattern) hit[v] |= __float_as_uint(yv);
            }
        }
    }
}

template <int V, bool kPattern>
__global__ __launch_bounds__(256) void spmm_narrow_kernel(int64_t n, int64_t batch, int64_t ld, int64_t gpx,
                                                          int64_t block_base,
                                                          const int64_t *__restrict__ fan_ptr,
                                                          const Edge *__restrict__ fan,
                                                          const float *__restrict__ bias, double ymax,
                                                          const float *__restrict__ yt, float *__restrict__ zt) {
    constexpr int P = kNarrowP, G = 64 / P;  // G neurons per wave
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int grp = lane / P, k = lane % P;
    // block b: XCD b % 8; chunk c for every XCD at once, neuron groups [x gpx, (x + 1) gpx) on XCD x
    const int64_t b = block_base + blockIdx.x;
    const int64_t local = b >> 3;
    const int64_t c = local / gpx;
    const int64_t g = (b & 7) * gpx + local % gpx;
    const int64_t j = (g * 4 + wave) * G + grp;
    const bool jv = j < n;
    const int64_t col = c * (P * V) + (int64_t)k * V;
    const bool active = jv && col < batch;  // batch is a multiple of V, so col < batch => col + V <= batch
    const int64_t colc = col < batch ? col : 0;  // lanes past the batch read a valid address and discard it
    const char *yl = reinterpret_cast<const char *>(yt + colc);
    const uint32_t pitch = (uint32_t)(ld * (int64_t)sizeof(float));
    int64_t eb = 0;
    int cnt = 0;
    if (jv) {
        eb = fan_ptr[j];
        cnt = (int)(fan_ptr[j + 1] - eb);
    }
    // the wave's shortest and longest list (every lane keeps running: the broadcasts read lanes of all groups)
    int lo = cnt, hi = cnt;
    static_for<0, G>([&](auto q) {
        const int cq = __builtin_amdgcn_readlane(cnt, q * P);
        lo = q == 0 ? cq : min(lo, cq);
        hi = q == 0 ? cq : max(hi, cq);
    });

    double acc[V];
    uint32_t hit[V];
#pragma unroll
    for (int v = 0; v < V; ++v) {
        acc[v] = 0.0;
        hit[v] = 0u;
    }
    Edge mine;
    mine.idx = 0;
    mine.w = 0.0f;
    if (k < cnt) mine = fan[eb + k];
    for (int base = 0; base < hi; base += P) {
        Edge next;  // the group's next P entries, loaded while these are used
        next.idx = 0;
        next.w = 0.0f;
        if (base + P + k < cnt) next = fan[eb + base + P + k];
        const int full = lo - base;
        narrow_batch<V, kPattern, 0>(mine, full, base, cnt, yl, pitch, acc, hit);
        if (hi - base > kNarrowUnroll)
            narrow_batch<V, kPattern, kNarrowUnroll>(mine, full, base, cnt, yl, pitch, acc, hit);
        mine = next;
    }
    if (!active) return;
    const double bj = (double)bias[j];
    float out[V];
#pragma unroll
    for (int v = 0; v < V; ++v)
        out[v] = (kPattern && (hit[v] & 0x7fffffffu) == 0u) ? 0.0f : activate(acc[v] + bj, ymax);
    store_v<V>(zt + j * ld + col, out);
}

// High fan-in variant: the same product with the gathered rows of Y^T served from LDS and each row read once
// per wave for all of the wave's neurons that use it.
//
// A workgroup (8 wave64s) owns 32 output neurons (4 per wave) and a chunk of 256 batch columns; lane l owns
// columns 4l..4l+3 of the chunk.  Input neurons are walked in tiles of 16 rows.  For every tile the
// workgroup stages the 16 x 256 slab of Y^T in LDS, widened to fp64 once (32 KiB, laid out so that both the
// staging stores and the reads are contiguous per wave); the next tile's slab is loaded into registers
// while the current one is multiplied.  A 16-bit mask per (tile, neuron), built at set-up, says which
// rows of the tile a fan-in list holds.  Each wave walks the 16 rows in order: it reads a row once (two
// ds_read_b128 per lane, at immediate offsets) and, for each of its 4 neurons whose mask has that row
// (a wave-uniform branch), takes the next list weight from the lane that loaded it (readlane) and does
// four fp64 FMAs.  Lists are sorted by input index, so every output is still summed in ascending input
// order.  At 50% density a row read feeds two list entries instead of one, which halves the LDS traffic
// per FMA, and the per-entry address arithmetic of a list walk disappears.
constexpr int kTileRows = 16;                       // input neurons per LDS tile (one mask bit each)
constexpr int kTiledCB = 256;                       // batch columns per workgroup (4 per lane)
constexpr int kTiledThreads = 512;
constexpr int kTiledNPW = 4;                        // output neurons per wave
constexpr int kTiledNJ = (kTiledThreads / 64) * kTiledNPW;
constexpr int kRowF4 = kTiledCB / 4;                // float4 per slab row (global side)
constexpr int kRowD2 = kTiledCB / 2;                // double2 per slab row (LDS side)
constexpr int kStageF4 = kTileRows * kRowF4 / kTiledThreads;
constexpr int kRowGroup = 2;                        // slab rows read ahead of their FMAs

// Row pitch of the per-(tile, neuron) arrays (masks, slot weights): n rounded up to a whole 64-neuron workgroup
// of the slot kernel, so every wave reads in bounds and the 64-bit mask loads stay 8-byte aligned; the padding
// stays zero.
__host__ __device__ inline int64_t mask_pitch(int64_t n) { return (n + 63) / 64 * 64; }

template <bool kPattern>
__global__ __launch_bounds__(kTiledThreads, 3) void spmm_tiled_kernel(
    int64_t n, int64_t batch, int64_t ld, int chunks, int ntiles, const int64_t *__restrict__ fan_ptr,
    const uint16_t *__restrict__ tile_mask, const Edge *__restrict__ fan, const float *__restrict__ bias,
    double ymax, const float *__restrict__ yt, float *__restrict__ zt) {
    __shared__ double2 slab[kTileRows * kRowD2];
    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);  // wave-uniform: masks and positions stay scalar
    // XCD-aware order: workgroups are dealt round-robin to the 8 XCDs, and the batch chunks of one neuron
    // group take consecutive slots of the same XCD, so they run together and read its fan-in lists from HBM
    // once (the group count is padded to a multiple of 8)
    const int64_t local = blockIdx.x / 8;
    const int64_t c = local % chunks;
    const int64_t g = (local / chunks) * 8 + blockIdx.x % 8;
    if (g * kTiledNJ >= n) return;  // padding group: the whole workgroup leaves before any barrier
    const int64_t jw = g * kTiledNJ + wave * kTiledNPW;  // first neuron of the wave
    const int64_t col0 = c * kTiledCB;
    const int64_t pitch = mask_pitch(n);

    double acc[kTiledNPW][4];
    uint32_t hit[kTiledNPW][4];  // pattern mode: OR of the inputs' high words (magnitude bits = nonzero)
#pragma unroll
    for (int q = 0; q < kTiledNPW; ++q)
#pragma unroll
        for (int v = 0; v < 4; ++v) {
            acc[q][v] = 0.0;
            hit[q][v] = 0u;
        }

    float4 st[kStageF4];
    auto load_slab = [&](int t) {
        const int64_t i0 = (int64_t)t * kTileRows;
#pragma unroll
        for (int s = 0; s < kStageF4; ++s) {
            const int q = s * kTiledThreads + tid;
            const int64_t gi = i0 + q / kRowF4, gc = col0 + (int64_t)(q % kRowF4) * 4;
            st[s] = (gi < n && gc < batch) ? *reinterpret_cast<const float4 *>(yt + gi * ld + gc)
                                           : make_float4(0.f, 0.f, 0.f, 0.f);
        }
    };
    auto stage = [&]() {
        // float4 q covers columns 4m..4m+3 of row q / 64 (m = q % 64): its two halves go to double2 slots m and
        // 64 + m of the row, so each store instruction writes 1 KiB contiguous
#pragma unroll
        for (int s = 0; s < kStageF4; ++s) {
            const int q = s * kTiledThreads + tid;
            const int row = q / kRowF4, m = q % kRowF4;
            slab[row * kRowD2 + m] = make_double2((double)st[s].x, (double)st[s].y);
            slab[row * kRowD2 + 64 + m] = make_double2((double)st[s].z, (double)st[s].w);
        }
    };
    // the 4 neurons' masks of tile t as one 64-bit scalar load; neurons past n read the zeroed padding
    auto load_mask = [&](int t) -> uint64_t {
        return jw < n ? *reinterpret_cast<const uint64_t *>(tile_mask + (int64_t)t * pitch + jw) : 0ull;
    };
    int64_t pos[kTiledNPW];  // next unread entry of each list
#pragma unroll
    for (int q = 0; q < kTiledNPW; ++q) pos[q] = jw + q < n ? fan_ptr[jw + q] : 0;
    float wn[kTiledNPW], wv[kTiledNPW];  // lane u holds the weight of the u-th list entry in the tile
    auto load_weights = [&](uint64_t mk) {
#pragma unroll
        for (int q = 0; q < kTiledNPW; ++q) {
            const int cnt = __builtin_popcount((uint32_t)(mk >> (16 * q)) & 0xffffu);
            wn[q] = lane < cnt ? fan[pos[q] + lane].w : 0.0f;
            pos[q] += cnt;
        }
    };

    uint64_t mk_cur = load_mask(0), mk_nxt = ntiles > 1 ? load_mask(1) : 0ull;
    load_slab(0);
    load_weights(mk_cur);
    stage();
    __syncthreads();
    const double2 *sl = slab + lane;
    for (int t = 0; t < ntiles; ++t) {
        const bool more = t + 1 < ntiles;
#pragma unroll
        for (int q = 0; q < kTiledNPW; ++q) wv[q] = wn[q];
        const uint64_t mk = mk_cur;
        if (more) {
            load_slab(t + 1);
            load_weights(mk_nxt);
            mk_cur = mk_nxt;
            if (t + 2 < ntiles) mk_nxt = load_mask(t + 2);
        }
        uint32_t m32[kTiledNPW];
        int kq[kTiledNPW];
#pragma unroll
        for (int q = 0; q < kTiledNPW; ++q) {
            m32[q] = __builtin_amdgcn_readfirstlane((uint32_t)(mk >> (16 * q)) & 0xffffu);
            kq[q] = 0;
        }
#pragma unroll
        for (int g = 0; g < kTileRows; g += kRowGroup) {
            double2 ya[kRowGroup], yb[kRowGroup];
#pragma unroll
            for (int k = 0; k < kRowGroup; ++k) {
                ya[k] = sl[(g + k) * kRowD2];
                yb[k] = sl[(g + k) * kRowD2 + 64];
            }
#pragma unroll
            for (int k = 0; k < kRowGroup; ++k) {
#pragma unroll
                for (int q = 0; q < kTiledNPW; ++q) {
                    if ((m32[q] >> (g + k)) & 1u) {
                        const double w = (double)__int_as_float(__builtin_amdgcn_readlane(__float_as_int(wv[q]), kq[q]));
                        ++kq[q];
                        acc[q][0] = __builtin_fma(ya[k].x, w, acc[q][0]);
                        acc[q][1] = __builtin_fma(ya[k].y, w, acc[q][1]);
                        acc[q][2] = __builtin_fma(yb[k].x, w, acc[q][2]);
                        acc[q][3] = __builtin_fma(yb[k].y, w, acc[q][3]);
                        if constexpr (kPattern) {
                            hit[q][0] |= (uint32_t)__double2hiint(ya[k].x);
                            hit[q][1] |= (uint32_t)__double2hiint(ya[k].y);
                            hit[q][2] |= (uint32_t)__double2hiint(yb[k].x);
                            hit[q][3] |= (uint32_t)__double2hiint(yb[k].y);
                        }
                    }
                }
            }
        }
        __syncthreads();  // every wave is done with this slab
        if (more) stage();
        __syncthreads();
    }
    const int64_t ca = col0 + 4 * lane;  // batch is a multiple of 4, so ca < batch => ca + 3 < batch
#pragma unroll
    for (int q = 0; q < kTiledNPW; ++q) {
        const int64_t j = jw + q;
        if (j >= n) break;
        const double bj = (double)bias[j];
        float f[4];
#pragma unroll
        for (int v = 0; v < 4; ++v)
            f[v] = (kPattern && (hit[q][v] & 0x7fffffffu) == 0u) ? 0.0f : activate(acc[q][v] + bj, ymax);
        if (ca < batch) *reinterpret_cast<float4 *>(zt + j * ld + ca) = make_float4(f[0], f[1], f[2], f[3]);
    }
}

// High fan-in variant with the weights in scalar registers (used when the n x n slot array below fits).
//
// The same product as the tiled kernel above, restructured after measuring gfx950: an fp64 FMA whose weight
// operand is a scalar register pair issues at about 1.25x the rate of one with three vector operands, and a
// readlane per list entry (the tiled kernel's way of broadcasting the weight) costs more than the FMAs it feeds.
// So the weights come from a "slot" array built at set-up: for input tile t (16 rows), phase h (2 rows) and
// output neuron j, the two fp64 weights W(16t + 2h + r, j), r = 0, 1, zero where the list has no entry, so a
// wave's 4 neurons find a phase's weights (16 scalar registers) in one 64-byte line, read with one scalar load.
//
// A workgroup is 16 wave64s owning 64 output neurons (4 per wave) and 256 batch columns (4 per lane); the
// 16 x 256 slab of Y^T is staged in LDS widened to fp64, double-buffered (one barrier per tile).  A tile is
// walked in phases of 2 rows; at the start of phase h a wave waits for phase h's data (the scalar weights and
// the two slab rows in registers), issues the loads of phase h + 1, then does the FMAs of phase h for every
// (row, neuron) whose mask bit is set.  Scalar loads may complete out of order, so the only safe wait on them
// is "all outstanding", which is why the loads of the next phase are issued only after that wait.  Every output
// is still summed in ascending input order (each FMA adds one product to one accumulator, rows in order).
constexpr int kSlotThreads = 1024;
constexpr int kSlotNPW = 4;                                  // output neurons per wave
constexpr int kSlotNJ = (kSlotThreads / 64) * kSlotNPW;      // 64 per workgroup
constexpr int kSlotPR = 2;                                   // slab rows per phase
constexpr int kSlotPhases = kTileRows / kSlotPR;             // phases per tile
constexpr int kSlotPrefetch = 1;                 // tiles ahead whose weight lines are pulled into L2
static_assert(kSlotNJ == 64, "mask_pitch() rounds n to whole workgroups");

template <bool kPattern>
__global__ __launch_bounds__(kSlotThreads, 1) void spmm_slots_kernel(
    int64_t n, int64_t batch, int64_t ld, int chunks, int ntiles, const uint16_t *__restrict__ tile_mask,
    const double *__restrict__ slots, const float *__restrict__ bias, double ymax, const float *__restrict__ yt,
    float *__restrict__ zt) {
    __shared__ double2 slab[2][kTileRows * kRowD2];
    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int64_t pitch = mask_pitch(n);
    // XCD-aware order as in the tiled kernel: the batch chunks of one neuron group run together on one XCD
    const int64_t local = blockIdx.x / 8;
    const int64_t c = local % chunks;
    const int64_t g = (local / chunks) * 8 + blockIdx.x % 8;
    if (g * kSlotNJ >= pitch) return;  // padding group: the whole workgroup leaves before any barrier
    const int64_t jw = g * kSlotNJ + wave * kSlotNPW;  // < pitch: masks and slots of padded neurons are zero
    const int64_t col0 = c * kTiledCB;

    double acc[kSlotNPW][4];
    uint32_t hit[kSlotNPW][4];  // pattern mode: OR of the inputs' high words (magnitude bits = nonzero)
#pragma unroll
    for (int q = 0; q < kSlotNPW; ++q)
#pragma unroll
        for (int v = 0; v < 4; ++v) {
            acc[q][v] = 0.0;
            hit[q][v] = 0u;
        }

    // staging: one float4 of the 16 x 256 slab per thread (row tid / 64, columns 4 (tid % 64) ..)
    const int srow = tid / kRowF4, sm = tid % kRowF4;
    const int64_t sgc = col0 + 4 * (int64_t)sm;
    float4 st;
    auto load_slab = [&](int t) {
        const int64_t gi = (int64_t)t * kTileRows + srow;
        st = (gi < n && sgc < batch) ? *reinterpret_cast<const float4 *>(yt + gi * ld + sgc)
                                     : make_float4(0.f, 0.f, 0.f, 0.f);
    };
    auto stage = [&](int buf) {
        slab[buf][srow * kRowD2 + sm] = make_double2((double)st.x, (double)st.y);
        slab[buf][srow * kRowD2 + 64 + sm] = make_double2((double)st.z, (double)st.w);
    };
    // weights of rows 2h, 2h + 1 of tile t for the wave's 4 neurons: one 64-byte line, one scalar load
    auto load_w = [&](int t, int h, double (&w)[kSlotNPW][kSlotPR]) {
        const double *wp = slots + (((int64_t)t * kSlotPhases + h) * pitch + jw) * kSlotPR;
#pragma unroll
        for (int q = 0; q < kSlotNPW; ++q)
#pragma unroll
            for (int r = 0; r < kSlotPR; ++r) w[q][r] = wp[q * kSlotPR + r];
    };
    auto load_y = [&](int buf, int h, double2 (&y)[kSlotPR][2]) {
        const double2 *sl = slab[buf] + lane;
#pragma unroll
        for (int r = 0; r < kSlotPR; ++r) {
            y[r][0] = sl[(kSlotPR * h + r) * kRowD2];
            y[r][1] = sl[(kSlotPR * h + r) * kRowD2 + 64];
        }
    };
    // an empty asm that reads the phase's registers: the compiler must complete their loads before it
    auto ready = [&](const double (&w)[kSlotNPW][kSlotPR], const double2 (&y)[kSlotPR][2]) {
#pragma unroll
        for (int q = 0; q < kSlotNPW; ++q)
#pragma unroll
            for (int r = 0; r < kSlotPR; ++r) asm volatile("" ::"s"(w[q][r]));
#pragma unroll
        for (int r = 0; r < kSlotPR; ++r)
            asm volatile("" ::"v"(y[r][0].x), "v"(y[r][0].y), "v"(y[r][1].x), "v"(y[r][1].y));
    };

    // two register sets, used alternately by even and odd phases, so no copies between phases
    double wa[kSlotNPW][kSlotPR], wb[kSlotNPW][kSlotPR];
    double2 ya[kSlotPR][2], yb[kSlotPR][2];
    uint32_t mk[kSlotNPW], mkn[kSlotNPW];  // each neuron's 16 mask bits of the current / next tile
    auto load_mask = [&](int t, uint32_t (&m)[kSlotNPW]) {
        const uint64_t v = *reinterpret_cast<const uint64_t *>(tile_mask + (int64_t)t * pitch + jw);
#pragma unroll
        for (int q = 0; q < kSlotNPW; ++q) m[q] = (uint32_t)(v >> (16 * q)) & 0xffffu;
    };
    // phase h of tile t: wait for (wc, yc), issue the loads of the next phase into (wn, yn), then the FMAs
    // (tn: the next tile, or the last tile again at the end, so that every load is unconditional and the
    // weights never pass through a branch merge, which would move them to vector registers)
    auto phase = [&](int t, int h, int tn, int buf, double (&wc)[kSlotNPW][kSlotPR], double2 (&yc)[kSlotPR][2],
                     double (&wn)[kSlotNPW][kSlotPR], double2 (&yn)[kSlotPR][2]) {
        ready(wc, yc);
        __builtin_amdgcn_sched_barrier(0);
        if (h + 1 < kSlotPhases) {
            load_w(t, h + 1, wn);
            load_y(buf, h + 1, yn);
        } else {
            load_w(tn, 0, wn);  // the next tile's rows are read after the barrier
        }
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int r = 0; r < kSlotPR; ++r) {
#pragma unroll
            for (int q = 0; q < kSlotNPW; ++q) {
                if (__builtin_expect((mk[q] >> (kSlotPR * h + r)) & 1u, 1u)) {
                    const double w = wc[q][r];
                    acc[q][0] = __builtin_fma(yc[r][0].x, w, acc[q][0]);
                    acc[q][1] = __builtin_fma(yc[r][0].y, w, acc[q][1]);
                    acc[q][2] = __builtin_fma(yc[r][1].x, w, acc[q][2]);
                    acc[q][3] = __builtin_fma(yc[r][1].y, w, acc[q][3]);
                    if constexpr (kPattern) {
                        hit[q][0] |= (uint32_t)__double2hiint(yc[r][0].x);
                        hit[q][1] |= (uint32_t)__double2hiint(yc[r][0].y);
                        hit[q][2] |= (uint32_t)__double2hiint(yc[r][1].x);
                        hit[q][3] |= (uint32_t)__double2hiint(yc[r][1].y);
                    }
                }
            }
        }
        __builtin_amdgcn_sched_barrier(0);
    };
    static_assert(kSlotPhases % 2 == 0, "a tile ends on an odd phase, so the next starts on set a");

    load_mask(0, mk);
    load_slab(0);
    stage(0);
    load_w(0, 0, wa);
    __syncthreads();
    load_y(0, 0, ya);
    for (int t = 0; t < ntiles; ++t) {
        const int tn = t + 1 < ntiles ? t + 1 : t;
        const int buf = t & 1;
        load_slab(tn);
        load_mask(tn, mkn);
        // Pull the weight lines of tile t + kSlotPrefetch into L2 with a vector load (lane h < 8: the wave's line of
        // phase h, lane 8: its masks): a scalar load that misses L2 stalls the whole phase, a vector load is waited
        // for only here, at the staging below.
        uint32_t pf = 0;
        if (t + kSlotPrefetch < ntiles && lane < kSlotPhases + 1) {
            pf = lane < kSlotPhases
                     ? *reinterpret_cast<const uint32_t *>(
                           slots + (((int64_t)(t + kSlotPrefetch) * kSlotPhases + lane) * pitch + jw) * kSlotPR)
                     : *reinterpret_cast<const uint32_t *>(tile_mask + (int64_t)(t + kSlotPrefetch) * pitch + jw);
        }
#pragma unroll
        for (int h = 0; h < kSlotPhases; h += 2) {
            phase(t, h, tn, buf, wa, ya, wb, yb);
            phase(t, h + 1, tn, buf, wb, yb, wa, ya);
        }
        stage((t + 1) & 1);          // that buffer was last read in tile t - 1, before the previous barrier
        asm volatile("" ::"v"(pf));  // keeps the prefetch load (its value is not needed)
#pragma unroll
        for (int q = 0; q < kSlotNPW; ++q) mk[q] = mkn[q];
        __syncthreads();
        load_y((t + 1) & 1, 0, ya);  // after the last tile: read and not used
    }
    const int64_t ca = col0 + 4 * lane;  // batch is a multiple of 4, so ca < batch => ca + 3 < batch
#pragma unroll
    for (int q = 0; q < kSlotNPW; ++q) {
        const int64_t j = jw + q;
        if (j >= n) break;
        const double bj = (double)bias[j];
        float f[4];
#pragma unroll
        for (int v = 0; v < 4; ++v)
            f[v] = (kPattern && (hit[q][v] & 0x7fffffffu) == 0u) ? 0.0f : activate(acc[q][v] + bj, ymax);
        if (ca < batch) *reinterpret_cast<float4 *>(zt + j * ld + ca) = make_float4(f[0], f[1], f[2], f[3]);
    }
}

// slots[((t * 8 + h) * pitch + j) * 2 + r] = W(16t + 2h + r, j): one wave per fan-in list, lanes over its entries.
__global__ void slots_kernel(int64_t n, const int64_t *__restrict__ fan_ptr, const Edge *__restrict__ fan,
                             double *__restrict__ slots) {
    const int64_t j = (int64_t)blockIdx.x * (blockDim.x / 64) + threadIdx.x / 64;
    if (j >= n) return;
    const int64_t pitch = mask_pitch(n);
    for (int64_t e = fan_ptr[j] + (threadIdx.x & 63); e < fan_ptr[j + 1]; e += 64) {
        const int64_t i = fan[e].idx;
        slots[((i / kSlotPR) * pitch + j) * kSlotPR + (i % kSlotPR)] = (double)fan[e].w;
    }
}

// tile_mask[t * pitch + j] bit r = list j holds input neuron t * 16 + r (lists are sorted by input index).
__global__ void tile_mask_kernel(int64_t n, const int64_t *__restrict__ fan_ptr, const Edge *__restrict__ fan,
                                 uint16_t *__restrict__ tile_mask) {
    const int64_t j = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (j >= n) return;
    const int64_t pitch = mask_pitch(n);
    int64_t t_cur = -1;
    uint32_t m = 0;
    for (int64_t e = fan_ptr[j]; e < fan_ptr[j + 1]; ++e) {
        const int64_t i = fan[e].idx;
        const int64_t t = i / kTileRows;
        if (t != t_cur) {
            if (t_cur >= 0) tile_mask[t_cur * pitch + j] = (uint16_t)m;
            t_cur = t;
            m = 0;
        }
        m |= 1u << (i % kTileRows);
    }
    if (t_cur >= 0) tile_mask[t_cur * pitch + j] = (uint16_t)m;
}

// T x T tile transpose through LDS (padded against bank conflicts): out (cols x rows) = in^T.  One workgroup per
// tile on a one-dimensional grid, tile b = (row tile b / col_tiles, column tile b % col_tiles).  Measured on
// MI355X: 32 x 32 tiles give small matrices enough workgroups (a 64 x 1024 activation block: 64 tiles, 3.2 us,
// against 16 tiles and 6.8 us at 64 x 64), while 64 x 64 tiles read whole 256-byte row segments and move a
// 34 GB matrix in 16.2 ms instead of 18.1.
template <int T>
__global__ __launch_bounds__(256) void transpose_kernel(const float *__restrict__ in, int64_t in_ld,
                                                        float *__restrict__ out, int64_t out_ld, int64_t rows,
                                                        int64_t cols, int64_t col_tiles) {
    __shared__ float tile[T][T + 1];
    constexpr int kStep = 256 / T;
    const int64_t r0 = (int64_t)(blockIdx.x / col_tiles) * T, c0 = (int64_t)(blockIdx.x % col_tiles) * T;
    const int tx = threadIdx.x % T, ty = threadIdx.x / T;
#pragma unroll
    for (int rr = ty; rr < T; rr += kStep) {
        const int64_t r = r0 + rr, c = c0 + tx;
        if (r < rows && c < cols) tile[rr][tx] = in[r * in_ld + c];
    }
    __syncthreads();
#pragma unroll
    for (int cc = ty; cc < T; cc += kStep) {
        const int64_t c = c0 + cc, r = r0 + tx;
        if (r < rows && c < cols) out[c * out_ld + r] = tile[tx][cc];
    }
}

}  // namespace

hipError_t launch_transpose(const float *in, int64_t in_ld, float *out, int64_t out_ld, int64_t rows, int64_t cols,
                            hipStream_t s) {
    if (rows == 0 || cols == 0) return hipSuccess;
    if (in_ld < cols || out_ld < rows) return hipErrorInvalidValue;
    const int T = rows * cols <= (int64_t(1) << 24) ? 32 : 64;
    const int64_t ct = (cols + T - 1) / T, rt = (rows + T - 1) / T;
    if (rt * ct > 0x7fffffffLL) return hipErrorInvalidValue;
    if (T == 32)
        transpose_kernel<32><<<(unsigned)(rt * ct), 256, 0, s>>>(in, in_ld, out, out_ld, rows, cols, ct);
    else
        transpose_kernel<64><<<(unsigned)(rt * ct), 256, 0, s>>>(in, in_ld, out, out_ld, rows, cols, ct);
    return hipGetLastError();
}

int spmm_tile_count(int64_t n) { return (int)((n + kTileRows - 1) / kTileRows); }

size_t spmm_tile_mask_elems(int64_t n) { return (size_t)spmm_tile_count(n) * (size_t)mask_pitch(n); }

// Kernel choice for a dense-Y layer.  Both LDS-tiled kernels visit every (input, output) slot, so their cost
// grows with n^2 and hardly with the density; the gather's grows with nnz.  Measured on MI355X (n = 4096,
// batch = 1024, per layer): the scalar-register kernel takes 0.51-0.54 ms from d = 0.15 to 0.5, the gather
// 0.47 ms at d = 0.2, 0.59 at 0.25, 0.70 at 0.3, so the former is used from d = 2/9; the readlane-fed kernel
// (for layers whose slot array would not fit) tied with the gather at d = 0.3 (0.69 ms) and took 0.83 ms at
// d = 0.5, so it is used from d = 0.3.  Thresholds on nnz / n^2 in exact integer arithmetic (n <= 65536).
static bool slots_fit(int64_t n);
bool spmm_wants_tiles(int64_t n, int64_t nnz) {
    if (n > 65536) return false;
    return slots_fit(n) ? 9 * nnz >= 2 * n * n : 10 * nnz >= 3 * n * n;
}

size_t spmm_slot_elems(int64_t n) { return (size_t)spmm_tile_count(n) * kTileRows * (size_t)mask_pitch(n); }

// The slot array holds every (input, output) pair in fp64: used while it stays at or below 2 GiB per layer.
static bool slots_fit(int64_t n) { return spmm_slot_elems(n) * sizeof(double) <= (size_t(1) << 31); }
bool spmm_wants_slots(int64_t n, int64_t nnz) { return spmm_wants_tiles(n, nnz) && slots_fit(n); }

hipError_t launch_spmm_slots(int64_t n, const int64_t *fan_ptr, const Edge *fan, double *slots, hipStream_t s) {
    hipError_t e = hipMemsetAsync(slots, 0, spmm_slot_elems(n) * sizeof(double), s);
    if (e != hipSuccess) return e;
    slots_kernel<<<(unsigned)((n + 3) / 4), 256, 0, s>>>(n, fan_ptr, fan, slots);
    return hipGetLastError();
}

hipError_t launch_spmm_tile_mask(int64_t n, const int64_t *fan_ptr, const Edge *fan, uint16_t *tile_mask,
                                 hipStream_t s) {
    hipError_t e = hipMemsetAsync(tile_mask, 0, spmm_tile_mask_elems(n) * sizeof(uint16_t), s);
    if (e != hipSuccess) return e;
    tile_mask_kernel<<<(unsigned)((n + 255) / 256), 256, 0, s>>>(n, fan_ptr, fan, tile_mask);
    return hipGetLastError();
}

hipError_t launch_spmm_fanin(int64_t n, int64_t batch, int64_t ld, const int64_t *fan_ptr, const Edge *fan,
                             const uint16_t *tile_mask, const double *slots, const float *bias, double ymax, int pattern,
                             const float *yt, float *zt, hipStream_t s, int *kind) {
    int kind_local = kKernGather;
    if (!kind) kind = &kind_local;
    *kind = kKernGather;
    if (n == 0 || batch == 0) return hipSuccess;
    if (slots && tile_mask && batch % 4 == 0 && batch >= 128) {
        *kind = kKernSlots;
        const int64_t chunks = (batch + kTiledCB - 1) / kTiledCB;
        const int64_t groups = mask_pitch(n) / kSlotNJ;
        const int64_t blocks = (groups + 7) / 8 * 8 * chunks;
        if (blocks > 0x7fffffffLL) return hipErrorInvalidValue;
        if (pattern)
            spmm_slots_kernel<true><<<(unsigned)blocks, kSlotThreads, 0, s>>>(
                n, batch, ld, (int)chunks, spmm_tile_count(n), tile_mask, slots, bias, ymax, yt, zt);
        else
            spmm_slots_kernel<false><<<(unsigned)blocks, kSlotThreads, 0, s>>>(
                n, batch, ld, (int)chunks, spmm_tile_count(n), tile_mask, slots, bias, ymax, yt, zt);
        return hipGetLastError();
    }
    if (tile_mask && batch % 4 == 0 && batch >= 128) {
        *kind = kKernTiled;
        const int64_t chunks = (batch + kTiledCB - 1) / kTiledCB;
        const int64_t groups = (n + kTiledNJ - 1) / kTiledNJ;
        const int64_t blocks = (groups + 7) / 8 * 8 * chunks;
        if (blocks > 0x7fffffffLL) return hipErrorInvalidValue;
        if (pattern)
            spmm_tiled_kernel<true><<<(unsigned)blocks, kTiledThreads, 0, s>>>(
                n, batch, ld, (int)chunks, spmm_tile_count(n), fan_ptr, tile_mask, fan, bias, ymax, yt, zt);
        else
            spmm_tiled_kernel<false><<<(unsigned)blocks, kTiledThreads, 0, s>>>(
                n, batch, ld, (int)chunks, spmm_tile_count(n), fan_ptr, tile_mask, fan, bias, ymax, yt, zt);
        return hipGetLastError();
    }
    // The narrow-chunk gather, for a batch of whole 16-byte lane loads: on wide layers whose 64-column slice
    // of Y^T (n x 256 bytes) fits an XCD's 4 MiB L2 (measured on MI355X at n = 16384, batch 4096: 0.58 ms per
    // layer against 0.93 for the kernel below; at n = 2^20, where neither slice fits, the kernel below is
    // slightly faster: 957 against 990 ms per very wide forward), and on batches under 256 from n = 4096 on,
    // where the kernel below would take one or two columns per lane (batch 64: 0.52-0.8x the time at
    // n = 32768, 0.65-0.9x at n = 4096 up to inverse sparsity 1024; below n = 4096 launches dominate and it
    // measured 1.1-1.3x)
    if (((n > 4096 && n <= 16384) || (batch < 256 && n >= 4096 && n <= (1 << 24))) && batch % 4 == 0 &&
        ld * 4 < (1 << 24)) {
        *kind = kKernNarrow;
        constexpr int V = 4;
        const int64_t chunks = (batch + kNarrowP * V - 1) / (kNarrowP * V);
        const int64_t groups = (n + 4 * (64 / kNarrowP) - 1) / (4 * (64 / kNarrowP));  // 16 neurons per workgroup
        const int64_t gpx = (groups + 7) / 8;  // per XCD
        const int64_t blocks = 8 * gpx * chunks;
        constexpr int64_t kSeg = 1ll << 23;  // a multiple of 8: a segment keeps every block's XCD
        for (int64_t base = 0; base < blocks; base += kSeg) {
            const unsigned nb = (unsigned)(blocks - base < kSeg ? blocks - base : kSeg);
            if (pattern)
                spmm_narrow_kernel<V, true><<<nb, 256, 0, s>>>(n, batch, ld, gpx, base, fan_ptr, fan, bias, ymax,
                                                                  yt, zt);
            else
                spmm_narrow_kernel<V, false><<<nb, 256, 0, s>>>(n, batch, ld, gpx, base, fan_ptr, fan, bias, ymax,
                                                                   yt, zt);
            hipError_t e = hipGetLastError();
            if (e != hipSuccess) return e;
        }
        return hipSuccess;
    }
    // Columns per lane: wide enough to keep 8 independent loads in flight, and a multiple that divides batch.
    // Columns per lane: four (one 16-byte load per lane, a 1 KiB row segment per wave) whenever the batch
    // allows; measured on MI355X at n = 4096, batch = 1024, four beat two by 1.4-1.6x at 0.1-10% density.
    int V = 1;
    if (batch % 4 == 0 && batch >= 256) V = 4;
    else if (batch % 2 == 0 && batch >= 128) V = 2;
    const int64_t chunks = (batch + 64 * V - 1) / (64 * V);
    const int64_t groups = (n + 3) / 4;
    // with 1, 2 or 4 chunks each row of 8 consecutive workgroups covers 8 / chunks groups of every chunk
    const int64_t blocks = (chunks < 8 && 8 % chunks == 0) ? (groups + 8 / chunks - 1) / (8 / chunks) * 8
                                                            : groups * chunks;
    if (chunks > 0x7fffffffLL) return hipErrorInvalidValue;
    // a launch holds at most 2^32 - 1 work-items: segments of 2^23 workgroups (a multiple of 8, so the
    // XCD of a workgroup, its linear index mod 8, is unchanged)
    constexpr int64_t kSeg = 1ll << 23;
    for (int64_t base = 0; base < blocks; base += kSeg) {
        const unsigned nb = (unsigned)(blocks - base < kSeg ? blocks - base : kSeg);
#define SDNN_GATHER(VV, PP) \
    spmm_fanin_kernel<VV, PP><<<nb, 256, 0, s>>>(n, batch, ld, (int)chunks, base, fan_ptr, fan, bias, ymax, yt, \
                                                 zt)
        switch (V * 2 + (pattern ? 1 : 0)) {
            case 8: SDNN_GATHER(4, false); break;
            case 9: SDNN_GATHER(4, true); break;
            case 4: SDNN_GATHER(2, false); break;
            case 5: SDNN_GATHER(2, true); break;
            case 3: SDNN_GATHER(1, true); break;
            default: SDNN_GATHER(1, false);
        }
#undef SDNN_GATHER
        hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    return hipGetLastError();
}

}  // namespace sdnn
