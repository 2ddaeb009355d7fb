// Dense-Y layer product for wide layers (and narrower ones with short lists), on a sample-blocked activation
// layout (Sec. III batched inference equation; Sec. IV loop body: the +.x product with the bias and ReLU fused
// into its epilogue).
//
// Layout.  The batch is cut into chunks of kBW = 32 samples; chunk c holds, for every neuron j, the 32
// values of samples 32c .. 32c + 31 in one 128-byte row: element (sample r, neuron i) sits at float
// ((r / 32) * n + i) * 32 + r % 32.  One chunk is a contiguous n x 128-byte block (128 MiB at n = 2^20),
// which the 256 MB Infinity Cache and the TLB hold while the whole chip works on it, and a row is one L2
// line.  With the neuron-major layout (n rows of `batch` samples) a chunk's slice is scattered over the
// whole activation buffer instead.
//
// Product.  Each wavefront owns eight output neurons, eight lanes each, four samples per lane (one 16-byte
// load of an input row per fan-in entry); all lanes walk their own neuron's fan-in list in step.  The eight
// neurons of a wave come from a per-layer order (set-up) that sorts every run of 4096 consecutive neurons by
// fan-in length, so the lists a wave walks together have nearly equal lengths: the common part runs without
// predication, the few remaining entries with a per-lane guard.  Products are exact in fp64 and summed in
// list order (ascending input index, as every other dense-Y kernel); bias, h and the single rounding are
// fused.  XCD-aware order: all workgroups of a chunk are dispatched before the next chunk's, and within a
// chunk XCD x (workgroup index mod 8) takes the x-th contiguous eighth of the neuron order, so the rows of
// the 4096-wide neighbourhood a block-structured layer reads stay in that XCD's L2 while the rest of the
// chunk is read from the Infinity Cache.
#include <algorithm>

#include <atomic>

#include "common.h"

namespace sdnn {

namespace {

constexpr int kBW = 32;          // samples per chunk (one 128-byte row per neuron)
constexpr int kSortSeg = 4096;   // neurons per sort segment of the processing order
#ifndef SDNN_BLOCKED_GROUPS
#define SDNN_BLOCKED_GROUPS 2
#endif
constexpr int kBWaves = 4;       // waves per workgroup of the product
constexpr int kBGroups = SDNN_BLOCKED_GROUPS;  // groups of eight neurons each wave takes in turn
constexpr int kBTile = kBWaves * kBGroups * 8;  // neurons per workgroup and chunk
#ifndef SDNN_BLOCKED_UNROLL
#define SDNN_BLOCKED_UNROLL 8
#endif
constexpr int kBUnroll = SDNN_BLOCKED_UNROLL;  // list entries per block (rows in flight per lane)
constexpr int kStageCap = 4096;  // entries of a workgroup's staged lists (32 KiB of LDS: five workgroups per CU)
constexpr int kStageAhead = 128;  // longest list the staged product walks; also how far past its region it loads

// ------------------------------------------------------------------------------------------ set-up

// Processing order: within each segment of kSortSeg consecutive neurons, by fan-in length (longest first,
// ties by index), so consecutive groups of eight have nearly equal lists.  One workgroup per segment:
// bitonic sort of 64-bit keys (complemented length, local index) in LDS.  The result is one schedule entry
// per position of the order (neuron, list length, list start), so the product reads it with one load;
// positions past n (up to the padded length) hold an empty list at the guard entry fan[nnz] and neuron -1.
__global__ __launch_bounds__(256) void blocked_order_kernel(int64_t n, int64_t padded, const int64_t *__restrict__ fan_ptr,
                                                            BlockedSched *__restrict__ sched) {
    __shared__ uint64_t key[kSortSeg];
    const int64_t base = (int64_t)blockIdx.x * kSortSeg;
    for (int t = threadIdx.x; t < kSortSeg; t += blockDim.x) {
        const int64_t j = base + t;
        if (j < n) {
            const int64_t len = fan_ptr[j + 1] - fan_ptr[j];
            const uint32_t lc = len > 0xffffffffLL ? 0u : 0xffffffffu - (uint32_t)len;
            key[t] = ((uint64_t)lc << 32) | (uint32_t)t;
        } else {
            key[t] = ~0ull;  // past the end: sorts last
        }
    }
    __syncthreads();
    for (int k = 2; k <= kSortSeg; k <<= 1) {
        for (int jj = k >> 1; jj > 0; jj >>= 1) {
            for (int t = threadIdx.x; t < kSortSeg; t += blockDim.x) {
                const int u = t ^ jj;
                if (u > t) {
                    const uint64_t a = key[t], b = key[u];
                    const bool up = (t & k) == 0;
                    if ((a > b) == up) {
                        key[t] = b;
                        key[u] = a;
                    }
                }
            }
            __syncthreads();
        }
    }
    const int64_t nnz = fan_ptr[n];
    for (int t = threadIdx.x; t < kSortSeg; t += blockDim.x) {
        const int64_t pos = base + t;
        if (pos >= padded) break;
        BlockedSched e;
        if (pos < n) {
            const int64_t j = base + (int64_t)(uint32_t)key[t];
            const int64_t len = fan_ptr[j + 1] - fan_ptr[j];
            e.j = (int32_t)j;
            e.len = (int32_t)len;
            e.e0 = len > 0 ? fan_ptr[j] : nnz;
        } else {
            e.j = -1;
            e.len = 0;
            e.e0 = nnz;
        }
        sched[pos] = e;
    }
}

// The workgroups' list regions: the padded size of each (its kBTile positions' lists, rounded up to an even
// entry count so that every region starts 16-byte aligned), then, after a scan of the sizes, one 64-thread
// workgroup per region copies its lists in schedule order (a wave prefix sum of the lengths places them),
// writes a zero entry into the padding, repoints the schedule's list starts and records the region.  The
// region's extent, its entries plus 2 * kStageAhead (the product loads kStageAhead entries past the region and
// reads up to a list's length past the last list's end), goes into region_max, or 2^30 when a list is longer
// than kStageAhead: the product stages the layer's lists only when every extent fits its LDS.
__global__ __launch_bounds__(256) void blocked_region_size_kernel(int64_t nreg, const BlockedSched *__restrict__ sched,
                                                                  int32_t *__restrict__ sizes) {
    const int64_t g = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (g >= nreg) return;
    int64_t cnt = 0;
    for (int k = 0; k < kBTile; ++k) cnt += sched[g * kBTile + k].len;
    sizes[g] = (int32_t)((cnt + 1) & ~1LL);
}

static_assert(kBTile == 64, "one wave per region in blocked_stage_kernel");

__global__ __launch_bounds__(64) void blocked_stage_kernel(const Edge *__restrict__ fan, BlockedSched *__restrict__ sched,
                                                           const int64_t *__restrict__ starts, Edge *__restrict__ stage,
                                                           BlockedRegion *__restrict__ regions, int32_t *region_max) {
    const int64_t g = blockIdx.x;
    const int lane = threadIdx.x;
    BlockedSched e = sched[g * kBTile + lane];
    int incl = e.len;
#pragma unroll
    for (int d = 1; d < 64; d <<= 1) {
        const int v = __shfl_up(incl, d);
        if (lane >= d) incl += v;
    }
    const int cnt = __shfl(incl, 63);
    int longest = e.len;
#pragma unroll
    for (int d = 1; d < 64; d <<= 1) longest = max(longest, __shfl_xor(longest, d));
    const int64_t base = starts[g];
    const int64_t dst = base + (incl - e.len);
    for (int i = 0; i < e.len; ++i) stage[dst + i] = fan[e.e0 + i];
    e.e0 = dst;
    sched[g * kBTile + lane] = e;
    if (lane == 0) {
        if (cnt & 1) stage[base + cnt] = Edge{0, 0.0f};
        BlockedRegion r;
        r.e0 = base;
        r.cnt = cnt;
        r.pad = 0;
        regions[g] = r;
        atomicMax(region_max, longest > kStageAhead ? (1 << 30) : ((cnt + 1) & ~1) + 2 * kStageAhead);
    }
}

// ------------------------------------------------------------------------------------------ product

__device__ __forceinline__ float4 load_row(const char *yc, int32_t i, uint32_t lo) {
    return *reinterpret_cast<const float4 *>(yc + ((uint32_t)i * (uint32_t)(kBW * 4) + lo));
}

template <bool kPattern>
__device__ __forceinline__ void fma4(const float4 &y, float w, double (&acc)[4], uint32_t (&hit)[4]) {
    const double wd = (double)w;
    acc[0] = __builtin_fma((double)y.x, wd, acc[0]);
    acc[1] = __builtin_fma((double)y.y, wd, acc[1]);
    acc[2] = __builtin_fma((double)y.z, wd, acc[2]);
    acc[3] = __builtin_fma((double)y.w, wd, acc[3]);
    if constexpr (kPattern) {
        hit[0] |= __float_as_uint(y.x);
        hit[1] |= __float_as_uint(y.y);
        hit[2] |= __float_as_uint(y.z);
        hit[3] |= __float_as_uint(y.w);
    }
}

// K entries t .. t + K - 1 of the lane's staged list: the K row loads are issued together, then the K
// products added in list order.  Entries past the list's end (up to kStageAhead of them: the next lists, or
// what was loaded after the region, all finite) load from an offset past the chunk, which reads zero without a
// memory access, so their products add zero.  No marked entry lies within a list's length.
template <int K, bool kPattern>
__device__ __forceinline__ void staged_block(const Edge *lst, int t, int len, __amdgpu_buffer_rsrc_t rs,
                                             uint32_t lo, uint32_t nrec, double (&acc)[4], uint32_t (&hit)[4]) {
    static_assert(K <= kBUnroll, "rows in flight per lane");
    float4 y[K];
    float w[K];
#pragma unroll
    for (int u = 0; u < K; ++u) {
        const Edge e = lst[t + u];
        const bool in = t + u < len;
        w[u] = e.w;
        y[u] = __builtin_bit_cast(
            float4, __builtin_amdgcn_raw_buffer_load_b128(rs, in ? (uint32_t)e.idx * (uint32_t)(kBW * 4) + lo : nrec, 0, 0));
    }
#pragma unroll
    for (int u = 0; u < K; ++u) fma4<kPattern>(y[u], w[u], acc, hit);
}

// Orders LDS writes and reads among the lanes of one wave (no other wave touches the region).
__device__ __forceinline__ void wave_lds_sync() {
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

// Wave-uniform minimum and maximum of a value that is equal within each group of eight lanes.
__device__ __forceinline__ void group8_min_max(int v, int &mn, int &mx) {
    int a = v, b = v;
#pragma unroll
    for (int off = 8; off < 64; off <<= 1) {
        a = min(a, __shfl_xor(a, off));
        b = max(b, __shfl_xor(b, off));
    }
    mn = __builtin_amdgcn_readfirstlane(a);
    mx = __builtin_amdgcn_readfirstlane(b);
}

// grid: nchunks * 8 * gpx workgroups of kBWaves waves; gpx = workgroups per XCD per chunk, tiles = workgroups
// per chunk (ceil(n / kBTile)).  Each wave takes kBGroups groups of eight consecutive positions of the
// schedule in turn (the next group's schedule entry is loaded while the current group runs).  A group's lists
// are walked in blocks of eight entries: the eight lanes of a neuron load the block's entries with one 8-byte
// load each (entry t + sub, clamped to the list's last entry), pass them through the wave's LDS slot, and
// read all eight back (a broadcast read), so the memory path carries each entry once per neuron rather than
// once per lane; the next block's entries are loaded while the current block's rows are in flight.
#ifndef SDNN_BLOCKED_WAVES_PER_EU
#define SDNN_BLOCKED_WAVES_PER_EU 1
#endif
// kStaged: the workgroup's lists sit in one region of the staged copy (`fan` then points to that copy); the
// workgroup loads the whole region into LDS at once (16 bytes per lane, straight to LDS) and reads every
// entry from there, so the only global loads of the loop are the rows.  Measured on the very wide layer: the
// per-block entry loads from HBM sat on each block's critical path (94 -> 79 ms per layer without them).
template <bool kPattern, bool kStaged>
__global__ __launch_bounds__(kBWaves * 64) __attribute__((amdgpu_waves_per_eu(SDNN_BLOCKED_WAVES_PER_EU, 8))) void spmm_blocked_kernel(
    int64_t n, int64_t gpx, int64_t tiles, int64_t nchunk, int xcd_chunks, const BlockedSched *__restrict__ sched,
    const Edge *__restrict__ fan, const BlockedRegion *__restrict__ regions, const uint32_t *__restrict__ nzrows,
    int64_t nz_words, const float *__restrict__ bias, double ymax, const float *__restrict__ yb, float *__restrict__ zb) {
    __shared__ __align__(16) Edge ent[kStaged ? kStageCap : kBWaves * kBUnroll * 8];
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int q = lane >> 3, sub = lane & 7;
    const int64_t b = blockIdx.x;
    const int64_t xcd = b & 7, local = b >> 3;
    int64_t c, g;
    if (xcd_chunks) {
        // whole chunks per XCD (chunk c on XCD c mod 8, its workgroups in schedule order), for chunks small
        // enough that one, with the next, stays in that XCD's L2
        c = xcd + 8 * (local / tiles);
        g = local - (local / tiles) * tiles;
        if (c >= nchunk) return;
    } else {
        c = local / gpx;
        g = xcd * gpx + (local - c * gpx);
        if (g >= tiles) return;
    }
    const char *yc = reinterpret_cast<const char *>(yb + c * n * kBW);
    float *zc = zb + c * n * kBW + sub * 4;
    const uint32_t lo = (uint32_t)sub * 16u;
    const BlockedSched *sp = sched + (g * kBWaves + wave) * (kBGroups * 8) + q;
    if constexpr (kStaged) {
        // the region (padded to an even count, 16-byte aligned) and more than kStageAhead entries after it (the
        // next regions, or the zeroed tail of the copy): a lane reads at most to index mx of its list (a tail
        // block's last slot), mx <= kStageAhead, so never past entry cnt + kStageAhead.  Each load instruction
        // moves 128 entries; the last ends before entry cnt + 2 * kStageAhead, within ent (the region's
        // extent, checked at set-up, is at most kStageCap) and within the copy (zeroed 2 * kStageAhead entries
        // past its last region)
        const BlockedRegion rg = regions[g];
        const Edge *src = fan + rg.e0;
        for (int base = wave * 128; base <= rg.cnt + kStageAhead; base += kBWaves * 128)
            __builtin_amdgcn_global_load_lds(reinterpret_cast<const void *>(src + base + 2 * lane),
                                             (__attribute__((address_space(3))) void *)(&ent[base]), 16,
                                             0, 0);
        __builtin_amdgcn_s_waitcnt(0x0F70);  // vmcnt(0): this wave's loads into LDS have landed
        __syncthreads();
        if (nzrows) {
            // a sparse input: entries whose input row is zero in this chunk are marked (bit 31 of the index;
            // n <= 2^24) and read nothing below
            // Eight entries per thread at a time, their map words loaded together (one round trip per eight
            // entries rather than per entry: the map is read at the start of every workgroup)
            const uint32_t *nzc = nzrows + c * nz_words;
            constexpr int kMarkU = 8;
            for (int k0 = threadIdx.x; k0 < rg.cnt; k0 += kMarkU * kBWaves * 64) {
                int32_t iv[kMarkU];
                uint32_t wv[kMarkU];
#pragma unroll
                for (int u = 0; u < kMarkU; ++u) {
                    const int k = k0 + u * kBWaves * 64;
                    iv[u] = k < rg.cnt ? ent[k].idx : 0;
                }
#pragma unroll
                for (int u = 0; u < kMarkU; ++u) wv[u] = nzc[iv[u] >> 5];
#pragma unroll
                for (int u = 0; u < kMarkU; ++u) {
                    const int k = k0 + u * kBWaves * 64;
                    if (k < rg.cnt && !((wv[u] >> (iv[u] & 31)) & 1u)) ent[k].idx = (int32_t)((uint32_t)iv[u] | 0x80000000u);
                }
            }
            __syncthreads();
        }
        // rows through buffer loads: an entry past its list's end, or marked, gets an offset past the chunk,
        // which reads zero without a memory access
        const uint32_t nrec = (uint32_t)n * (uint32_t)(kBW * 4);
        const __amdgpu_buffer_rsrc_t rs = __builtin_amdgcn_make_buffer_rsrc((void *)yc, (short)0, (int)nrec, 0x00020000);
        for (int gi = 0; gi < kBGroups; ++gi) {
            const BlockedSched cur = sp[8 * gi];
            int len = cur.len;
            Edge *lst = ent + (cur.e0 - rg.e0);
            int mn, mx;
            group8_min_max(len, mn, mx);
            if (nzrows) {
                // drop the marked entries: each neuron's 8 lanes move its unmarked ones to the front of its
                // list, in order (reads of a block happen before its writes, which land at or before them)
                int kept = 0;
                for (int t = 0; t < mx; t += 8) {
                    const int tt = t + sub;
                    Edge e;
                    e.idx = -1;
                    e.w = 0.0f;
                    if (tt < len) e = lst[tt];
                    const bool keep = tt < len && e.idx >= 0;
                    const uint32_t seg = (uint32_t)(__ballot(keep) >> (8 * q)) & 0xffu;
                    wave_lds_sync();
                    if (keep) lst[kept + __popc(seg & ((1u << sub) - 1u))] = e;
                    kept += __popc(seg);
                    wave_lds_sync();
                }
                len = kept;
                group8_min_max(len, mn, mx);
            }
            double acc[4] = {0.0, 0.0, 0.0, 0.0};
            uint32_t hit[4] = {0u, 0u, 0u, 0u};
            int t = 0;
            for (; t + kBUnroll <= mx; t += kBUnroll) staged_block<kBUnroll, kPattern>(lst, t, len, rs, lo, nrec, acc, hit);
            // the last mx - t (< kBUnroll, the same for the whole wave) entries: one block of the smallest even
            // size that covers them, since loads past the longest list still occupy the address and data units
            const int rem = mx - t;
            if (rem > 6)
                staged_block<8, kPattern>(lst, t, len, rs, lo, nrec, acc, hit);
            else if (rem > 4)
                staged_block<6, kPattern>(lst, t, len, rs, lo, nrec, acc, hit);
            else if (rem > 2)
                staged_block<4, kPattern>(lst, t, len, rs, lo, nrec, acc, hit);
            else if (rem > 0)
                staged_block<2, kPattern>(lst, t, len, rs, lo, nrec, acc, hit);
            if (cur.j >= 0) {
                const double bd = (double)bias[cur.j];
                float4 out;
                out.x = (kPattern && (hit[0] & 0x7fffffffu) == 0u) ? 0.0f : activate(acc[0] + bd, ymax);
                out.y = (kPattern && (hit[1] & 0x7fffffffu) == 0u) ? 0.0f : activate(acc[1] + bd, ymax);
                out.z = (kPattern && (hit[2] & 0x7fffffffu) == 0u) ? 0.0f : activate(acc[2] + bd, ymax);
                out.w = (kPattern && (hit[3] & 0x7fffffffu) == 0u) ? 0.0f : activate(acc[3] + bd, ymax);
                *reinterpret_cast<float4 *>(zc + (int64_t)cur.j * kBW) = out;
            }
        }
        return;
    }
    Edge *slot = &ent[wave * kBUnroll * 8];
    BlockedSched cur = sp[0];
    for (int gi = 0; gi < kBGroups; ++gi) {
        const BlockedSched nxt = sp[8 * min(gi + 1, kBGroups - 1)];
        const float bj = bias[cur.j >= 0 ? cur.j : 0];
        const int len = cur.len;
        const Edge *lst = fan + cur.e0;
        const int last = len > 0 ? len - 1 : 0;
        int mn, mx;
        group8_min_max(len, mn, mx);
        double acc[4] = {0.0, 0.0, 0.0, 0.0};
        uint32_t hit[4] = {0u, 0u, 0u, 0u};
        constexpr int kR = kBUnroll / 8;  // entries each lane loads per block
        Edge mine[kR];
#pragma unroll
        for (int r = 0; r < kR; ++r) mine[r] = lst[min(8 * r + sub, last)];
        for (int t = 0; t < mx; t += kBUnroll) {
            // this block's entries of the lane's neuron: entry t + 8r + u at slot[64r + 8q + u]
#pragma unroll
            for (int r = 0; r < kR; ++r) slot[64 * r + lane] = mine[r];
            wave_lds_sync();
            Edge e[kBUnroll];
#pragma unroll
            for (int r = 0; r < kR; ++r)
#pragma unroll
                for (int u = 0; u < 8; ++u) e[8 * r + u] = slot[64 * r + q * 8 + u];
            wave_lds_sync();
            float4 y[kBUnroll];
#pragma unroll
            for (int u = 0; u < kBUnroll; ++u) y[u] = load_row(yc, e[u].idx, lo);
#pragma unroll
            for (int r = 0; r < kR; ++r) mine[r] = lst[min(t + kBUnroll + 8 * r + sub, last)];  // the next block's
            __builtin_amdgcn_sched_barrier(0);
            if (t + kBUnroll <= mn) {
#pragma unroll
                for (int u = 0; u < kBUnroll; ++u) fma4<kPattern>(y[u], e[u].w, acc, hit);
            } else {
                // entries past a lane's end add a zeroed input, which leaves its sum unchanged
#pragma unroll
                for (int u = 0; u < kBUnroll; ++u) {
                    float4 yv = y[u];
                    if (t + u >= len) yv = make_float4(0.f, 0.f, 0.f, 0.f);
                    fma4<kPattern>(yv, e[u].w, acc, hit);
                }
            }
        }
        if (cur.j >= 0) {
            const double bd = (double)bj;
            float4 out;
            out.x = (kPattern && (hit[0] & 0x7fffffffu) == 0u) ? 0.0f : activate(acc[0] + bd, ymax);
            out.y = (kPattern && (hit[1] & 0x7fffffffu) == 0u) ? 0.0f : activate(acc[1] + bd, ymax);
            out.z = (kPattern && (hit[2] & 0x7fffffffu) == 0u) ? 0.0f : activate(acc[2] + bd, ymax);
            out.w = (kPattern && (hit[3] & 0x7fffffffu) == 0u) ? 0.0f : activate(acc[3] + bd, ymax);
            *reinterpret_cast<float4 *>(zc + (int64_t)cur.j * kBW) = out;
        }
        cur = nxt;
    }
}

// ------------------------------------------------------------------------------------------ format changes

// Sparse rows -> blocked activations.  One workgroup per (chunk, part of the neurons); 16 threads per sample.
// The part is walked in ranges of kDensR neurons: the range's 32 x kDensR tile is zeroed in LDS, each
// sample's entries that fall in the range are written into it (the sample's cursor moves forward through
// its sorted row), and the tile is stored as kDensR whole 128-byte rows.  The first entry of the part is
// found by a binary search per sample.  Row extents are checked as in the other format changes, and the
// part-0 workgroups also check every column of their samples.
constexpr int kDensR = 256;
constexpr int kDensThreads = 512;

__global__ __launch_bounds__(kDensThreads) void densify_blocked_kernel(
    int64_t n, int64_t batch, int64_t part_len, const int64_t *__restrict__ in_row_ptr,
    const int32_t *__restrict__ in_cnt, const int32_t *__restrict__ in_col, const float *__restrict__ in_val,
    float *__restrict__ yb, uint32_t *__restrict__ nzrows, int64_t nz_words, uint32_t *err) {
    __shared__ __align__(16) float tile[kDensR * kBW];
    __shared__ uint32_t rowbits[kDensR / 32];  // rows of the range that receive a nonzero
    const int64_t nparts = (n + part_len - 1) / part_len;
    const int64_t c = blockIdx.x / nparts, part = blockIdx.x % nparts;
    const int s = threadIdx.x >> 4, k = threadIdx.x & 15;  // sample of the chunk, thread within the sample
    const int64_t r = c * kBW + s;
    const int64_t a0 = part * part_len, a1 = min(n, a0 + part_len);
    int64_t rb = 0, re = 0;
    if (r < batch) {
        if (in_row_ptr) {
            const int64_t nnz = (in_col && in_val) ? in_row_ptr[batch] : 0;
            rb = in_row_ptr[r];
            re = in_row_ptr[r + 1];
            if (rb < 0 || re < rb || re - rb > n || re > nnz) {
                if (k == 0 && part == 0) atomicOr(err, 1u);
                rb = re = 0;
            }
        } else {
            rb = r * n;
            re = rb + in_cnt[r];
        }
    }
    if (part == 0)
        for (int64_t t = rb + k; t < re; t += 16) {
            const int32_t i = in_col[t];
            if (i < 0 || i >= n) atomicOr(err, 1u);
        }
    // first entry with column >= a0 (columns ascending within a row)
    int64_t lo = rb, hi = re;
    while (lo < hi) {
        const int64_t mid = (lo + hi) >> 1;
        if (in_col[mid] < a0) lo = mid + 1;
        else hi = mid;
    }
    int64_t cur = lo;  // equal across the sample's 16 threads
    for (int64_t a = a0; a < a1; a += kDensR) {
        const int64_t ra = min<int64_t>(kDensR, a1 - a);
        for (int t = threadIdx.x; t < kDensR * kBW; t += kDensThreads) tile[t] = 0.0f;
        if (threadIdx.x < kDensR / 32) rowbits[threadIdx.x] = 0u;
        __syncthreads();
        // entries of this range: [cur, next) with next the first column >= a + kDensR
        int64_t next = cur;
        for (;;) {
            const int64_t t = next + k;
            const int32_t i = t < re ? in_col[t] : 0x7fffffff;
            const bool in = i < a + ra;
            if (in && i >= a) {
                const float v = in_val[t];
                tile[(i - a) * kBW + s] = v;
                if (nzrows && v != 0.0f) atomicOr(&rowbits[(i - a) >> 5], 1u << ((i - a) & 31));
            }
            // the 16 threads of a sample share one ballot segment: advance past the leading run that is in range
            const uint64_t m = __ballot(in);
            const uint32_t seg = (uint32_t)(m >> (threadIdx.x & 48)) & 0xffffu;
            const int run = __builtin_ctz(~seg | 0x10000u);
            next += run;
            if (run < 16) break;
        }
        cur = next;
        __syncthreads();
        // bit i of the chunk's map: row a + i holds a nonzero
        if (nzrows && threadIdx.x < kDensR / 32) nzrows[c * nz_words + (a >> 5) + threadIdx.x] = rowbits[threadIdx.x];
        // with the map, only the rows that hold a nonzero are stored: the product that takes the map reads no
        // other row, so the zero rows (about half of them at 2% density) cost no write
        float4 *dst = reinterpret_cast<float4 *>(yb + (c * n + a) * kBW);
        const float4 *srct = reinterpret_cast<const float4 *>(tile);
        for (int t = threadIdx.x; t < ra * (kBW / 4); t += kDensThreads) {
            const int row = t / (kBW / 4);
            if (!nzrows || ((rowbits[row >> 5] >> (row & 31)) & 1u)) dst[t] = srct[t];
        }
        __syncthreads();
    }
}

// Blocked activations -> CSR rows, in three steps.  Count: one wavefront per (chunk, part of kPackR
// neurons) counts each sample's nonzeros in the part (lane = neuron, one ballot per sample).  Scan: per
// sample, the part counts become offsets within the row and the row total goes to cnt.  Pack: one
// workgroup per (chunk, part) moves the part's 32 x kPackR values into LDS transposed, and each wave, for
// each of its samples, compacts the survivors in ascending neuron order into its LDS area and then writes
// the run at row_ptr[r] + offset with whole-wave stores aligned to 128-byte lines (a run of a few hundred
// entries is written in whole lines but for its two ends).
constexpr int kPackR = 512;
constexpr int kTileLd = kBW + 1;  // LDS row pitch of a transposed 64 x 32 tile (conflict-free column reads)

// Rows a .. a + 63 of chunk c (rows from a1 on read as zero) into v: lane l gets row a + l, all 32 samples.
// The global reads are coalesced (each instruction takes eight whole rows, 1 KiB) and the transpose goes
// through the wave's LDS tile.
__device__ __forceinline__ void load_tile(const float *yb, int64_t c, int64_t n, int64_t a, int64_t a1, float *tile,
                                          int lane, float (&v)[kBW]) {
    const float4 *src = reinterpret_cast<const float4 *>(yb + (c * n + a) * kBW);
    const int64_t rows = a1 - a < 64 ? a1 - a : 64;
#pragma unroll
    for (int u = 0; u < 8; ++u) {
        const int r = 8 * u + (lane >> 3);
        float4 f = make_float4(0.f, 0.f, 0.f, 0.f);
        if (r < rows) f = src[64 * u + lane];
        float *d = tile + r * kTileLd + (lane & 7) * 4;
        d[0] = f.x;
        d[1] = f.y;
        d[2] = f.z;
        d[3] = f.w;
    }
    wave_lds_sync();
#pragma unroll
    for (int s = 0; s < kBW; ++s) v[s] = tile[lane * kTileLd + s];
    wave_lds_sync();
}

__global__ __launch_bounds__(256) void blocked_count_kernel(int64_t n, int64_t batch, int64_t nparts,
                                                            const float *__restrict__ yb, int32_t *__restrict__ pcnt) {
    __shared__ float tiles[4][64 * kTileLd];
    const int lane = threadIdx.x & 63;
    const int64_t w = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
    const int64_t nchunks = (batch + kBW - 1) / kBW;
    if (w >= nchunks * nparts) return;
    float *tile = tiles[threadIdx.x >> 6];
    const int64_t c = w / nparts, part = w % nparts;
    const int64_t a0 = part * kPackR, a1 = min(n, a0 + kPackR);
    int cnt[kBW];
#pragma unroll
    for (int s = 0; s < kBW; ++s) cnt[s] = 0;
    for (int64_t a = a0; a < a1; a += 64) {
        float v[kBW];
        load_tile(yb, c, n, a, a1, tile, lane, v);
#pragma unroll
        for (int s = 0; s < kBW; ++s) cnt[s] += __popcll(__ballot(v[s] != 0.0f));
    }
#pragma unroll
    for (int s = 0; s < kBW; ++s) {
        const int64_t r = c * kBW + s;
        if (lane == s && r < batch) pcnt[part * batch + r] = cnt[s];
    }
}

// per sample: part counts -> exclusive offsets within the row (in place); row totals -> cnt
__global__ __launch_bounds__(256) void blocked_scan_kernel(int64_t batch, int64_t nparts, int32_t *__restrict__ pcnt,
                                                           int32_t *__restrict__ cnt) {
    const int64_t r = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (r >= batch) return;
    int32_t run = 0;
    for (int64_t p = 0; p < nparts; ++p) {
        const int32_t v = pcnt[p * batch + r];
        pcnt[p * batch + r] = run;
        run += v;
    }
    cnt[r] = run;
}

constexpr int kPackThreads = 1024;
constexpr int kPackLd = kPackR + 1;  // LDS pitch (floats) of one sample's values in the transposed part
constexpr size_t kPackLds = (size_t)kBW * kPackLd * sizeof(float) + (size_t)(kPackThreads / 64) * kPackR * 8;

__global__ __launch_bounds__(kPackThreads) void blocked_pack_kernel(int64_t n, int64_t batch, int64_t nparts,
                                                                    const float *__restrict__ yb,
                                                                    const int32_t *__restrict__ poff,
                                                                    const int64_t *__restrict__ row_ptr,
                                                                    int32_t *__restrict__ out_col,
                                                                    float *__restrict__ out_val) {
    extern __shared__ __align__(16) float pack_lds[];
    float *in = pack_lds;  // [kBW][kPackLd]: sample s's value of neuron a0 + j at s * kPackLd + j
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    int32_t *scol = reinterpret_cast<int32_t *>(pack_lds + kBW * kPackLd) + wave * 2 * kPackR;
    float *sval = reinterpret_cast<float *>(scol + kPackR);
    const int64_t c = blockIdx.x / nparts, part = blockIdx.x % nparts;
    const int64_t a0 = part * kPackR;
    const int rows = (int)(n - a0 < kPackR ? n - a0 : kPackR);
    // the part's rows (32 samples each, 128 bytes) as 16-byte pieces, coalesced; rows past n read as zero
    const float4 *src = reinterpret_cast<const float4 *>(yb + (c * n + a0) * kBW);
    for (int t = tid; t < kPackR * (kBW / 4); t += kPackThreads) {
        const int row = t / (kBW / 4), q = (t % (kBW / 4)) * 4;
        float4 f = make_float4(0.f, 0.f, 0.f, 0.f);
        if (row < rows) f = src[t];
        in[(q + 0) * kPackLd + row] = f.x;
        in[(q + 1) * kPackLd + row] = f.y;
        in[(q + 2) * kPackLd + row] = f.z;
        in[(q + 3) * kPackLd + row] = f.w;
    }
    __syncthreads();
    for (int s = wave; s < kBW; s += kPackThreads / 64) {
        const int64_t r = c * kBW + s;
        if (r >= batch) break;  // uniform in the wave; later samples are past the end too
        int cnt = 0;
        for (int j0 = 0; j0 < kPackR; j0 += 64) {
            const float v = in[s * kPackLd + j0 + lane];
            const bool keep = v != 0.0f;
            const uint64_t m = __ballot(keep);
            if (keep) {
                const int o = cnt + lane_rank(m);
                scol[o] = (int32_t)(a0 + j0 + lane);
                sval[o] = v;
            }
            cnt += __popcll(m);
        }
        wave_lds_sync();
        const int64_t base = row_ptr[r] + poff[part * batch + r];
        // entry e goes to base + e; the lanes start at the 128-byte line holding base, so each store
        // instruction covers two whole lines
        const int lead = (int)(base & 31);
        for (int e = lane - lead; e < cnt; e += 64) {
            if (e >= 0) {
                out_col[base + e] = scol[e];
                out_val[base + e] = sval[e];
            }
        }
        wave_lds_sync();  // the run's LDS area is rewritten for the wave's next sample
    }
}

// Batch-major rows (batch x n, row pitch ld_in) <-> blocked.  One workgroup per (chunk, 128 neurons): the
// 32 x 128 tile goes through LDS; samples past the batch end are written as zeros.
constexpr int kTrN = 128;

__global__ __launch_bounds__(256) void to_blocked_kernel(int64_t n, int64_t batch, int64_t ld_in,
                                                         const float *__restrict__ y, float *__restrict__ yb) {
    __shared__ float tile[kBW][kTrN + 1];
    const int64_t ntiles = (n + kTrN - 1) / kTrN;
    const int64_t c = blockIdx.x / ntiles, j0 = (blockIdx.x % ntiles) * kTrN;
    for (int t = threadIdx.x; t < kBW * kTrN; t += 256) {
        const int s = t / kTrN, jj = t % kTrN;
        const int64_t r = c * kBW + s, j = j0 + jj;
        tile[s][jj] = (r < batch && j < n) ? y[r * ld_in + j] : 0.0f;
    }
    __syncthreads();
    for (int t = threadIdx.x; t < kBW * kTrN; t += 256) {
        const int jj = t / kBW, s = t % kBW;
        const int64_t j = j0 + jj;
        if (j < n) yb[(c * n + j) * kBW + s] = tile[s][jj];
    }
}

__global__ __launch_bounds__(256) void from_blocked_kernel(int64_t n, int64_t batch, int64_t ld_out,
                                                           const float *__restrict__ yb, float *__restrict__ y) {
    __shared__ float tile[kBW][kTrN + 1];
    const int64_t ntiles = (n + kTrN - 1) / kTrN;
    const int64_t c = blockIdx.x / ntiles, j0 = (blockIdx.x % ntiles) * kTrN;
    for (int t = threadIdx.x; t < kBW * kTrN; t += 256) {
        const int jj = t / kBW, s = t % kBW;
        const int64_t j = j0 + jj;
        tile[s][jj] = j < n ? yb[(c * n + j) * kBW + s] : 0.0f;
    }
    __syncthreads();
    for (int t = threadIdx.x; t < kBW * kTrN; t += 256) {
        const int s = t / kTrN, jj = t % kTrN;
        const int64_t r = c * kBW + s, j = j0 + jj;
        if (r < batch && j < n) y[r * ld_out + j] = tile[s][jj];
    }
}

}  // namespace

int64_t blocked_chunks(int64_t batch) { return (batch + kBW - 1) / kBW; }

size_t blocked_elems(int64_t n, int64_t batch) { return (size_t)blocked_chunks(batch) * kBW * (size_t)n; }

bool blocked_wanted(int64_t n, int64_t batch) { return n > 4096 && n <= (1 << 24) && batch >= 256; }

bool blocked_only(int64_t n) { return n > 16384 && n <= (1 << 24); }

// Up to 16384 neurons the blocked product pays only on short lists (measured at n 16384, 32 entries per
// neuron, batch 4096: 0.43 ms per layer against 0.53 in the narrow-chunk gather); dense-ish layers keep the
// scalar-register and tiled products, so only layers averaging at most 48 entries per neuron get the schedule.
bool blocked_planned(int64_t n, int64_t nnz) { return blocked_only(n) || (n > 4096 && nnz <= 48 * n); }

size_t blocked_pack_elems(int64_t n, int64_t batch) { return (size_t)((n + kPackR - 1) / kPackR) * (size_t)batch; }

int64_t blocked_sched_elems(int64_t n) { return (n + kBTile - 1) / kBTile * kBTile; }

hipError_t launch_blocked_order(int64_t n, const int64_t *fan_ptr, BlockedSched *sched, hipStream_t s) {
    if (n == 0) return hipSuccess;
    const int64_t padded = blocked_sched_elems(n);
    blocked_order_kernel<<<(unsigned)((padded + kSortSeg - 1) / kSortSeg), 256, 0, s>>>(n, padded, fan_ptr, sched);
    return hipGetLastError();
}

int64_t blocked_regions(int64_t n) { return blocked_sched_elems(n) / kBTile; }

int64_t blocked_nz_words(int64_t n) { return (n + kDensR - 1) / kDensR * (kDensR / 32); }

size_t blocked_stage_elems(int64_t n, int64_t nnz) {
    return (size_t)nnz + (size_t)blocked_regions(n) + 2 * kStageAhead;
}

int32_t blocked_stage_cap() { return kStageCap; }

hipError_t launch_blocked_stage(int64_t n, int64_t nnz, const Edge *fan, BlockedSched *sched, Edge *stage,
                                BlockedRegion *regions, int32_t *sizes, int64_t *starts, int64_t *scan_tmp,
                                int32_t *region_max, hipStream_t s) {
    if (n == 0) return hipSuccess;
    const int64_t nreg = blocked_regions(n);
    blocked_region_size_kernel<<<(unsigned)((nreg + 255) / 256), 256, 0, s>>>(nreg, sched, sizes);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    e = launch_exclusive_scan_i32_to_i64(nreg, sizes, starts, scan_tmp, s);
    if (e != hipSuccess) return e;
    // the regions end between nnz and nnz + nreg entries (one padding entry at most per region): zeroing from
    // nnz to the end of the copy leaves zeros in the 2 * kStageAhead entries after the last region, which the
    // staging loads of the last regions may read
    e = hipMemsetAsync(stage + nnz, 0, ((size_t)nreg + 2 * kStageAhead) * sizeof(Edge), s);
    if (e != hipSuccess) return e;
    e = hipMemsetAsync(region_max, 0, sizeof(int32_t), s);
    if (e != hipSuccess) return e;
    blocked_stage_kernel<<<(unsigned)nreg, 64, 0, s>>>(fan, sched, starts, stage, regions, region_max);
    return hipGetLastError();
}

hipError_t launch_spmm_blocked(int64_t n, int64_t batch, const BlockedSched *sched, const Edge *fan,
                               const BlockedRegion *regions, const uint32_t *nzrows, const float *bias, double ymax,
                               int pattern, const float *yb, float *zb, hipStream_t s) {
    if (n == 0 || batch == 0) return hipSuccess;
    if (n > (1 << 24)) return hipErrorInvalidValue;  // 32-bit row offsets within a chunk
    const int64_t nchunks = blocked_chunks(batch);
    const int64_t groups = (n + kBTile - 1) / kBTile;
    const int64_t gpx = (groups + 7) / 8;
    // chunks of at most 2 MiB (n <= 16384) go whole to one XCD each (measured on n = 16384, batch 4096: all 8
    // XCDs sharing each chunk keep about 2.5 chunks in flight, more than one XCD's 4 MB L2 holds); wider
    // chunks are split over the XCDs as above
    const int xcd_chunks = n * kBW * 4 <= (int64_t(2) << 20) ? 1 : 0;
    // workgroups per chunk (n <= 2^24: at most 2^19 + 8); in the XCD-chunk order 8 chunks are launched as a
    // unit, the workgroups of missing chunks of the last unit return at once
    const int64_t per_chunk = xcd_chunks ? groups : 8 * gpx;
    const int64_t unit = xcd_chunks ? 8 : 1;
    // launches of whole units, at most 2^23 workgroups each; every launch numbers its workgroups from 0, so
    // the data pointers move to its first chunk
    const int64_t chunks_per_launch = std::max<int64_t>(unit, (int64_t(1) << 23) / (per_chunk * unit) * unit);
    for (int64_t c0 = 0; c0 < nchunks; c0 += chunks_per_launch) {
        const int64_t nc = std::min(chunks_per_launch, nchunks - c0);
        const unsigned nb = (unsigned)((nc + unit - 1) / unit * unit * per_chunk);
        const float *y0 = yb + c0 * n * kBW;
        float *z0 = zb + c0 * n * kBW;
        const int64_t words = blocked_nz_words(n);
        const uint32_t *nz0 = (regions && nzrows) ? nzrows + c0 * words : nullptr;
        if (regions) {
            if (pattern)
                spmm_blocked_kernel<true, true><<<nb, kBWaves * 64, 0, s>>>(n, gpx, groups, nc, xcd_chunks, sched, fan, regions, nz0, words, bias, ymax, y0, z0);
            else
                spmm_blocked_kernel<false, true><<<nb, kBWaves * 64, 0, s>>>(n, gpx, groups, nc, xcd_chunks, sched, fan, regions, nz0, words, bias, ymax, y0, z0);
        } else if (pattern) {
            spmm_blocked_kernel<true, false><<<nb, kBWaves * 64, 0, s>>>(n, gpx, groups, nc, xcd_chunks, sched, fan, nullptr, nullptr, 0, bias, ymax, y0, z0);
        } else {
            spmm_blocked_kernel<false, false><<<nb, kBWaves * 64, 0, s>>>(n, gpx, groups, nc, xcd_chunks, sched, fan, nullptr, nullptr, 0, bias, ymax, y0, z0);
        }
        hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    return hipSuccess;
}

hipError_t launch_densify_blocked(int64_t n, int64_t batch, const int64_t *in_row_ptr, const int32_t *in_cnt,
                                  const int32_t *in_col, const float *in_val, float *yb, uint32_t *nzrows, uint32_t *err,
                                  hipStream_t s) {
    if (n == 0 || batch == 0) return hipSuccess;
    const int64_t nchunks = blocked_chunks(batch);
    // enough parts for about eight workgroups per CU on the widest layers, whole ranges per part
    int64_t part_len = (n + 7) / 8;
    part_len = (part_len + kDensR - 1) / kDensR * kDensR;
    const int64_t nparts = (n + part_len - 1) / part_len;
    const int64_t blocks = nchunks * nparts;
    if (blocks > 0x7fffffffLL) return hipErrorInvalidValue;
    densify_blocked_kernel<<<(unsigned)blocks, kDensThreads, 0, s>>>(n, batch, part_len, in_row_ptr, in_cnt, in_col,
                                                                      in_val, yb, nzrows, blocked_nz_words(n), err);
    return hipGetLastError();
}

hipError_t launch_blocked_to_csr(int64_t n, int64_t batch, const float *yb, int32_t *pcnt, int32_t *cnt,
                                 int64_t *row_ptr, int64_t *scan_tmp, int32_t *out_col, float *out_val, hipStream_t s) {
    if (batch == 0) return hipSuccess;
    const int64_t nparts = (n + kPackR - 1) / kPackR;
    const int64_t waves = blocked_chunks(batch) * nparts;
    const int64_t blocks = (waves + 3) / 4;
    if (blocks > 0x7fffffffLL) return hipErrorInvalidValue;
    blocked_count_kernel<<<(unsigned)blocks, 256, 0, s>>>(n, batch, nparts, yb, pcnt);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    blocked_scan_kernel<<<(unsigned)((batch + 255) / 256), 256, 0, s>>>(batch, nparts, pcnt, cnt);
    e = hipGetLastError();
    if (e != hipSuccess) return e;
    e = launch_exclusive_scan_i32_to_i64(batch, cnt, row_ptr, scan_tmp, s);
    if (e != hipSuccess) return e;
    // the pack's LDS exceeds the default dynamic limit: raise it once per device (bit d of attr_devices;
    // devices beyond 63 set it on every call)
    static std::atomic<unsigned long long> attr_devices{0};
    int dev = 0;
    e = hipGetDevice(&dev);
    if (e != hipSuccess) return e;
    const unsigned long long bit = dev >= 0 && dev < 64 ? 1ull << dev : 0ull;
    if (!bit || !(attr_devices.load(std::memory_order_acquire) & bit)) {
        e = hipFuncSetAttribute((const void *)blocked_pack_kernel, hipFuncAttributeMaxDynamicSharedMemorySize,
                                (int)kPackLds);
        if (e != hipSuccess) return e;
        attr_devices.fetch_or(bit, std::memory_order_release);
    }
    const int64_t groups = blocked_chunks(batch) * nparts;
    if (groups > 0x7fffffffLL) return hipErrorInvalidValue;
    blocked_pack_kernel<<<(unsigned)groups, kPackThreads, kPackLds, s>>>(n, batch, nparts, yb, pcnt, row_ptr, out_col,
                                                                        out_val);
    return hipGetLastError();
}

hipError_t launch_to_blocked(int64_t n, int64_t batch, int64_t ld_in, const float *y, float *yb, hipStream_t s) {
    if (n == 0 || batch == 0) return hipSuccess;
    const int64_t blocks = blocked_chunks(batch) * ((n + kTrN - 1) / kTrN);
    if (blocks > 0x7fffffffLL) return hipErrorInvalidValue;
    to_blocked_kernel<<<(unsigned)blocks, 256, 0, s>>>(n, batch, ld_in, y, yb);
    return hipGetLastError();
}

hipError_t launch_from_blocked(int64_t n, int64_t batch, int64_t ld_out, const float *yb, float *y, hipStream_t s) {
    if (n == 0 || batch == 0) return hipSuccess;
    const int64_t blocks = blocked_chunks(batch) * ((n + kTrN - 1) / kTrN);
    if (blocks > 0x7fffffffLL) return hipErrorInvalidValue;
    from_blocked_kernel<<<(unsigned)blocks, 256, 0, s>>>(n, batch, ld_out, yb, y);
    return hipGetLastError();
}

}  // namespace sdnn
