// Layer set-up kernels: CSR validation, the fan-in (transposed) copy of W_k used by the dense-Y
// product, and an int32 -> int64 scan.
//
// Set-up runs once per layer and is not part of the timed forward pass.  The paper's library keeps
// weights in CSR distributed by rows (Sec. V.A); the dense-Y product instead needs, for every output
// neuron, the list of its inputs, i.e. W_k^T in CSR.  The lists are built here by a stable LSD radix sort
// of the entries by column (8-bit digits: tile histograms, a scan per digit, a stable scatter), which
// leaves every list in ascending input order, so the stored order, and with it the fp64 summation order of
// the forward pass, does not depend on atomic timing.  List pointers come from a column count and a scan.
#include "common.h"

namespace sdnn {

namespace {

constexpr uint32_t kFlagIndex = 1u;    // CSR structure invalid
constexpr uint32_t kFlagValue = 2u;    // non-finite weight or bias
constexpr uint32_t kFlagPosBias = 4u;  // some bias > 0 (informational)

// flags[2] receives the largest bias as an order-preserving key (bits of a negative float complemented, of a
// positive one with the sign bit set: unsigned order is float order), flags[3] the complement of the smallest
// key (so that both start from zero), one atomic each per wave.
__global__ void validate_layer_kernel(int64_t n, int64_t nnz, const int64_t *__restrict__ row_ptr,
                                      const int32_t *__restrict__ col, const float *__restrict__ val,
                                      const float *__restrict__ bias, uint32_t *flags) {
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    uint32_t key = 0u, nkey = 0u;
    if (i < n) {
        const uint32_t u = __float_as_uint(bias[i]);
        key = (u & 0x80000000u) ? ~u : (u | 0x80000000u);
        nkey = ~key;
    }
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) {
        key = max(key, (uint32_t)__shfl_xor((int)key, off));
        nkey = max(nkey, (uint32_t)__shfl_xor((int)nkey, off));
    }
    if ((threadIdx.x & 63) == 0) {
        atomicMax(&flags[2], key);
        atomicMax(&flags[3], nkey);
    }
    if (i >= n) return;
    uint32_t f = 0;
    const int64_t b = row_ptr[i], e = row_ptr[i + 1];
    if (i == 0 && b != 0) f |= kFlagIndex;
    if (i == n - 1 && e != nnz) f |= kFlagIndex;
    if (b < 0 || e < b || e > nnz) {
        f |= kFlagIndex;
    } else {
        int32_t prev = -1;
        for (int64_t t = b; t < e; ++t) {
            const int32_t c = col[t];
            if (c < 0 || c >= n || c <= prev) f |= kFlagIndex;
            prev = c;
            if (!isfinite(val[t])) f |= kFlagValue;
        }
    }
    const float bi = bias[i];
    if (!isfinite(bi)) f |= kFlagValue;
    if (bi > 0.0f) {
        f |= kFlagPosBias;
        atomicAdd(&flags[1], 1u);  // number of neurons with a positive bias
    }
    if (f) atomicOr(flags, f);
}

__global__ void fanin_count_kernel(int64_t nnz, const int32_t *__restrict__ col, int32_t *counts) {
    const int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (e < nnz) atomicAdd(&counts[col[e]], 1);
}

// ------------------------------------------------------------------ exclusive scan (int32 -> int64)

constexpr int kScanThreads = 256;
constexpr int kScanPerThread = 16;
constexpr int64_t kScanChunk = (int64_t)kScanThreads * kScanPerThread;  // 4096 elements per block

template <typename T>
__device__ int64_t block_exclusive_scan(int64_t v, int64_t *lds) {
    // lds: kScanThreads int64 entries; returns the exclusive prefix of v over the block, lds[last] = total
    const int t = threadIdx.x;
    lds[t] = v;
    __syncthreads();
    for (int off = 1; off < kScanThreads; off <<= 1) {
        const int64_t add = t >= off ? lds[t - off] : 0;
        __syncthreads();
        lds[t] += add;
        __syncthreads();
    }
    const int64_t incl = lds[t];
    return incl - v;
}

// Sum of each 4096-element chunk.
template <typename T>
__global__ void scan_reduce_kernel(int64_t count, const T *__restrict__ in, int64_t *__restrict__ sums) {
    __shared__ int64_t lds[kScanThreads];
    const int64_t base = (int64_t)blockIdx.x * kScanChunk + (int64_t)threadIdx.x * kScanPerThread;
    int64_t s = 0;
    for (int q = 0; q < kScanPerThread; ++q) {
        const int64_t idx = base + q;
        if (idx < count) s += (int64_t)in[idx];
    }
    lds[threadIdx.x] = s;
    __syncthreads();
    for (int off = kScanThreads / 2; off > 0; off >>= 1) {
        if ((int)threadIdx.x < off) lds[threadIdx.x] += lds[threadIdx.x + off];
        __syncthreads();
    }
    if (threadIdx.x == 0) sums[blockIdx.x] = lds[0];
}

// In-place exclusive scan of the chunk sums (at most 4096 of them) by one block.
__global__ void scan_sums_kernel(int64_t nsums, int64_t *sums) {
    __shared__ int64_t lds[kScanThreads];
    const int64_t base = (int64_t)threadIdx.x * kScanPerThread;
    int64_t loc[kScanPerThread];
    int64_t s = 0;
    for (int q = 0; q < kScanPerThread; ++q) {
        const int64_t idx = base + q;
        loc[q] = idx < nsums ? sums[idx] : 0;
        s += loc[q];
    }
    int64_t run = block_exclusive_scan<int64_t>(s, lds);
    for (int q = 0; q < kScanPerThread; ++q) {
        const int64_t idx = base + q;
        if (idx < nsums) sums[idx] = run;
        run += loc[q];
    }
}

// out[i] = sum(in[0..i)) for i in [0, count]; out[count] = total.
template <typename T>
__global__ void scan_apply_kernel(int64_t count, const T *__restrict__ in, const int64_t *__restrict__ sums,
                                  int64_t *__restrict__ out) {
    __shared__ int64_t lds[kScanThreads];
    const int64_t base = (int64_t)blockIdx.x * kScanChunk + (int64_t)threadIdx.x * kScanPerThread;
    int64_t loc[kScanPerThread];
    int64_t s = 0;
    for (int q = 0; q < kScanPerThread; ++q) {
        const int64_t idx = base + q;
        loc[q] = idx < count ? (int64_t)in[idx] : 0;
        s += loc[q];
    }
    int64_t run = block_exclusive_scan<T>(s, lds) + sums[blockIdx.x];
    for (int q = 0; q < kScanPerThread; ++q) {
        const int64_t idx = base + q;
        if (idx < count) out[idx] = run;
        run += loc[q];
        if (idx == count - 1) out[count] = run;
    }
}

// ------------------------------------------------------------------ fan-in lists

// Fan-in lists by a stable LSD radix sort of the entries of W_k by output column.  The entries start in
// CSR order (rows ascending), so a stable sort by column leaves each list sorted by input index: the fp64
// summation order of the dense-Y kernels is then fixed, and any fan-in length is handled.
constexpr int kSortThreads = 256;
constexpr int kSortPer = 16;                              // entries per thread per tile
constexpr int kSortTile = kSortThreads * kSortPer;        // 4096 entries per tile
constexpr int kRadix = 256;                               // 8-bit digits

// keys[e] = column of entry e, vals[e] = (row of e, weight): one thread per row.
__global__ void sort_expand_kernel(int64_t n, const int64_t *__restrict__ row_ptr, const int32_t *__restrict__ col,
                                   const float *__restrict__ val, int32_t *__restrict__ keys, Edge *__restrict__ vals) {
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= n) return;
    for (int64_t e = row_ptr[i]; e < row_ptr[i + 1]; ++e) {
        keys[e] = col[e];
        Edge ed;
        ed.idx = (int32_t)i;
        ed.w = val[e];
        vals[e] = ed;
    }
}

// counts[d * ntiles + tile] = entries of the tile whose digit is d.
__global__ __launch_bounds__(kSortThreads) void sort_hist_kernel(int64_t nnz, int shift, int64_t ntiles,
                                                                 const int32_t *__restrict__ keys,
                                                                 int32_t *__restrict__ counts) {
    __shared__ int32_t h[kRadix];
    const int64_t tile = blockIdx.x;
    h[threadIdx.x] = 0;
    __syncthreads();
    const int64_t base = tile * kSortTile;
    for (int k = 0; k < kSortPer; ++k) {
        const int64_t e = base + k * kSortThreads + threadIdx.x;
        if (e < nnz) atomicAdd(&h[(keys[e] >> shift) & (kRadix - 1)], 1);
    }
    __syncthreads();
    counts[(int64_t)threadIdx.x * ntiles + tile] = h[threadIdx.x];
}

// One workgroup per digit: exclusive scan of its tile counts in place, digit total to totals[d].
__global__ __launch_bounds__(kSortThreads) void sort_scan_kernel(int64_t ntiles, int32_t *__restrict__ counts,
                                                                 int64_t *__restrict__ totals) {
    __shared__ int64_t wsum[kSortThreads / 64];
    const int d = blockIdx.x, lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    int32_t *row = counts + (int64_t)d * ntiles;
    int64_t run = 0;
    for (int64_t b0 = 0; b0 < ntiles; b0 += kSortThreads) {
        const int64_t t = b0 + threadIdx.x;
        const int64_t v = t < ntiles ? row[t] : 0;
        int64_t incl = v;
#pragma unroll
        for (int o = 1; o < 64; o <<= 1) {
            const int64_t u = __shfl_up(incl, o);
            if (lane >= o) incl += u;
        }
        if (lane == 63) wsum[wave] = incl;
        __syncthreads();
        int64_t before = 0, all = 0;
#pragma unroll
        for (int w = 0; w < kSortThreads / 64; ++w) {
            before += w < wave ? wsum[w] : 0;
            all += wsum[w];
        }
        if (t < ntiles) row[t] = (int32_t)(run + before + incl - v);
        run += all;
        __syncthreads();
    }
    if (threadIdx.x == 0) totals[d] = run;
}

// Stable scatter of one tile: round k handles entries base + k * 256 + t in order; within a wave the rank
// among equal digits comes from a match mask built from 8 ballots, across waves from per-wave digit counts.
__global__ __launch_bounds__(kSortThreads) void sort_scatter_kernel(int64_t nnz, int shift, int64_t ntiles,
                                                                    const int32_t *__restrict__ counts,
                                                                    const int64_t *__restrict__ totals,
                                                                    const int32_t *__restrict__ keys_in,
                                                                    const Edge *__restrict__ vals_in,
                                                                    int32_t *__restrict__ keys_out,
                                                                    Edge *__restrict__ vals_out) {
    __shared__ int64_t start[kRadix];             // where digit d of this tile goes next
    __shared__ int32_t wcnt[kSortThreads / 64][kRadix];
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int64_t tile = blockIdx.x;
    {
        // digit base = entries with a smaller digit (all tiles) + entries of this digit in earlier tiles
        int64_t base = 0;
        for (int d = 0; d < tid; ++d) base += totals[d];
        start[tid] = base + counts[(int64_t)tid * ntiles + tile];
    }
    for (int w = 0; w < kSortThreads / 64; ++w) wcnt[w][tid] = 0;
    __syncthreads();
    const uint64_t lt = (lane == 0) ? 0ull : (~0ull >> (64 - lane));
    for (int k = 0; k < kSortPer; ++k) {
        const int64_t e = tile * kSortTile + (int64_t)k * kSortThreads + tid;
        const bool valid = e < nnz;
        const int32_t key = valid ? keys_in[e] : 0;
        const int d = (key >> shift) & (kRadix - 1);
        uint64_t match = __ballot(valid);
#pragma unroll
        for (int b = 0; b < 8; ++b) {
            const uint64_t m = __ballot((d >> b) & 1);
            match &= ((d >> b) & 1) ? m : ~m;
        }
        const int rank = __popcll(match & lt);
        // the last lane of each digit group publishes the wave's count for that digit
        if (valid && (match >> lane) == 1ull) wcnt[wave][d] = __popcll(match);
        __syncthreads();
        if (valid) {
            int64_t pos = start[d] + rank;
            for (int w = 0; w < wave; ++w) pos += wcnt[w][d];
            keys_out[pos] = key;
            vals_out[pos] = vals_in[e];
        }
        __syncthreads();
        {
            int32_t add = 0;
            for (int w = 0; w < kSortThreads / 64; ++w) {
                add += wcnt[w][tid];
                wcnt[w][tid] = 0;
            }
            start[tid] += add;
        }
        __syncthreads();
    }
}

__global__ void max_segment_kernel(int64_t n, const int64_t *__restrict__ ptr, int32_t *out) {
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i < n) atomicMax(out, (int32_t)(ptr[i + 1] - ptr[i]));
}

__global__ void pack_edges_kernel(int64_t nnz, const int32_t *__restrict__ col, const float *__restrict__ val,
                                  Edge *__restrict__ out) {
    const int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (e < nnz) {
        Edge ed;
        ed.idx = col[e];
        ed.w = val[e];
        out[e] = ed;
    }
}

inline unsigned blocks_for(int64_t count, int threads) { return (unsigned)((count + threads - 1) / threads); }

}  // namespace

hipError_t launch_validate_layer(int64_t n, int64_t nnz, const int64_t *row_ptr, const int32_t *col,
                                 const float *val, const float *bias, uint32_t *flags, hipStream_t s) {
    validate_layer_kernel<<<blocks_for(n, 256), 256, 0, s>>>(n, nnz, row_ptr, col, val, bias, flags);
    return hipGetLastError();
}

hipError_t launch_fanin_counts(int64_t nnz, const int32_t *col, int32_t *counts, hipStream_t s) {
    if (nnz == 0) return hipSuccess;
    fanin_count_kernel<<<blocks_for(nnz, 256), 256, 0, s>>>(nnz, col, counts);
    return hipGetLastError();
}

int64_t scan_tmp_elems(int64_t count) { return (count + kScanChunk - 1) / kScanChunk + 1; }

hipError_t launch_exclusive_scan_i32_to_i64(int64_t count, const int32_t *in, int64_t *out, int64_t *tmp,
                                            hipStream_t s) {
    if (count == 0) return hipMemsetAsync(out, 0, sizeof(int64_t), s);
    const int64_t nblocks = (count + kScanChunk - 1) / kScanChunk;
    if (nblocks > kScanChunk) return hipErrorInvalidValue;  // more than 16.7M elements: not needed here
    scan_reduce_kernel<int32_t><<<(unsigned)nblocks, kScanThreads, 0, s>>>(count, in, tmp);
    scan_sums_kernel<<<1, kScanThreads, 0, s>>>(nblocks, tmp);
    scan_apply_kernel<int32_t><<<(unsigned)nblocks, kScanThreads, 0, s>>>(count, in, tmp, out);
    return hipGetLastError();
}

hipError_t launch_max_segment(int64_t n, const int64_t *ptr, int32_t *out, hipStream_t s) {
    max_segment_kernel<<<blocks_for(n, 256), 256, 0, s>>>(n, ptr, out);
    return hipGetLastError();
}

size_t fanin_sort_bytes(int64_t nnz) {
    const int64_t ntiles = (nnz + kSortTile - 1) / kSortTile;
    return 2 * (size_t)nnz * sizeof(int32_t) + (size_t)nnz * sizeof(Edge) +
           (size_t)kRadix * (size_t)ntiles * sizeof(int32_t) + kRadix * sizeof(int64_t) + 1024;
}

hipError_t launch_fanin_lists(int64_t n, int64_t nnz, const int64_t *row_ptr, const int32_t *col, const float *val,
                              Edge *fan, void *scratch, hipStream_t s) {
    if (nnz == 0) return hipSuccess;
    const int64_t ntiles = (nnz + kSortTile - 1) / kSortTile;
    if (ntiles > 0x7fffffffLL) return hipErrorInvalidValue;
    char *p = (char *)scratch;
    int32_t *keys[2];
    keys[0] = (int32_t *)p;
    p += (size_t)nnz * sizeof(int32_t);
    keys[1] = (int32_t *)p;
    p += (size_t)nnz * sizeof(int32_t);
    Edge *tmp = (Edge *)p;
    p += (size_t)nnz * sizeof(Edge);
    int32_t *counts = (int32_t *)p;
    p += (size_t)kRadix * (size_t)ntiles * sizeof(int32_t);
    int64_t *totals = (int64_t *)(((uintptr_t)p + 7) & ~(uintptr_t)7);
    int passes = 0;
    while ((int64_t)1 << (8 * passes) < n) ++passes;
    if (passes == 0) passes = 1;
    // the last pass must land in fan: start in fan when the pass count is even, in tmp when it is odd
    Edge *vals[2] = {passes % 2 ? tmp : fan, passes % 2 ? fan : tmp};
    sort_expand_kernel<<<blocks_for(n, 256), 256, 0, s>>>(n, row_ptr, col, val, keys[0], vals[0]);
    for (int pass = 0; pass < passes; ++pass) {
        const int a = pass & 1, b = a ^ 1;
        sort_hist_kernel<<<(unsigned)ntiles, kSortThreads, 0, s>>>(nnz, 8 * pass, ntiles, keys[a], counts);
        sort_scan_kernel<<<kRadix, kSortThreads, 0, s>>>(ntiles, counts, totals);
        sort_scatter_kernel<<<(unsigned)ntiles, kSortThreads, 0, s>>>(nnz, 8 * pass, ntiles, counts, totals, keys[a],
                                                                     vals[a], keys[b], vals[b]);
    }
    return hipGetLastError();
}

hipError_t launch_pack_edges(int64_t nnz, const int32_t *col, const float *val, Edge *out, hipStream_t s) {
    if (nnz == 0) return hipSuccess;
    pack_edges_kernel<<<blocks_for(nnz, 256), 256, 0, s>>>(nnz, col, val, out);
    return hipGetLastError();
}

}  // namespace sdnn
