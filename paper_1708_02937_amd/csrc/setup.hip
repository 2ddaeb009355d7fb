// Layer set-up kernels: CSR validation, the fan-in (transposed) copy of W_k used by the dense-Y
// product, and an int32 -> int64 scan.
//
// Set-up runs once per layer and is not part of the timed forward pass.  The paper's library keeps
// weights in CSR distributed by rows (Sec. V.A); the dense-Y product instead needs, for every output
// neuron, the list of its inputs, i.e. W_k^T in CSR.  That list is built here with a counting sort
// (count, scan, scatter) followed by a per-list sort by input index, so the stored order, and with it
// the fp64 summation order of the forward pass, does not depend on atomic timing.
#include "common.h"

namespace sdnn {

namespace {

constexpr uint32_t kFlagIndex = 1u;    // CSR structure invalid
constexpr uint32_t kFlagValue = 2u;    // non-finite weight or bias
constexpr uint32_t kFlagPosBias = 4u;  // some bias > 0 (informational)

__global__ void validate_layer_kernel(int64_t n, int64_t nnz, const int64_t *__restrict__ row_ptr,
                                      const int32_t *__restrict__ col, const float *__restrict__ val,
                                      const float *__restrict__ bias, uint32_t *flags) {
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
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

// One thread per source row i: append (i, W(i, j)) to the list of every output j it reaches.
__global__ void fanin_scatter_kernel(int64_t n, const int64_t *__restrict__ row_ptr, const int32_t *__restrict__ col,
                                     const float *__restrict__ val, const int64_t *__restrict__ fan_ptr,
                                     int32_t *cursor, Edge *__restrict__ fan) {
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= n) return;
    for (int64_t e = row_ptr[i]; e < row_ptr[i + 1]; ++e) {
        const int32_t j = col[e];
        const int32_t pos = atomicAdd(&cursor[j], 1);
        Edge ed;
        ed.idx = (int32_t)i;
        ed.w = val[e];
        fan[fan_ptr[j] + pos] = ed;
    }
}

// One wave per list: stage it in LDS, place each entry at its rank by input index (indices are distinct).
__global__ void fanin_sort_kernel(int64_t n, const int64_t *__restrict__ fan_ptr, Edge *__restrict__ fan) {
    extern __shared__ Edge seg[];
    const int64_t j = blockIdx.x;
    if (j >= n) return;
    const int64_t b = fan_ptr[j];
    const int len = (int)(fan_ptr[j + 1] - b);
    if (len <= 1) return;
    for (int t = threadIdx.x; t < len; t += blockDim.x) seg[t] = fan[b + t];
    __syncthreads();
    for (int t = threadIdx.x; t < len; t += blockDim.x) {
        const int32_t key = seg[t].idx;
        int rank = 0;
        for (int u = 0; u < len; ++u) rank += seg[u].idx < key;
        fan[b + rank] = seg[t];
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

hipError_t launch_fanin_scatter(int64_t n, const int64_t *row_ptr, const int32_t *col, const float *val,
                                const int64_t *fan_ptr, int32_t *cursor, Edge *fan, hipStream_t s) {
    fanin_scatter_kernel<<<blocks_for(n, 256), 256, 0, s>>>(n, row_ptr, col, val, fan_ptr, cursor, fan);
    return hipGetLastError();
}

hipError_t launch_max_segment(int64_t n, const int64_t *ptr, int32_t *out, hipStream_t s) {
    max_segment_kernel<<<blocks_for(n, 256), 256, 0, s>>>(n, ptr, out);
    return hipGetLastError();
}

// Caller guarantees every list is at most 8192 entries (64 KiB of LDS).
hipError_t launch_fanin_sort(int64_t n, int32_t max_len, const int64_t *fan_ptr, Edge *fan, hipStream_t s) {
    if (max_len <= 1) return hipSuccess;
    if (max_len > 8192) return hipErrorInvalidValue;
    fanin_sort_kernel<<<(unsigned)n, 64, (size_t)max_len * sizeof(Edge), s>>>(n, fan_ptr, fan);
    return hipGetLastError();
}

hipError_t launch_pack_edges(int64_t nnz, const int32_t *col, const float *val, Edge *out, hipStream_t s) {
    if (nnz == 0) return hipSuccess;
    pack_edges_kernel<<<blocks_for(nnz, 256), 256, 0, s>>>(nnz, col, val, out);
    return hipGetLastError();
}

}  // namespace sdnn
