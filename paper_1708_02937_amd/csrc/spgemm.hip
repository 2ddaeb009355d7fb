// Sparse-Y layer product (row-wise Gustavson SpGEMM) with the bias, activation and zero pruning fused.
//
// Row r of Y_{k+1} is h(sum_i Y(r,i) W(i,:) + b): every stored entry of the sample scales the fan-out
// row of its neuron into a dense accumulator (Sec. II.D matrix multiply over +.x, computed row by row).
// One workgroup (16 waves) owns one sample.  The accumulator is an fp64 array in LDS covering a window
// of 16384 output columns (128 KiB of gfx950's 160 KiB); wider layers are processed window by window.
// Products are exact in fp64 and added with LDS fp64 atomics.
//
// The epilogue walks the window in column order: z = acc + b_j, h(z), one rounding to fp32, and the
// entries that are not zero (Sec. II.E: zeros are not stored) are compacted with a wave ballot, a
// per-lane bit count below the lane, and a scan of the eight wave totals.  Rows are written to fixed
// slots of the output buffer (row r starts at r * n, its length goes to cnt[r]), so the next layer
// reads them without any global scan; only the final layer is packed into contiguous CSR.
//
// When every b_j <= 0 an empty sample stays empty (h(b_j) = 0), so such rows skip all work.
#include "common.h"

namespace sdnn {

namespace {

constexpr int kThreads = 1024;
constexpr int kWaves = kThreads / 64;
constexpr int kTile = 16384;  // fp64 accumulator window: 128 KiB of LDS

// One stored entry of the sample with the extent of its fan-out row (wave-private LDS staging).
struct RowRef {
    double y;
    int64_t start;
    int32_t len;
    int32_t pad;
};

__global__ __launch_bounds__(kThreads) void spgemm_row_kernel(
    int64_t n, int64_t batch, const int64_t *__restrict__ in_row_ptr, const int32_t *__restrict__ in_cnt,
    const int32_t *__restrict__ in_col, const float *__restrict__ in_val, const int64_t *__restrict__ w_ptr,
    const Edge *__restrict__ w, const float *__restrict__ bias, int bias_nonpos, double ymax,
    int32_t *__restrict__ out_cnt, int32_t *__restrict__ out_col, float *__restrict__ out_val, uint32_t *err) {
    extern __shared__ double acc[];
    __shared__ int wave_tot[kWaves];
    __shared__ RowRef refs[kThreads];

    const int64_t r = blockIdx.x;
    int64_t yb, ylen;
    if (in_row_ptr) {
        // caller-provided CSR: a row that does not lie inside [0, nnz) is flagged and read as empty,
        // and out-of-range column indices are flagged and skipped, so no access leaves the arrays
        const int64_t nnz = (in_col && in_val) ? in_row_ptr[batch] : 0;  // no arrays: every row must be empty
        yb = in_row_ptr[r];
        ylen = in_row_ptr[r + 1] - yb;
        if (yb < 0 || ylen < 0 || ylen > n || yb + ylen > nnz) {
            if (threadIdx.x == 0) atomicOr(err, 1u);
            ylen = 0;
        }
    } else {
        yb = r * n;
        ylen = in_cnt[r];
    }
    if (ylen == 0 && bias_nonpos) {
        if (threadIdx.x == 0) out_cnt[r] = 0;
        return;
    }
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int half = lane >> 5, hl = lane & 31;
    const int64_t ob = r * n;
    int64_t written = 0;

    for (int64_t c0 = 0; c0 < n; c0 += kTile) {
        const int64_t c1 = (c0 + kTile < n) ? c0 + kTile : n;
        const int width = (int)(c1 - c0);
        for (int t = threadIdx.x; t < width; t += kThreads) acc[t] = 0.0;
        __syncthreads();
        // scatter: each wave takes 64 stored entries of the sample at once (one per lane, coalesced),
        // gathers the extents of their fan-out rows and parks (y, row start, row length) in its own LDS
        // area; then each half-wave reads one fan-out row with 32 lanes (a coalesced 256-byte load),
        // four rows per half in flight, and adds the exact products into the accumulator
        RowRef *my = refs + wave * 64;
        for (int64_t base = (int64_t)wave * 64; base < ylen; base += kThreads) {
            const int64_t t = base + lane;
            RowRef ref;
            ref.y = 0.0;
            ref.start = 0;
            ref.len = 0;
            if (t < ylen) {
                const int32_t i = in_col[yb + t];
                if (i >= 0 && i < n) {
                    ref.y = (double)in_val[yb + t];
                    ref.start = w_ptr[i];
                    ref.len = (int32_t)(w_ptr[i + 1] - ref.start);
                } else {
                    atomicOr(err, 1u);
                }
            }
            my[lane] = ref;
            const int rows = (int)((ylen - base) < 64 ? (ylen - base) : 64);
            for (int r = 0; r < rows; r += 8) {
                RowRef rr[4];
#pragma unroll
                for (int p = 0; p < 4; ++p) {
                    const int row = r + 2 * p + half;
                    rr[p] = my[row < rows ? row : 0];
                    if (row >= rows) rr[p].len = 0;
                }
                int maxl = 0;
#pragma unroll
                for (int p = 0; p < 4; ++p) maxl = rr[p].len > maxl ? rr[p].len : maxl;
                maxl = max(maxl, __shfl_xor(maxl, 32));
                for (int c = 0; c < maxl; c += 32) {
                    Edge ed[4];
#pragma unroll
                    for (int p = 0; p < 4; ++p) {
                        ed[p].idx = -1;
                        ed[p].w = 0.0f;
                        if (c + hl < rr[p].len) ed[p] = w[rr[p].start + c + hl];
                    }
#pragma unroll
                    for (int p = 0; p < 4; ++p)
                        if (ed[p].idx >= c0 && ed[p].idx < c1)
                            atomicAdd(&acc[ed[p].idx - c0], rr[p].y * (double)ed[p].w);
                }
            }
        }
        __syncthreads();
        // epilogue and compaction, in column order
        for (int base = 0; base < width; base += kThreads) {
            const int t = base + (int)threadIdx.x;
            float f = 0.0f;
            if (t < width) f = activate(acc[t] + (double)bias[c0 + t], ymax);
            const bool keep = (t < width) && (f != 0.0f);
            const uint64_t m = __ballot(keep);
            const int pre = lane_rank(m);
            if (lane == 0) wave_tot[wave] = __popcll(m);
            __syncthreads();
            int off = 0, tot = 0;
#pragma unroll
            for (int u = 0; u < kWaves; ++u) {
                const int v = wave_tot[u];
                off += (u < wave) ? v : 0;
                tot += v;
            }
            if (keep) {
                const int64_t pos = ob + written + off + pre;
                out_col[pos] = (int32_t)(c0 + t);
                out_val[pos] = f;
            }
            written += tot;
            __syncthreads();
        }
    }
    if (threadIdx.x == 0) out_cnt[r] = (int32_t)written;
}

// Pack slot rows into contiguous CSR: row r moves from [r*n, r*n + cnt[r]) to [row_ptr[r], row_ptr[r+1]).
__global__ __launch_bounds__(256) void compact_rows_kernel(int64_t n, const int32_t *__restrict__ cnt,
                                                           const int64_t *__restrict__ row_ptr,
                                                           const int32_t *__restrict__ in_col,
                                                           const float *__restrict__ in_val,
                                                           int32_t *__restrict__ out_col,
                                                           float *__restrict__ out_val) {
    const int64_t r = blockIdx.x;
    const int64_t len = cnt[r], src = r * n, dst = row_ptr[r];
    for (int64_t t = threadIdx.x; t < len; t += blockDim.x) {
        out_col[dst + t] = in_col[src + t];
        out_val[dst + t] = in_val[src + t];
    }
}

// Dense activations from a batch of sparse rows: yt (n x batch, neuron-major, zero-filled by the caller)
// receives every stored entry.  Input is either caller CSR (row extents checked as in the SpGEMM) or
// slot rows written by a previous layer.
__global__ __launch_bounds__(256) void densify_kernel(int64_t n, int64_t batch, const int64_t *__restrict__ in_row_ptr,
                                                      const int32_t *__restrict__ in_cnt,
                                                      const int32_t *__restrict__ in_col,
                                                      const float *__restrict__ in_val, float *__restrict__ yt,
                                                      uint32_t *err) {
    const int64_t r = blockIdx.x;
    int64_t yb, ylen;
    if (in_row_ptr) {
        const int64_t nnz = (in_col && in_val) ? in_row_ptr[batch] : 0;
        yb = in_row_ptr[r];
        ylen = in_row_ptr[r + 1] - yb;
        if (yb < 0 || ylen < 0 || ylen > n || yb + ylen > nnz) {
            if (threadIdx.x == 0) atomicOr(err, 1u);
            ylen = 0;
        }
    } else {
        yb = r * n;
        ylen = in_cnt[r];
    }
    for (int64_t t = threadIdx.x; t < ylen; t += blockDim.x) {
        const int32_t i = in_col[yb + t];
        if (i < 0 || i >= n) {
            atomicOr(err, 1u);
            continue;
        }
        yt[(int64_t)i * batch + r] = in_val[yb + t];
    }
}

// Slot rows from dense batch-major activations (already h(.)-applied): keep the nonzeros of row r in
// column order at [r*n, r*n + cnt[r]), compacted with a wave ballot and a scan of the wave totals.
__global__ __launch_bounds__(kThreads) void dense_to_slots_kernel(int64_t n, const float *__restrict__ y,
                                                                  int32_t *__restrict__ out_cnt,
                                                                  int32_t *__restrict__ out_col,
                                                                  float *__restrict__ out_val) {
    __shared__ int wave_tot[kWaves];
    const int64_t r = blockIdx.x;
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const float *row = y + r * n;
    const int64_t ob = r * n;
    int64_t written = 0;
    for (int64_t base = 0; base < n; base += kThreads) {
        const int64_t j = base + threadIdx.x;
        const float f = j < n ? row[j] : 0.0f;
        const bool keep = f != 0.0f;
        const uint64_t m = __ballot(keep);
        const int pre = lane_rank(m);
        if (lane == 0) wave_tot[wave] = __popcll(m);
        __syncthreads();
        int off = 0, tot = 0;
#pragma unroll
        for (int u = 0; u < kWaves; ++u) {
            const int v = wave_tot[u];
            off += (u < wave) ? v : 0;
            tot += v;
        }
        if (keep) {
            out_col[ob + written + off + pre] = (int32_t)j;
            out_val[ob + written + off + pre] = f;
        }
        written += tot;
        __syncthreads();
    }
    if (threadIdx.x == 0) out_cnt[r] = (int32_t)written;
}

}  // namespace

size_t spgemm_lds_bytes(int64_t n) { return (size_t)(n < kTile ? n : kTile) * sizeof(double); }

hipError_t launch_spgemm_layer(int64_t n, int64_t batch, const int64_t *in_row_ptr, const int32_t *in_cnt,
                               const int32_t *in_col, const float *in_val, const int64_t *w_ptr, const Edge *w,
                               const float *bias, int bias_nonpos, double ymax, int32_t *out_cnt, int32_t *out_col,
                               float *out_val, uint32_t *err, hipStream_t s) {
    if (batch == 0) return hipSuccess;
    if (batch > 0x7fffffffLL) return hipErrorInvalidValue;
    static bool attr_set = false;
    if (!attr_set) {
        hipError_t e = hipFuncSetAttribute((const void *)spgemm_row_kernel, hipFuncAttributeMaxDynamicSharedMemorySize,
                                           (int)((size_t)kTile * sizeof(double)));
        if (e != hipSuccess) return e;
        attr_set = true;
    }
    spgemm_row_kernel<<<(unsigned)batch, kThreads, spgemm_lds_bytes(n), s>>>(
        n, batch, in_row_ptr, in_cnt, in_col, in_val, w_ptr, w, bias, bias_nonpos, ymax, out_cnt, out_col, out_val, err);
    return hipGetLastError();
}

hipError_t launch_compact_rows(int64_t n, int64_t batch, const int32_t *cnt, const int64_t *row_ptr,
                               const int32_t *in_col, const float *in_val, int32_t *out_col, float *out_val,
                               hipStream_t s) {
    if (batch == 0) return hipSuccess;
    compact_rows_kernel<<<(unsigned)batch, 256, 0, s>>>(n, cnt, row_ptr, in_col, in_val, out_col, out_val);
    return hipGetLastError();
}

hipError_t launch_densify(int64_t n, int64_t batch, const int64_t *in_row_ptr, const int32_t *in_cnt,
                          const int32_t *in_col, const float *in_val, float *yt, uint32_t *err, hipStream_t s) {
    if (batch == 0) return hipSuccess;
    hipError_t e = hipMemsetAsync(yt, 0, (size_t)n * (size_t)batch * sizeof(float), s);
    if (e != hipSuccess) return e;
    densify_kernel<<<(unsigned)batch, 256, 0, s>>>(n, batch, in_row_ptr, in_cnt, in_col, in_val, yt, err);
    return hipGetLastError();
}

hipError_t launch_dense_to_slots(int64_t n, int64_t batch, const float *y, int32_t *out_cnt, int32_t *out_col,
                                 float *out_val, hipStream_t s) {
    if (batch == 0) return hipSuccess;
    dense_to_slots_kernel<<<(unsigned)batch, kThreads, 0, s>>>(n, y, out_cnt, out_col, out_val);
    return hipGetLastError();
}

}  // namespace sdnn
