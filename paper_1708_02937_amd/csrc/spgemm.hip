// Sparse-Y layer product (row-wise Gustavson SpGEMM) with the bias, activation and zero pruning fused.
//
// Row r of Y_{k+1} is h(sum_i Y(r,i) W(i,:) + b): every stored entry of the sample scales the fan-out
// row of its neuron into a dense accumulator (Sec. II.D matrix multiply over +.x, computed row by row).
// A workgroup (16 waves) owns one sample at a time.  The accumulator is an fp64 array in LDS covering a
// window of 16384 output columns (128 KiB of gfx950's 160 KiB); wider layers are processed window by
// window, reading only the window's part of each fan-out row (per-row window offsets built at set-up).
// Products are exact in fp64 and added with LDS fp64 atomics.
//
// Scheduling: one persistent workgroup per CU takes chunks of samples from a device counter (every
// workgroup leaves once the counter passes the last chunk).  A chunk is classified 64 samples at a time:
// when every b_j <= 0 an empty sample stays empty (h(b_j) = 0) and costs one store.
//
// The epilogue visits the window in column order: z = acc + b_j, h(z), one rounding to fp32, and the
// entries that are not zero (Sec. II.E: zeros are not stored) are compacted with a wave prefix sum of
// per-thread survivor counts and a scan of the wave totals.  It zeroes what it reads, so the
// accumulator needs no separate clearing.  When every b_j <= 0 only touched columns can survive: for
// samples with few products the scatter also marks a bitmap and the epilogue walks only marked columns;
// windows that received no product are skipped.  Rows go to fixed slots of the output buffer (row r
// starts at r * n, its length goes to cnt[r]), so the next layer reads them without a global scan; only
// the final layer is packed into contiguous CSR.
#include "common.h"

namespace sdnn {

namespace {

constexpr int kThreads = 1024;
constexpr int kWaves = kThreads / 64;
constexpr int kTile = 16384;  // fp64 accumulator window: 128 KiB of LDS
constexpr int kBitWords = kTile / 32;

// One stored entry of the sample with the extent of its fan-out row segment (wave-private LDS staging).
struct RowRef {
    double y;
    int32_t start;
    int32_t len;
};

struct RowIn {
    int64_t yb, ylen;
};

// Extent of sample r of the input; caller CSR rows outside [0, nnz) or longer than n are flagged and read
// as empty, so no access leaves the arrays.
__device__ __forceinline__ RowIn input_row(int64_t r, int64_t n, int64_t batch, const int64_t *in_row_ptr,
                                           const int32_t *in_cnt, const int32_t *in_col, const float *in_val,
                                           uint32_t *err) {
    RowIn ri;
    if (in_row_ptr) {
        const int64_t nnz = (in_col && in_val) ? in_row_ptr[batch] : 0;  // no arrays: every row must be empty
        ri.yb = in_row_ptr[r];
        ri.ylen = in_row_ptr[r + 1] - ri.yb;
        if (ri.yb < 0 || ri.ylen < 0 || ri.ylen > n || ri.yb + ri.ylen > nnz) {
            atomicOr(err, 1u);
            ri.ylen = 0;
        }
    } else {
        ri.yb = r * n;
        ri.ylen = in_cnt[r];
    }
    return ri;
}

__global__ __launch_bounds__(kThreads) void spgemm_row_kernel(
    int64_t n, int64_t batch, int nwin, int chunk, const int64_t *__restrict__ in_row_ptr,
    const int32_t *__restrict__ in_cnt, const int32_t *__restrict__ in_col, const float *__restrict__ in_val,
    const int64_t *__restrict__ w_ptr, const int32_t *__restrict__ w_seg, const Edge *__restrict__ w,
    const float *__restrict__ bias, int bias_nonpos, int64_t sparse_limit, int lane_segments, double ymax,
    int32_t *__restrict__ out_cnt, int32_t *__restrict__ out_col, float *__restrict__ out_val, uint32_t *err,
    unsigned long long *work) {
    extern __shared__ double acc[];
    __shared__ RowRef refs[kThreads];
    __shared__ uint32_t bits[kBitWords];
    __shared__ int wave_tot[kWaves];
    __shared__ int64_t rows[64];
    __shared__ int nrows;
    __shared__ unsigned long long chunk_id;
    __shared__ int any;

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int half = lane >> 5, hl = lane & 31;
    const int width0 = (int)(n < kTile ? n : kTile);
    for (int t = tid; t < width0; t += kThreads) acc[t] = 0.0;
    for (int t = tid; t < kBitWords; t += kThreads) bits[t] = 0u;
    if (tid == 0) any = 0;
    const unsigned long long nchunks = (unsigned long long)((batch + chunk - 1) / chunk);

    for (;;) {
        if (tid == 0) chunk_id = atomicAdd(work, 1ull);
        __syncthreads();
        const unsigned long long ch = chunk_id;
        if (ch >= nchunks) break;  // uniform: every workgroup reaches this once the counter passes the end
        if (wave == 0) {
            const int64_t r = (int64_t)ch * chunk + lane;
            const bool valid = lane < chunk && r < batch;
            int64_t ylen = 0;
            if (valid) ylen = input_row(r, n, batch, in_row_ptr, in_cnt, in_col, in_val, err).ylen;
            const bool todo = valid && (ylen > 0 || !bias_nonpos);
            if (valid && !todo) out_cnt[r] = 0;
            const uint64_t m = __ballot(todo);
            if (todo) rows[lane_rank(m)] = r;
            if (lane == 0) nrows = __popcll(m);
        }
        __syncthreads();
        const int nr = nrows;
        for (int q = 0; q < nr; ++q) {
            const int64_t r = rows[q];
            const RowIn ri = input_row(r, n, batch, in_row_ptr, in_cnt, in_col, in_val, err);
            const int64_t yb = ri.yb, ylen = ri.ylen;
            const bool sparse = bias_nonpos && ylen <= sparse_limit;
            const int64_t ob = r * n;
            int64_t written = 0;
            for (int win = 0; win < nwin; ++win) {
                const int64_t c0 = (int64_t)win * kTile;
                const int64_t c1 = (c0 + kTile < n) ? c0 + kTile : n;
                const int width = (int)(c1 - c0);
                // scatter: each wave takes 64 stored entries of the sample at once (one per lane,
                // coalesced), gathers the extents of their fan-out row segments and parks (y, start,
                // length) in its own LDS area; then each half-wave reads one segment with 32 lanes (a
                // coalesced load), four segments per half in flight, and adds the exact products
                bool mine_any = false;
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
                            const int64_t rb = w_ptr[i];
                            if (w_seg) {
                                const int32_t *sg = w_seg + (int64_t)i * (nwin + 1) + win;
                                ref.start = (int32_t)(rb + sg[0]);
                                ref.len = sg[1] - sg[0];
                            } else {
                                ref.start = (int32_t)rb;
                                ref.len = (int32_t)(w_ptr[i + 1] - rb);
                            }
                        } else {
                            atomicOr(err, 1u);
                        }
                    }
                    if (lane_segments) {
                        // short segments: every lane walks its own (it spans one or two cache lines),
                        // eight weight loads in flight per lane
                        int maxl = ref.len;
#pragma unroll
                        for (int off = 32; off >= 1; off >>= 1) maxl = max(maxl, __shfl_xor(maxl, off));
                        for (int cc = 0; cc < maxl; cc += 8) {
                            Edge ed[8];
#pragma unroll
                            for (int u = 0; u < 8; ++u) {
                                ed[u].idx = -1;
                                ed[u].w = 0.0f;
                                if (cc + u < ref.len) ed[u] = w[ref.start + cc + u];
                            }
#pragma unroll
                            for (int u = 0; u < 8; ++u) {
                                if (ed[u].idx >= c0 && ed[u].idx < c1) {
                                    const int col = ed[u].idx - (int)c0;
                                    atomicAdd(&acc[col], ref.y * (double)ed[u].w);
                                    if (sparse) atomicOr(&bits[col >> 5], 1u << (col & 31));
                                    mine_any = true;
                                }
                            }
                        }
                        continue;
                    }
                    my[lane] = ref;
                    const int nref = (int)((ylen - base) < 64 ? (ylen - base) : 64);
                    for (int rr0 = 0; rr0 < nref; rr0 += 8) {
                        RowRef rr[4];
#pragma unroll
                        for (int p = 0; p < 4; ++p) {
                            const int row = rr0 + 2 * p + half;
                            rr[p] = my[row < nref ? row : 0];
                            if (row >= nref) rr[p].len = 0;
                        }
                        int maxl = 0;
#pragma unroll
                        for (int p = 0; p < 4; ++p) maxl = rr[p].len > maxl ? rr[p].len : maxl;
                        maxl = max(maxl, __shfl_xor(maxl, 32));
                        for (int cc = 0; cc < maxl; cc += 32) {
                            Edge ed[4];
#pragma unroll
                            for (int p = 0; p < 4; ++p) {
                                ed[p].idx = -1;
                                ed[p].w = 0.0f;
                                if (cc + hl < rr[p].len) ed[p] = w[rr[p].start + cc + hl];
                            }
#pragma unroll
                            for (int p = 0; p < 4; ++p) {
                                if (ed[p].idx >= c0 && ed[p].idx < c1) {
                                    const int col = ed[p].idx - (int)c0;
                                    atomicAdd(&acc[col], rr[p].y * (double)ed[p].w);
                                    if (sparse) atomicOr(&bits[col >> 5], 1u << (col & 31));
                                    mine_any = true;
                                }
                            }
                        }
                    }
                }
                if (mine_any) any = 1;
                __syncthreads();
                const bool touched = any != 0;
                if (sparse) {
                    if (touched) {
                        // epilogue over marked columns: count survivors per bitmap word, scan, write
                        const int nw = (width + 31) >> 5;
                        uint32_t word = tid < nw ? bits[tid] : 0u;
                        int keep = 0;
                        for (uint32_t m = word; m; m &= m - 1) {
                            const int col = tid * 32 + __builtin_ctz(m);
                            keep += activate(acc[col] + (double)bias[c0 + col], ymax) != 0.0f;
                        }
                        int incl = keep;
#pragma unroll
                        for (int d = 1; d < 64; d <<= 1) {
                            const int v = __shfl_up(incl, d);
                            if (lane >= d) incl += v;
                        }
                        if (lane == 63) wave_tot[wave] = incl;
                        __syncthreads();
                        int off = 0, tot = 0;
#pragma unroll
                        for (int u = 0; u < kWaves; ++u) {
                            const int v = wave_tot[u];
                            off += (u < wave) ? v : 0;
                            tot += v;
                        }
                        int64_t pos = ob + written + off + incl - keep;
                        for (uint32_t m = word; m; m &= m - 1) {
                            const int col = tid * 32 + __builtin_ctz(m);
                            const float f = activate(acc[col] + (double)bias[c0 + col], ymax);
                            acc[col] = 0.0;
                            if (f != 0.0f) {
                                out_col[pos] = (int32_t)(c0 + col);
                                out_val[pos] = f;
                                ++pos;
                            }
                        }
                        if (tid < nw) bits[tid] = 0u;
                        written += tot;
                    }
                } else if (touched || !bias_nonpos) {
                    // epilogue over the whole window in column order, 4 consecutive columns per thread
                    // (4096 per round); reads and zeroes the accumulator
                    for (int base = 0; base < width; base += 4 * kThreads) {
                        const int t0 = base + 4 * tid;
                        float f[4];
                        int keep = 0;
#pragma unroll
                        for (int v = 0; v < 4; ++v) {
                            f[v] = 0.0f;
                            if (t0 + v < width) {
                                f[v] = activate(acc[t0 + v] + (double)bias[c0 + t0 + v], ymax);
                                acc[t0 + v] = 0.0;
                            }
                            keep += f[v] != 0.0f;
                        }
                        int incl = keep;
#pragma unroll
                        for (int d = 1; d < 64; d <<= 1) {
                            const int v = __shfl_up(incl, d);
                            if (lane >= d) incl += v;
                        }
                        if (lane == 63) wave_tot[wave] = incl;
                        __syncthreads();
                        int off = 0, tot = 0;
#pragma unroll
                        for (int u = 0; u < kWaves; ++u) {
                            const int v = wave_tot[u];
                            off += (u < wave) ? v : 0;
                            tot += v;
                        }
                        int64_t pos = ob + written + off + incl - keep;
#pragma unroll
                        for (int v = 0; v < 4; ++v) {
                            if (f[v] != 0.0f) {
                                out_col[pos] = (int32_t)(c0 + t0 + v);
                                out_val[pos] = f[v];
                                ++pos;
                            }
                        }
                        written += tot;
                        __syncthreads();
                    }
                }
                __syncthreads();
                if (tid == 0) any = 0;
                __syncthreads();
            }
            if (tid == 0) out_cnt[r] = (int32_t)written;
        }
        __syncthreads();  // rows[] and chunk_id are rewritten for the next chunk
    }
}

// w_seg[i * (nwin + 1) + t] = offset, within fan-out row i, of its first column >= t * kTile.
__global__ void window_seg_kernel(int64_t n, int nwin, const int64_t *__restrict__ w_ptr,
                                  const int32_t *__restrict__ col, int32_t *__restrict__ w_seg) {
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= n) return;
    const int64_t b = w_ptr[i], e = w_ptr[i + 1];
    int64_t p = b;
    for (int t = 0; t <= nwin; ++t) {
        const int64_t bound = (int64_t)t * kTile;
        while (p < e && col[p] < bound) ++p;
        w_seg[i * (nwin + 1) + t] = (int32_t)(p - b);
    }
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

int spgemm_windows(int64_t n) { return (int)((n + kTile - 1) / kTile); }

bool spgemm_wants_window_index(int64_t n) { return spgemm_windows(n) > 1 && spgemm_windows(n) <= 16; }

hipError_t launch_window_seg(int64_t n, const int64_t *w_ptr, const int32_t *col, int32_t *w_seg, hipStream_t s) {
    window_seg_kernel<<<(unsigned)((n + 255) / 256), 256, 0, s>>>(n, spgemm_windows(n), w_ptr, col, w_seg);
    return hipGetLastError();
}

hipError_t launch_spgemm_layer(int64_t n, int64_t batch, const int64_t *in_row_ptr, const int32_t *in_cnt,
                               const int32_t *in_col, const float *in_val, const int64_t *w_ptr, const int32_t *w_seg,
                               const Edge *w, int64_t w_nnz, const float *bias, int bias_nonpos, double ymax,
                               int32_t *out_cnt, int32_t *out_col, float *out_val, uint32_t *err,
                               unsigned long long *work, int num_cu, hipStream_t s) {
    if (batch == 0) return hipSuccess;
    if (batch > 0x7fffffffLL) return hipErrorInvalidValue;
    static bool attr_set = false;
    if (!attr_set) {
        hipError_t e = hipFuncSetAttribute((const void *)spgemm_row_kernel, hipFuncAttributeMaxDynamicSharedMemorySize,
                                           (int)((size_t)kTile * sizeof(double)));
        if (e != hipSuccess) return e;
        attr_set = true;
    }
    const int nwin = spgemm_windows(n);
    const int64_t grid = batch < num_cu ? batch : num_cu;
    int64_t chunk = batch / (grid * 16);
    chunk = chunk < 1 ? 1 : (chunk > 64 ? 64 : chunk);
    // the bitmap epilogue pays off while a window gets at most ~2048 products
    const double per_win = (double)w_nnz / (double)n / (double)nwin;
    const int64_t sparse_limit = per_win > 0 ? (int64_t)(2048.0 / per_win) : n;
    // segments of at most ~16 entries are walked lane by lane, longer ones by half-waves
    const int lane_segments = (w_seg || nwin == 1) && per_win <= 16.0 ? 1 : 0;
    spgemm_row_kernel<<<(unsigned)grid, kThreads, spgemm_lds_bytes(n), s>>>(
        n, batch, nwin, (int)chunk, in_row_ptr, in_cnt, in_col, in_val, w_ptr, w_seg, w, bias, bias_nonpos,
        sparse_limit, lane_segments, ymax, out_cnt, out_col, out_val, err, work);
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
