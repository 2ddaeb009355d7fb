// Sparse-Y layer product (row-wise Gustavson SpGEMM) with the bias, activation and zero pruning fused.
//
// Row r of Y_{k+1} is h(sum_i Y(r,i) W(i,:) + b): every stored entry of the sample scales the fan-out
// row of its neuron into a dense accumulator (Sec. II.D matrix multiply over +.x, computed row by row).
// A workgroup (16 waves) owns one sample at a time.  The accumulator is an fp64 array in LDS covering a
// window of 16384 output columns (128 KiB of gfx950's 160 KiB); wider layers are processed window by
// window, reading only the window's part of each fan-out row (per-row window offsets built at set-up).
// Products are exact in fp64 and added with LDS fp64 atomics.
//
// Scheduling: a planning pass sorts the samples of a layer into three classes.  When every b_j <= 0 an
// empty sample stays empty (h(b_j) = 0) and costs one store; a sample whose products fit a wave's share of
// LDS (at most 1024) goes to the small-sample kernel, one wavefront per sample; every other sample goes to
// the workgroup kernel below, where one persistent workgroup per CU takes chunks of the list from a device
// counter (every workgroup leaves once the counter passes the last chunk).  Samples of at most 1024 entries
// keep them in registers (one per thread); with three or four windows and only marked columns to read, they
// go to a pipelined instance that loads every window's data a window ahead (described at that kernel), which
// also takes samples of up to 2048 entries.
//
// The epilogue visits the window in column order: z = acc + b_j, h(z), one rounding to fp32, and the
// entries that are not zero (Sec. II.E: zeros are not stored) are compacted with a wave prefix sum of
// per-thread survivor counts and a scan of the wave totals.  It zeroes what it reads, so the
// accumulator needs no separate clearing.  When every b_j <= 0 only touched columns can survive: for
// samples with few products the scatter also marks a bitmap and the epilogue walks only marked columns;
// windows that received no product are skipped.  Then also a sum at most -max_j b_j is zero after h in every
// column, so for the other samples the scatter's atomics return the previous sum and mark a column when an
// addition lifts it above that bound: the epilogue reads only the marked columns (a handful per window on a
// sparse network) and clears the window with 16-byte stores.  Rows go to fixed slots of the output buffer (row r
// starts at r * n, its length goes to cnt[r]), so the next layer reads them without a global scan; only
// the final layer is packed into contiguous CSR.
#include <atomic>

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

constexpr int kSmallCap = 1024;   // products per sample in the small-sample kernel (a power of two)
constexpr int kSmallWaves = 4;    // wavefronts per workgroup of the small-sample kernel

// Per-layer counters kept by the sparse layer kernels (one row of the net's statistics array).
enum : int { kStatSmall = 0, kStatLarge = 1, kStatNnz = 2, kStatWork = 3, kStatResident = 4, kStatResidentWork = 5 };

// Planning pass: one thread per sample.  When only touched columns can be nonzero (every b_j <= 0, or the
// bias applies only on the structural pattern), empty samples are finished here (cnt = 0); the others are
// appended, with one atomic per wave and list, to the small list (lists[0 ..)), the list of samples the
// workgroup kernel can keep in registers (lists[2 batch ..)) or the general list (lists[batch ..)).
__global__ __launch_bounds__(256) void spgemm_plan_kernel(int64_t n, int64_t batch, const int64_t *__restrict__ in_row_ptr,
                                                          const int32_t *__restrict__ in_cnt,
                                                          const int32_t *__restrict__ in_col,
                                                          const float *__restrict__ in_val, int only_touched,
                                                          int64_t small_len, int64_t resident_len,
                                                          int32_t *__restrict__ out_cnt, int32_t *__restrict__ lists,
                                                          unsigned long long *stats, uint32_t *err) {
    const int64_t r = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    const int lane = threadIdx.x & 63;
    const bool valid = r < batch;
    int64_t ylen = 0;
    if (valid) ylen = input_row(r, n, batch, in_row_ptr, in_cnt, in_col, in_val, err).ylen;
    const bool skip = valid && only_touched && ylen == 0;
    const bool small = valid && only_touched && ylen > 0 && ylen <= small_len;
    const bool resident = valid && !skip && !small && ylen <= resident_len;
    const bool large = valid && !skip && !small && !resident;
    if (skip) out_cnt[r] = 0;
    const uint64_t ms = __ballot(small), ml = __ballot(large), mr = __ballot(resident);
    unsigned long long bs = 0, bl = 0, br = 0;
    if (lane == 0) {
        if (ms) bs = atomicAdd(&stats[kStatSmall], (unsigned long long)__popcll(ms));
        if (ml) bl = atomicAdd(&stats[kStatLarge], (unsigned long long)__popcll(ml));
        if (mr) br = atomicAdd(&stats[kStatResident], (unsigned long long)__popcll(mr));
    }
    bs = __shfl(bs, 0);
    bl = __shfl(bl, 0);
    br = __shfl(br, 0);
    if (small) lists[bs + lane_rank(ms)] = (int32_t)r;
    if (large) lists[batch + bl + lane_rank(ml)] = (int32_t)r;
    if (resident) lists[2 * batch + br + lane_rank(mr)] = (int32_t)r;
}

// Orders this wave's earlier LDS accesses before its later ones (the lanes of one wave exchange data
// through LDS between the phases of the small-sample kernel).
__device__ __forceinline__ void wave_lds_sync() {
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

// Value of lane (l ^ M) for lane l of the wave: DPP quad permutations for M = 1, 2, DPP row shifts (lanes
// l - M and l + M within each row of 16) for M = 4, 8, a swizzle within 32 lanes for M = 16, a permute for
// M = 32.
template <int M>
__device__ __forceinline__ int xor_lanes(int v, int lane) {
    if constexpr (M == 1) {
        return __builtin_amdgcn_update_dpp(0, v, 0xB1, 0xF, 0xF, false);  // quad_perm [1, 0, 3, 2]
    } else if constexpr (M == 2) {
        return __builtin_amdgcn_update_dpp(0, v, 0x4E, 0xF, 0xF, false);  // quad_perm [2, 3, 0, 1]
    } else if constexpr (M == 4 || M == 8) {
        const int hi = __builtin_amdgcn_update_dpp(0, v, 0x100 + M, 0xF, 0xF, false);  // row_shl: lane l + M
        const int lo = __builtin_amdgcn_update_dpp(0, v, 0x110 + M, 0xF, 0xF, false);  // row_shr: lane l - M
        return (lane & M) ? lo : hi;
    } else if constexpr (M == 16) {
        return __builtin_amdgcn_ds_swizzle(v, (16 << 10) | 0x1F);  // and 0x1f, or 0, xor 16
    } else {
        return __builtin_amdgcn_ds_bpermute((lane ^ M) << 2, v);
    }
}
template <int M>
__device__ __forceinline__ double xor_lanes(double v, int lane) {
    const long long b = __double_as_longlong(v);
    const int lo = xor_lanes<M>((int)b, lane), hi = xor_lanes<M>((int)(b >> 32), lane);
    return __longlong_as_double(((long long)hi << 32) | (uint32_t)lo);
}

// One stage (block size KK, distance J) of a bitonic sort of 64 * P (key, value) pairs held by a wave, lane
// l holding elements l * P .. l * P + P - 1: distances below P stay inside a lane, the others exchange with
// lane l ^ (J / P).  Equal keys keep their places within each compared pair, so every element survives.
template <int P, int KK, int J, bool kVals>
__device__ __forceinline__ void bitonic_stages(int32_t (&k)[P], double (&v)[P], int lane) {
    if constexpr (J >= P) {
        constexpr int LJ = J / P;
        const bool lower = (lane & LJ) == 0;
#pragma unroll
        for (int r = 0; r < P; ++r) {
            const bool up = ((lane * P + r) & KK) == 0;
            const int32_t pk = xor_lanes<LJ>(k[r], lane);
            const bool take = (lower == up) ? pk < k[r] : pk > k[r];
            if constexpr (kVals) {
                const double pv = xor_lanes<LJ>(v[r], lane);
                if (take) v[r] = pv;
            }
            if (take) k[r] = pk;
        }
    } else {
#pragma unroll
        for (int r = 0; r < P; ++r) {
            const int r2 = r ^ J;
            if (r2 > r) {
                const bool up = ((lane * P + r) & KK) == 0;
                if (up ? k[r] > k[r2] : k[r] < k[r2]) {
                    const int32_t tk = k[r];
                    k[r] = k[r2];
                    k[r2] = tk;
                    if constexpr (kVals) {
                        const double tv = v[r];
                        v[r] = v[r2];
                        v[r2] = tv;
                    }
                }
            }
        }
    }
    if constexpr (J > 1) bitonic_stages<P, KK, J / 2, kVals>(k, v, lane);
}
template <int P, int KK, bool kVals>
__device__ __forceinline__ void bitonic_blocks(int32_t (&k)[P], double (&v)[P], int lane) {
    bitonic_stages<P, KK, KK / 2, kVals>(k, v, lane);
    if constexpr (KK < 64 * P) bitonic_blocks<P, KK * 2, kVals>(k, v, lane);
}

// Bitonic sort by key of the 64 * P (key, value) pairs in keys/vals (one wave), in registers, with one
// 32-bit word per pair in the network: (key << 9) | position (keys below 2^22 - 1, at most 512 pairs;
// 0x7fffffff pads), the values fetched by position afterwards.  Words are unique (equal keys keep their
// order of position), and an exchange moves one register instead of three.
template <int P>
__device__ __forceinline__ void wave_sort_packed(int32_t *keys, double *vals, int lane) {
    static_assert(64 * P <= 512, "nine position bits");
    int32_t k[P];
    double v[P];
#pragma unroll
    for (int r = 0; r < P; ++r) {
        const int e = lane * P + r;
        const int32_t c = keys[e];
        k[r] = c == 0x7fffffff ? c : (int32_t)(((uint32_t)c << 9) | (uint32_t)e);
    }
    bitonic_blocks<P, 2, false>(k, v, lane);
#pragma unroll
    for (int r = 0; r < P; ++r) v[r] = k[r] == 0x7fffffff ? 0.0 : vals[k[r] & 511];
    wave_lds_sync();  // every lane has read the values at their old places
#pragma unroll
    for (int r = 0; r < P; ++r) {
        keys[lane * P + r] = k[r] == 0x7fffffff ? 0x7fffffff : (int32_t)((uint32_t)k[r] >> 9);
        vals[lane * P + r] = v[r];
    }
}

// Small samples (every b_j <= 0, at most kSmallCap products): one wavefront per sample, no accumulator
// window.  The wave expands the sample's products (column, exact fp64 product) into its own LDS area
// (a wave prefix sum of the fan-out row lengths gives each entry its place), sorts them by column with a
// bitonic network held in registers, then each run of equal columns is summed, biased, activated and rounded once, and the
// survivors are compacted in column order with a ballot.  Only touched columns can survive when
// b_j <= 0 or when the bias applies only on the structural pattern, so nothing else is visited.
// kUniformBias: every b_j is the same value, read once from bias[0] (no bias load per run).
template <bool kUniformBias>
__global__ __launch_bounds__(kSmallWaves * 64) void spgemm_small_kernel(
    int64_t n, int64_t batch, const int64_t *__restrict__ in_row_ptr, const int32_t *__restrict__ in_cnt,
    const int32_t *__restrict__ in_col, const float *__restrict__ in_val, const int64_t *__restrict__ w_ptr,
    const Edge *__restrict__ w, const float *__restrict__ bias, double zero_below, double ymax,
    const int32_t *__restrict__ list, unsigned long long *stats, int32_t *__restrict__ out_cnt,
    int32_t *__restrict__ out_col, float *__restrict__ out_val, uint32_t *err) {
    __shared__ int32_t keys_all[kSmallWaves][kSmallCap];
    __shared__ double vals_all[kSmallWaves][kSmallCap];
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    int32_t *keys = keys_all[wave];
    double *vals = vals_all[wave];
    const int64_t count = (int64_t)stats[kStatSmall];
    const double b_uni = kUniformBias ? (double)bias[0] : 0.0;
    const int64_t stride = (int64_t)gridDim.x * kSmallWaves;
    for (int64_t q = (int64_t)blockIdx.x * kSmallWaves + wave; q < count; q += stride) {
        const int64_t r = list[q];
        const RowIn ri = input_row(r, n, batch, in_row_ptr, in_cnt, in_col, in_val, err);
        // expand: the planner guarantees ylen * (longest fan-out row) <= kSmallCap
        int total = 0;
        for (int64_t base = 0; base < ri.ylen; base += 64) {
            const int64_t t = base + lane;
            double y = 0.0;
            int64_t start = 0;
            int len = 0;
            if (t < ri.ylen) {
                const int32_t i = in_col[ri.yb + t];
                if (i >= 0 && i < n) {
                    y = (double)in_val[ri.yb + t];
                    start = w_ptr[i];
                    // a zero input adds nothing and is no structural entry: its products are not expanded
                    len = y != 0.0 ? (int)(w_ptr[i + 1] - start) : 0;
                } else {
                    atomicOr(err, 1u);
                }
            }
            int incl = len;
#pragma unroll
            for (int d = 1; d < 64; d <<= 1) {
                const int v = __shfl_up(incl, d);
                if (lane >= d) incl += v;
            }
            int pos = total + incl - len;
            total += __shfl(incl, 63);
            for (int k0 = 0; k0 < len; k0 += 8) {
                Edge ed[8];
#pragma unroll
                for (int u = 0; u < 8; ++u)
                    if (k0 + u < len) ed[u] = w[start + k0 + u];
#pragma unroll
                for (int u = 0; u < 8; ++u)
                    if (k0 + u < len) {
                        keys[pos + k0 + u] = ed[u].idx;
                        vals[pos + k0 + u] = y * (double)ed[u].w;
                    }
            }
        }
        int size = 64;
        while (size < total) size <<= 1;
        for (int e = total + lane; e < size; e += 64) keys[e] = 0x7fffffff;
        wave_lds_sync();
        // bitonic sort of (key, value) pairs by key over [0, size): in registers up to 512 pairs (more would
        // cost the kernel's occupancy; columns below 2^22 - 1), through LDS otherwise
        if (size <= 512 && n < (1 << 22)) {
            switch (size) {
                case 64: wave_sort_packed<1>(keys, vals, lane); break;
                case 128: wave_sort_packed<2>(keys, vals, lane); break;
                case 256: wave_sort_packed<4>(keys, vals, lane); break;
                default: wave_sort_packed<8>(keys, vals, lane); break;
            }
        } else {
            for (int k = 2; k <= size; k <<= 1) {
                for (int j = k >> 1; j > 0; j >>= 1) {
                    for (int p = lane; p < (size >> 1); p += 64) {
                        const int i = ((p & ~(j - 1)) << 1) | (p & (j - 1));
                        const int l = i + j;
                        const int32_t ki = keys[i], kl = keys[l];
                        const bool up = (i & k) == 0;
                        if ((ki > kl) == up && ki != kl) {
                            keys[i] = kl;
                            keys[l] = ki;
                            const double vi = vals[i];
                            vals[i] = vals[l];
                            vals[l] = vi;
                        }
                    }
                    wave_lds_sync();
                }
            }
        }
        wave_lds_sync();
        // runs of equal columns: the first element of a run sums it, then h, one rounding, compaction
        const int64_t ob = r * n;
        int written = 0;
        for (int base = 0; base < total; base += 64) {
            const int e = base + lane;
            float f = 0.0f;
            int32_t key = 0;
            if (e < total) {
                key = keys[e];
                if (e == 0 || keys[e - 1] != key) {
                    double z = 0.0;
                    for (int u = e; u < total && keys[u] == key; ++u) z += vals[u];
                    f = z > zero_below ? activate(z + (kUniformBias ? b_uni : (double)bias[key]), ymax) : 0.0f;
                }
            }
            const bool keep = f != 0.0f;
            const uint64_t m = __ballot(keep);
            if (keep) {
                const int64_t o = ob + written + lane_rank(m);
                out_col[o] = key;
                out_val[o] = f;
            }
            written += __popcll(m);
        }
        if (lane == 0) {
            out_cnt[r] = written;
            if (written) atomicAdd(&stats[kStatNnz], (unsigned long long)written);
        }
        wave_lds_sync();  // the next sample rewrites this wave's LDS area
    }
}

constexpr int kRounds = kTile / (4 * kThreads);  // dense-epilogue rounds of 4 columns per thread
constexpr int kRoundCols = 4 * kThreads;          // columns per dense-epilogue round
static_assert(kTile % kRoundCols == 0, "whole rounds per window");

// LDS position of accumulator column `col` of a window: within each round of 4096 columns, column 4t + v sits
// at v * 1024 + t, so when thread t reads its 4 consecutive columns in the dense epilogue the 64 lanes of a
// wave touch 64 consecutive doubles (column-major per thread would put the lanes 32 bytes apart: an 8-way
// bank conflict on every read and write).  The scatter uses the same map.
__device__ __forceinline__ int acc_pos(int col) {
    return (col & ~(kRoundCols - 1)) | ((col & 3) * kThreads) | ((col & (kRoundCols - 1)) >> 2);
}
// Add product v to column col of the window.  mark_all (bitmap epilogue): mark every column a nonzero entry
// touches.  cross (every b_j <= 0, dense samples): the sum starts at 0 <= zero_below, so a column whose final
// sum exceeds zero_below was pushed across it by some addition; that addition reads the previous sum back and
// marks the column, and only marked columns can survive.  The thread's add rounds like the LDS unit's, so no
// crossing goes unmarked; a column that crosses and falls back is marked and dropped by the epilogue.
template <int K, bool kLinear = false>
__device__ __forceinline__ void add_products(double *acc, uint32_t *bits, const int (&col)[K], const double (&v)[K],
                                             const bool (&ok)[K], bool mark_all, bool cross, double zero_below) {
    // kLinear: column c of the window at position c (instances without the dense epilogue)
    auto at = [](int c) { return kLinear ? c : acc_pos(c); };
    if (cross) {
        double old[K];
#pragma unroll
        for (int u = 0; u < K; ++u) old[u] = ok[u] ? atomicAdd(&acc[at(col[u])], v[u]) : 0.0;
#pragma unroll
        for (int u = 0; u < K; ++u)
            if (ok[u] && old[u] <= zero_below && old[u] + v[u] > zero_below)
                atomicOr(&bits[col[u] >> 5], 1u << (col[u] & 31));
    } else {
#pragma unroll
        for (int u = 0; u < K; ++u)
            if (ok[u]) {
                atomicAdd(&acc[at(col[u])], v[u]);
                if (mark_all) atomicOr(&bits[col[u] >> 5], 1u << (col[u] & 31));
            }
    }
}
constexpr int kRes = 1;                           // stored entries a thread keeps in registers (resident mode)
constexpr int kResLoads = 4;                      // weight loads in flight per resident entry
constexpr int kPre = 8;                           // entries of each window's segment loaded a window ahead

template <bool kResident>
__global__ __launch_bounds__(kThreads) void spgemm_row_kernel(
    int64_t n, int64_t batch, int nwin, const int64_t *__restrict__ in_row_ptr,
    const int32_t *__restrict__ in_cnt, const int32_t *__restrict__ in_col, const float *__restrict__ in_val,
    const int64_t *__restrict__ w_ptr, const int32_t *__restrict__ w_seg, const Edge *__restrict__ w,
    const float *__restrict__ bias, int bias_nonpos, double zero_below, int pattern, int64_t sparse_limit,
    int lane_segments, double ymax, const int32_t *__restrict__ list, unsigned long long *stats, int32_t *__restrict__ out_cnt,
    int32_t *__restrict__ out_col, float *__restrict__ out_val, uint32_t *err) {
    // bias_nonpos: only touched columns can be nonzero (every b_j <= 0, or pattern mode); pattern: the
    // bias applies only on the structural pattern, so the touched-column bitmap is always kept
    extern __shared__ __align__(16) double acc[];
    __shared__ RowRef refs[kThreads];
    __shared__ uint32_t bits[kBitWords];
    __shared__ int wave_tot[kWaves];
    __shared__ unsigned long long wave_tot4[kWaves];
    __shared__ unsigned long long chunk_id;
    __shared__ int any;

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int half = lane >> 5, hl = lane & 31;
    // this instance's list was filled by the planning pass of the layer; chunks of it are taken in turn.  An
    // empty list (every later layer of a net whose activations have died out) ends the workgroup before it
    // clears its accumulator (the same count in every workgroup)
    const int64_t count = (int64_t)stats[kResident ? kStatResident : kStatLarge];
    if (count == 0) return;
    // the accumulator covers whole rounds (the positions of a partial round's columns spread over the round)
    const int width0 = (int)(n < kTile ? (n + kRoundCols - 1) / kRoundCols * kRoundCols : kTile);
    for (int t = tid; t < width0; t += kThreads) acc[t] = 0.0;
    for (int t = tid; t < kBitWords; t += kThreads) bits[t] = 0u;
    if (tid == 0) any = 0;
    int64_t chunk = count / ((int64_t)gridDim.x * 16);
    chunk = chunk < 1 ? 1 : (chunk > 64 ? 64 : chunk);
    const unsigned long long nchunks = (unsigned long long)((count + chunk - 1) / chunk);
    const int32_t *large = list + (kResident ? 2 : 1) * batch;

    for (;;) {
        if (tid == 0) chunk_id = atomicAdd(&stats[kResident ? kStatResidentWork : kStatWork], 1ull);
        __syncthreads();
        const unsigned long long ch = chunk_id;
        if (ch >= nchunks) break;  // uniform: every workgroup reaches this once the counter passes the end
        const int64_t q0 = (int64_t)ch * chunk;
        const int nr = (int)((count - q0) < chunk ? (count - q0) : chunk);
        for (int q = 0; q < nr; ++q) {
            const int64_t r = large[q0 + q];
            const RowIn ri = input_row(r, n, batch, in_row_ptr, in_cnt, in_col, in_val, err);
            const int64_t yb = ri.yb, ylen = ri.ylen;
            const bool sparse = pattern || (bias_nonpos && ylen <= sparse_limit);
            const bool cross = !sparse && zero_below >= 0.0;
            // resident instance: up to kRes stored entries per thread, kept in registers across the
            // windows; the thread's fan-out segment for window w is [s_lo, s_hi), and the next window's
            // segment starts where this one ends, so each window costs one more offset load, issued a
            // window ahead.  The planner sends only samples that fit here (and short fan-out segments).
            constexpr bool resident = kResident;
            double my_y[kRes];
            int32_t my_i[kRes];
            int64_t my_rb[kRes], s_lo[kRes], s_hi[kRes];
#pragma unroll
            for (int k = 0; k < kRes; ++k) {
                my_y[k] = 0.0;
                my_i[k] = -1;
                my_rb[k] = s_lo[k] = s_hi[k] = 0;
                const int64_t t = tid + (int64_t)k * kThreads;
                if (resident && t < ylen) {
                    const int32_t i = in_col[yb + t];
                    if (i >= 0 && i < n) {
                        my_i[k] = i;
                        my_y[k] = (double)in_val[yb + t];
                        my_rb[k] = w_ptr[i];
                        s_lo[k] = my_rb[k];
                        s_hi[k] = w_seg ? my_rb[k] + w_seg[(int64_t)i * (nwin + 1) + 1] : w_ptr[i + 1];
                    } else {
                        atomicOr(err, 1u);
                    }
                }
            }
            const int64_t ob = r * n;
            int64_t written = 0;
            // resident instance: the first kPre entries of each window's segment are loaded a window ahead
            // (the first window's right after the set-up), so that the previous window's epilogue covers
            // their latency; longer segments load the rest kResLoads at a time
            Edge pre[kRes][kPre];
            if constexpr (kResident) {
#pragma unroll
                for (int k = 0; k < kRes; ++k)
#pragma unroll
                    for (int u = 0; u < kPre; ++u) {
                        pre[k][u].idx = 0;
                        pre[k][u].w = 0.0f;
                        if (s_lo[k] + u < s_hi[k]) pre[k][u] = w[s_lo[k] + u];
                    }
            }
            for (int win = 0; win < nwin; ++win) {
                const int64_t c0 = (int64_t)win * kTile;
                const int64_t c1 = (c0 + kTile < n) ? c0 + kTile : n;
                const int width = (int)(c1 - c0);
                bool mine_any = false;
                if constexpr (kResident) {
#pragma unroll
                    for (int k = 0; k < kRes; ++k) {
                        const int64_t lo = s_lo[k], hi = s_hi[k];
                        if (win + 1 < nwin && my_i[k] >= 0) {
                            s_lo[k] = s_hi[k];
                            s_hi[k] = my_rb[k] + w_seg[(int64_t)my_i[k] * (nwin + 1) + win + 2];
                        }
                        int64_t e = lo;
                        {
                            int col[kPre];
                            double v[kPre];
                            bool ok[kPre];
#pragma unroll
                            for (int u = 0; u < kPre; ++u) {
                                ok[u] = e + u < hi;
                                col[u] = pre[k][u].idx - (int)c0;
                                v[u] = my_y[k] * (double)pre[k][u].w;
                                mine_any |= ok[u];
                            }
                            add_products(acc, bits, col, v, ok, sparse && my_y[k] != 0.0, cross, zero_below);
                            e += kPre;
                        }
                        for (; e < hi; e += kResLoads) {
                            Edge ed[kResLoads];
#pragma unroll
                            for (int u = 0; u < kResLoads; ++u)
                                if (e + u < hi) ed[u] = w[e + u];
                            int col[kResLoads];
                            double v[kResLoads];
                            bool ok[kResLoads];
#pragma unroll
                            for (int u = 0; u < kResLoads; ++u) {
                                ok[u] = e + u < hi;
                                col[u] = ed[u].idx - (int)c0;
                                v[u] = my_y[k] * (double)ed[u].w;
                                mine_any |= ok[u];
                            }
                            add_products(acc, bits, col, v, ok, sparse && my_y[k] != 0.0, cross, zero_below);
                        }
                        // the next window's segment is [s_lo, s_hi) now: start its loads
                        if (win + 1 < nwin) {
#pragma unroll
                            for (int u = 0; u < kPre; ++u)
                                if (s_lo[k] + u < s_hi[k]) pre[k][u] = w[s_lo[k] + u];
                        }
                    }
                } else {
                    // each wave takes 64 stored entries of the sample at once (one per lane, coalesced),
                    // gathers the extents of their fan-out row segments and parks (y, start, length) in
                    // its own LDS area; then each half-wave reads one segment with 32 lanes (a coalesced
                    // load), four segments per half in flight, and adds the exact products
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
                            // short segments: every lane walks its own (it spans one or two cache
                            // lines), eight weight loads in flight per lane
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
                                int col[8];
                                double v[8];
                                bool ok[8];
#pragma unroll
                                for (int u = 0; u < 8; ++u) {
                                    ok[u] = ed[u].idx >= c0 && ed[u].idx < c1;
                                    col[u] = ed[u].idx - (int)c0;
                                    v[u] = ref.y * (double)ed[u].w;
                                    mine_any |= ok[u];
                                }
                                add_products(acc, bits, col, v, ok, sparse && ref.y != 0.0, cross, zero_below);
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
                                int col[4];
                                double v[4];
                                bool ok[4];
#pragma unroll
                                for (int p = 0; p < 4; ++p) {
                                    ok[p] = ed[p].idx >= c0 && ed[p].idx < c1;
                                    col[p] = ed[p].idx - (int)c0;
                                    v[p] = rr[p].y * (double)ed[p].w;
                                    mine_any |= ok[p];
                                }
                                if (cross) {
                                    add_products(acc, bits, col, v, ok, false, true, zero_below);
                                } else {
#pragma unroll
                                    for (int p = 0; p < 4; ++p)
                                        if (ok[p]) {
                                            atomicAdd(&acc[acc_pos(col[p])], v[p]);
                                            if (sparse && rr[p].y != 0.0) atomicOr(&bits[col[p] >> 5], 1u << (col[p] & 31));
                                        }
                                }
                            }
                        }
                    }
                }
                if (mine_any) any = 1;
                __syncthreads();
                const bool touched = any != 0;
                if (sparse || cross) {
                    if (touched) {
                        // epilogue over marked columns (every touched column, or in cross mode those whose
                        // sum crossed zero_below): count survivors per bitmap word, scan, write
                        const int nw = (width + 31) >> 5;
                        uint32_t word = tid < nw ? bits[tid] : 0u;
                        int keep = 0;
                        for (uint32_t m = word; m; m &= m - 1) {
                            const int col = tid * 32 + __builtin_ctz(m);
                            const double a = acc[acc_pos(col)];
                            keep += a > zero_below && activate(a + (double)bias[c0 + col], ymax) != 0.0f;
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
                            const double a = acc[acc_pos(col)];
                            const float f = a > zero_below ? activate(a + (double)bias[c0 + col], ymax) : 0.0f;
                            if (!cross) acc[acc_pos(col)] = 0.0;
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
                    // epilogue over the whole window in column order (round rd: thread t owns columns
                    // rd * 4096 + 4t .. +3), in two passes so that no output value is held across the scan:
                    // the first counts the survivors of each round (the counts travel in 16-bit fields of
                    // one integer, one scan for all rounds), marks them in a per-thread mask and clears
                    // every other slot it found nonzero; the second writes the marked columns in order and
                    // clears them.
                    unsigned long long packed = 0;
                    uint32_t smask = 0;  // bit 4 rd + v: column rd * 4096 + 4 tid + v survives
#pragma unroll
                    for (int rd = 0; rd < kRounds; ++rd) {
                        int keep = 0;
#pragma unroll
                        for (int v = 0; v < 4; ++v) {
                            const int t = rd * 4 * kThreads + 4 * tid + v;
                            const int at = rd * kRoundCols + v * kThreads + tid;  // acc_pos(t)
                            if (t < width) {
                                const double a = acc[at];
                                if (a > zero_below && activate(a + (double)bias[c0 + t], ymax) != 0.0f) {
                                    ++keep;
                                    smask |= 1u << (4 * rd + v);
                                } else if (__double_as_longlong(a) != 0) {
                                    acc[at] = 0.0;
                                }
                            }
                        }
                        packed |= (unsigned long long)keep << (16 * rd);
                    }
                    unsigned long long incl = packed;
#pragma unroll
                    for (int d = 1; d < 64; d <<= 1) {
                        const unsigned long long v = __shfl_up(incl, d);
                        if (lane >= d) incl += v;
                    }
                    if (lane == 63) wave_tot4[wave] = incl;
                    __syncthreads();
                    unsigned long long before = 0, all = 0;
#pragma unroll
                    for (int u = 0; u < kWaves; ++u) {
                        const unsigned long long v = wave_tot4[u];
                        before += (u < wave) ? v : 0ull;
                        all += v;
                    }
                    const unsigned long long excl = incl - packed;
                    int64_t round_base = ob + written;
                    for (int rd = 0; rd < kRounds; ++rd) {
                        const int sh = 16 * rd;
                        if ((smask >> (4 * rd)) & 15u) {
                            int64_t pos = round_base + (int64_t)((before >> sh) & 0xffff) + (int64_t)((excl >> sh) & 0xffff);
#pragma unroll
                            for (int v = 0; v < 4; ++v) {
                                if ((smask >> (4 * rd + v)) & 1u) {
                                    const int t = rd * 4 * kThreads + 4 * tid + v;
                                    const int at = rd * kRoundCols + v * kThreads + tid;
                                    out_col[pos] = (int32_t)(c0 + t);
                                    out_val[pos] = activate(acc[at] + (double)bias[c0 + t], ymax);
                                    ++pos;
                                    acc[at] = 0.0;
                                }
                            }
                        }
                        round_base += (int64_t)((all >> sh) & 0xffff);
                    }
                    written = round_base - ob;
                }
                __syncthreads();
                if (tid == 0) any = 0;
                if (cross && touched) {
                    // cross mode leaves the unmarked sums in place: clear the window with 16-byte stores
                    double2 *acc2 = reinterpret_cast<double2 *>(acc);
                    for (int t = tid; t < width0 / 2; t += kThreads) acc2[t] = make_double2(0.0, 0.0);
                }
                __syncthreads();
            }
            if (tid == 0) {
                out_cnt[r] = (int32_t)written;
                if (written) atomicAdd(&stats[kStatNnz], (unsigned long long)written);
            }
        }
        __syncthreads();  // chunk_id is rewritten for the next chunk
    }
}

// Pipelined register-resident instance, for layers whose windows only marked columns leave (every b_j <= 0,
// so the scatter marks threshold crossings, or the bias on the structural pattern, so it marks every touched
// column) and three or four accumulator windows (per-row window offsets).  Per sample and window the work is
// short (a few products per thread), so what bounds it is the chain of dependent loads: the sample's entry,
// its fan-out row's window offsets, the segment itself, each a round trip to memory.  Here every load is
// issued at least one window before its value is read.  Workgroup g takes the samples g, g + G, g + 2G, ...
// of the list (G workgroups).  Every window issues the same loads in the same order: at its start the
// entries of its own segment beyond the buffered ones (the address unit has nothing else queued then);
// after its products the first kPipePre entries of the next window's segment (in the last window, of the
// next sample's first window) into the other of two register buffers, the fan-out row starts and window
// offsets of the next sample's entries (read a window earlier), and the next sample's entries.  The
// last two are real in one window each (the entries in the first, the rows in the second, kept from the
// third on) and read one shared address in the others, so the instruction stream, and with it the count of
// loads issued after each one, is the same in every window (each wait is for its own load only) while the
// memory requests stay those the sample needs.  Lanes with nothing to load read w[0] and ignore it (the
// layer has at least one weight).  Samples of up to 2 * kThreads entries give each thread a second entry,
// read without the pipeline (its offsets at the sample's first window, its segment in every window).
// kUniformBias: every b_j is the same value, read once from bias[0], so the epilogue issues no load of its own
// (a bias load there would also wait for the prefetch issued before it).
constexpr int kPipeWin = 4;   // accumulator windows (n <= 4 * 16384)
constexpr int kPipePre = 8;   // entries of a window's segment loaded a window ahead
constexpr int kPipeRem = 8;   // entries beyond those, loaded at the start of their window

// Two consecutive fan-out entries, read with one 16-byte load (8-byte aligned; the packed array has one
// entry of padding, so the pair that starts at a row's last entry stays inside it).
struct __attribute__((aligned(8))) EdgePair {
    Edge e[2];
};

// One stored entry of a sample as the pipelined instance keeps it: the value, the start of the neuron's
// fan-out row, and the offsets of the row's window segments from the current window on (shifted down one
// place per window, so that every index is a constant).  ok = false: no entry (or an invalid one); its
// offsets are then ignored.
struct PipeEntry {
    double y;
    int64_t rb;
    int32_t so[kPipeWin + 1];
    bool ok;
};

template <bool kUniformBias>
__global__ __launch_bounds__(kThreads) void spgemm_pipe_kernel(
    int64_t n, int64_t batch, int nwin, const int64_t *__restrict__ in_row_ptr, const int32_t *__restrict__ in_cnt,
    const int32_t *__restrict__ in_col, const float *__restrict__ in_val, const int64_t *__restrict__ w_ptr,
    const int32_t *__restrict__ w_seg, const Edge *__restrict__ w, const float *__restrict__ bias, double zero_below,
    int pattern, int64_t sparse_limit, double ymax, const int32_t *__restrict__ list, unsigned long long *stats,
    int32_t *__restrict__ out_cnt, int32_t *__restrict__ out_col, float *__restrict__ out_val, uint32_t *err) {
    extern __shared__ __align__(16) double acc[];
    __shared__ uint32_t bits[kBitWords];
    __shared__ int wave_tot[kWaves];
    __shared__ int any;

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int64_t count = (int64_t)stats[kStatResident];
    const int64_t grid = gridDim.x;
    if ((int64_t)blockIdx.x >= count) return;  // uniform: no sample for this workgroup
    const int width0 = (int)(n < kTile ? (n + kRoundCols - 1) / kRoundCols * kRoundCols : kTile);
    for (int t = tid; t < width0; t += kThreads) acc[t] = 0.0;
    for (int t = tid; t < kBitWords; t += kThreads) bits[t] = 0u;
    if (tid == 0) any = 0;
    const int32_t *res = list + 2 * batch;
    const double b_uni = kUniformBias ? (double)bias[0] : 0.0;

    // the samples' rows, 64 at a time: lane l of every wave holds sample s0 + l of this workgroup
    int32_t ref_r = 0, ref_len = 0;
    int64_t ref_yb = 0;
    auto load_refs = [&](int64_t s0) {
        const int64_t j = (int64_t)blockIdx.x + (s0 + lane) * grid;
        ref_r = 0;
        ref_yb = 0;
        ref_len = 0;
        if (j < count) {
            ref_r = res[j];
            const RowIn ri = input_row(ref_r, n, batch, in_row_ptr, in_cnt, in_col, in_val, err);
            ref_yb = ri.yb;
            ref_len = (int32_t)ri.ylen;
        }
        __builtin_amdgcn_s_waitcnt(0);  // once per 64 samples: read at once
    };
    struct Sample {
        int64_t r, yb, ylen;
    };
    auto sample_at = [&](int64_t s) {
        const int k = (int)(s & 63);
        Sample sm;
        sm.r = __builtin_amdgcn_readlane(ref_r, k);
        sm.ylen = __builtin_amdgcn_readlane(ref_len, k);
        sm.yb = (int64_t)(((uint64_t)(uint32_t)__builtin_amdgcn_readlane((int)(ref_yb >> 32), k) << 32) |
                          (uint32_t)__builtin_amdgcn_readlane((int)ref_yb, k));
        return sm;
    };
    // this thread's stored entry of a sample (the row's first entry for lanes past its end; the planning pass
    // sends no empty sample here, and the input then has an entry 0)
    auto entry_load = [&](const Sample &sm, int32_t &ri, float &ry, bool real) {
        const int64_t t = real && sm.ylen > 0 ? sm.yb + (tid < sm.ylen ? tid : 0) : 0;
        ri = in_col[t];
        ry = in_val[t];
    };
    // the entry's fan-out row start and window offsets (row 0 for lanes without a valid entry)
    auto entry_rows = [&](const Sample &sm, int32_t ri, float ry, PipeEntry &e, bool real) {
        const bool has = tid < sm.ylen;
        e.ok = has && ri >= 0 && ri < n;
        if (real && has && !e.ok) atomicOr(err, 1u);
        const int64_t i = real && e.ok ? ri : 0;
        e.y = e.ok ? (double)ry : 0.0;
        e.rb = w_ptr[i];
        const int32_t *sg = w_seg + i * (nwin + 1);  // nwin + 1 = 4 or 5 offsets
#pragma unroll
        for (int t = 0; t < 4; ++t) e.so[t] = sg[t];
        e.so[4] = sg[nwin == 4 ? 4 : 3];
    };
    // entries u < kPipePre of the segment [lo, lo + len) of the row starting at rb, in pairs (w[0], w[1]
    // past its end)
    auto prefetch = [&](int64_t rb, int32_t lo, int32_t len, EdgePair(&buf)[kPipePre / 2]) {
        const Edge *row = w + rb + lo;
#pragma unroll
        for (int u = 0; u < kPipePre / 2; ++u)
            buf[u] = *reinterpret_cast<const EdgePair *>(2 * u < len ? row + 2 * u : w);
    };

    int64_t s = 0;
    load_refs(0);
    Sample cur = sample_at(0), nxt = cur;
    PipeEntry E, N;
    int32_t ni = 0;
    float ny = 0.0f;
    entry_load(cur, ni, ny, true);
    entry_rows(cur, ni, ny, E, true);
    N = E;
    PipeEntry T = E;
    EdgePair bufA[kPipePre / 2], bufB[kPipePre / 2];
    prefetch(E.rb, E.so[0], E.ok ? E.so[1] - E.so[0] : 0, bufA);
    int win = 0;
    int64_t written = 0;
    bool has_next = false;
    // samples of more than kThreads entries: thread t also takes entry t + kThreads, loaded at the sample's
    // first window and read window by window without the pipeline (one round trip per window)
    double y2 = 0.0;
    int64_t rb2 = 0;
    int32_t so2[kPipeWin + 1] = {0, 0, 0, 0, 0};
    bool ok2 = false;

    auto step = [&](EdgePair(&cb)[kPipePre / 2], EdgePair(&pb)[kPipePre / 2]) -> bool {
        const int64_t c0 = (int64_t)win * kTile;
        const int64_t c1 = (c0 + kTile < n) ? c0 + kTile : n;
        const int width = (int)(c1 - c0);
        const bool mark_all = pattern || cur.ylen <= sparse_limit;
        const bool last = win + 1 == nwin;
        if (win == 0) {
            has_next = (int64_t)blockIdx.x + (s + 1) * grid < count;
            if (has_next && ((s + 1) & 63) == 0) load_refs(s + 1);
            nxt = has_next ? sample_at(s + 1) : cur;
        }
        const bool two = cur.ylen > kThreads;  // uniform
        if (two && win == 0) {
            const int64_t t2 = tid + (int64_t)kThreads;
            ok2 = false;
            y2 = 0.0;
            rb2 = 0;
            if (t2 < cur.ylen) {
                const int32_t i2 = in_col[cur.yb + t2];
                const float v2 = in_val[cur.yb + t2];
                if (i2 >= 0 && i2 < n) {
                    ok2 = true;
                    y2 = (double)v2;
                    rb2 = w_ptr[i2];
                    const int32_t *sg = w_seg + (int64_t)i2 * (nwin + 1);
#pragma unroll
                    for (int t = 0; t < 4; ++t) so2[t] = sg[t];
                    so2[4] = sg[nwin == 4 ? 4 : 3];
                } else {
                    atomicOr(err, 1u);
                }
            }
        }
        const int32_t lo = E.so[0], len = E.ok ? E.so[1] - lo : 0;
        const Edge *row = w + E.rb + lo;
        if (win == 2) N = T;  // the next sample's rows, loaded in the second window
        // this window's entries beyond the buffered ones (the other loads follow the products)
        EdgePair rem[kPipeRem / 2];
#pragma unroll
        for (int u = 0; u < kPipeRem / 2; ++u)
            rem[u] = *reinterpret_cast<const EdgePair *>(kPipePre + 2 * u < len ? row + kPipePre + 2 * u : w);
        // the products of this window's segment (buffered ones four at a time)
        bool mine_any = len > 0;
#pragma unroll
        for (int h = 0; h < kPipePre; h += 4) {
            int col[4];
            double v[4];
            bool ok[4];
#pragma unroll
            for (int u = 0; u < 4; ++u) {
                const Edge &ed = cb[(h + u) >> 1].e[(h + u) & 1];
                ok[u] = h + u < len;
                col[u] = ed.idx - (int)c0;
                v[u] = E.y * (double)ed.w;
            }
            add_products<4, true>(acc, bits, col, v, ok, mark_all && E.y != 0.0, !mark_all, zero_below);
        }
#pragma unroll
        for (int h = 0; h < kPipeRem; h += 4) {
            int col[4];
            double v[4];
            bool ok[4];
#pragma unroll
            for (int u = 0; u < 4; ++u) {
                const Edge &ed = rem[(h + u) >> 1].e[(h + u) & 1];
                ok[u] = kPipePre + h + u < len;
                col[u] = ed.idx - (int)c0;
                v[u] = E.y * (double)ed.w;
            }
            add_products<4, true>(acc, bits, col, v, ok, mark_all && E.y != 0.0, !mark_all, zero_below);
        }
        // rare: segments longer than kPipePre + kPipeRem
        for (int e = kPipePre + kPipeRem; e < len; e += 4) {
            EdgePair ep[2];
#pragma unroll
            for (int u = 0; u < 2; ++u)
                ep[u] = *reinterpret_cast<const EdgePair *>(e + 2 * u < len ? row + e + 2 * u : w);
            int col[4];
            double v[4];
            bool ok[4];
#pragma unroll
            for (int u = 0; u < 4; ++u) {
                const Edge &ed = ep[u >> 1].e[u & 1];
                ok[u] = e + u < len;
                col[u] = ed.idx - (int)c0;
                v[u] = E.y * (double)ed.w;
            }
            add_products<4, true>(acc, bits, col, v, ok, mark_all && E.y != 0.0, !mark_all, zero_below);
        }
        if (two) {
            // the second entry's segment of this window
            const int32_t len2 = ok2 ? so2[1] - so2[0] : 0;
            const Edge *row2 = w + rb2 + so2[0];
            mine_any |= len2 > 0;
            for (int e = 0; e < len2; e += 4) {
                EdgePair ep[2];
#pragma unroll
                for (int u = 0; u < 2; ++u)
                    ep[u] = *reinterpret_cast<const EdgePair *>(e + 2 * u < len2 ? row2 + e + 2 * u : w);
                int col[4];
                double v[4];
                bool ok[4];
#pragma unroll
                for (int u = 0; u < 4; ++u) {
                    const Edge &ed = ep[u >> 1].e[u & 1];
                    ok[u] = e + u < len2;
                    col[u] = ed.idx - (int)c0;
                    v[u] = y2 * (double)ed.w;
                }
                add_products<4, true>(acc, bits, col, v, ok, mark_all && y2 != 0.0, !mark_all, zero_below);
            }
        }
        // the next window's (or sample's) buffered entries and the next sample's rows and entries
        {
            const bool nx = last && has_next;
            const int64_t rb = last ? N.rb : E.rb;
            const int32_t plo = last ? N.so[0] : E.so[1];
            const int32_t plen = (last ? (nx && N.ok) : E.ok) ? (last ? N.so[1] : E.so[2]) - plo : 0;
            prefetch(rb, plo, plen, pb);
        }
        entry_rows(nxt, ni, ny, T, win == 1);
        entry_load(nxt, ni, ny, win == 0);
        if (mine_any) any = 1;
        __syncthreads();
        const bool touched = any != 0;
        if (touched) {
            // survivors among the marked columns: count per bitmap word, scan, write in column order
            const int nw = (width + 31) >> 5;
            const uint32_t word = tid < nw ? bits[tid] : 0u;
            int keep = 0;
            for (uint32_t m = word; m; m &= m - 1) {
                const int col = tid * 32 + __builtin_ctz(m);
                const double a = acc[col];
                keep += a > zero_below && activate(a + (kUniformBias ? b_uni : (double)bias[c0 + col]), ymax) != 0.0f;
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
            int64_t pos = cur.r * n + written + off + incl - keep;
            for (uint32_t m = word; m; m &= m - 1) {
                const int col = tid * 32 + __builtin_ctz(m);
                const double a = acc[col];
                const float f = a > zero_below ? activate(a + (kUniformBias ? b_uni : (double)bias[c0 + col]), ymax) : 0.0f;
                if (mark_all) acc[col] = 0.0;
                if (f != 0.0f) {
                    out_col[pos] = (int32_t)(c0 + col);
                    out_val[pos] = f;
                    ++pos;
                }
            }
            if (tid < nw) bits[tid] = 0u;
            written += tot;
            if (tid == 0) any = 0;  // every thread read it before the scan's barrier
            if (!mark_all) {
                // crossing marks leave the other sums in place.  Wave v read only the marked columns of its
                // bitmap words, columns 2048 v .. 2048 v + 2047: once its reads are done it clears that
                // range itself with 16-byte stores, so no workgroup barrier sits between reads and clear
                wave_lds_sync();
                if (wave * 64 * 32 < width0) {
                    double2 *acc2 = reinterpret_cast<double2 *>(acc) + wave * 64 * 16;
                    for (int t = lane; t < 64 * 16; t += 64) acc2[t] = make_double2(0.0, 0.0);
                }
            }
        }
        __syncthreads();  // the window's epilogue is done before the next window's products
        if (!last) {
#pragma unroll
            for (int t = 0; t < kPipeWin; ++t) {
                E.so[t] = E.so[t + 1];
                so2[t] = so2[t + 1];
            }
            ++win;
            return true;
        }
        if (tid == 0) {
            out_cnt[cur.r] = (int32_t)written;
            if (written) atomicAdd(&stats[kStatNnz], (unsigned long long)written);
        }
        if (!has_next) return false;
        ++s;
        cur = nxt;
        E = N;
        win = 0;
        written = 0;
        return true;
    };
    for (;;) {
        if (!step(bufA, bufB)) break;
        if (!step(bufB, bufA)) break;
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

// Dense activations from a batch of sparse rows: element (r, i) of y (zero-filled by the caller) is at
// r * rs + i * cs and receives every stored entry.  Input is either caller CSR (row extents checked as in the
// SpGEMM) or slot rows written by a previous layer.
__global__ __launch_bounds__(256) void densify_kernel(int64_t n, int64_t batch, int64_t rs, int64_t cs,
                                                      const int64_t *__restrict__ in_row_ptr,
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
        yt[r * rs + (int64_t)i * cs] = in_val[yb + t];
    }
}

// Slot rows from dense batch-major activations (already h(.)-applied): keep the nonzeros of row r in
// column order at [r*n, r*n + cnt[r]), compacted with a wave ballot and a scan of the wave totals.
constexpr int kSlotThreads = 1024;
constexpr int kSlotWaves = kSlotThreads / 64;

__global__ __launch_bounds__(kSlotThreads) void dense_to_slots_kernel(int64_t n, const float *__restrict__ y,
                                                                  int32_t *__restrict__ out_cnt,
                                                                  int32_t *__restrict__ out_col,
                                                                  float *__restrict__ out_val) {
    __shared__ int wave_tot[kSlotWaves];
    const int64_t r = blockIdx.x;
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const float *row = y + r * n;
    const int64_t ob = r * n;
    int64_t written = 0;
    for (int64_t base = 0; base < n; base += kSlotThreads) {
        const int64_t j = base + threadIdx.x;
        const float f = j < n ? row[j] : 0.0f;
        const bool keep = f != 0.0f;
        const uint64_t m = __ballot(keep);
        const int pre = lane_rank(m);
        if (lane == 0) wave_tot[wave] = __popcll(m);
        __syncthreads();
        int off = 0, tot = 0;
#pragma unroll
        for (int u = 0; u < kSlotWaves; ++u) {
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

// The same with four consecutive columns per thread (one 16-byte load; rows 16-byte aligned, n % 4 == 0): a
// lane's survivor count (0-4) is scanned across the wave by three bit-sliced ballots, so an iteration covers
// 4096 columns with the same two barriers.  Row r's survivors go to [row_off[r], ...) when row_off is given
// (rows packed back to back: the final CSR), else to [r*n, ...).
__global__ __launch_bounds__(kSlotThreads) void dense_to_slots4_kernel(int64_t n, const float *__restrict__ y,
                                                                   const int64_t *__restrict__ row_off,
                                                                   int32_t *__restrict__ out_cnt,
                                                                   int32_t *__restrict__ out_col,
                                                                   float *__restrict__ out_val) {
    __shared__ int wave_tot[kSlotWaves];
    const int64_t r = blockIdx.x;
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const float4 *row = reinterpret_cast<const float4 *>(y + r * n);
    const int64_t ob = row_off ? row_off[r] : r * n, n4 = n / 4;
    int64_t written = 0;
    for (int64_t base = 0; base < n4; base += kSlotThreads) {
        const int64_t q = base + threadIdx.x;
        const float4 f = q < n4 ? row[q] : make_float4(0.f, 0.f, 0.f, 0.f);
        const float v[4] = {f.x, f.y, f.z, f.w};
        int c = 0;
#pragma unroll
        for (int e = 0; e < 4; ++e) c += v[e] != 0.0f ? 1 : 0;
        const uint64_t b0 = __ballot(c & 1), b1 = __ballot(c & 2), b2 = __ballot(c & 4);
        const int pre = lane_rank(b0) + 2 * lane_rank(b1) + 4 * lane_rank(b2);
        if (lane == 0) wave_tot[wave] = __popcll(b0) + 2 * __popcll(b1) + 4 * __popcll(b2);
        __syncthreads();
        int off = 0, tot = 0;
#pragma unroll
        for (int u = 0; u < kSlotWaves; ++u) {
            const int t = wave_tot[u];
            off += (u < wave) ? t : 0;
            tot += t;
        }
        int64_t o = ob + written + off + pre;
#pragma unroll
        for (int e = 0; e < 4; ++e)
            if (v[e] != 0.0f) {
                out_col[o] = (int32_t)(4 * q + e);
                out_val[o] = v[e];
                ++o;
            }
        written += tot;
        __syncthreads();
    }
    if (threadIdx.x == 0) out_cnt[r] = (int32_t)written;
}

// Nonzeros of each dense batch-major row (n % 4 == 0), for packing the rows straight into CSR.
__global__ __launch_bounds__(kSlotThreads) void dense_count4_kernel(int64_t n, const float *__restrict__ y,
                                                                int32_t *__restrict__ cnt) {
    __shared__ int wave_tot[kSlotWaves];
    const int64_t r = blockIdx.x;
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const float4 *row = reinterpret_cast<const float4 *>(y + r * n);
    int c = 0;
    for (int64_t q = threadIdx.x; q < n / 4; q += kSlotThreads) {
        const float4 f = row[q];
        c += (f.x != 0.0f ? 1 : 0) + (f.y != 0.0f ? 1 : 0) + (f.z != 0.0f ? 1 : 0) + (f.w != 0.0f ? 1 : 0);
    }
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) c += __shfl_xor(c, off);
    if (lane == 0) wave_tot[wave] = c;
    __syncthreads();
    if (threadIdx.x == 0) {
        int t = 0;
#pragma unroll
        for (int u = 0; u < kSlotWaves; ++u) t += wave_tot[u];
        cnt[r] = t;
    }
}

}  // namespace

size_t spgemm_lds_bytes(int64_t n) {
    return (size_t)(n < kTile ? (n + kRoundCols - 1) / kRoundCols * kRoundCols : kTile) * sizeof(double);
}

int spgemm_windows(int64_t n) { return (int)((n + kTile - 1) / kTile); }

bool spgemm_wants_window_index(int64_t n) { return spgemm_windows(n) > 1 && spgemm_windows(n) <= 16; }

hipError_t launch_window_seg(int64_t n, const int64_t *w_ptr, const int32_t *col, int32_t *w_seg, hipStream_t s) {
    window_seg_kernel<<<(unsigned)((n + 255) / 256), 256, 0, s>>>(n, spgemm_windows(n), w_ptr, col, w_seg);
    return hipGetLastError();
}

int64_t spgemm_small_len(int64_t n, int32_t max_fanout) {
    return max_fanout > 0 ? kSmallCap / max_fanout : n;
}

hipError_t launch_spgemm_layer(int64_t n, int64_t batch, const int64_t *in_row_ptr, const int32_t *in_cnt,
                               const int32_t *in_col, const float *in_val, const int64_t *w_ptr, const int32_t *w_seg,
                               const Edge *w, int64_t w_nnz, int32_t max_fanout, const float *bias, int bias_nonpos,
                               int bias_uniform, double zero_below, int pattern, double ymax, int32_t *out_cnt,
                               int32_t *out_col, float *out_val, int32_t *lists, unsigned long long *stats, uint32_t *err,
                               int num_cu, hipStream_t s) {
    if (batch == 0) return hipSuccess;
    const int only_touched = bias_nonpos || pattern;
    if (batch > 0x7fffffffLL) return hipErrorInvalidValue;
    // the accumulator window exceeds the default dynamic LDS limit: raise it once per device (bit d of
    // attr_devices; devices beyond 63 set it on every call)
    static std::atomic<unsigned long long> attr_devices{0};
    int dev = 0;
    hipError_t ed = hipGetDevice(&dev);
    if (ed != hipSuccess) return ed;
    const unsigned long long bit = dev >= 0 && dev < 64 ? 1ull << dev : 0ull;
    if (!bit || !(attr_devices.load(std::memory_order_acquire) & bit)) {
        for (const void *f : {(const void *)spgemm_row_kernel<true>, (const void *)spgemm_row_kernel<false>,
                              (const void *)spgemm_pipe_kernel<true>, (const void *)spgemm_pipe_kernel<false>}) {
            hipError_t e = hipFuncSetAttribute(f, hipFuncAttributeMaxDynamicSharedMemorySize,
                                               (int)((size_t)kTile * sizeof(double)));
            if (e != hipSuccess) return e;
        }
        attr_devices.fetch_or(bit, std::memory_order_release);
    }
    const int nwin = spgemm_windows(n);
    // the bitmap epilogue pays off while a window gets at most ~2048 products
    const double per_win = (double)w_nnz / (double)n / (double)nwin;
    const int64_t sparse_limit = per_win > 0 ? (int64_t)(2048.0 / per_win) : n;
    // segments of at most ~16 entries are walked lane by lane, longer ones by half-waves
    const int lane_segments = (w_seg || nwin == 1) && per_win <= 16.0 ? 1 : 0;
    const int64_t small_len = spgemm_small_len(n, max_fanout);
    // the pipelined instance: three or four windows, and only marked columns leave them; it also takes
    // samples of up to 2 * kThreads entries (a second entry per thread, loaded without the pipeline)
    const bool pipe = w_seg && nwin >= 3 && nwin <= kPipeWin && w_nnz > 0 && (pattern || zero_below >= 0.0);
    const int64_t resident_len = lane_segments ? (int64_t)(pipe ? 2 : kRes) * kThreads : 0;
    spgemm_plan_kernel<<<(unsigned)((batch + 255) / 256), 256, 0, s>>>(
        n, batch, in_row_ptr, in_cnt, in_col, in_val, only_touched, small_len, resident_len, out_cnt, lists, stats,
        err);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    if (only_touched) {
        // each wave strides through the small list (a static share), so launch no more workgroups than the
        // CUs hold at once (the LDS areas bound it to 3 per CU): a workgroup that had to wait for another to
        // finish would start its whole share late
        static std::atomic<int> per_cu_cache[2] = {{0}, {0}};
        int per_cu = per_cu_cache[bias_uniform ? 1 : 0].load(std::memory_order_relaxed);
        if (per_cu <= 0) {
            e = hipOccupancyMaxActiveBlocksPerMultiprocessor(
                &per_cu,
                bias_uniform ? (const void *)spgemm_small_kernel<true> : (const void *)spgemm_small_kernel<false>,
                kSmallWaves * 64, 0);
            if (e != hipSuccess) return e;
            if (per_cu < 1) per_cu = 1;
            per_cu_cache[bias_uniform ? 1 : 0].store(per_cu, std::memory_order_relaxed);
        }
        const int64_t want = (batch + kSmallWaves - 1) / kSmallWaves;
        const int64_t cap = (int64_t)num_cu * per_cu;
        const unsigned blocks = (unsigned)(want < cap ? want : cap);
        if (bias_uniform)
            spgemm_small_kernel<true><<<blocks, kSmallWaves * 64, 0, s>>>(
                n, batch, in_row_ptr, in_cnt, in_col, in_val, w_ptr, w, bias, zero_below, ymax, lists, stats, out_cnt,
                out_col, out_val, err);
        else
            spgemm_small_kernel<false><<<blocks, kSmallWaves * 64, 0, s>>>(
                n, batch, in_row_ptr, in_cnt, in_col, in_val, w_ptr, w, bias, zero_below, ymax, lists, stats, out_cnt,
                out_col, out_val, err);
        e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    const int64_t grid = batch < num_cu ? batch : num_cu;
    if (resident_len > 0 && pipe) {
        if (bias_uniform)
            spgemm_pipe_kernel<true><<<(unsigned)grid, kThreads, spgemm_lds_bytes(n), s>>>(
                n, batch, nwin, in_row_ptr, in_cnt, in_col, in_val, w_ptr, w_seg, w, bias, zero_below, pattern,
                sparse_limit, ymax, lists, stats, out_cnt, out_col, out_val, err);
        else
            spgemm_pipe_kernel<false><<<(unsigned)grid, kThreads, spgemm_lds_bytes(n), s>>>(
                n, batch, nwin, in_row_ptr, in_cnt, in_col, in_val, w_ptr, w_seg, w, bias, zero_below, pattern,
                sparse_limit, ymax, lists, stats, out_cnt, out_col, out_val, err);
        e = hipGetLastError();
        if (e != hipSuccess) return e;
    } else if (resident_len > 0) {
        spgemm_row_kernel<true><<<(unsigned)grid, kThreads, spgemm_lds_bytes(n), s>>>(
            n, batch, nwin, in_row_ptr, in_cnt, in_col, in_val, w_ptr, w_seg, w, bias, only_touched, zero_below,
            pattern, sparse_limit, lane_segments, ymax, lists, stats, out_cnt, out_col, out_val, err);
        e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    spgemm_row_kernel<false><<<(unsigned)grid, kThreads, spgemm_lds_bytes(n), s>>>(
        n, batch, nwin, in_row_ptr, in_cnt, in_col, in_val, w_ptr, w_seg, w, bias, only_touched, zero_below,
        pattern, sparse_limit, lane_segments, ymax, lists, stats, out_cnt, out_col, out_val, err);
    return hipGetLastError();
}

hipError_t launch_compact_rows(int64_t n, int64_t batch, const int32_t *cnt, const int64_t *row_ptr,
                               const int32_t *in_col, const float *in_val, int32_t *out_col, float *out_val,
                               hipStream_t s) {
    if (batch == 0) return hipSuccess;
    compact_rows_kernel<<<(unsigned)batch, 256, 0, s>>>(n, cnt, row_ptr, in_col, in_val, out_col, out_val);
    return hipGetLastError();
}

hipError_t launch_densify(int64_t n, int64_t batch, int64_t ld, const int64_t *in_row_ptr, const int32_t *in_cnt,
                          const int32_t *in_col, const float *in_val, float *yt, float *tmp, uint32_t *err,
                          hipStream_t s) {
    if (batch == 0) return hipSuccess;
    if (!tmp) {
        hipError_t e = hipMemsetAsync(yt, 0, (size_t)n * (size_t)ld * sizeof(float), s);
        if (e != hipSuccess) return e;
        densify_kernel<<<(unsigned)batch, 256, 0, s>>>(n, batch, 1, ld, in_row_ptr, in_cnt, in_col, in_val, yt, err);
        return hipGetLastError();
    }
    // batch-major first (a sample's entries land in one contiguous row, so its stores coalesce; scattered
    // straight into Y^T every 4-byte store hits another row), then one tiled transpose
    hipError_t e = hipMemsetAsync(tmp, 0, (size_t)n * (size_t)batch * sizeof(float), s);
    if (e != hipSuccess) return e;
    densify_kernel<<<(unsigned)batch, 256, 0, s>>>(n, batch, n, 1, in_row_ptr, in_cnt, in_col, in_val, tmp, err);
    e = hipGetLastError();
    if (e != hipSuccess) return e;
    return launch_transpose(tmp, n, yt, ld, batch, n, s);
}

hipError_t launch_dense_to_csr(int64_t n, int64_t batch, const float *y, int32_t *cnt, int64_t *row_ptr,
                               int64_t *scan_tmp, int32_t *out_col, float *out_val, hipStream_t s) {
    if (batch == 0 || n % 4 != 0) return hipErrorInvalidValue;
    dense_count4_kernel<<<(unsigned)batch, kSlotThreads, 0, s>>>(n, y, cnt);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    e = launch_exclusive_scan_i32_to_i64(batch, cnt, row_ptr, scan_tmp, s);
    if (e != hipSuccess) return e;
    dense_to_slots4_kernel<<<(unsigned)batch, kSlotThreads, 0, s>>>(n, y, row_ptr, cnt, out_col, out_val);
    return hipGetLastError();
}

hipError_t launch_dense_to_slots(int64_t n, int64_t batch, const float *y, int32_t *out_cnt, int32_t *out_col,
                                 float *out_val, hipStream_t s) {
    if (batch == 0) return hipSuccess;
    if (n % 4 == 0)
        dense_to_slots4_kernel<<<(unsigned)batch, kSlotThreads, 0, s>>>(n, y, nullptr, out_cnt, out_col, out_val);
    else
        dense_to_slots_kernel<<<(unsigned)batch, kSlotThreads, 0, s>>>(n, y, out_cnt, out_col, out_val);
    return hipGetLastError();
}

}  // namespace sdnn
