// Shared definitions of the HIP library (kernels and host runtime).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace sdnn {

// A weight entry packed for one 64-bit load: the other end of the edge and its fp32 value.
struct __align__(8) Edge {
    int32_t idx;
    float w;
};

constexpr int kWave = 64;

// The kernels (or kernel sequences) a forward call launches, as the library's profiling log names them.
enum KernelKind : int {
    kKernTranspose = 0,   // dense batch-major <-> neuron-major activations
    kKernGather = 1,      // dense-Y product: fan-in gather, one wave per neuron and 64 to 256 samples
    kKernNarrow = 2,      // dense-Y product: narrow-chunk gather, 16 lanes per neuron, 64 samples
    kKernSlots = 3,       // dense-Y product: LDS tiles with scalar-register fp64 weights
    kKernTiled = 4,       // dense-Y product: LDS tiles, weights broadcast from lanes
    kKernDenseGemm = 5,   // dense-W arm on the fp64 matrix cores
    kKernSpgemm = 6,      // sparse-Y product: planning, small-sample and workgroup SpGEMM kernels
    kKernDensify = 7,     // sparse rows -> dense neuron-major activations
    kKernPack = 8,        // dense activations -> CSR result
    kKernCompact = 9,     // sparse slot rows -> CSR result
    kKernBlocked = 10,    // dense-Y product on the sample-blocked layout
    kKernDenseGemm32 = 11 // dense-W arm on the fp32 matrix cores
};

// Wave-local exclusive count of set bits below this lane in a 64-bit ballot.
__device__ __forceinline__ int lane_rank(uint64_t mask) {
    return __builtin_amdgcn_mbcnt_hi((uint32_t)(mask >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)mask, 0u));
}

// h(z) = min(max(z, 0), ymax) in fp64, then one round-to-nearest-even to fp32.
__device__ __forceinline__ float activate(double z, double ymax) {
    if (z < 0.0) z = 0.0;
    if (z > ymax) z = ymax;
    return (float)z;
}

// ---------------------------------------------------------------- launchers (defined in the .hip files)

// setup.hip
hipError_t launch_validate_layer(int64_t n, int64_t nnz, const int64_t *row_ptr, const int32_t *col,
                                 const float *val, const float *bias, uint32_t *flags, hipStream_t s);
hipError_t launch_fanin_counts(int64_t nnz, const int32_t *col, int32_t *counts, hipStream_t s);
hipError_t launch_exclusive_scan_i32_to_i64(int64_t count, const int32_t *in, int64_t *out, int64_t *tmp,
                                            hipStream_t s);
int64_t scan_tmp_elems(int64_t count);
// Fan-in lists (W_k^T, each list sorted by input index) by a stable radix sort of the entries by column;
// scratch holds fanin_sort_bytes(nnz) bytes.
size_t fanin_sort_bytes(int64_t nnz);
hipError_t launch_fanin_lists(int64_t n, int64_t nnz, const int64_t *row_ptr, const int32_t *col, const float *val,
                              Edge *fan, void *scratch, hipStream_t s);
hipError_t launch_max_segment(int64_t n, const int64_t *ptr, int32_t *out, hipStream_t s);
hipError_t launch_pack_edges(int64_t nnz, const int32_t *col, const float *val, Edge *out, hipStream_t s);

// Row pitch (floats) of the neuron-major activation buffers Y^T (n rows of `batch` samples).  Lines taken one
// per row at a power-of-two byte pitch fall into a fraction of an XCD's L2 sets (measured on MI355X: at a
// 16 KiB pitch a 1 MiB working set already misses about half the time, at 16 KiB + 256 B a 3 MiB one stays
// resident), so for wide layers (n > 4096) of 256 samples or more the pitch is an odd multiple of 64 floats
// (256 bytes).  At n = 4096, batch 1024 the padding measured 1-3% slower per layer, so narrower layers keep
// the dense pitch.
inline int64_t act_ld(int64_t n, int64_t batch) {
    return (n <= 4096 || batch < 256) ? batch : (((batch + 63) / 64) | 1) * 64;
}

// spmm.hip
// rows x cols (row pitch in_ld >= cols) -> cols x rows (row pitch out_ld >= rows)
hipError_t launch_transpose(const float *in, int64_t in_ld, float *out, int64_t out_ld, int64_t rows, int64_t cols,
                            hipStream_t s);
int spmm_tile_count(int64_t n);
size_t spmm_tile_mask_elems(int64_t n);
bool spmm_wants_tiles(int64_t n, int64_t nnz);
hipError_t launch_spmm_tile_mask(int64_t n, const int64_t *fan_ptr, const Edge *fan, uint16_t *tile_mask,
                                 hipStream_t s);
// fp64 weight slots of every (input, output) pair for the scalar-register SpMM (zero where W has no entry).
size_t spmm_slot_elems(int64_t n);
bool spmm_wants_slots(int64_t n, int64_t nnz);
hipError_t launch_spmm_slots(int64_t n, const int64_t *fan_ptr, const Edge *fan, double *slots, hipStream_t s);
// pattern != 0: the bias and h apply only where some fan-in entry meets a nonzero input (else 0).
// tile_mask / slots: the high fan-in structures when the layer has them (else null).
// yt, zt: n x batch at row pitch ld (act_ld(n, batch)).
// kind (may be null) receives which product kernel ran (a KernelKind).
hipError_t launch_spmm_fanin(int64_t n, int64_t batch, int64_t ld, const int64_t *fan_ptr, const Edge *fan,
                             const uint16_t *tile_mask, const double *slots, const float *bias, double ymax, int pattern,
                             const float *yt, float *zt, hipStream_t s, int *kind = nullptr);

// gemm.hip
hipError_t launch_dense_from_fanin(int64_t n, const int64_t *fan_ptr, const Edge *fan, double *wt, hipStream_t s);
int gemm_splits(int64_t n, int64_t batch, int num_cu);
size_t gemm_partial_bytes(int64_t n, int64_t batch, int num_cu);
// partial: gemm_partial_bytes(n, batch, num_cu) bytes of scratch (unused when that is 0).
hipError_t launch_gemm_dense_layer(int64_t n, int64_t batch, int64_t ld, const double *wt, const float *bias, double ymax,
                                   const float *yt, float *zt, double *partial, int num_cu, hipStream_t s);

// fp32 copy and the fp32 matrix-core arm (partial: gemm_partial_bytes scratch, used as fp32)
hipError_t launch_dense32_from_fanin(int64_t n, const int64_t *fan_ptr, const Edge *fan, float *wt, hipStream_t s);
hipError_t launch_gemm32_dense_layer(int64_t n, int64_t batch, int64_t ld, const float *wt, const float *bias,
                                     double ymax, const float *yt, float *zt, float *partial, int num_cu, hipStream_t s);

// spgemm.hip
size_t spgemm_lds_bytes(int64_t n);
int spgemm_windows(int64_t n);
bool spgemm_wants_window_index(int64_t n);
hipError_t launch_window_seg(int64_t n, const int64_t *w_ptr, const int32_t *col, int32_t *w_seg, hipStream_t s);
// ylen limit of the small-sample SpGEMM kernel for a layer whose longest fan-out row has max_fanout entries.
int64_t spgemm_small_len(int64_t n, int32_t max_fanout);
// One sparse layer: planning pass, small-sample kernel, the two workgroup kernels (entries kept in
// registers, general).  lists holds 3 * batch int32; stats points to the layer's kSpgemmStats counters
// (zero on entry); counter kSpgemmStatNnz receives the output nnz.
constexpr int kSpgemmStats = 8;
constexpr int kSpgemmStatNnz = 2;
// pattern != 0: the bias and h apply only on the structural pattern of Y_k W_k.  zero_below: a sum z with
// z <= zero_below gives h(z + b_j) = 0 for every j (-max_j b_j when every b_j <= 0, else -infinity), so the
// epilogues read no bias for such a column.  bias_uniform != 0: every b_j equals bias[0].
hipError_t launch_spgemm_layer(int64_t n, int64_t batch, const int64_t *in_row_ptr, const int32_t *in_cnt,
                               const int32_t *in_col, const float *in_val, const int64_t *w_ptr, const int32_t *w_seg,
                               const Edge *w, int64_t w_nnz, int32_t max_fanout, const float *bias, int bias_nonpos,
                               int bias_uniform, double zero_below, int pattern, double ymax, int32_t *out_cnt,
                               int32_t *out_col, float *out_val, int32_t *lists, unsigned long long *stats, uint32_t *err,
                               int num_cu, hipStream_t s);
// Y^T (n x batch at row pitch ld) from sparse rows; tmp (batch x n floats, may be null) stages them batch-major.
hipError_t launch_densify(int64_t n, int64_t batch, int64_t ld, const int64_t *in_row_ptr, const int32_t *in_cnt,
                          const int32_t *in_col, const float *in_val, float *yt, float *tmp, uint32_t *err,
                          hipStream_t s);
hipError_t launch_dense_to_slots(int64_t n, int64_t batch, const float *y, int32_t *out_cnt, int32_t *out_col,
                                 float *out_val, hipStream_t s);
// Dense batch-major rows (n % 4 == 0) straight to CSR: counts, their exclusive scan into row_ptr[batch + 1],
// then the survivors of each row at row_ptr[r] in column order.
hipError_t launch_dense_to_csr(int64_t n, int64_t batch, const float *y, int32_t *cnt, int64_t *row_ptr,
                               int64_t *scan_tmp, int32_t *out_col, float *out_val, hipStream_t s);
hipError_t launch_compact_rows(int64_t n, int64_t batch, const int32_t *cnt, const int64_t *row_ptr,
                               const int32_t *in_col, const float *in_val, int32_t *out_col, float *out_val,
                               hipStream_t s);

// blocked.hip: the sample-blocked activation layout of wide layers (chunks of 32 samples, each chunk an
// n x 32 block: element (r, i) at ((r / 32) * n + i) * 32 + r % 32) and its product.
int64_t blocked_chunks(int64_t batch);
size_t blocked_elems(int64_t n, int64_t batch);   // floats of one blocked activation buffer
bool blocked_wanted(int64_t n, int64_t batch);     // the dense-Y path can use the blocked layout
bool blocked_only(int64_t n);                      // ... and always does (no other dense-Y product this wide)
bool blocked_planned(int64_t n, int64_t nnz);      // set-up builds a layer's schedule and staged lists
size_t blocked_pack_elems(int64_t n, int64_t batch);  // int32 scratch of launch_blocked_to_csr
// Schedule of the blocked product (set-up): neurons sorted by fan-in length within runs of 4096, one entry
// per position (neuron or -1, list length, list start; an empty list starts at the guard entry fan[nnz],
// which set-up zeroes), padded to blocked_sched_elems(n) positions.
struct __align__(16) BlockedSched {
    int32_t j;
    int32_t len;
    int64_t e0;
};
int64_t blocked_sched_elems(int64_t n);
hipError_t launch_blocked_order(int64_t n, const int64_t *fan_ptr, BlockedSched *sched, hipStream_t s);
// The lists of each workgroup of the product (kBlockedTile consecutive schedule positions) copied into one
// contiguous region, in schedule order, so that the product stages them into LDS at once (set-up).  A
// region starts 16-byte aligned (its length is padded to an even count with a zero entry); stage holds
// blocked_stage_elems(n, nnz) entries (the last 128, zeroed, cover the staging loads' overrun).  The schedule's
// list starts are rewritten to point into stage; region_max receives the largest region extent (entries the
// product needs in LDS, 2^30 when a list is too long to stage).
// sizes: blocked_regions(n) int32 of scratch; starts: blocked_regions(n) + 1 int64.
struct __align__(16) BlockedRegion {
    int64_t e0;   // first entry of the region in the staged copy
    int32_t cnt;  // entries of the region (unpadded)
    int32_t pad;
};
int64_t blocked_regions(int64_t n);
size_t blocked_stage_elems(int64_t n, int64_t nnz);
int32_t blocked_stage_cap();  // largest region extent the product stages in LDS
hipError_t launch_blocked_stage(int64_t n, int64_t nnz, const Edge *fan, BlockedSched *sched, Edge *stage,
                                BlockedRegion *regions, int32_t *sizes, int64_t *starts, int64_t *scan_tmp,
                                int32_t *region_max, hipStream_t s);
// regions: the staged lists (null when a region exceeds blocked_stage_cap(): entries come from fan instead).
// nzrows (with regions only, may be null): per chunk a map of blocked_nz_words(n) words, bit i set when
// input row i holds a nonzero; the product then reads no row that is zero in its chunk.
int64_t blocked_nz_words(int64_t n);
hipError_t launch_spmm_blocked(int64_t n, int64_t batch, const BlockedSched *sched, const Edge *fan,
                               const BlockedRegion *regions, const uint32_t *nzrows, const float *bias, double ymax,
                               int pattern, const float *yb, float *zb, hipStream_t s);
// sparse rows (caller CSR, or slot rows with counts) -> blocked; every element is written, except that when
// nzrows is not null the rows of a chunk that hold no nonzero are not stored (only a product given the same map,
// which reads no such row, may consume the result), and the nonzero-row map of every chunk
// (blocked_chunks(batch) * blocked_nz_words(n) words) is written
hipError_t launch_densify_blocked(int64_t n, int64_t batch, const int64_t *in_row_ptr, const int32_t *in_cnt,
                                  const int32_t *in_col, const float *in_val, float *yb, uint32_t *nzrows, uint32_t *err,
                                  hipStream_t s);
// blocked -> CSR: pcnt holds blocked_pack_elems int32, cnt batch int32, row_ptr batch + 1
hipError_t launch_blocked_to_csr(int64_t n, int64_t batch, const float *yb, int32_t *pcnt, int32_t *cnt,
                                 int64_t *row_ptr, int64_t *scan_tmp, int32_t *out_col, float *out_val, hipStream_t s);
// batch-major (row pitch ld) <-> blocked
hipError_t launch_to_blocked(int64_t n, int64_t batch, int64_t ld_in, const float *y, float *yb, hipStream_t s);
hipError_t launch_from_blocked(int64_t n, int64_t batch, int64_t ld_out, const float *yb, float *y, hipStream_t s);

// semiring.hip
enum : int { kSemiringPlusTimes = 0, kSemiringMaxPlus = 1, kSemiringMaxMin = 2, kSemiringMinMax = 3, kSemiringXorAnd = 4 };
float semiring_zero(int semiring);
// Z^T = (Y (+).(x) W)^T from Y^T (n x batch, row pitch ld) over the fan-in lists; no bias, no activation.
hipError_t launch_semiring_mxm(int semiring, int64_t n, int64_t batch, int64_t ld, const int64_t *fan_ptr, const Edge *fan,
                               const float *yt, float *zt, hipStream_t s);
// Z (batch x n, row-major) = Y (+).(x) W for CSR rows Y, row by row from W's packed fan-out rows (w_ptr = W's
// row pointers, w = (column, weight) pairs), without densifying Y (extents and columns checked, flagged in err).
hipError_t launch_semiring_rows(int semiring, int64_t n, int64_t batch, const int64_t *row_ptr, const int32_t *col,
                                const float *val, const int64_t *w_ptr, const Edge *w, float *z, uint32_t *err,
                                hipStream_t s);
}  // namespace sdnn
