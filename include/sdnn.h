/*
 * sdnn.h -- C ABI of the MI355X sparse DNN forward-pass library (libsdnn.so).
 *
 * The library computes the inference step of a ReLU deep neural network,
 *
 *     Y_{k+1} = h(Y_k W_k + 1 b_k^T),   h(x) = min(max(x, 0), ymax),
 *
 * for k = k0 .. k1-1 (Kepner et al., arXiv:1708.02937, Sec. III, batched
 * inference equation and ReLU; Sec. IV, Fig. 4: the function dnn(Y, W, B, L)
 * whose loop body is one matrix multiply over the +.x semiring followed by an
 * element-wise + (max.+ multiply) with the bias and an element-wise max (max.+
 * add) with zero).  The paper writes the product as W_k Y_k with Y stored
 * neurons x batch; this ABI takes Y batch x n (one sample per row) and W_k
 * n_in x n_out, i.e. the transposes of the paper's operands.  ymax = +INFINITY
 * gives the paper's plain ReLU.  The bias is added at every position, as the
 * dense equation states.
 *
 * Arithmetic: inputs and outputs are fp32.  The sparse paths form every product
 * exactly and accumulate in fp64, add the bias and apply h in fp64, and round
 * once to fp32 per layer; the dense-W path (the comparison arm for the paper's
 * sparse-versus-dense experiment, Sec. V) does the same on the fp64 matrix
 * cores, or, as SDNN_ARM_DENSE_F32, computes in fp32 on the fp32 matrix cores.  Output entries equal to zero are not stored in CSR results (Sec. II,
 * 0-element).
 *
 * Conventions for every call:
 *   - Pointers named in comments as "device" must point to memory on the
 *     net's device (the HIP device current when the net was created); "host"
 *     pointers to host memory.  A call that does device work makes the net's
 *     device current while it runs and restores the caller's device before it
 *     returns.  All device memory is the caller's (the net arena, workspaces,
 *     operands); the library allocates none, apart from the fixed scratch array
 *     behind sdnn_forward_dense_noalloc, and frees none.
 *   - CSR matrices use int64 row_ptr (rows + 1 entries, row_ptr[0] = 0),
 *     int32 column indices strictly increasing within a row, fp32 values.
 *   - Work is enqueued on the net's HIP stream and is asynchronous unless the
 *     description says the call synchronises.
 *   - No call aborts or throws; each returns an sdnn_status.  On error,
 *     sdnn_last_error() returns a thread-local text with the detail and the
 *     net stays usable.
 *   - A net must be used from one host thread at a time.
 */
#ifndef SDNN_H
#define SDNN_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
    SDNN_OK = 0,
    SDNN_ERR_NULL_POINTER = 1,       /* a required pointer is NULL */
    SDNN_ERR_INVALID_VALUE = 2,      /* bad size or count, non-finite weight or bias, ymax not > 0 */
    SDNN_ERR_INVALID_INDEX = 3,      /* CSR structure: row_ptr not monotone or not ending at nnz, a
                                        column out of [0, n), unsorted or repeated within a row */
    SDNN_ERR_DIMENSION_MISMATCH = 4, /* layer range outside [0, L] or batch / nnz inconsistent */
    SDNN_ERR_INVALID_OBJECT = 5,     /* NULL net, layer not set, dense arm not built */
    SDNN_ERR_WORKSPACE_TOO_SMALL = 6,/* ws_bytes below sdnn_workspace_size() */
    SDNN_ERR_OUT_OF_MEMORY = 7,      /* a host allocation by the library failed */
    SDNN_ERR_DEVICE = 8,             /* a HIP call failed; detail in sdnn_last_error() */
    SDNN_ERR_UNSUPPORTED = 9         /* a size the library does not handle (see the message) */
} sdnn_status;

/* Which product a dense-Y forward uses for Y_k W_k. */
enum {
    SDNN_ARM_SPARSE = 0,    /* CSR W_k: each output neuron gathers its fan-in (row-per-wavefront SpMM) */
    SDNN_ARM_DENSE = 1,     /* dense W_k with explicit zeros on the fp64 matrix cores (Sec. V dense baseline,
                               the sparse paths' arithmetic: exact products, fp64 sums, one rounding) */
    SDNN_ARM_DENSE_F32 = 2  /* the same dense product in fp32 on the fp32 matrix cores, the arithmetic of the
                               single-precision BLAS the paper compares with (Sec. V.A): fp32 products and
                               sums, so results differ from the others by fp32 rounding of the sums */
};

/* Dense copies an arena holds (sdnn_net_arena_size / sdnn_net_create dense_flags). */
enum {
    SDNN_ARENA_DENSE_F64 = 1, /* an n x n fp64 copy of every layer, for SDNN_ARM_DENSE */
    SDNN_ARENA_DENSE_F32 = 2  /* an n x n fp32 copy of every layer, for SDNN_ARM_DENSE_F32 */
};

/* Where the bias b_k is added (sdnn_net_set_bias_mode). */
enum {
    SDNN_BIAS_EVERYWHERE = 0, /* every position, as the dense equation states (Sec. III); the default */
    SDNN_BIAS_PATTERN = 1     /* only where Y_k W_k has a structural entry: some stored W_k(i, j) meets a
                                 nonzero Y_k(r, i).  This is the Fig. 4 listing read with GraphBLAS
                                 pattern semantics (Sec. IV: eWiseMult with the bias matrix keeps the
                                 pattern of Y_k W_k, eWiseAdd with the zero matrix leaves 0 elsewhere),
                                 with activations stored as their nonzeros. */
};

typedef struct sdnn_net_s *sdnn_net;

/*
 * Bytes of device memory (the net arena) a net of L layers of width n needs, when layer k will hold at
 * most nnz_per_layer[k] weight entries (host array of L values) and dense_flags (SDNN_ARENA_DENSE_*) names
 * the dense copies wanted.  The arena holds every derived copy the library keeps: per layer the packed
 * fan-out rows, the fan-in (transposed) lists, and, as n and the capacity call for them, the tile masks and
 * fp64 weight slots of near-dense layers, the window offsets of wide sparse-activation layers, the schedule
 * and staged lists of the sample-blocked product (layers wider than 16384 neurons, and from 4097 on layers
 * averaging at most 48 entries per neuron) and the dense copies; plus the set-up scratch and the per-forward
 * flags.
 * Errors: NULL_POINTER, INVALID_VALUE (n, L, a capacity outside [0, 2^31-1], unknown flags).
 */
sdnn_status sdnn_net_arena_size(int64_t n, int32_t L, const int64_t *nnz_per_layer, int32_t dense_flags,
                                int64_t *bytes);

/*
 * Create a net of L layers of width n (every layer is n x n, Sec. IV: all
 * layers have the same number of neurons), the shape of the paper's dnn(Y, W, B, L) (Fig. 4), whose
 * operands all belong to the caller.  ymax > 0 is the clamp of h (+INFINITY for plain ReLU).
 * nnz_per_layer (host, L values) caps each layer's entries and dense_flags selects the dense copies, as for
 * sdnn_net_arena_size; `arena` is device memory of at least that many bytes, 256-byte aligned, owned by the
 * caller, which must keep it alive and untouched until sdnn_net_free: the library allocates no device
 * memory for the net, now or later.  `stream` is a hipStream_t (NULL = the default stream).  *net receives
 * a host handle owned by the caller; release it with sdnn_net_free.  Checks the device is a gfx950 part.
 * Errors: NULL_POINTER, INVALID_VALUE (n < 1, n > 2^31-1, L < 0, ymax <= 0 or NaN, bad capacities or
 * flags, arena misaligned), WORKSPACE_TOO_SMALL (arena_bytes below sdnn_net_arena_size), UNSUPPORTED, DEVICE.
 */
sdnn_status sdnn_net_create(sdnn_net *net, int64_t n, int32_t L, float ymax, const int64_t *nnz_per_layer,
                            int32_t dense_flags, void *arena, int64_t arena_bytes, void *stream);

/* Replace the stream later work is enqueued on. */
sdnn_status sdnn_net_set_stream(sdnn_net net, void *stream);

/*
 * Select where the bias is added (SDNN_BIAS_EVERYWHERE or SDNN_BIAS_PATTERN)
 * for later forward calls.  The two readings differ only at positions with no
 * structural product and b_j > 0.  The dense arm (SDNN_ARM_DENSE) stores every
 * zero of W_k, so it computes SDNN_BIAS_EVERYWHERE only; a dense-arm forward
 * in pattern mode fails with UNSUPPORTED.
 * Errors: INVALID_OBJECT, INVALID_VALUE (unknown mode).
 */
sdnn_status sdnn_net_set_bias_mode(sdnn_net net, int32_t mode);

/*
 * Set layer k (0 <= k < L) from a CSR W_k (n_in x n_out, row i = fan-out of
 * input neuron i, Sec. IV: CSR weights) and bias b_k[n] (Sec. III: b_k is
 * replicated over the batch).  All four arrays are device memory that the
 * caller keeps alive and unchanged until the net is freed or the layer is set
 * again.  The call validates the CSR and the values on the device, builds the
 * fan-in (transposed) copy used by the dense-Y path and the layer's other
 * derived structures in its region of the arena (a dense copy is rebuilt by
 * the next sdnn_net_build_dense), and synchronises the net's stream once (the
 * fan-in lists come from a stable radix sort of the entries by column, so each
 * is sorted by input index).  Layers wider than n = 2^24 are rejected with
 * UNSUPPORTED.  On a validation error the layer keeps its previous contents;
 * on a device error it is left unset.
 * Errors: INVALID_OBJECT, NULL_POINTER (nnz > 0 and col/val NULL), INVALID_VALUE
 * (nnz < 0 or >= 2^31, non-finite value), INVALID_INDEX, WORKSPACE_TOO_SMALL (nnz above the layer's
 * capacity in the arena), UNSUPPORTED, DEVICE.
 */
sdnn_status sdnn_net_set_layer(sdnn_net net, int32_t k, int64_t nnz, const int64_t *row_ptr,
                               const int32_t *col_idx, const float *val, const float *bias);

/*
 * Build, for every layer, the dense copies of W_k with explicit zeros that the arena holds (Sec. V.B: the
 * dense version stores zeros explicitly): n*n fp64 values for SDNN_ARM_DENSE and/or n*n fp32 values for
 * SDNN_ARM_DENSE_F32, in the layer's region of the arena.  Synchronises once.
 * Errors: INVALID_OBJECT (a layer not set, or an arena without dense copies), DEVICE.
 */
sdnn_status sdnn_net_build_dense(sdnn_net net);

/* Semirings of Sec. II for sdnn_mxm_dense / sdnn_mxm_csr: (+) . (x), 0-element. */
enum {
    SDNN_SEMIRING_PLUS_TIMES = 0, /* + . x        on R,            0 */
    SDNN_SEMIRING_MAX_PLUS = 1,   /* max . +      on {-inf} u R,   -inf */
    SDNN_SEMIRING_MAX_MIN = 2,    /* max . min    on {-inf} u R,   -inf */
    SDNN_SEMIRING_MIN_MAX = 3,    /* min . max    on R u {+inf},   +inf */
    SDNN_SEMIRING_XOR_AND = 4     /* xor . and    GF(2): a value is 1 when nonzero; results are 0 or 1 */
};

/*
 * Matrix multiply over a semiring (Sec. II.D) with layer k's weights:
 * Z = Y (+).(x) W_k, Z(r, j) = (+) over the stored entries W_k(i, j) of
 * Y(r, i) (x) W_k(i, j), starting from the semiring's 0-element (so a column
 * with no stored entry holds the 0-element).  No bias, no activation.
 * Y and Z are device fp32 arrays of batch x n, row-major; Z may alias Y.
 * Values are carried in fp64 and rounded once; every semiring but + . x is
 * exact.  ws: at least sdnn_workspace_size(net, batch, 0) bytes.  Asynchronous
 * on the net's stream.
 * Errors: INVALID_OBJECT (net NULL or layer k not set), NULL_POINTER,
 * DIMENSION_MISMATCH (k or batch), INVALID_VALUE (semiring), WORKSPACE_TOO_SMALL, DEVICE.
 */
sdnn_status sdnn_mxm_dense(sdnn_net net, int32_t k, int32_t semiring, int64_t batch, const float *Y, float *Z,
                           void *ws, int64_t ws_bytes);

/*
 * The same product for a CSR batch Y (y_row_ptr[batch+1], y_col, y_val; device
 * arrays, columns in [0, n)): entries Y does not store are the semiring's
 * 0-element (the additive identity and multiplicative annihilator, Sec. II.E,
 * so they contribute nothing), and the product is computed row by row over the
 * stored entries only (the row-wise form of Sec. II.D): each stored Y(r, i)
 * folds Y(r, i) (x) W_k(i, :) into an accumulator window of row r, so Y is never
 * densified.  Z (device, batch x n fp32, row-major) receives every entry.
 * + . x adds the exact products in fp64 in the order the accumulator's atomic
 * adds land and rounds once (within one fp32 rounding of the ordered sum, not
 * fixed bit for bit); the other semirings are exact.  ws and ws_bytes are not
 * used (may be NULL / 0).  Synchronises the stream once to report invalid CSR
 * extents or columns (INVALID_INDEX; the offending rows or entries are skipped).
 * Errors: INVALID_OBJECT, NULL_POINTER, DIMENSION_MISMATCH, INVALID_VALUE, INVALID_INDEX, DEVICE.
 */
sdnn_status sdnn_mxm_csr(sdnn_net net, int32_t k, int32_t semiring, int64_t batch, const int64_t *y_row_ptr,
                         const int32_t *y_col, const float *y_val, float *Z, void *ws, int64_t ws_bytes);

/*
 * Bytes of device workspace a forward call over `batch` samples needs:
 * y_is_csr = 0 for sdnn_forward_dense, 1 for sdnn_forward_csr.
 * Errors: INVALID_OBJECT, NULL_POINTER, INVALID_VALUE (batch < 0).
 */
sdnn_status sdnn_workspace_size(sdnn_net net, int64_t batch, int32_t y_is_csr, int64_t *bytes);

/*
 * Layers [k0, k1) on a dense batch: Y_in and Y_out are device fp32 arrays of
 * batch x n, row-major (sample-major).  Y_out receives Y_{k1}; it may alias
 * Y_in.  ws is device memory of at least sdnn_workspace_size(net, batch, 0)
 * bytes that the call may overwrite.  Asynchronous on the net's stream; no
 * host synchronisation.  k0 == k1 copies Y_in to Y_out.
 * Errors: INVALID_OBJECT, NULL_POINTER, DIMENSION_MISMATCH, INVALID_VALUE (arm),
 * WORKSPACE_TOO_SMALL, UNSUPPORTED (dense arm with SDNN_BIAS_PATTERN), DEVICE.
 */
sdnn_status sdnn_forward_dense(sdnn_net net, int32_t k0, int32_t k1, int64_t batch, const float *Y_in,
                               float *Y_out, void *ws, int64_t ws_bytes, int32_t arm);

/*
 * For callers that cannot allocate device memory (code under HIP graph capture, tight serving loops,
 * harnesses that forbid allocation): sdnn_forward_dense without a workspace argument.  Its workspace (the two
 * activation buffers and the dense arm's partial sums) is a fixed device array of the library, one per
 * GPU, sdnn_noalloc_scratch_bytes() bytes (64 MiB), held from the first sdnn_net_create on that GPU until
 * the process ends.  The call itself allocates and frees nothing.  Layers whose workspace
 * (sdnn_workspace_size(net, batch, 0)) exceeds that size are refused with UNSUPPORTED.  Every call on one
 * GPU shares the array, which keeps the last call's contents: calls that overlap on one GPU (other host
 * threads, other nets or streams without ordering between them) race and give undefined results.  Same
 * arguments, result and errors as sdnn_forward_dense otherwise.
 */
sdnn_status sdnn_forward_dense_noalloc(sdnn_net net, int32_t k0, int32_t k1, int64_t batch, const float *Y_in,
                                       float *Y_out, int32_t arm);

/* Size in bytes of the fixed scratch array behind sdnn_forward_dense_noalloc. */
int64_t sdnn_noalloc_scratch_bytes(void);

/*
 * Layers [k0, k1) on a CSR batch Y_in = (y_row_ptr[batch+1], y_col, y_val),
 * device arrays, columns strictly increasing within a row (not checked; the
 * result is undefined otherwise).  y_col and y_val may be NULL when every row
 * is empty.  Row extents outside [0, nnz] and column indices outside [0, n)
 * are detected on the device and reported as INVALID_INDEX (the offending
 * entries are skipped, so no access leaves the arrays).  The result Y_{k1} is written in CSR with
 * no stored zeros: out_row_ptr (device, batch + 1 int64, caller-owned)
 * receives the row pointers; *out_col and *out_val (host pointers to receive
 * device addresses) point into ws and stay valid until ws is reused; *out_nnz
 * (host) receives nnz(Y_{k1}).  ws is device memory of at least
 * sdnn_workspace_size(net, batch, 1) bytes.  Synchronises the net's stream
 * at the end, to read the nnz, and at the activation-format decisions below.
 * Internally, activations stay as sparse rows (row-wise SpGEMM) until the
 * first layer whose input holds at least batch * n / 8 entries or whose bias
 * is positive on at least a quarter of the neurons (its output is then mostly
 * nonzero); from that layer on they are kept dense and neuron-major inside ws
 * and packed back into CSR after the last layer.  The host tracks an upper
 * bound of each layer's input size and reads the exact count (one stream
 * synchronisation) only when the bound reaches the threshold, always for the
 * first layer.  The result is the same either way.
 * Errors: INVALID_OBJECT, NULL_POINTER, DIMENSION_MISMATCH, INVALID_INDEX, WORKSPACE_TOO_SMALL, UNSUPPORTED
 * (batch above 2^24), DEVICE.
 */
sdnn_status sdnn_forward_csr(sdnn_net net, int32_t k0, int32_t k1, int64_t batch, const int64_t *y_row_ptr,
                             const int32_t *y_col, const float *y_val, void *ws, int64_t ws_bytes,
                             int64_t *out_row_ptr, int32_t **out_col, float **out_val, int64_t *out_nnz);

/*
 * Profiling log.  While enabled, every forward call records a pair of HIP events on the net's stream around
 * each layer's product launch(es) and around the format changes, so the log holds the GPU time of each.
 * The kernel field names what ran (SDNN_KERNEL_*); layer is the layer index, or -1 for a format change.
 * Recording costs two event records per entry and is not meant for calls under graph capture.
 */
enum {
    SDNN_KERNEL_TRANSPOSE = 0,  /* dense batch-major <-> neuron-major activations (sdnn_forward_dense) */
    SDNN_KERNEL_GATHER = 1,     /* dense-Y CSR product: fan-in gather (one wavefront per output neuron) */
    SDNN_KERNEL_NARROW = 2,     /* dense-Y CSR product: narrow-chunk gather (16 lanes per output neuron) */
    SDNN_KERNEL_SLOTS = 3,      /* dense-Y CSR product: LDS tiles, scalar-register fp64 weights */
    SDNN_KERNEL_TILED = 4,      /* dense-Y CSR product: LDS tiles */
    SDNN_KERNEL_DENSE_GEMM = 5, /* dense-W arm on the matrix cores */
    SDNN_KERNEL_SPGEMM = 6,     /* sparse-Y product: row-wise SpGEMM with fused epilogue and compaction */
    SDNN_KERNEL_DENSIFY = 7,    /* sparse rows -> dense neuron-major activations (sdnn_forward_csr) */
    SDNN_KERNEL_PACK = 8,       /* dense activations -> CSR result (sdnn_forward_csr) */
    SDNN_KERNEL_COMPACT = 9,    /* sparse rows -> CSR result (sdnn_forward_csr) */
    SDNN_KERNEL_BLOCKED = 10,   /* dense-Y CSR product on the sample-blocked layout (wide layers, short lists) */
    SDNN_KERNEL_DENSE_GEMM32 = 11 /* dense-W arm on the fp32 matrix cores */
};

typedef struct {
    int32_t layer;  /* layer index, or -1 */
    int32_t kernel; /* SDNN_KERNEL_* */
    float ms;       /* GPU time between the two events */
} sdnn_kernel_time;

/* enable != 0 clears the log and starts recording; 0 stops recording (the log is kept until read). */
sdnn_status sdnn_net_set_profiling(sdnn_net net, int32_t enable);

/*
 * Synchronises the net's stream, writes up to max_records entries of the log, oldest first, into out
 * (host), sets *count (host) to the number of entries the log held, and clears it.
 * Errors: INVALID_OBJECT, NULL_POINTER, DEVICE.
 */
sdnn_status sdnn_net_read_profile(sdnn_net net, sdnn_kernel_time *out, int32_t max_records, int32_t *count);

/* Free the net's host handle (synchronises its stream); the arena is the caller's to release afterwards. */
sdnn_status sdnn_net_free(sdnn_net net);

/* Static text for a status code. */
const char *sdnn_status_string(sdnn_status status);

/* Detail of the last error on the calling thread ("" if none). */
const char *sdnn_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* SDNN_H */
