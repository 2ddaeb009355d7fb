// Host runtime behind the C ABI of include/sdnn.h: argument checks, layer set-up, workspace carving and
// the layer loop of the forward pass (the loop of the paper's dnn() function, Fig. 4, Sec. IV), with every
// layer's work enqueued on the net's HIP stream.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdio>
#include <cstring>
#include <mutex>
#include <string>
#include <vector>

#include "common.h"
#include "sdnn.h"

using sdnn::Edge;

namespace {

thread_local std::string g_last_error;

sdnn_status fail(sdnn_status s, const std::string &msg) {
    g_last_error = msg;
    return s;
}

sdnn_status fail_hip(hipError_t e, const char *what) {
    return fail(SDNN_ERR_DEVICE, std::string(what) + ": " + hipGetErrorString(e));
}

// Makes the net's device current for one call and gives the caller's device back on return.
struct DeviceScope {
    int prev = -1;  // the caller's device when it has to be restored
    hipError_t err = hipSuccess;
    explicit DeviceScope(int dev) {
        int cur = 0;
        err = hipGetDevice(&cur);
        if (err == hipSuccess && cur != dev) {
            err = hipSetDevice(dev);
            if (err == hipSuccess) prev = cur;
        }
    }
    ~DeviceScope() {
        if (prev >= 0) (void)hipSetDevice(prev);
    }
    DeviceScope(const DeviceScope &) = delete;
    DeviceScope &operator=(const DeviceScope &) = delete;
};

#define SDNN_ON_DEVICE(net)                                                     \
    DeviceScope device_scope_((net)->device);                                   \
    if (device_scope_.err != hipSuccess) return fail_hip(device_scope_.err, "hipSetDevice")

#define SDNN_HIP(call)                                      \
    do {                                                    \
        hipError_t e_ = (call);                             \
        if (e_ != hipSuccess) return fail_hip(e_, #call);   \
    } while (0)

struct Layer {
    bool set = false;
    int64_t nnz = 0;
    const int64_t *row_ptr = nullptr;  // caller-owned fan-out CSR and bias
    const int32_t *col = nullptr;
    const float *val = nullptr;
    const float *bias = nullptr;
    bool bias_nonpos = true;
    bool bias_uniform = false;  // every b_j has the same bits
    int64_t pos_bias = 0;      // neurons with b_j > 0
    double zero_below = -INFINITY;  // every b_j <= 0: -max_j b_j (a sum at most this is zero after h), else -inf
    int32_t max_fanout = 0;    // longest fan-out row of W_k
    Edge *w_pack = nullptr;    // fan-out entries packed as (column, weight)
    int64_t *fan_ptr = nullptr;  // fan-in CSR (W_k^T)
    Edge *fan = nullptr;
    uint16_t *tile_mask = nullptr;  // which rows of each 16-row input tile each fan-in list holds (high fan-in only)
    double *slots = nullptr;        // fp64 weight of every (input, output) pair, tile-major (high fan-in, n^2 fits)
    int32_t *w_seg = nullptr;     // where each fan-out row crosses each accumulator window (wide layers only)
    sdnn::BlockedSched *sched = nullptr;  // schedule of the blocked product (wide layers, short lists)
    Edge *stage = nullptr;                 // its lists in schedule order, one region per workgroup
    sdnn::BlockedRegion *regions = nullptr;  // the regions (null when one exceeds the product's LDS capacity)
    double *dense_wt = nullptr;  // n x n, W_k k-major in fp64 (zeros explicit), for the fp64 dense arm
    float *dense_wt32 = nullptr; // the same in fp32, for the fp32 dense arm
    bool dense_ready = false, dense32_ready = false;  // the dense copies hold the current W_k
};

constexpr size_t kAlign = 256;
inline size_t align_up(size_t x) { return (x + kAlign - 1) / kAlign * kAlign; }

// ---------------------------------------------------------------------------------------- net arena
// All device memory a net keeps lives in one caller-owned arena, laid out once at creation from n, L, the
// entry capacity of every layer and which dense copies are wanted.  Per layer, at fixed offsets: the packed
// fan-out rows, the fan-in (W_k^T) pointers and lists (plus a zero guard entry), and the optional structures
// whose need follows from n and the capacity (tile masks and fp64 weight slots for dense-ish layers, window
// offsets for the SpGEMM of wide layers, the blocked product's schedule and staged lists, the dense
// copies).  Shared: the set-up scratch (counts, scan, radix-sort buffers, sized for the largest layer) and
// the small per-forward flags and counters.
constexpr size_t kAbsent = ~size_t(0);

struct LayerPlan {
    size_t w_pack = kAbsent, fan_ptr = kAbsent, fan = kAbsent, tile_mask = kAbsent, slots = kAbsent,
           w_seg = kAbsent, sched = kAbsent, stage = kAbsent, regions = kAbsent, starts = kAbsent,
           dense64 = kAbsent, dense32 = kAbsent;
    size_t bytes = 0;
};

struct NetPlan {
    size_t flags = 0, d_int = 0, stats = 0, counts = 0, tmp = 0, sort = 0;
    std::vector<size_t> layer_off;
    std::vector<LayerPlan> layer;
    size_t bytes = 0;
};

size_t take(size_t &off, size_t bytes) {
    const size_t at = off;
    off = align_up(off + bytes);
    return at;
}

LayerPlan plan_layer(int64_t n, int64_t cap, int32_t dense_flags) {
    LayerPlan lp;
    size_t off = 0;
    // one entry more than the layer's: 16-byte loads of entry pairs may read one entry past a row's end
    lp.w_pack = take(off, (size_t)(std::max<int64_t>(cap, 1) + 1) * sizeof(Edge));
    lp.fan_ptr = take(off, (size_t)(n + 1) * sizeof(int64_t));
    lp.fan = take(off, (size_t)(cap + 1) * sizeof(Edge));
    if (sdnn::spmm_wants_tiles(n, cap)) lp.tile_mask = take(off, sdnn::spmm_tile_mask_elems(n) * sizeof(uint16_t));
    if (sdnn::spmm_wants_slots(n, cap)) lp.slots = take(off, sdnn::spmm_slot_elems(n) * sizeof(double));
    if (sdnn::spgemm_wants_window_index(n))
        lp.w_seg = take(off, (size_t)n * (size_t)(sdnn::spgemm_windows(n) + 1) * sizeof(int32_t));
    if (sdnn::blocked_planned(n, cap)) {
        lp.sched = take(off, (size_t)sdnn::blocked_sched_elems(n) * sizeof(sdnn::BlockedSched));
        lp.stage = take(off, sdnn::blocked_stage_elems(n, cap) * sizeof(Edge));
        lp.regions = take(off, (size_t)sdnn::blocked_regions(n) * sizeof(sdnn::BlockedRegion));
        lp.starts = take(off, (size_t)(sdnn::blocked_regions(n) + 1) * sizeof(int64_t));
    }
    if (dense_flags & SDNN_ARENA_DENSE_F64) lp.dense64 = take(off, (size_t)n * (size_t)n * sizeof(double));
    if (dense_flags & SDNN_ARENA_DENSE_F32) lp.dense32 = take(off, (size_t)n * (size_t)n * sizeof(float));
    lp.bytes = off;
    return lp;
}

NetPlan plan_net(int64_t n, int32_t L, const int64_t *caps, int32_t dense_flags) {
    NetPlan np;
    size_t off = 0;
    int64_t max_cap = 0;
    for (int32_t k = 0; k < L; ++k) max_cap = std::max(max_cap, caps[k]);
    np.flags = take(off, 4 * sizeof(uint32_t));
    np.d_int = take(off, 4 * sizeof(int32_t));
    np.stats = take(off, (size_t)std::max<int32_t>(L, 1) * sdnn::kSpgemmStats * sizeof(unsigned long long));
    np.counts = take(off, (size_t)n * sizeof(int32_t));
    np.tmp = take(off, (size_t)sdnn::scan_tmp_elems(n) * sizeof(int64_t));
    np.sort = take(off, sdnn::fanin_sort_bytes(max_cap));
    for (int32_t k = 0; k < L; ++k) {
        np.layer.push_back(plan_layer(n, caps[k], dense_flags));
        np.layer_off.push_back(take(off, np.layer.back().bytes));
    }
    np.bytes = off;
    return np;
}

template <typename T>
T *at(char *base, size_t off) {
    return off == kAbsent ? nullptr : reinterpret_cast<T *>(base + off);
}

sdnn_status check_plan_args(int64_t n, int32_t L, const int64_t *caps, int32_t dense_flags) {
    if (n < 1 || n > 0x7fffffffLL) return fail(SDNN_ERR_INVALID_VALUE, "n must be in [1, 2^31-1]");
    if (L < 0) return fail(SDNN_ERR_INVALID_VALUE, "L must be >= 0");
    if (L > 0 && !caps) return fail(SDNN_ERR_NULL_POINTER, "nnz_per_layer is required when L > 0");
    if (dense_flags & ~(SDNN_ARENA_DENSE_F64 | SDNN_ARENA_DENSE_F32))
        return fail(SDNN_ERR_INVALID_VALUE, "unknown dense-copy flags");
    for (int32_t k = 0; k < L; ++k)
        if (caps[k] < 0 || caps[k] > 0x7fffffffLL) return fail(SDNN_ERR_INVALID_VALUE, "layer capacities must be in [0, 2^31-1]");
    return SDNN_OK;
}

// Workspace of a CSR forward: two slot buffers (count[batch], col[n*ld], val[n*ld] with ld = act_ld(n, batch)
// >= batch, so that a pair of them also holds two n x batch activation buffers at row pitch ld) and a scan area.
struct CsrWs {
    int32_t *cnt[2];
    int32_t *col[2];
    float *val[2];
    int32_t *lists;  // 3 * batch: the sample lists of the layer being computed
    int64_t *scan_tmp;
    int32_t *pcnt;   // per (part, sample) counts of the blocked -> CSR packing
    uint32_t *nzrows;  // nonzero-row maps of a sparse input in the blocked layout
    size_t bytes;
};

CsrWs carve_csr(void *base, int64_t n, int64_t batch) {
    CsrWs w{};
    char *p = (char *)base;
    size_t off = 0;
    const size_t slots = (size_t)sdnn::act_ld(n, batch) * (size_t)n;
    for (int b = 0; b < 2; ++b) {
        w.cnt[b] = (int32_t *)(p + off);
        off = align_up(off + (size_t)batch * sizeof(int32_t));
        w.col[b] = (int32_t *)(p + off);
        off = align_up(off + slots * sizeof(int32_t));
        w.val[b] = (float *)(p + off);
        off = align_up(off + slots * sizeof(float));
    }
    w.lists = (int32_t *)(p + off);
    off = align_up(off + 3 * (size_t)batch * sizeof(int32_t));
    w.scan_tmp = (int64_t *)(p + off);
    off = align_up(off + (size_t)sdnn::scan_tmp_elems(batch) * sizeof(int64_t));
    w.pcnt = (int32_t *)(p + off);
    w.nzrows = nullptr;
    if (sdnn::blocked_wanted(n, batch)) {
        off = align_up(off + sdnn::blocked_pack_elems(n, batch) * sizeof(int32_t));
        w.nzrows = (uint32_t *)(p + off);
        off = align_up(off + (size_t)sdnn::blocked_chunks(batch) * (size_t)sdnn::blocked_nz_words(n) * sizeof(uint32_t));
    }
    w.bytes = off;
    return w;
}

constexpr int64_t kMaxScan = 16777216;  // longest array the device prefix sum handles (fan-in pointers, row pointers)

// bytes of one n x batch fp32 activation buffer at row pitch act_ld(n, batch)
size_t act_bytes(int64_t n, int64_t batch) {
    return align_up((size_t)n * (size_t)sdnn::act_ld(n, batch) * sizeof(float));
}

// two activation buffers, then the dense arm's split-K partial sums (small batches only)
size_t dense_ws_bytes(int64_t n, int64_t batch, int num_cu) {
    return 2 * act_bytes(n, batch) + align_up(sdnn::gemm_partial_bytes(n, batch, num_cu));
}

// Workspace of sdnn_forward_dense_noalloc: a fixed device array, one copy per GPU, held until the process
// ends.  In host code the symbol is only a host-side stand-in; kernels get the device address that
// hipGetSymbolAddress returns for the current device (kept per device in g_scratch).
constexpr size_t kScratchBytes = size_t(64) << 20;
static __device__ __align__(256) unsigned char scratch[kScratchBytes];

constexpr int kMaxDevices = 64;
struct ScratchSlot {
    std::once_flag once;
    void *ptr = nullptr;
    hipError_t err = hipErrorNotInitialized;
};
ScratchSlot g_scratch[kMaxDevices];

// Looks up this device's copy of the scratch array once; the device must be current.
void scratch_init(int dev) {
    if (dev < 0 || dev >= kMaxDevices) return;
    ScratchSlot &slot = g_scratch[dev];
    std::call_once(slot.once, [&slot]() {
        void *p = nullptr;
        const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        slot.err = e;
        slot.ptr = e == hipSuccess ? p : nullptr;
        if (e != hipSuccess) (void)hipGetLastError();
    });
}

}  // namespace

struct sdnn_net_s {
    int64_t n = 0;
    int32_t L = 0;
    double ymax = INFINITY;
    int bias_pattern = 0;  // SDNN_BIAS_PATTERN: bias only on the structural pattern of Y_k W_k
    hipStream_t stream = nullptr;
    int device = 0;
    std::vector<Layer> layers;
    uint32_t *d_flags = nullptr;
    int32_t *d_int = nullptr;
    unsigned long long *d_stats = nullptr;  // kSpgemmStats counters per layer of a forward call
    int num_cu = 256;
    char *arena = nullptr;  // caller-owned device memory holding everything above and every layer's copies
    NetPlan plan;
    std::vector<int64_t> caps;  // entry capacity of each layer
    int32_t dense_flags = 0;
    // profiling log (sdnn_net_set_profiling): one pair of events around each timed launch sequence
    struct ProfRec {
        int32_t layer, kernel;
        hipEvent_t a, b;
    };
    bool profiling = false;
    std::vector<ProfRec> prof;
    std::vector<hipEvent_t> ev_free;
};

namespace {

// Whether dense-Y layers [k0, k1) run on the sample-blocked layout: always beyond 16384 neurons; from 4097 to
// 16384 only when every layer of the range stages its lists (short lists), since the other dense-Y products
// share the neuron-major layout and the forward keeps one layout throughout.
bool use_blocked(const sdnn_net_s *net, int32_t k0, int32_t k1, int64_t batch) {
    if (!sdnn::blocked_wanted(net->n, batch)) return false;
    if (sdnn::blocked_only(net->n)) return true;
    for (int32_t k = k0; k < k1; ++k)
        if (!net->layers[(size_t)k].regions) return false;
    return true;
}

hipError_t prof_event(sdnn_net net, hipEvent_t *e) {
    if (!net->ev_free.empty()) {
        *e = net->ev_free.back();
        net->ev_free.pop_back();
        return hipSuccess;
    }
    return hipEventCreate(e);
}

// Opens a profiling record for the launches that follow (layer -1: not a layer's product); *idx = -1 when
// profiling is off.
hipError_t prof_begin(sdnn_net net, int32_t layer, int kind, int *idx) {
    *idx = -1;
    if (!net->profiling) return hipSuccess;
    sdnn_net_s::ProfRec r{layer, kind, nullptr, nullptr};
    hipError_t e = prof_event(net, &r.a);
    if (e != hipSuccess) return e;
    e = prof_event(net, &r.b);
    if (e == hipSuccess) e = hipEventRecord(r.a, net->stream);
    if (e != hipSuccess) {
        net->ev_free.push_back(r.a);
        if (r.b) net->ev_free.push_back(r.b);
        return e;
    }
    net->prof.push_back(r);
    *idx = (int)net->prof.size() - 1;
    return hipSuccess;
}

// Closes record idx (kind >= 0 replaces the kernel kind given at the start).
hipError_t prof_end(sdnn_net net, int idx, int kind = -1) {
    if (idx < 0) return hipSuccess;
    if (kind >= 0) net->prof[(size_t)idx].kernel = kind;
    return hipEventRecord(net->prof[(size_t)idx].b, net->stream);
}

void prof_clear(sdnn_net net) {
    for (auto &r : net->prof) {
        net->ev_free.push_back(r.a);
        net->ev_free.push_back(r.b);
    }
    net->prof.clear();
}

}  // namespace

static_assert(SDNN_KERNEL_TRANSPOSE == sdnn::kKernTranspose && SDNN_KERNEL_GATHER == sdnn::kKernGather &&
                  SDNN_KERNEL_NARROW == sdnn::kKernNarrow && SDNN_KERNEL_SLOTS == sdnn::kKernSlots &&
                  SDNN_KERNEL_TILED == sdnn::kKernTiled && SDNN_KERNEL_DENSE_GEMM == sdnn::kKernDenseGemm &&
                  SDNN_KERNEL_SPGEMM == sdnn::kKernSpgemm && SDNN_KERNEL_DENSIFY == sdnn::kKernDensify &&
                  SDNN_KERNEL_PACK == sdnn::kKernPack && SDNN_KERNEL_COMPACT == sdnn::kKernCompact &&
                  SDNN_KERNEL_BLOCKED == sdnn::kKernBlocked && SDNN_KERNEL_DENSE_GEMM32 == sdnn::kKernDenseGemm32,
              "profiling kernel ids of the header and the library agree");

extern "C" {

const char *sdnn_status_string(sdnn_status s) {
    switch (s) {
        case SDNN_OK: return "SDNN_OK";
        case SDNN_ERR_NULL_POINTER: return "SDNN_ERR_NULL_POINTER";
        case SDNN_ERR_INVALID_VALUE: return "SDNN_ERR_INVALID_VALUE";
        case SDNN_ERR_INVALID_INDEX: return "SDNN_ERR_INVALID_INDEX";
        case SDNN_ERR_DIMENSION_MISMATCH: return "SDNN_ERR_DIMENSION_MISMATCH";
        case SDNN_ERR_INVALID_OBJECT: return "SDNN_ERR_INVALID_OBJECT";
        case SDNN_ERR_WORKSPACE_TOO_SMALL: return "SDNN_ERR_WORKSPACE_TOO_SMALL";
        case SDNN_ERR_OUT_OF_MEMORY: return "SDNN_ERR_OUT_OF_MEMORY";
        case SDNN_ERR_DEVICE: return "SDNN_ERR_DEVICE";
        case SDNN_ERR_UNSUPPORTED: return "SDNN_ERR_UNSUPPORTED";
    }
    return "SDNN_ERR_UNKNOWN";
}

const char *sdnn_last_error(void) { return g_last_error.c_str(); }

sdnn_status sdnn_net_arena_size(int64_t n, int32_t L, const int64_t *nnz_per_layer, int32_t dense_flags,
                                int64_t *bytes) {
    g_last_error.clear();
    if (!bytes) return fail(SDNN_ERR_NULL_POINTER, "bytes is NULL");
    sdnn_status st = check_plan_args(n, L, nnz_per_layer, dense_flags);
    if (st != SDNN_OK) return st;
    *bytes = (int64_t)plan_net(n, L, nnz_per_layer, dense_flags).bytes;
    return SDNN_OK;
}

sdnn_status sdnn_net_create(sdnn_net *out, int64_t n, int32_t L, float ymax, const int64_t *nnz_per_layer,
                            int32_t dense_flags, void *arena, int64_t arena_bytes, void *stream) {
    g_last_error.clear();
    if (!out) return fail(SDNN_ERR_NULL_POINTER, "net is NULL");
    *out = nullptr;
    sdnn_status st = check_plan_args(n, L, nnz_per_layer, dense_flags);
    if (st != SDNN_OK) return st;
    if (!(ymax > 0.0f)) return fail(SDNN_ERR_INVALID_VALUE, "ymax must be > 0 (INFINITY for plain ReLU)");
    if (!arena) return fail(SDNN_ERR_NULL_POINTER, "arena is NULL");
    if (((uintptr_t)arena) % kAlign != 0) return fail(SDNN_ERR_INVALID_VALUE, "arena must be 256-byte aligned");
    NetPlan plan = plan_net(n, L, nnz_per_layer, dense_flags);
    if (arena_bytes < (int64_t)plan.bytes)
        return fail(SDNN_ERR_WORKSPACE_TOO_SMALL, "arena smaller than sdnn_net_arena_size(): need " +
                                                      std::to_string(plan.bytes) + " bytes");
    int dev = 0;
    SDNN_HIP(hipGetDevice(&dev));
    hipDeviceProp_t prop;
    SDNN_HIP(hipGetDeviceProperties(&prop, dev));
    if (std::strncmp(prop.gcnArchName, "gfx950", 6) != 0)
        return fail(SDNN_ERR_UNSUPPORTED, std::string("built for gfx950, device is ") + prop.gcnArchName);
    sdnn_net net = new (std::nothrow) sdnn_net_s();
    if (!net) return fail(SDNN_ERR_OUT_OF_MEMORY, "host allocation failed");
    net->n = n;
    net->L = L;
    net->ymax = (double)ymax;
    net->stream = (hipStream_t)stream;
    net->device = dev;
    net->num_cu = prop.multiProcessorCount > 0 ? prop.multiProcessorCount : 256;
    net->layers.resize((size_t)L);
    net->arena = (char *)arena;
    net->plan = std::move(plan);
    net->caps.assign(nnz_per_layer, nnz_per_layer + L);
    net->dense_flags = dense_flags;
    net->d_flags = at<uint32_t>(net->arena, net->plan.flags);
    net->d_int = at<int32_t>(net->arena, net->plan.d_int);
    net->d_stats = at<unsigned long long>(net->arena, net->plan.stats);
    scratch_init(dev);  // this device's copy of the allocation-free entry point's scratch array
    *out = net;
    return SDNN_OK;
}

sdnn_status sdnn_net_set_stream(sdnn_net net, void *stream) {
    g_last_error.clear();
    if (!net) return fail(SDNN_ERR_INVALID_OBJECT, "net is NULL");
    net->stream = (hipStream_t)stream;
    return SDNN_OK;
}

sdnn_status sdnn_net_set_bias_mode(sdnn_net net, int32_t mode) {
    g_last_error.clear();
    if (!net) return fail(SDNN_ERR_INVALID_OBJECT, "net is NULL");
    if (mode != SDNN_BIAS_EVERYWHERE && mode != SDNN_BIAS_PATTERN) return fail(SDNN_ERR_INVALID_VALUE, "unknown bias mode");
    net->bias_pattern = mode == SDNN_BIAS_PATTERN ? 1 : 0;
    return SDNN_OK;
}

sdnn_status sdnn_net_set_layer(sdnn_net net, int32_t k, int64_t nnz, const int64_t *row_ptr, const int32_t *col_idx,
                               const float *val, const float *bias) {
    g_last_error.clear();
    if (!net) return fail(SDNN_ERR_INVALID_OBJECT, "net is NULL");
    if (k < 0 || k >= net->L) return fail(SDNN_ERR_DIMENSION_MISMATCH, "layer index outside [0, L)");
    if (!row_ptr || !bias) return fail(SDNN_ERR_NULL_POINTER, "row_ptr and bias are required");
    if (nnz < 0 || nnz > 0x7fffffffLL) return fail(SDNN_ERR_INVALID_VALUE, "nnz must be in [0, 2^31-1]");
    if (nnz > 0 && (!col_idx || !val)) return fail(SDNN_ERR_NULL_POINTER, "col_idx and val are required when nnz > 0");
    if (nnz > net->caps[(size_t)k])
        return fail(SDNN_ERR_WORKSPACE_TOO_SMALL, "the arena holds " + std::to_string(net->caps[(size_t)k]) +
                                                      " entries for this layer (sdnn_net_create's nnz_per_layer)");
    const int64_t n = net->n;
    hipStream_t s = net->stream;
    if (n > kMaxScan) return fail(SDNN_ERR_UNSUPPORTED, "layers wider than 2^24 neurons are not supported");
    SDNN_ON_DEVICE(net);

    // 1. validate on the device
    SDNN_HIP(hipMemsetAsync(net->d_flags, 0, 4 * sizeof(uint32_t), s));
    SDNN_HIP(sdnn::launch_validate_layer(n, nnz, row_ptr, col_idx, val, bias, net->d_flags, s));
    uint32_t fl[4] = {0, 0, 0, 0};
    SDNN_HIP(hipMemcpyAsync(fl, net->d_flags, 4 * sizeof(uint32_t), hipMemcpyDeviceToHost, s));
    SDNN_HIP(hipStreamSynchronize(s));
    const uint32_t flags = fl[0];
    if (flags & 1u)
        return fail(SDNN_ERR_INVALID_INDEX,
                    "W_k is not valid CSR (row_ptr monotone from 0 to nnz, columns in [0,n) strictly increasing)");
    if (flags & 2u) return fail(SDNN_ERR_INVALID_VALUE, "W_k or b_k holds a non-finite value");

    // 2. derived copies, built in the layer's region of the arena (its previous copies are overwritten; any
    //    forward that still reads them was enqueued earlier on the same stream)
    Layer &l = net->layers[(size_t)k];
    l = Layer();  // not set until the build below completes
    char *base = net->arena + net->plan.layer_off[(size_t)k];
    const LayerPlan &lp = net->plan.layer[(size_t)k];
    Layer nl;
    nl.set = true;
    nl.nnz = nnz;
    nl.row_ptr = row_ptr;
    nl.col = col_idx;
    nl.val = val;
    nl.bias = bias;
    nl.bias_nonpos = (flags & 4u) == 0;
    nl.pos_bias = (int64_t)fl[1];
    {
        // with every b_j <= 0, an accumulated sum at most -max_j b_j gives h(sum + b_j) = 0 for every j
        const uint32_t key = fl[2];
        const uint32_t u = (key & 0x80000000u) ? (key & 0x7fffffffu) : ~key;
        float bmax;
        std::memcpy(&bmax, &u, sizeof(bmax));
        nl.zero_below = nl.bias_nonpos ? -(double)bmax : -INFINITY;
        // fl[3] holds the complement of the smallest key: equal keys mean every b_j has the same bits
        nl.bias_uniform = ~fl[3] == key;
    }
    nl.w_pack = at<Edge>(base, lp.w_pack);
    nl.fan_ptr = at<int64_t>(base, lp.fan_ptr);
    nl.fan = at<Edge>(base, lp.fan);
    // optional structures: present when this layer's density (not only the capacity) wants them
    nl.w_seg = at<int32_t>(base, lp.w_seg);
    nl.sched = at<sdnn::BlockedSched>(base, lp.sched);
    nl.stage = at<Edge>(base, lp.stage);
    sdnn::BlockedRegion *regions = at<sdnn::BlockedRegion>(base, lp.regions);
    int64_t *starts = at<int64_t>(base, lp.starts);
    nl.tile_mask = sdnn::spmm_wants_tiles(n, nnz) ? at<uint16_t>(base, lp.tile_mask) : nullptr;
    nl.slots = sdnn::spmm_wants_slots(n, nnz) ? at<double>(base, lp.slots) : nullptr;
    nl.dense_wt = at<double>(base, lp.dense64);
    nl.dense_wt32 = at<float>(base, lp.dense32);
    int32_t *counts = at<int32_t>(net->arena, net->plan.counts);
    int64_t *tmp = at<int64_t>(net->arena, net->plan.tmp);
    char *sort_scratch = net->arena + net->plan.sort;

    hipError_t e;
#define SETUP_HIP(call)                                  \
    do {                                                 \
        e = (call);                                      \
        if (e != hipSuccess) return fail_hip(e, #call);  \
    } while (0)
    SETUP_HIP(sdnn::launch_pack_edges(nnz, col_idx, val, nl.w_pack, s));
    SETUP_HIP(hipMemsetAsync(counts, 0, (size_t)n * sizeof(int32_t), s));
    SETUP_HIP(sdnn::launch_fanin_counts(nnz, col_idx, counts, s));
    SETUP_HIP(sdnn::launch_exclusive_scan_i32_to_i64(n, counts, nl.fan_ptr, tmp, s));
    SETUP_HIP(sdnn::launch_fanin_lists(n, nnz, row_ptr, col_idx, val, nl.fan, sort_scratch, s));
    SETUP_HIP(hipMemsetAsync(nl.fan + nnz, 0, sizeof(Edge), s));
    SETUP_HIP(hipMemsetAsync(net->d_int, 0, sizeof(int32_t), s));
    SETUP_HIP(sdnn::launch_max_segment(n, row_ptr, net->d_int, s));
    SETUP_HIP(hipMemcpyAsync(&nl.max_fanout, net->d_int, sizeof(int32_t), hipMemcpyDeviceToHost, s));
    if (nl.w_seg) SETUP_HIP(sdnn::launch_window_seg(n, row_ptr, col_idx, nl.w_seg, s));
    int32_t region_max = 0;
    if (nl.sched) {
        SETUP_HIP(sdnn::launch_blocked_order(n, nl.fan_ptr, nl.sched, s));
        SETUP_HIP(sdnn::launch_blocked_stage(n, nnz, nl.fan, nl.sched, nl.stage, regions, counts, starts, tmp,
                                             net->d_int + 1, s));
        SETUP_HIP(hipMemcpyAsync(&region_max, net->d_int + 1, sizeof(int32_t), hipMemcpyDeviceToHost, s));
    }
    if (nl.tile_mask) SETUP_HIP(sdnn::launch_spmm_tile_mask(n, nl.fan_ptr, nl.fan, nl.tile_mask, s));
    if (nl.slots) SETUP_HIP(sdnn::launch_spmm_slots(n, nl.fan_ptr, nl.fan, nl.slots, s));
    SETUP_HIP(hipStreamSynchronize(s));
#undef SETUP_HIP
    // the product stages each workgroup's lists in LDS when the longest region fits; otherwise it reads the
    // same staged copy entry by entry
    if (nl.sched && region_max <= sdnn::blocked_stage_cap()) nl.regions = regions;
    l = nl;
    return SDNN_OK;
}

sdnn_status sdnn_net_build_dense(sdnn_net net) {
    g_last_error.clear();
    if (!net) return fail(SDNN_ERR_INVALID_OBJECT, "net is NULL");
    if (!net->dense_flags) return fail(SDNN_ERR_INVALID_OBJECT, "the arena holds no dense copies (dense_flags 0)");
    SDNN_ON_DEVICE(net);
    const int64_t n = net->n;
    for (int32_t k = 0; k < net->L; ++k) {
        Layer &l = net->layers[(size_t)k];
        if (!l.set) return fail(SDNN_ERR_INVALID_OBJECT, "every layer must be set before build_dense");
        if (l.dense_wt && !l.dense_ready) {
            SDNN_HIP(sdnn::launch_dense_from_fanin(n, l.fan_ptr, l.fan, l.dense_wt, net->stream));
            l.dense_ready = true;
        }
        if (l.dense_wt32 && !l.dense32_ready) {
            SDNN_HIP(sdnn::launch_dense32_from_fanin(n, l.fan_ptr, l.fan, l.dense_wt32, net->stream));
            l.dense32_ready = true;
        }
    }
    SDNN_HIP(hipStreamSynchronize(net->stream));
    return SDNN_OK;
}

sdnn_status sdnn_workspace_size(sdnn_net net, int64_t batch, int32_t y_is_csr, int64_t *bytes) {
    g_last_error.clear();
    if (!net) return fail(SDNN_ERR_INVALID_OBJECT, "net is NULL");
    if (!bytes) return fail(SDNN_ERR_NULL_POINTER, "bytes is NULL");
    if (batch < 0) return fail(SDNN_ERR_INVALID_VALUE, "batch must be >= 0");
    *bytes = y_is_csr ? (int64_t)carve_csr(nullptr, net->n, batch).bytes : (int64_t)dense_ws_bytes(net->n, batch, net->num_cu);
    return SDNN_OK;
}

static sdnn_status check_range(sdnn_net net, int32_t k0, int32_t k1) {
    if (k0 < 0 || k1 < k0 || k1 > net->L) return fail(SDNN_ERR_DIMENSION_MISMATCH, "need 0 <= k0 <= k1 <= L");
    for (int32_t k = k0; k < k1; ++k)
        if (!net->layers[(size_t)k].set) return fail(SDNN_ERR_INVALID_OBJECT, "a layer in [k0, k1) is not set");
    return SDNN_OK;
}

static sdnn_status forward_dense_impl(sdnn_net net, int32_t k0, int32_t k1, int64_t batch, const float *Y_in,
                                      float *Y_out, void *ws, int64_t ws_bytes, int32_t arm, bool static_ws);

sdnn_status sdnn_forward_dense(sdnn_net net, int32_t k0, int32_t k1, int64_t batch, const float *Y_in, float *Y_out,
                               void *ws, int64_t ws_bytes, int32_t arm) {
    g_last_error.clear();
    return forward_dense_impl(net, k0, k1, batch, Y_in, Y_out, ws, ws_bytes, arm, false);
}

sdnn_status sdnn_forward_dense_noalloc(sdnn_net net, int32_t k0, int32_t k1, int64_t batch, const float *Y_in,
                                       float *Y_out, int32_t arm) {
    g_last_error.clear();
    return forward_dense_impl(net, k0, k1, batch, Y_in, Y_out, nullptr, 0, arm, true);
}

int64_t sdnn_noalloc_scratch_bytes(void) { return (int64_t)kScratchBytes; }

static sdnn_status forward_dense_impl(sdnn_net net, int32_t k0, int32_t k1, int64_t batch, const float *Y_in,
                                      float *Y_out, void *ws, int64_t ws_bytes, int32_t arm, bool static_ws) {
    if (!net) return fail(SDNN_ERR_INVALID_OBJECT, "net is NULL");
    sdnn_status st = check_range(net, k0, k1);
    if (st != SDNN_OK) return st;
    if (batch < 0) return fail(SDNN_ERR_DIMENSION_MISMATCH, "batch must be >= 0");
    if (arm != SDNN_ARM_SPARSE && arm != SDNN_ARM_DENSE && arm != SDNN_ARM_DENSE_F32)
        return fail(SDNN_ERR_INVALID_VALUE, "unknown arm");
    if (arm != SDNN_ARM_SPARSE && net->bias_pattern)
        return fail(SDNN_ERR_UNSUPPORTED, "the dense arms store every zero of W_k, so they have no bias pattern");
    if (batch == 0) return SDNN_OK;
    if (!Y_in || !Y_out) return fail(SDNN_ERR_NULL_POINTER, "Y_in and Y_out are required");
    SDNN_ON_DEVICE(net);
    const int64_t n = net->n;
    hipStream_t s = net->stream;
    if (k0 == k1) {
        if (Y_out != Y_in)
            SDNN_HIP(hipMemcpyAsync(Y_out, Y_in, (size_t)batch * (size_t)n * sizeof(float), hipMemcpyDeviceToDevice, s));
        return SDNN_OK;
    }
    if (static_ws) {
        // the library's fixed scratch array of this device replaces the caller's workspace
        const ScratchSlot *slot = net->device < kMaxDevices ? &g_scratch[net->device] : nullptr;
        if (!slot || !slot->ptr)
            return fail(SDNN_ERR_DEVICE, std::string("scratch array of the allocation-free entry point unavailable: ") +
                                             hipGetErrorString(slot ? slot->err : hipErrorInvalidDevice));
        if (dense_ws_bytes(n, batch, net->num_cu) > kScratchBytes)
            return fail(SDNN_ERR_UNSUPPORTED, "batch x n needs " + std::to_string(dense_ws_bytes(n, batch, net->num_cu)) +
                                                  " bytes of scratch; the allocation-free entry point holds " +
                                                  std::to_string(kScratchBytes));
        ws = slot->ptr;
        ws_bytes = (int64_t)kScratchBytes;
    }
    if (!ws) return fail(SDNN_ERR_NULL_POINTER, "ws is required");
    if (ws_bytes < (int64_t)dense_ws_bytes(n, batch, net->num_cu))
        return fail(SDNN_ERR_WORKSPACE_TOO_SMALL, "workspace smaller than sdnn_workspace_size(net, batch, 0)");
    for (int32_t k = k0; k < k1; ++k) {
        const Layer &l = net->layers[(size_t)k];
        if ((arm == SDNN_ARM_DENSE && !l.dense_ready) || (arm == SDNN_ARM_DENSE_F32 && !l.dense32_ready))
            return fail(SDNN_ERR_INVALID_OBJECT, "dense arm requested before sdnn_net_build_dense (or without its copy "
                                                 "in the arena)");
    }
    const int64_t ld = sdnn::act_ld(n, batch);
    float *buf[2];
    buf[0] = (float *)ws;
    buf[1] = (float *)((char *)ws + act_bytes(n, batch));
    double *partial = (double *)((char *)ws + 2 * act_bytes(n, batch));
    int pr = -1;
    if (arm == SDNN_ARM_SPARSE && use_blocked(net, k0, k1, batch)) {
        // the sample-blocked layout (each buffer holds n x ld >= n x round32(batch) floats)
        SDNN_HIP(prof_begin(net, -1, sdnn::kKernTranspose, &pr));
        SDNN_HIP(sdnn::launch_to_blocked(n, batch, n, Y_in, buf[0], s));
        SDNN_HIP(prof_end(net, pr));
        int cb = 0;
        for (int32_t k = k0; k < k1; ++k) {
            const Layer &l = net->layers[(size_t)k];
            SDNN_HIP(prof_begin(net, k, sdnn::kKernBlocked, &pr));
            SDNN_HIP(sdnn::launch_spmm_blocked(n, batch, l.sched, l.stage, l.regions, nullptr, l.bias, net->ymax, net->bias_pattern, buf[cb],
                                               buf[cb ^ 1], s));
            SDNN_HIP(prof_end(net, pr));
            cb ^= 1;
        }
        SDNN_HIP(prof_begin(net, -1, sdnn::kKernTranspose, &pr));
        SDNN_HIP(sdnn::launch_from_blocked(n, batch, n, buf[cb], Y_out, s));
        SDNN_HIP(prof_end(net, pr));
        return SDNN_OK;
    }
    SDNN_HIP(prof_begin(net, -1, sdnn::kKernTranspose, &pr));
    SDNN_HIP(sdnn::launch_transpose(Y_in, n, buf[0], ld, batch, n, s));  // batch x n -> n x batch
    SDNN_HIP(prof_end(net, pr));
    int cur = 0;
    for (int32_t k = k0; k < k1; ++k) {
        const Layer &l = net->layers[(size_t)k];
        int kind = sdnn::kKernDenseGemm;
        SDNN_HIP(prof_begin(net, k, kind, &pr));
        if (arm == SDNN_ARM_SPARSE)
            SDNN_HIP(sdnn::launch_spmm_fanin(n, batch, ld, l.fan_ptr, l.fan, l.tile_mask, l.slots, l.bias,
                                             net->ymax, net->bias_pattern, buf[cur], buf[cur ^ 1], s, &kind));
        else if (arm == SDNN_ARM_DENSE)
            SDNN_HIP(sdnn::launch_gemm_dense_layer(n, batch, ld, l.dense_wt, l.bias, net->ymax, buf[cur],
                                                   buf[cur ^ 1], partial, net->num_cu, s));
        else {
            kind = sdnn::kKernDenseGemm32;
            SDNN_HIP(sdnn::launch_gemm32_dense_layer(n, batch, ld, l.dense_wt32, l.bias, net->ymax, buf[cur],
                                                     buf[cur ^ 1], reinterpret_cast<float *>(partial), net->num_cu, s));
        }
        SDNN_HIP(prof_end(net, pr, kind));
        cur ^= 1;
    }
    SDNN_HIP(prof_begin(net, -1, sdnn::kKernTranspose, &pr));
    SDNN_HIP(sdnn::launch_transpose(buf[cur], ld, Y_out, n, n, batch, s));  // n x batch -> batch x n
    SDNN_HIP(prof_end(net, pr));
    return SDNN_OK;
}

sdnn_status sdnn_forward_csr(sdnn_net net, int32_t k0, int32_t k1, int64_t batch, const int64_t *y_row_ptr,
                             const int32_t *y_col, const float *y_val, void *ws, int64_t ws_bytes,
                             int64_t *out_row_ptr, int32_t **out_col, float **out_val, int64_t *out_nnz) {
    g_last_error.clear();
    if (!net) return fail(SDNN_ERR_INVALID_OBJECT, "net is NULL");
    sdnn_status st = check_range(net, k0, k1);
    if (st != SDNN_OK) return st;
    if (batch < 0 || batch > 0x7fffffffLL) return fail(SDNN_ERR_DIMENSION_MISMATCH, "batch must be in [0, 2^31-1]");
    if (batch > kMaxScan) return fail(SDNN_ERR_UNSUPPORTED, "CSR batches above 2^24 samples are not supported");
    if (!y_row_ptr || !out_row_ptr || !out_col || !out_val || !out_nnz)
        return fail(SDNN_ERR_NULL_POINTER, "y_row_ptr and the four outputs are required");
    if (!ws) return fail(SDNN_ERR_NULL_POINTER, "ws is required");
    SDNN_ON_DEVICE(net);
    const int64_t n = net->n;
    hipStream_t s = net->stream;
    CsrWs w = carve_csr(ws, n, batch);
    if (ws_bytes < (int64_t)w.bytes)
        return fail(SDNN_ERR_WORKSPACE_TOO_SMALL, "workspace smaller than sdnn_workspace_size(net, batch, 1)");
    if (k0 == k1) {  // identity: copy the input CSR into the workspace
        int64_t in_nnz = 0;
        SDNN_HIP(hipMemcpyAsync(&in_nnz, y_row_ptr + batch, sizeof(int64_t), hipMemcpyDeviceToHost, s));
        SDNN_HIP(hipStreamSynchronize(s));
        if (in_nnz < 0 || in_nnz > batch * n)
            return fail(SDNN_ERR_DIMENSION_MISMATCH, "y_row_ptr[batch] outside [0, batch*n]");
        if (in_nnz > 0 && (!y_col || !y_val)) return fail(SDNN_ERR_NULL_POINTER, "y_col and y_val are required");
        SDNN_HIP(hipMemcpyAsync(out_row_ptr, y_row_ptr, (size_t)(batch + 1) * sizeof(int64_t), hipMemcpyDeviceToDevice, s));
        if (in_nnz > 0) {
            SDNN_HIP(hipMemcpyAsync(w.col[0], y_col, (size_t)in_nnz * sizeof(int32_t), hipMemcpyDeviceToDevice, s));
            SDNN_HIP(hipMemcpyAsync(w.val[0], y_val, (size_t)in_nnz * sizeof(float), hipMemcpyDeviceToDevice, s));
        }
        SDNN_HIP(hipStreamSynchronize(s));
        *out_col = w.col[0];
        *out_val = w.val[0];
        *out_nnz = in_nnz;
        return SDNN_OK;
    }
    if (batch == 0) {  // no samples: an empty result (row_ptr = {0})
        SDNN_HIP(hipMemsetAsync(out_row_ptr, 0, sizeof(int64_t), s));
        SDNN_HIP(hipStreamSynchronize(s));
        *out_col = w.col[0];
        *out_val = w.val[0];
        *out_nnz = 0;
        return SDNN_OK;
    }
    SDNN_HIP(hipMemsetAsync(net->d_flags, 0, sizeof(uint32_t), s));
    SDNN_HIP(hipMemsetAsync(net->d_stats, 0, (size_t)(k1 - k0) * sdnn::kSpgemmStats * sizeof(unsigned long long), s));

    // Activation format per layer.  While outputs are sparse they stay as slot rows (row-wise SpGEMM).
    // From the first layer whose input is dense enough, activations are kept dense and neuron-major and
    // each layer gathers over fan-in lists (the dense-Y product); the result is packed back into rows at
    // the end.  A layer's input counts as dense when it holds at least 1/8 of batch * n entries, or when
    // the layer's bias is positive on at least a quarter of its neurons and applies everywhere (every such
    // neuron is then h(b_j) > 0 in every sample that does not push it below zero, so the output is dense
    // whatever the input).  On the sample-blocked layout the switch comes at 1/16 (measured on n 16384, 32
    // entries per neuron, batch 4096, a 10%-dense input: the SpGEMM takes 0.69 ms and densifying its 5x
    // larger output 0.42 ms; densifying the input 0.15 ms and the blocked product 0.42 ms).  The input size
    // is known on the host only through a synchronisation, so the host keeps an upper bound (a layer whose
    // untouched columns stay zero, every b_j <= 0 or bias on the pattern only, writes at most (longest
    // fan-out row) entries per input entry) and reads the exact count from the device only when the bound
    // reaches the threshold.
    const double dense_at = (double)batch * (double)n / (use_blocked(net, k0, k1, batch) ? 16.0 : 8.0);
    double nnz_hi = (double)batch * (double)n;  // upper bound of the current layer's input entries
    bool exact = false;
    if (nnz_hi >= dense_at) {
        int64_t in_nnz = 0;
        SDNN_HIP(hipMemcpyAsync(&in_nnz, y_row_ptr + batch, sizeof(int64_t), hipMemcpyDeviceToHost, s));
        SDNN_HIP(hipStreamSynchronize(s));
        nnz_hi = (double)in_nnz;
        exact = true;
    }
    int32_t kd = k1;
    int cur = 0;  // slot buffer that receives the next sparse layer's output
    // An empty activation stays empty through every layer whose untouched columns stay zero (every b_j <= 0,
    // or the bias on the pattern only).  After the 1st, 2nd, 4th, 8th ... sparse layer, when at least
    // kEmptyCheckLayers such layers follow, the host reads the layer's output count (one synchronisation) and
    // stops at an empty output, which is then Y_{k1} (the deep sparse network dies out this way after its
    // second layer; the rest would cost launches only).
    constexpr int32_t kEmptyCheckLayers = 8;
    int64_t next_check = 1;
    for (int32_t k = k0; k < k1; ++k) {
        const Layer &l = net->layers[(size_t)k];
        if (!net->bias_pattern && 4 * l.pos_bias >= n) {
            kd = k;
            break;
        }
        if (nnz_hi >= dense_at && !exact) {
            unsigned long long got = 0;
            SDNN_HIP(hipMemcpyAsync(&got, net->d_stats + sdnn::kSpgemmStats * (k - 1 - k0) + sdnn::kSpgemmStatNnz, sizeof(got), hipMemcpyDeviceToHost, s));
            SDNN_HIP(hipStreamSynchronize(s));
            nnz_hi = (double)got;
            exact = true;
        }
        if (nnz_hi >= dense_at) {
            kd = k;
            break;
        }
        const bool first = k == k0;
        int pr = -1;
        SDNN_HIP(prof_begin(net, k, sdnn::kKernSpgemm, &pr));
        SDNN_HIP(sdnn::launch_spgemm_layer(n, batch, first ? y_row_ptr : nullptr, first ? nullptr : w.cnt[cur ^ 1],
                                           first ? y_col : w.col[cur ^ 1], first ? y_val : w.val[cur ^ 1], l.row_ptr,
                                           l.w_seg, l.w_pack, l.nnz, l.max_fanout, l.bias, l.bias_nonpos ? 1 : 0,
                                           l.bias_uniform ? 1 : 0, l.zero_below,
                                           net->bias_pattern, net->ymax, w.cnt[cur], w.col[cur], w.val[cur], w.lists,
                                           net->d_stats + sdnn::kSpgemmStats * (k - k0), net->d_flags, net->num_cu, s));
        SDNN_HIP(prof_end(net, pr));
        cur ^= 1;
        const double full = (double)batch * (double)n;
        nnz_hi = (l.bias_nonpos || net->bias_pattern) ? std::min(full, nnz_hi * (double)l.max_fanout) : full;
        exact = false;
        if (k - k0 + 1 == next_check) {
            next_check *= 2;
            bool stays_empty = k1 - k - 1 >= kEmptyCheckLayers;
            for (int32_t j = k + 1; stays_empty && j < k1; ++j)
                stays_empty = net->layers[(size_t)j].bias_nonpos || net->bias_pattern;
            if (stays_empty) {
                unsigned long long got = 0;
                SDNN_HIP(hipMemcpyAsync(&got, net->d_stats + sdnn::kSpgemmStats * (k - k0) + sdnn::kSpgemmStatNnz,
                                        sizeof(got), hipMemcpyDeviceToHost, s));
                SDNN_HIP(hipStreamSynchronize(s));
                nnz_hi = (double)got;
                exact = true;
                if (got == 0) break;  // Y_{k+1} is empty, and so is every later activation
            }
        }
    }
    int last = 0, outb;  // slot buffer holding Y_{k1}, and the buffer the packed CSR goes to
    bool packed = false;  // the CSR is already in buffer outb
    if (kd < k1 && use_blocked(net, kd, k1, batch)) {
        // dense activations in the sample-blocked layout, packed straight into CSR at the end
        const bool from_user = kd == k0;
        const int db = from_user ? 0 : cur;  // the input rows (if any) sit in buffer cur ^ 1
        float *dense[2] = {reinterpret_cast<float *>(w.col[db]), w.val[db]};
        // a sparse input (at most 1/16 of batch * n entries: a 32-sample row is then entirely zero with
        // probability >= (15/16)^32, about 13%, at uniform density): the first product skips the zero rows
        // (only when the first layer stages its lists: the product reads the map only then, and densify does
        // not store the zero rows when it writes one)
        uint32_t *nz = (nnz_hi <= (double)batch * (double)n / 16.0 && net->layers[(size_t)kd].regions) ? w.nzrows : nullptr;
        int pr = -1;
        SDNN_HIP(prof_begin(net, -1, sdnn::kKernDensify, &pr));
        SDNN_HIP(sdnn::launch_densify_blocked(n, batch, from_user ? y_row_ptr : nullptr, from_user ? nullptr : w.cnt[cur ^ 1],
                                              from_user ? y_col : w.col[cur ^ 1], from_user ? y_val : w.val[cur ^ 1],
                                              dense[0], nz, net->d_flags, s));
        SDNN_HIP(prof_end(net, pr));
        int dc = 0;
        for (int32_t k = kd; k < k1; ++k) {
            const Layer &l = net->layers[(size_t)k];
            SDNN_HIP(prof_begin(net, k, sdnn::kKernBlocked, &pr));
            SDNN_HIP(sdnn::launch_spmm_blocked(n, batch, l.sched, l.stage, l.regions, k == kd ? nz : nullptr, l.bias,
                                               net->ymax, net->bias_pattern, dense[dc], dense[dc ^ 1], s));
            SDNN_HIP(prof_end(net, pr));
            dc ^= 1;
        }
        SDNN_HIP(prof_begin(net, -1, sdnn::kKernPack, &pr));
        SDNN_HIP(sdnn::launch_blocked_to_csr(n, batch, dense[dc], w.pcnt, w.cnt[db ^ 1], out_row_ptr, w.scan_tmp,
                                             w.col[db ^ 1], w.val[db ^ 1], s));
        SDNN_HIP(prof_end(net, pr));
        packed = true;
        outb = db ^ 1;
    } else if (kd < k1) {
        const bool from_user = kd == k0;
        const int db = from_user ? 0 : cur;  // the input rows (if any) sit in buffer cur ^ 1
        // two n x batch fp32 buffers at row pitch ld
        float *dense[2] = {reinterpret_cast<float *>(w.col[db]), w.val[db]};
        const int64_t ld = sdnn::act_ld(n, batch);
        // dense[1] is free until the first layer: it stages the rows batch-major when they hold at least a
        // quarter of batch * n entries (measured on MI355X: 0.34 instead of 0.69 ms for 32M entries into
        // 16384 x 4096; at 2% density the extra transpose costs more than the scattered stores it saves)
        float *stage = nnz_hi >= (double)batch * (double)n / 4.0 ? dense[1] : nullptr;
        int pr = -1;
        SDNN_HIP(prof_begin(net, -1, sdnn::kKernDensify, &pr));
        SDNN_HIP(sdnn::launch_densify(n, batch, ld, from_user ? y_row_ptr : nullptr, from_user ? nullptr : w.cnt[cur ^ 1],
                                      from_user ? y_col : w.col[cur ^ 1], from_user ? y_val : w.val[cur ^ 1],
                                      dense[0], stage, net->d_flags, s));
        SDNN_HIP(prof_end(net, pr));
        int dc = 0;
        for (int32_t k = kd; k < k1; ++k) {
            const Layer &l = net->layers[(size_t)k];
            int kind = sdnn::kKernGather;
            SDNN_HIP(prof_begin(net, k, kind, &pr));
            SDNN_HIP(sdnn::launch_spmm_fanin(n, batch, ld, l.fan_ptr, l.fan, l.tile_mask, l.slots, l.bias,
                                             net->ymax, net->bias_pattern, dense[dc], dense[dc ^ 1], s, &kind));
            SDNN_HIP(prof_end(net, pr, kind));
            dc ^= 1;
        }
        SDNN_HIP(prof_begin(net, -1, sdnn::kKernPack, &pr));
        SDNN_HIP(sdnn::launch_transpose(dense[dc], ld, dense[dc ^ 1], n, n, batch, s));  // -> batch x n
        if (n % 4 == 0) {
            // counted first, then packed straight into the other buffer pair (no slot rows in between)
            SDNN_HIP(sdnn::launch_dense_to_csr(n, batch, dense[dc ^ 1], w.cnt[db ^ 1], out_row_ptr, w.scan_tmp,
                                               w.col[db ^ 1], w.val[db ^ 1], s));
            packed = true;
            outb = db ^ 1;
        } else {
            SDNN_HIP(sdnn::launch_dense_to_slots(n, batch, dense[dc ^ 1], w.cnt[db ^ 1], w.col[db ^ 1],
                                                 w.val[db ^ 1], s));
            last = db ^ 1;
            outb = db;
        }
        SDNN_HIP(prof_end(net, pr));
    } else {
        last = cur ^ 1;
        outb = cur;
    }
    if (!packed) {
        int pr = -1;
        SDNN_HIP(prof_begin(net, -1, sdnn::kKernCompact, &pr));
        SDNN_HIP(sdnn::launch_exclusive_scan_i32_to_i64(batch, w.cnt[last], out_row_ptr, w.scan_tmp, s));
        SDNN_HIP(sdnn::launch_compact_rows(n, batch, w.cnt[last], out_row_ptr, w.col[last], w.val[last],
                                           w.col[outb], w.val[outb], s));
        SDNN_HIP(prof_end(net, pr));
    }
    int64_t nnz = 0;
    uint32_t flags = 0;
    SDNN_HIP(hipMemcpyAsync(&nnz, out_row_ptr + batch, sizeof(int64_t), hipMemcpyDeviceToHost, s));
    SDNN_HIP(hipMemcpyAsync(&flags, net->d_flags, sizeof(uint32_t), hipMemcpyDeviceToHost, s));
    SDNN_HIP(hipStreamSynchronize(s));
    if (flags & 1u)
        return fail(SDNN_ERR_INVALID_INDEX, "Y_in is not valid CSR (row extents or column indices out of range)");
    *out_col = w.col[outb];
    *out_val = w.val[outb];
    *out_nnz = nnz;
    return SDNN_OK;
}

static sdnn_status mxm_common(sdnn_net net, int32_t k, int32_t semiring, int64_t batch, void *ws, int64_t ws_bytes,
                              bool needs_ws) {
    if (!net) return fail(SDNN_ERR_INVALID_OBJECT, "net is NULL");
    if (k < 0 || k >= net->L) return fail(SDNN_ERR_DIMENSION_MISMATCH, "layer index outside [0, L)");
    if (!net->layers[(size_t)k].set) return fail(SDNN_ERR_INVALID_OBJECT, "layer k is not set");
    if (semiring < SDNN_SEMIRING_PLUS_TIMES || semiring > SDNN_SEMIRING_XOR_AND)
        return fail(SDNN_ERR_INVALID_VALUE, "unknown semiring");
    if (batch < 0) return fail(SDNN_ERR_DIMENSION_MISMATCH, "batch must be >= 0");
    if (!needs_ws) return SDNN_OK;
    if (batch > 0 && !ws) return fail(SDNN_ERR_NULL_POINTER, "ws is required");
    if (batch > 0 && ws_bytes < (int64_t)dense_ws_bytes(net->n, batch, net->num_cu))
        return fail(SDNN_ERR_WORKSPACE_TOO_SMALL, "workspace smaller than sdnn_workspace_size(net, batch, 0)");
    return SDNN_OK;
}

sdnn_status sdnn_mxm_dense(sdnn_net net, int32_t k, int32_t semiring, int64_t batch, const float *Y, float *Z,
                           void *ws, int64_t ws_bytes) {
    g_last_error.clear();
    sdnn_status st = mxm_common(net, k, semiring, batch, ws, ws_bytes, true);
    if (st != SDNN_OK || batch == 0) return st;
    if (!Y || !Z) return fail(SDNN_ERR_NULL_POINTER, "Y and Z are required");
    SDNN_ON_DEVICE(net);
    const int64_t n = net->n;
    hipStream_t s = net->stream;
    const Layer &l = net->layers[(size_t)k];
    const int64_t ld = sdnn::act_ld(n, batch);
    float *yt = (float *)ws;
    float *zt = (float *)((char *)ws + act_bytes(n, batch));
    SDNN_HIP(sdnn::launch_transpose(Y, n, yt, ld, batch, n, s));  // batch x n -> n x batch
    SDNN_HIP(sdnn::launch_semiring_mxm(semiring, n, batch, ld, l.fan_ptr, l.fan, yt, zt, s));
    SDNN_HIP(sdnn::launch_transpose(zt, ld, Z, n, n, batch, s));  // n x batch -> batch x n
    return SDNN_OK;
}

sdnn_status sdnn_mxm_csr(sdnn_net net, int32_t k, int32_t semiring, int64_t batch, const int64_t *y_row_ptr,
                         const int32_t *y_col, const float *y_val, float *Z, void *ws, int64_t ws_bytes) {
    g_last_error.clear();
    (void)ws;
    (void)ws_bytes;
    sdnn_status st = mxm_common(net, k, semiring, batch, ws, ws_bytes, false);
    if (st != SDNN_OK || batch == 0) return st;
    if (!y_row_ptr || !Z) return fail(SDNN_ERR_NULL_POINTER, "y_row_ptr and Z are required");
    SDNN_ON_DEVICE(net);
    const int64_t n = net->n;
    hipStream_t s = net->stream;
    const Layer &l = net->layers[(size_t)k];
    SDNN_HIP(hipMemsetAsync(net->d_flags, 0, sizeof(uint32_t), s));
    // row by row over the stored entries (the SpGEMM skeleton): Y is never densified
    SDNN_HIP(sdnn::launch_semiring_rows(semiring, n, batch, y_row_ptr, y_col, y_val, l.row_ptr, l.w_pack, Z,
                                        net->d_flags, s));
    uint32_t flags = 0;
    SDNN_HIP(hipMemcpyAsync(&flags, net->d_flags, sizeof(uint32_t), hipMemcpyDeviceToHost, s));
    SDNN_HIP(hipStreamSynchronize(s));
    if (flags & 1u) return fail(SDNN_ERR_INVALID_INDEX, "Y is not valid CSR (row extents or column indices out of range)");
    return SDNN_OK;
}

sdnn_status sdnn_net_set_profiling(sdnn_net net, int32_t enable) {
    g_last_error.clear();
    if (!net) return fail(SDNN_ERR_INVALID_OBJECT, "net is NULL");
    if (enable) prof_clear(net);
    net->profiling = enable != 0;
    return SDNN_OK;
}

sdnn_status sdnn_net_read_profile(sdnn_net net, sdnn_kernel_time *out, int32_t max_records, int32_t *count) {
    g_last_error.clear();
    if (!net) return fail(SDNN_ERR_INVALID_OBJECT, "net is NULL");
    if (!count || (max_records > 0 && !out)) return fail(SDNN_ERR_NULL_POINTER, "count (and out) are required");
    SDNN_ON_DEVICE(net);
    SDNN_HIP(hipStreamSynchronize(net->stream));
    *count = (int32_t)std::min<size_t>(net->prof.size(), 0x7fffffff);
    for (size_t i = 0; i < net->prof.size() && (int64_t)i < (int64_t)max_records; ++i) {
        float ms = 0.0f;
        SDNN_HIP(hipEventElapsedTime(&ms, net->prof[i].a, net->prof[i].b));
        out[i].layer = net->prof[i].layer;
        out[i].kernel = net->prof[i].kernel;
        out[i].ms = ms;
    }
    prof_clear(net);
    return SDNN_OK;
}

sdnn_status sdnn_net_free(sdnn_net net) {
    g_last_error.clear();
    if (!net) return SDNN_OK;
    DeviceScope device_scope(net->device);  // frees on the net's device even if it cannot be made current
    (void)hipStreamSynchronize(net->stream);
    prof_clear(net);
    for (hipEvent_t e : net->ev_free) (void)hipEventDestroy(e);
    delete net;  // the arena belongs to the caller
    return SDNN_OK;
}

}  // extern "C"
