// C ABI of libfbdt (declared in include/fbdt.h) and the host runtime around
// the kernels: argument checks, per-device scratch, the stream-ordered
// boosting loop, model storage and kernel timing.
#include "fbdt.h"
#include "fbdt_internal.h"

#include <hip/hip_runtime.h>

#include <algorithm>
#include <atomic>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <mutex>
#include <string>
#include <vector>

using namespace fbdt;

struct fbdt_model {
    int32_t n_trees = 0, depth = 0, n_features = 0, n_bins = 0;
    double f0 = 0.0;
    std::vector<uint8_t> cut_feature, cut_bin;
    std::vector<double> gain, leaf;
    // missing values (section 4.2): boost weights of the inner nodes [T][2^D - 1];
    // an event whose code of a node's cut feature is the missing code stops there
    bool missing = false;
    std::vector<double> inner;
    std::vector<float> boundaries;
    // device copies of the forest for apply, one per device used
    struct DeviceCopy {
        int device;
        uint16_t *cuts;
        double *leaves;
        int nodes_stride;   // tile stride the node records were made for (0: none)
        uint32_t *nodes;    // [T][16] node records of shallow forests, or null
        uint2 *frec;        // [T][2^D - 1] (feature, threshold) for float apply, or null
        double *gains;      // [T][2^D - 1] separation gains, or null
        // float apply of shallow forests: per-feature threshold table and the
        // node records (threshold ranks) for the tile stride fnodes_stride
        uint32_t *ftab;
        int ftab_words;
        uint32_t *fnodes;
        int fnodes_stride;
    };
    std::mutex mu;
    std::vector<DeviceCopy> copies;
};

namespace {

thread_local std::string g_error;

int fail(int code, const char *fmt, ...) {
    char buf[512];
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(buf, sizeof buf, fmt, ap);
    va_end(ap);
    g_error = buf;
    return code;
}

#define HIP_TRY(expr)                                                                    \
    do {                                                                                 \
        hipError_t e_ = (expr);                                                          \
        if (e_ != hipSuccess)                                                            \
            return fail(FBDT_E_DEVICE, "%s failed: %s", #expr, hipGetErrorString(e_));   \
    } while (0)

// Scratch of fbdt_best_cuts_noalloc, the entry point that allocates nothing:
// the candidate cut of every (node, feature) of a call, float64 gains
// [n_nodes][d] then int32 cut bins [n_nodes][d] from byte offset
// kNoAllocGainBytes.  A file-scope device array, so each device holds its
// own copy for the life of the process.  In host code the name `scratch`
// is a host-side stand-in: kernels and copies take the device address that
// hipGetSymbolAddress returned for the current device (DeviceInfo::scratch).
constexpr size_t kNoAllocCandidates = 64 * 256;
constexpr size_t kNoAllocGainBytes = kNoAllocCandidates * sizeof(double);
constexpr size_t kNoAllocScratchBytes = kNoAllocGainBytes + kNoAllocCandidates * sizeof(int32_t);
static_assert(kNoAllocGainBytes % 256 == 0, "the cut array starts 256-byte aligned");
__device__ __align__(256) unsigned char scratch[kNoAllocScratchBytes];

struct DeviceInfo {
    int cu_count = 0;
    size_t max_lds = 0;
    void *scratch = nullptr;                  // device address of `scratch` on this device
    hipError_t scratch_status = hipSuccess;   // hipGetSymbolAddress's result
};

std::mutex g_dev_mu;
std::vector<DeviceInfo> g_dev_info(64);

int device_info(int dev, DeviceInfo *out) {
    if (dev < 0 || dev >= 64) return fail(FBDT_E_DEVICE, "device id %d out of range", dev);
    std::lock_guard<std::mutex> lk(g_dev_mu);
    DeviceInfo &di = g_dev_info[dev];
    if (di.cu_count == 0) {
        int cu = 0, lds = 0;
        HIP_TRY(hipDeviceGetAttribute(&cu, hipDeviceAttributeMultiprocessorCount, dev));
        HIP_TRY(hipDeviceGetAttribute(&lds, hipDeviceAttributeMaxSharedMemoryPerBlock, dev));
        HIP_TRY(prepare_kernels((size_t)lds));
        // the no-allocation scratch of this device (dev is the current
        // device here: callers pass the id hipGetDevice returned)
        void *sp = nullptr;
        di.scratch_status = hipGetSymbolAddress(&sp, HIP_SYMBOL(scratch));
        di.scratch = di.scratch_status == hipSuccess ? sp : nullptr;
        di.cu_count = cu;
        di.max_lds = (size_t)lds;
    }
    *out = di;
    return FBDT_OK;
}

// ---- options --------------------------------------------------------------
// Forced allocation failure (tests of the error path): while positive, each
// device allocation the library would make fails instead, as an exhausted
// device would make it fail, and the count goes down by one.
std::atomic<int64_t> opt_fail_alloc{0};

hipError_t device_alloc(void **p, size_t bytes) {
    int64_t left = opt_fail_alloc.load();
    while (left > 0) {
        if (opt_fail_alloc.compare_exchange_weak(left, left - 1)) {
            *p = nullptr;
            return hipErrorOutOfMemory;
        }
    }
    return hipMalloc(p, bytes);
}

std::atomic<int64_t> opt_hist_fpg{0}, opt_hist_chunks{0}, opt_hist_threads{0}, opt_hist_copies{0},
    opt_apply_threads{0}, opt_fit_graphs{1}, opt_hist_timeline{0};
// event lists below the root: 0 = the fit decides (kListAutoWork), 1 =
// never, 2 = always; and the list pass's launch-shape overrides
std::atomic<int64_t> opt_hist_lists{0}, opt_list_fpg{0}, opt_list_parts{0}, opt_list_copies{0};
// fits with events x (depth - 2) of at least this histogram the layers below
// the root from event lists.  Measured on 10M x 40 events (fits of 20 trees,
// streaming / lists): depth 3 breaks even near 10M events (1.18 at 2M, 0.98
// at 10M), depth 4 near 4-5M (0.99 at 4M), depth 6 near 2.5M (1.04 at 2M,
// 0.93 at 3M, 0.77 at 10M): the deeper layers that lists speed up most
// grow with the depth, while the extra route pass per layer costs about
// the same at every layer.
constexpr int64_t kListAutoWork = 10000000;

// Phase timeline of the histogram launches of the last fit made with option
// hist_timeline (host copy): [launches][max_blocks][kTimelineStamps].
struct Timeline {
    std::mutex mu;
    int64_t launches = 0;
    int32_t max_blocks = 0;
    int64_t rate_khz = 0;
    std::vector<int32_t> blocks;          // grid of each launch
    std::vector<uint64_t> stamps;
};
Timeline g_timeline;

HistOverrides hist_overrides() {
    HistOverrides ov;
    ov.fpg = (int)opt_hist_fpg.load();
    ov.chunks = (int)opt_hist_chunks.load();
    ov.threads = (int)opt_hist_threads.load();
    ov.copies = (int)opt_hist_copies.load();
    return ov;
}

// ---- timing ---------------------------------------------------------------
struct PendingTiming {
    int kind;
    hipEvent_t start, stop;
    double bytes;
};
std::mutex g_t_mu;
std::atomic<int> g_timing{0};   // bit k set: time launches of kind k
std::vector<PendingTiming> g_pending;
std::vector<hipEvent_t> g_event_pool;
int64_t g_t_launches[FBDT_K_COUNT];
double g_t_ms[FBDT_K_COUNT];
double g_t_bytes[FBDT_K_COUNT];

hipEvent_t take_event() {
    std::lock_guard<std::mutex> lk(g_t_mu);
    if (!g_event_pool.empty()) {
        hipEvent_t e = g_event_pool.back();
        g_event_pool.pop_back();
        return e;
    }
    // timing-only events: no system-scope fence (no cache write-back and
    // invalidate around the timed kernel)
    hipEvent_t e = nullptr;
    if (hipEventCreateWithFlags(&e, hipEventDisableSystemFence) != hipSuccess) return nullptr;
    return e;
}

// Brackets one kernel launch with events when timing is on.
struct Timed {
    int kind;
    double bytes;
    hipStream_t s;
    hipEvent_t a = nullptr;
    Timed(int k, hipStream_t st, double b = 0.0) : kind(k), bytes(b), s(st) {
        if ((g_timing.load(std::memory_order_relaxed) >> k) & 1) {
            a = take_event();
            if (a && hipEventRecord(a, s) != hipSuccess) a = nullptr;
        }
    }
    void done() {
        if (!a) return;
        hipEvent_t b = take_event();
        if (!b || hipEventRecord(b, s) != hipSuccess) return;
        std::lock_guard<std::mutex> lk(g_t_mu);
        g_pending.push_back({kind, a, b, bytes});
        a = nullptr;
    }
};

// ---- per-device scratch ---------------------------------------------------
// Launch sequence of a fit's boosting loop, captured once per distinct set
// of arguments and replayed (kernel launches only).
struct GraphKey {
    const void *xb, *y, *w;
    int64_t n, ldb;
    int d, n_bins, depth, n_trees, scale, lblocks;
    double eta, alpha;
    uint64_t seed;
    int64_t fpg, chunks, threads, copies;
    bool signed_w, missing;
    bool lists;
    int64_t list_fpg, list_parts, list_copies;
    bool operator==(const GraphKey &o) const {
        return xb == o.xb && y == o.y && w == o.w && n == o.n && ldb == o.ldb && d == o.d &&
               n_bins == o.n_bins && depth == o.depth && n_trees == o.n_trees &&
               scale == o.scale && lblocks == o.lblocks && eta == o.eta && alpha == o.alpha &&
               seed == o.seed && fpg == o.fpg && chunks == o.chunks && threads == o.threads &&
               copies == o.copies && signed_w == o.signed_w && missing == o.missing &&
               lists == o.lists && list_fpg == o.list_fpg && list_parts == o.list_parts &&
               list_copies == o.list_copies;
    }
};

struct Arena {
    std::mutex mu;
    void *ptr = nullptr;
    size_t size = 0;
    std::vector<std::pair<GraphKey, hipGraphExec_t>> graphs;  // oldest first
    hipStream_t capture = nullptr;  // records launches only; never runs work
};
Arena g_arena[64];
constexpr size_t kMaxGraphs = 4;

void drop_graphs(Arena &a) {
    for (auto &g : a.graphs) (void)hipGraphExecDestroy(g.second);
    a.graphs.clear();
}

int arena_reserve(Arena &a, size_t bytes) {
    if (bytes <= a.size) return FBDT_OK;
    drop_graphs(a);  // captured launches point into the old allocation
    if (a.ptr) {
        HIP_TRY(hipFree(a.ptr));
        a.ptr = nullptr;
        a.size = 0;
    }
    size_t want = bytes + bytes / 4 + (1 << 20);
    HIP_TRY(device_alloc(&a.ptr, want));
    a.size = want;
    return FBDT_OK;
}

// Frees the scratch of every device (after the device has finished with it:
// hipFree waits) and the fit graphs that point into it.
int release_scratch() {
    int cur = -1;
    HIP_TRY(hipGetDevice(&cur));
    for (int dev = 0; dev < 64; ++dev) {
        Arena &a = g_arena[dev];
        std::lock_guard<std::mutex> lk(a.mu);
        if (!a.ptr) continue;
        HIP_TRY(hipSetDevice(dev));
        drop_graphs(a);
        const hipError_t e = hipFree(a.ptr);
        a.ptr = nullptr;
        a.size = 0;
        if (e != hipSuccess) {
            (void)hipSetDevice(cur);
            return fail(FBDT_E_DEVICE, "hipFree of the scratch failed: %s", hipGetErrorString(e));
        }
    }
    HIP_TRY(hipSetDevice(cur));
    return FBDT_OK;
}

// Carves 256-byte aligned sub-buffers out of one allocation.
struct Carver {
    size_t off = 0;
    std::vector<std::pair<void **, size_t>> items;
    template <typename T>
    void add(T **p, size_t count) {
        items.push_back({reinterpret_cast<void **>(p), count * sizeof(T)});
        off += (count * sizeof(T) + 255) & ~(size_t)255;
    }
    void assign(void *base) {
        size_t o = 0;
        for (auto &it : items) {
            *it.first = static_cast<char *>(base) + o;
            o += (it.second + 255) & ~(size_t)255;
        }
    }
};

// ---- argument checks ------------------------------------------------------
bool aligned16(const void *p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

int check_codes(const uint8_t *xb, int64_t n, int32_t d, int64_t ldb) {
    if (!xb) return fail(FBDT_E_INVAL, "xb is NULL");
    if (n < 1) return fail(FBDT_E_INVAL, "n = %lld must be >= 1", (long long)n);
    if (n > (int64_t)1 << 40) return fail(FBDT_E_INVAL, "n = %lld too large", (long long)n);
    if (d < 1 || d > 255) return fail(FBDT_E_INVAL, "d = %d must be in [1, 255]", d);
    if (ldb < n || ldb % 16 != 0)
        return fail(FBDT_E_INVAL, "ldb = %lld must be a multiple of 16 and >= n = %lld",
                    (long long)ldb, (long long)n);
    if (!aligned16(xb)) return fail(FBDT_E_INVAL, "xb must be 16-byte aligned");
    return FBDT_OK;
}

int check_bins(int32_t n_bins) {
    if (n_bins < 2 || n_bins > 256)
        return fail(FBDT_E_INVAL, "n_bins = %d must be in [2, 256]", n_bins);
    return FBDT_OK;
}

int current_device(int *dev, DeviceInfo *di) {
    HIP_TRY(hipGetDevice(dev));
    return device_info(*dev, di);
}

int read_err(int *err_dev, hipStream_t s, int *out) {
    HIP_TRY(hipMemcpyAsync(out, err_dev, sizeof(int), hipMemcpyDeviceToHost, s));
    HIP_TRY(hipStreamSynchronize(s));
    return FBDT_OK;
}

double hist_algorithmic_bytes(int64_t n, int d, int n_bins, int layer, bool routed,
                              bool sibling) {
    double b = (double)n * d + 4.0 * n;                 // bin codes + weights
    if (routed) {
        if (layer >= 2) b += (double)n;                 // parent ids
        if (layer >= 1) b += 2.0 * n;                   // routing code + ids written
    } else {
        b += (double)n;                                 // node ids
    }
    // the histograms written: below the root a sibling pass writes one child
    // per parent (the other is parent - child)
    const int hnodes = sibling && layer >= 1 ? 1 << (layer - 1) : 1 << layer;
    b += (double)hnodes * d * n_bins * 2 * 8;
    return b;
}

// Bytes a list pass of layer `layer` needs at the least: for each expected
// entry (a sampled event, alpha n of them at the root, about half of them
// in the listed children with sib) its 8-byte entry and d codes, plus the
// histograms written.
double list_algorithmic_bytes(int64_t n, double alpha, int d, int n_bins, int layer, bool sib) {
    const double entries = alpha * (double)n * (sib ? 0.5 : 1.0);
    const int hnodes = sib ? 1 << (layer - 1) : 1 << layer;
    return entries * (8.0 + d) + (double)hnodes * d * n_bins * 2 * 8;
}

}  // namespace

// ===========================================================================
extern "C" {

const char *fbdt_last_error(void) { return g_error.c_str(); }

int fbdt_set_option(const char *name, int64_t value) {
    if (!name) return fail(FBDT_E_INVAL, "option name is NULL");
    if (value < 0) return fail(FBDT_E_INVAL, "option %s: value must be >= 0", name);
    if (!strcmp(name, "hist_features_per_group")) {
        if (value != 0 && !hist_fpg_supported((int)value))
            return fail(FBDT_E_INVAL, "hist_features_per_group must be 0, 1, 2, 4, 5 or 8");
        opt_hist_fpg = value;
    } else if (!strcmp(name, "hist_event_chunks")) {
        opt_hist_chunks = value;
    } else if (!strcmp(name, "hist_threads")) {
        if (value != 0 && (value % 64 != 0 || value > 1024))
            return fail(FBDT_E_INVAL, "hist_threads must be a multiple of 64, <= 1024");
        opt_hist_threads = value;
    } else if (!strcmp(name, "hist_copies")) {
        if (value != 0 && value != 1 && value != 2 && value != 4)
            return fail(FBDT_E_INVAL, "hist_copies must be 0, 1, 2 or 4");
        opt_hist_copies = value;
    } else if (!strcmp(name, "hist_lists")) {
        if (value > 2) return fail(FBDT_E_INVAL, "hist_lists must be 0 (auto), 1 (off) or 2 (on)");
        opt_hist_lists = value;
    } else if (!strcmp(name, "list_features_per_group")) {
        if (value != 0 && !list_fpg_supported((int)value))
            return fail(FBDT_E_INVAL,
                        "list_features_per_group must be 0, 4, 8, 12, 20, 28, 36 or 40");
        opt_list_fpg = value;
    } else if (!strcmp(name, "list_parts")) {
        if (value > 4096) return fail(FBDT_E_INVAL, "list_parts must be <= 4096");
        opt_list_parts = value;
    } else if (!strcmp(name, "list_copies")) {
        if (value != 0 && value != 1 && value != 2 && value != 4)
            return fail(FBDT_E_INVAL, "list_copies must be 0, 1, 2 or 4");
        opt_list_copies = value;
    } else if (!strcmp(name, "hist_timeline")) {
        opt_hist_timeline = value != 0;
    } else if (!strcmp(name, "fail_alloc")) {
        // the scratch the library holds is released first, so that the next
        // call that needs scratch allocates (and fails)
        if (value > 0) {
            const int rc = release_scratch();
            if (rc) return rc;
        }
        opt_fail_alloc = value;
    } else if (!strcmp(name, "fit_graphs")) {
        opt_fit_graphs = value != 0;
    } else if (!strcmp(name, "apply_threads")) {
        if (value != 0 && (value % 64 != 0 || value > 1024))
            return fail(FBDT_E_INVAL, "apply_threads must be a multiple of 64, <= 1024");
        opt_apply_threads = value;
    } else {
        return fail(FBDT_E_INVAL, "unknown option %s", name);
    }
    return FBDT_OK;
}

int fbdt_timing_enable(int32_t kinds) {
    std::lock_guard<std::mutex> lk(g_t_mu);
    for (auto &p : g_pending) {
        (void)hipEventSynchronize(p.stop);
        g_event_pool.push_back(p.start);
        g_event_pool.push_back(p.stop);
    }
    g_pending.clear();
    for (int k = 0; k < FBDT_K_COUNT; ++k) {
        g_t_launches[k] = 0;
        g_t_ms[k] = 0.0;
        g_t_bytes[k] = 0.0;
    }
    g_timing = kinds & ((1 << FBDT_K_COUNT) - 1);
    return FBDT_OK;
}

int fbdt_timing_read(int32_t kind, int64_t *launches, double *total_ms, double *bytes) {
    if (kind < 0 || kind >= FBDT_K_COUNT) return fail(FBDT_E_INVAL, "kernel kind %d", kind);
    std::lock_guard<std::mutex> lk(g_t_mu);
    for (auto &p : g_pending) {
        HIP_TRY(hipEventSynchronize(p.stop));
        float ms = 0.f;
        HIP_TRY(hipEventElapsedTime(&ms, p.start, p.stop));
        g_t_launches[p.kind] += 1;
        g_t_ms[p.kind] += ms;
        g_t_bytes[p.kind] += p.bytes;
        g_event_pool.push_back(p.start);
        g_event_pool.push_back(p.stop);
    }
    g_pending.clear();
    if (launches) *launches = g_t_launches[kind];
    if (total_ms) *total_ms = g_t_ms[kind];
    if (bytes) *bytes = g_t_bytes[kind];
    return FBDT_OK;
}

// ---- binning --------------------------------------------------------------
static int encode_with(const float *x, int64_t n, int32_t d, int64_t ldx, int32_t n_bins,
                       const float *host_bounds, uint8_t *xb, int64_t ldb, hipStream_t s) {
    int dev;
    DeviceInfo di;
    int rc = current_device(&dev, &di);
    if (rc) return rc;
    Arena &a = g_arena[dev];
    std::lock_guard<std::mutex> lk(a.mu);
    const size_t nb = (size_t)d * (n_bins - 1);
    Carver cv;
    float *bounds;
    int *err;
    cv.add(&bounds, std::max<size_t>(nb, 1));
    cv.add(&err, 1);
    if ((rc = arena_reserve(a, cv.off))) return rc;
    cv.assign(a.ptr);
    HIP_TRY(hipMemcpyAsync(bounds, host_bounds, nb * sizeof(float), hipMemcpyHostToDevice, s));
    HIP_TRY(launch_fill_u32(err, 0u, 1, s));
    {
        Timed t(FBDT_K_ENCODE, s, (double)n * d * 5.0);
        HIP_TRY(launch_encode(x, ldx, n, d, bounds, n_bins, xb, ldb, err, s));
        t.done();
    }
    int h_err = 0;
    if ((rc = read_err(err, s, &h_err))) return rc;
    if (h_err & kErrNan) return fail(FBDT_E_NAN, "NaN among the feature values needs n_bins <= 255");
    return FBDT_OK;
}

// Training boundaries [d][n_bins - 1]: no NaN, non-decreasing per feature.
static int check_boundaries(const float *b, int32_t d, int32_t n_bins) {
    for (int j = 0; j < d; ++j) {
        const float *r = b + (size_t)j * (n_bins - 1);
        for (int k = 0; k < n_bins - 1; ++k) {
            if (std::isnan(r[k])) return fail(FBDT_E_INVAL, "boundary %d of feature %d is NaN", k, j);
            if (k > 0 && !(r[k - 1] <= r[k]))
                return fail(FBDT_E_INVAL, "boundaries of feature %d are not ascending", j);
        }
    }
    return FBDT_OK;
}

static int check_float_input(const float *x, int64_t n, int32_t d, int64_t ldx) {
    if (!x) return fail(FBDT_E_INVAL, "x is NULL");
    if (ldx < n) return fail(FBDT_E_INVAL, "ldx = %lld < n", (long long)ldx);
    (void)d;
    return FBDT_OK;
}

int fbdt_bin(const float *x, int64_t n, int32_t d, int64_t ldx, int32_t n_bins,
             float *boundaries, uint8_t *xb, int64_t ldb, void *stream) {
    int rc;
    if ((rc = check_codes(xb, n, d, ldb)) || (rc = check_bins(n_bins)) ||
        (rc = check_float_input(x, n, d, ldx)))
        return rc;
    if (!boundaries) return fail(FBDT_E_INVAL, "boundaries is NULL");
    hipStream_t s = static_cast<hipStream_t>(stream);
    int dev;
    DeviceInfo di;
    if ((rc = current_device(&dev, &di))) return rc;
    // Exact order statistics on the device: boundary k of feature j is the
    // value of rank floor(k n / B) of the feature (section 2.2), read off a
    // radix sort of the feature's values; then every value is encoded.
    QuantileScratch qs;
    HIP_TRY(quantile_scratch(n, d, &qs));
    const size_t nb = (size_t)d * (n_bins - 1);
    Arena &a = g_arena[dev];
    std::lock_guard<std::mutex> lk(a.mu);
    Carver cv;
    uint64_t *keys_a, *keys_b;
    char *temp;
    unsigned long long *nan_count;
    float *bounds;
    int *err;
    cv.add(&keys_a, qs.key_elems);
    cv.add(&keys_b, qs.key_elems);
    cv.add(&temp, std::max<size_t>(qs.temp_bytes, 1));
    cv.add(&nan_count, (size_t)d);
    cv.add(&bounds, nb);
    cv.add(&err, 1);
    if ((rc = arena_reserve(a, cv.off))) return rc;
    cv.assign(a.ptr);
    HIP_TRY(launch_fill_u32(err, 0u, 1, s));
    HIP_TRY(launch_quantile_boundaries(x, ldx, n, d, n_bins, qs, keys_a, keys_b, temp, nan_count,
                                       bounds, err, s));
    int h_err = 0;
    if ((rc = read_err(err, s, &h_err))) return rc;
    if (h_err & kErrNan)
        return fail(FBDT_E_NAN, "NaN among the feature values needs n_bins <= 255");
    {
        Timed t(FBDT_K_ENCODE, s, (double)n * d * 5.0);
        HIP_TRY(launch_encode(x, ldx, n, d, bounds, n_bins, xb, ldb, err, s));
        t.done();
    }
    std::vector<float> host(nb);
    HIP_TRY(hipMemcpyAsync(host.data(), bounds, nb * sizeof(float), hipMemcpyDeviceToHost, s));
    if ((rc = read_err(err, s, &h_err))) return rc;
    if (h_err & kErrNan) return fail(FBDT_E_NAN, "NaN among the feature values needs n_bins <= 255");
    std::memcpy(boundaries, host.data(), nb * sizeof(float));
    return FBDT_OK;
}

int fbdt_bin_transform(const float *x, int64_t n, int32_t d, int64_t ldx, int32_t n_bins,
                       const float *boundaries, uint8_t *xb, int64_t ldb, void *stream) {
    int rc;
    if ((rc = check_codes(xb, n, d, ldb)) || (rc = check_bins(n_bins)) ||
        (rc = check_float_input(x, n, d, ldx)))
        return rc;
    if (!boundaries) return fail(FBDT_E_INVAL, "boundaries is NULL");
    for (int j = 0; j < d; ++j)
        for (int k = 1; k < n_bins - 1; ++k)
            if (!(boundaries[(size_t)j * (n_bins - 1) + k - 1] <=
                  boundaries[(size_t)j * (n_bins - 1) + k]))
                return fail(FBDT_E_INVAL, "boundaries of feature %d are not ascending", j);
    return encode_with(x, n, d, ldx, n_bins, boundaries, xb, ldb, static_cast<hipStream_t>(stream));
}

// ---- fit ------------------------------------------------------------------
int fbdt_fit(const uint8_t *xb, int64_t n, int32_t d, int64_t ldb, int32_t n_bins,
             const int8_t *y, const float *w, const fbdt_fit_params *p, fbdt_model **out,
             double *score_out, void *stream) {
    int rc;
    if ((rc = check_codes(xb, n, d, ldb)) || (rc = check_bins(n_bins))) return rc;
    if (!y) return fail(FBDT_E_INVAL, "y is NULL");
    if (!p) return fail(FBDT_E_INVAL, "params is NULL");
    if (!out) return fail(FBDT_E_INVAL, "out is NULL");
    if (p->depth < 1 || p->depth > 7) return fail(FBDT_E_INVAL, "depth %d not in [1, 7]", p->depth);
    if (p->n_trees < 1) return fail(FBDT_E_INVAL, "n_trees %d < 1", p->n_trees);
    if (!(p->shrinkage > 0.0) || !std::isfinite(p->shrinkage))
        return fail(FBDT_E_INVAL, "shrinkage must be finite and > 0");
    if (!(p->subsample > 0.0 && p->subsample <= 1.0))
        return fail(FBDT_E_INVAL, "subsample must be in (0, 1]");

    int dev;
    DeviceInfo di;
    if ((rc = current_device(&dev, &di))) return rc;
    hipStream_t s = static_cast<hipStream_t>(stream);
    const int D = p->depth, T = p->n_trees;
    const int nin = (1 << D) - 1, nleaf = 1 << D;
    const int64_t npad = (n + 15) & ~(int64_t)15;

    // missing values (section 4.2) are possible with at most 255 bins; the
    // scan of the codes decides, so the plans and buffers below fit either mode
    const bool may_miss = n_bins <= kMissingCode;
    // below the root the routed pass histograms one child per parent (the
    // other is parent - child), except with missing values: an event that
    // stops at a parent is in the parent's histograms but in neither child's,
    // so both children are histogrammed
    std::vector<HistShape> plans_sib(D), plans_both(may_miss ? D : 0);
    size_t partial_elems = 0;
    for (int mode = 0; mode < (may_miss ? 2 : 1); ++mode) {
        std::vector<HistShape> &pl = mode == 0 ? plans_sib : plans_both;
        for (int l = 0; l < D; ++l) {
            pl[l] = plan_histogram(n, d, n_bins, l, mode == 0, di.cu_count, di.max_lds,
                                   hist_overrides());
            pl[l].prefix = true;   // the cut scan reads prefix-summed rows
            const size_t hnodes = pl[l].sibling ? (size_t)1 << (l - 1) : (size_t)1 << l;
            partial_elems =
                std::max(partial_elems, (size_t)pl[l].chunks * hnodes * d * n_bins * 2);
            if (pl[l].lds_bytes + kHistStaticLdsReserve > di.max_lds)
                return fail(FBDT_E_INVAL, "layer %d needs %zu bytes of LDS, the device has %zu", l,
                            pl[l].lds_bytes, di.max_lds);
        }
    }
    // layers 1 .. D-1 of large fits histogram event lists (the lighter child
    // of every parent, or with missing values every node of the layer)
    // (the phase timeline measures the streaming pass: a fit that records
    // it streams every layer)
    const int64_t lists_opt = opt_hist_lists.load();
    const bool lists = D >= 2 && npad <= kListMaxEvents && opt_hist_timeline.load() == 0 &&
                       (lists_opt == 2 || (lists_opt == 0 && n * (D - 2) >= kListAutoWork));
    std::vector<ListShape> lplans_sib(lists ? D : 0), lplans_both(lists && may_miss ? D : 0);
    for (int l = 1; lists && l < D; ++l) {
        for (int mode = 0; mode < (may_miss ? 2 : 1); ++mode) {
            const int nl = mode == 0 ? 1 << (l - 1) : 1 << l;
            ListShape &ls = (mode == 0 ? lplans_sib : lplans_both)[l];
            ls = plan_list_histogram(d, nl, di.cu_count, di.max_lds, (int)opt_list_fpg.load(),
                                     (int)opt_list_parts.load(), (int)opt_list_copies.load());
            partial_elems =
                std::max(partial_elems, (size_t)ls.parts * d * n_bins * 2);
            if (ls.lds_bytes > di.max_lds)
                return fail(FBDT_E_INVAL, "the list pass of layer %d needs %zu bytes of LDS", l,
                            ls.lds_bytes);
        }
    }
    const int lblocks_plain = leaf_blocks(n, D, false, di.cu_count);
    const int lblocks_miss = may_miss ? leaf_blocks(n, D, true, di.cu_count) : 0;
    const size_t slots_max = may_miss ? (size_t)2 * nleaf - 1 : (size_t)nleaf;
    const size_t leaf_partial_elems =
        std::max((size_t)lblocks_plain * 2 * nleaf, (size_t)lblocks_miss * 2 * slots_max);
    const bool fused = D <= kFusedLeafDepth;
    const int max_nodes = 1 << (D - 1);

    Arena &a = g_arena[dev];
    std::lock_guard<std::mutex> lk(a.mu);
    FitBuffers fb{};
    Carver cv;
    cv.add(&fb.F, npad);
    cv.add(&fb.w, npad);
    cv.add(&fb.yts, npad);
    if (w) cv.add(&fb.v, npad);
    if (w) cv.add(&fb.vsign, npad);
    cv.add(&fb.node[0], npad);
    cv.add(&fb.node[1], npad);
    cv.add(&fb.partial, partial_elems);
    // summed histograms of the layers that have children (all but the last)
    const size_t hfull_elems = D >= 2 ? ((size_t)1 << (D - 2)) * d * n_bins * 2 : 1;
    cv.add(&fb.hfull[0], hfull_elems);
    cv.add(&fb.hfull[1], hfull_elems);
    // side histograms of the weights below the fixed-point grid, by the
    // parity of the layer's index in the whole fit (tree * D + layer)
    const size_t small_elems = (size_t)max_nodes * d * n_bins * 2;
    cv.add(&fb.small[0], small_elems);
    cv.add(&fb.small[1], small_elems);
    const int S = cut_slices(n_bins);
    cv.add(&fb.cand_gain, (size_t)max_nodes * d * S);
    cv.add(&fb.cand_cut, (size_t)max_nodes * d * S);
    cv.add(&fb.leaf_partial, leaf_partial_elems);
    cv.add(&fb.class_partial, 3 * kValidateBlocks);
    cv.add(&fb.f0, 2);
    cv.add(&fb.err, 1);
    cv.add(&fb.cut_feature, (size_t)T * nin);
    cv.add(&fb.cut_bin, (size_t)T * nin);
    cv.add(&fb.gain, (size_t)T * nin);
    cv.add(&fb.leaf, (size_t)T * slots_max);
    // event lists: the event-major codes, the lists (a list holds at most
    // the sampled events of its node's parent: one list per parent, or with
    // missing values two), per layer 64 cursors + 64 node counts, the lists'
    // starts, caps and listed children, and their partial rows for the cut
    // scan
    uint8_t *xr = nullptr;
    uint2 *list = nullptr, *lchunks = nullptr;
    uint32_t *lctr = nullptr, *lstart = nullptr, *lcap = nullptr, *lside = nullptr;
    const size_t lctr_count = (size_t)D * 2 * kListMaxSlots;
    if (lists) {
        cv.add(&xr, list_codes_bytes(n, d));
        cv.add(&list, (size_t)(may_miss ? 2 : 1) * npad);
        cv.add(&lctr, lctr_count);
        cv.add(&lstart, kListMaxSlots);
        cv.add(&lcap, kListMaxSlots);
        cv.add(&lside, kListMaxSlots);
        cv.add(&lchunks, kListMaxSlots);
    }
    // phase timeline of every histogram launch (measurement option)
    const bool timeline = opt_hist_timeline.load() != 0;
    int tl_blocks = 0;
    for (int mode = 0; mode < (may_miss ? 2 : 1); ++mode)
        for (const HistShape &h : mode == 0 ? plans_sib : plans_both)
            tl_blocks = std::max(tl_blocks, h.blocks);
    const size_t tl_count = timeline ? (size_t)T * D * tl_blocks * kTimelineStamps : 0;
    unsigned long long *tl = nullptr;
    if (timeline) cv.add(&tl, tl_count);
    cv.add(&fb.sany, 2);   // last: the other buffers keep their offsets
    cv.add(&fb.keys, 2 * kKeyWords);
    if ((rc = arena_reserve(a, cv.off))) return rc;
    cv.assign(a.ptr);
    if (timeline) HIP_TRY(launch_fill_u32(tl, 0u, 2 * tl_count, s));

    HIP_TRY(launch_fill_u32(fb.err, 0u, 1, s));
    HIP_TRY(launch_fill_u32(fb.small[0], 0u, 2 * small_elems, s));
    HIP_TRY(launch_fill_u32(fb.small[1], 0u, 2 * small_elems, s));
    HIP_TRY(launch_fill_u32(fb.sany, 0u, 2, s));
    HIP_TRY(launch_fill_u32(reinterpret_cast<uint32_t *>(fb.keys), 0u, 2 * 2 * kKeyWords, s));
    // the histogram and leaf passes read whole steps of events: padded events
    // weigh 0 and have no pseudo-response
    HIP_TRY(launch_fill_u32(fb.w, 0u, (size_t)npad, s));
    HIP_TRY(launch_fill_u32(fb.yts, 0u, 2 * (size_t)npad, s));
    if (w) {
        HIP_TRY(launch_fill_u32(fb.v, 0u, (size_t)npad, s));
        HIP_TRY(hipMemcpyAsync(fb.v, w, (size_t)n * sizeof(float), hipMemcpyDeviceToDevice, s));
    }
    HIP_TRY(launch_validate(y, w, n, fb.class_partial, fb.err, s));
    if (may_miss) HIP_TRY(launch_find_code(xb, ldb, n, d, (uint8_t)kMissingCode, kHasMissing, fb.err, s));
    HIP_TRY(launch_initial_score(fb.class_partial, fb.f0, fb.err, s));
    int h_err = 0;
    double h_f0[2] = {0.0, 0.0};
    HIP_TRY(hipMemcpyAsync(h_f0, fb.f0, sizeof h_f0, hipMemcpyDeviceToHost, s));
    if ((rc = read_err(fb.err, s, &h_err))) return rc;
    if (h_err & kErrLabel) return fail(FBDT_E_LABEL, "labels must be +1 or -1");
    if (h_err & kErrWeight) return fail(FBDT_E_WEIGHT, "weights must be finite");
    if (h_err & kErrClass)
        return fail(FBDT_E_LABEL, "a class has no positive total weight");
    // every histogram weight has |w| = |fl32(v |y~|)| < 2 |v| (1 + 2^-24):
    // twice the sum of |v| bounds the magnitude of every (partial) bin sum
    const int scale = histogram_scale(2.0 * h_f0[1] * (1.0 + 1e-6));
    // negative event weights (section 4.1): their signs travel in bytes
    // beside the weights, and the histogram passes subtract those events
    const bool signed_w = (h_err & kNegWeights) != 0;
    const bool missing = may_miss && (h_err & kHasMissing) != 0;
    if (missing && leaf_lds_bytes(D, true) > kLeafMaxLds)
        return fail(FBDT_E_INVAL, "the leaf pass of depth %d with missing values (code %d) "
                    "needs more LDS than the device has", D, kMissingCode);
    const int nslots = missing ? 2 * nleaf - 1 : nleaf;   // boost weights per tree
    const int lblocks = missing ? lblocks_miss : lblocks_plain;
    if (signed_w) HIP_TRY(launch_sign_bytes(w, n, npad, fb.vsign, s));
    const uint8_t *vsign = signed_w ? fb.vsign : nullptr;
    const std::vector<HistShape> &plans = missing ? plans_both : plans_sib;
    const std::vector<ListShape> &lplans = missing ? lplans_both : lplans_sib;
    if (lists) HIP_TRY(launch_transpose_codes(xb, ldb, n, d, xr, s));

    const uint64_t seed = p->seed;
    const double alpha = p->subsample, eta = p->shrinkage;
    // every launch of the boosting loop, in stream order (no host sync)
    auto enqueue_trees = [&](hipStream_t st) -> int {
        for (int t = 0; t < T; ++t) {
            {
                Timed tm(FBDT_K_TREE_PREP, st, (double)n * 30.0);
                // the previous tree's boost weights: summed here from the leaf
                // pass partials (shallow trees; workgroup 0 records them), or
                // from the model after leaf_finalize
                double *prev = t == 0 ? nullptr : fb.leaf + (size_t)(t - 1) * nslots;
                HIP_TRY(launch_tree_prep(y, w, fb.F, t == 0 ? fb.f0 : nullptr,
                                         t == 0 ? nullptr : fb.node[D & 1], fused ? nullptr : prev,
                                         t > 0 && fused ? fb.leaf_partial : nullptr, lblocks, eta,
                                         fused ? prev : nullptr, D, missing, n, seed, t, alpha,
                                         fb.w, fb.yts, nullptr, di.cu_count, st));
                tm.done();
            }
            uint8_t *cf = fb.cut_feature + (size_t)t * nin;
            uint8_t *cc = fb.cut_bin + (size_t)t * nin;
            double *cg = fb.gain + (size_t)t * nin;
            // best-cut keys of layer gl = t * D + l (by gl's parity)
            auto keys = [&](int gl) { return fb.keys + (size_t)(gl & 1) * kKeyWords; };
            for (int l = 0; l < D; ++l) {
                const int gl = t * D + l;   // side histograms alternate by gl's parity
                // the previous layer's best cuts are the ones this pass routes
                // with; workgroup 0 records them in the model
                const int plo = l >= 1 ? (1 << (l - 1)) - 1 : 0;
                ParentCuts pc;
                if (l >= 1)
                    pc = ParentCuts{fb.cand_gain, keys(gl - 1), S, cf + plo, cc + plo, cg + plo};
                if (lists && l >= 1) {
                    // route with list output, then histogram the lists
                    const ListShape &ls = lplans[l];
                    const int lmode = missing ? kCutStopped : kCutSibling;
                    uint32_t *ctr = lctr + (size_t)l * 2 * kListMaxSlots;
                    const uint32_t *cap_prev =
                        l >= 2 ? lctr + (size_t)(l - 1) * 2 * kListMaxSlots + kListMaxSlots : nullptr;
                    {
                        Timed tm(FBDT_K_ROUTE, st, 3.0 * (double)n);
                        HIP_TRY(launch_route_list(
                            xb, ldb, n, d, n_bins, l >= 2 ? fb.node[(l - 1) & 1] : nullptr,
                            fb.node[l & 1], fb.w, vsign, pc, l, n_bins <= kMissingCode, lmode,
                            fb.hfull[(l - 1) & 1], scale, cap_prev, (uint32_t)npad, ctr, lstart,
                            lcap, lside, list, fb.small[gl & 1], fb.sany + (gl & 1), fb.err, st));
                        tm.done();
                    }
                    {
                        Timed tm(FBDT_K_HISTOGRAM, st,
                                 list_algorithmic_bytes(n, alpha, d, n_bins, l, !missing));
                        HIP_TRY(launch_hist_list(ls, lmode, list, lstart, lcap, ctr, lside, xr, d,
                                                 n_bins, vsign != nullptr, scale, lchunks,
                                                 fb.partial, fb.err,
                                                 l + 1 < D ? ctr + kListMaxSlots : nullptr, st));
                        tm.done();
                    }
                    {
                        Timed tm(FBDT_K_BEST_CUTS, st);
                        const size_t next_count =
                            (size_t)(l + 1 < D ? 1 << (l + 1) : 1) * d * n_bins * 2;
                        HIP_TRY(launch_cut_scan(fb.partial, 0, scale, fb.small[gl & 1],
                                                fb.sany + (gl & 1), fb.small[(gl + 1) & 1],
                                                fb.sany + ((gl + 1) & 1), next_count, ls.lists, d,
                                                n_bins, lmode, fb.cand_gain, fb.cand_cut,
                                                fb.hfull[(l - 1) & 1],
                                                l + 1 < D ? fb.hfull[l & 1] : nullptr, st,
                                                lchunks, nullptr, 0, keys(gl), keys(gl + 1)));
                        tm.done();
                    }
                    continue;
                }
                // layers with many parents are routed by a pass of their own
                // (one code gather per event instead of one per feature group)
                const bool own_route = l >= 1 && (1 << (l - 1)) > kRoutedMaxParents;
                if (own_route) {
                    Timed tm(FBDT_K_ROUTE, st, 3.0 * (double)n);
                    HIP_TRY(launch_route_layer(xb, ldb, n, d, fb.node[(l - 1) & 1],
                                               fb.node[l & 1], pc, l, n_bins <= kMissingCode,
                                               fb.err, di.cu_count, st));
                    tm.done();
                }
                {
                    Timed tm(FBDT_K_HISTOGRAM, st,
                             hist_algorithmic_bytes(n, d, n_bins, l, !own_route,
                                                    plans[l].sibling));
                    HIP_TRY(launch_histogram(
                        plans[l], xb, ldb, n, d, n_bins,
                        own_route ? fb.node[l & 1] : l >= 2 ? fb.node[(l - 1) & 1] : nullptr,
                        !own_route && l >= 1 ? fb.node[l & 1] : nullptr, fb.w, vsign,
                        own_route ? ParentCuts{} : pc, l, !own_route, scale, fb.partial,
                        fb.small[gl & 1], fb.err, st,
                        tl ? tl + (size_t)(t * D + l) * tl_blocks * kTimelineStamps : nullptr));
                    tm.done();
                }
                {
                    Timed tm(FBDT_K_BEST_CUTS, st);
                    // right children below the root: parent - left child (the
                    // parents' summed rows are kept for that; fits with missing
                    // values histogram both children); the next layer's side
                    // histogram (next tree's root after the last layer) is
                    // cleared on the way
                    const bool sib = plans[l].sibling;
                    const int cmode = sib ? kCutSibling : kCutPlain;
                    const size_t next_count =
                        (size_t)(l + 1 < D ? 1 << (l + 1) : 1) * d * n_bins * 2;
                    // the root's scan also clears the counters of the tree's
                    // list passes (layers 1 .. D-1 follow it)
                    const bool clear = lists && l == 0;
                    HIP_TRY(launch_cut_scan(fb.partial, plans[l].chunks, scale, fb.small[gl & 1],
                                            nullptr, fb.small[(gl + 1) & 1],
                                            fb.sany + ((gl + 1) & 1), next_count,
                                            sib ? 1 << (l - 1) : 1 << l, d, n_bins, cmode,
                                            fb.cand_gain, fb.cand_cut,
                                            cmode != kCutPlain ? fb.hfull[(l - 1) & 1] : nullptr,
                                            l + 1 < D ? fb.hfull[l & 1] : nullptr, st, nullptr,
                                            clear ? lctr : nullptr, clear ? (int)lctr_count : 0,
                                            keys(gl), keys(gl + 1)));
                    tm.done();
                }
            }
            {
                const int plo = (1 << (D - 1)) - 1;
                const ParentCuts pc{fb.cand_gain, keys(t * D + D - 1), S, cf + plo, cc + plo,
                                    cg + plo};
                // the leaves of deep trees are routed by a pass of their own,
                // like the deep layers
                const bool own_route = (1 << (D - 1)) > kRoutedMaxParents;
                if (own_route) {
                    Timed tm(FBDT_K_ROUTE, st, 3.0 * (double)n);
                    HIP_TRY(launch_route_layer(xb, ldb, n, d, fb.node[(D - 1) & 1],
                                               fb.node[D & 1], pc, D, n_bins <= kMissingCode,
                                               fb.err, di.cu_count, st));
                    tm.done();
                }
                Timed tm(FBDT_K_LEAF, st);
                HIP_TRY(launch_leaf(xb, ldb, n, d,
                                    own_route ? fb.node[D & 1]
                                              : D >= 2 ? fb.node[(D - 1) & 1] : nullptr,
                                    own_route ? nullptr : fb.node[D & 1],
                                    own_route ? ParentCuts{} : pc, D, missing, !own_route, fb.v,
                                    fb.yts, lblocks, fb.leaf_partial, fb.err, st));
                if (!fused || t == T - 1)
                    HIP_TRY(launch_leaf_finalize(fb.leaf_partial, lblocks, D, missing, eta,
                                                 fb.leaf + (size_t)t * nslots, st));
                tm.done();
            }
        }
        return FBDT_OK;
    };
    const int timed_kinds = (1 << FBDT_K_TREE_PREP) | (1 << FBDT_K_HISTOGRAM) |
                            (1 << FBDT_K_BEST_CUTS) | (1 << FBDT_K_LEAF) | (1 << FBDT_K_ROUTE);
    if (opt_fit_graphs.load() && !timeline && !(g_timing.load() & timed_kinds)) {
        const GraphKey key{xb, y, w, n, ldb, d, n_bins, D, T, scale, lblocks, eta, alpha, seed,
                           opt_hist_fpg.load(), opt_hist_chunks.load(), opt_hist_threads.load(),
                           opt_hist_copies.load(), signed_w, missing, lists,
                           opt_list_fpg.load(), opt_list_parts.load(), opt_list_copies.load()};
        hipGraphExec_t exec = nullptr;
        for (auto &g : a.graphs)
            if (g.first == key) exec = g.second;
        if (!exec) {
            // captured on a stream of the library's own, since the caller's may
            // be the null stream, which cannot be captured; the graph then runs
            // on the caller's stream
            if (!a.capture) HIP_TRY(hipStreamCreateWithFlags(&a.capture, hipStreamNonBlocking));
            HIP_TRY(hipStreamBeginCapture(a.capture, hipStreamCaptureModeThreadLocal));
            const int qrc = enqueue_trees(a.capture);
            hipGraph_t graph = nullptr;
            const hipError_t ce = hipStreamEndCapture(a.capture, &graph);
            if (qrc != FBDT_OK || ce != hipSuccess) {
                if (graph) (void)hipGraphDestroy(graph);
                if (qrc != FBDT_OK) return qrc;
                return fail(FBDT_E_DEVICE, "capturing the boosting loop failed: %s",
                            hipGetErrorString(ce));
            }
            const hipError_t ie = hipGraphInstantiate(&exec, graph, nullptr, nullptr, 0);
            (void)hipGraphDestroy(graph);
            if (ie != hipSuccess)
                return fail(FBDT_E_DEVICE, "instantiating the boosting loop failed: %s",
                            hipGetErrorString(ie));
            if (a.graphs.size() >= kMaxGraphs) {
                (void)hipGraphExecDestroy(a.graphs.front().second);
                a.graphs.erase(a.graphs.begin());
            }
            a.graphs.push_back({key, exec});
        }
        HIP_TRY(hipGraphLaunch(exec, s));
    } else if ((rc = enqueue_trees(s))) {
        return rc;
    }
    if (score_out)
        HIP_TRY(launch_tree_prep(y, w, fb.F, nullptr, fb.node[D & 1],
                                 fb.leaf + (size_t)(T - 1) * nslots, nullptr, 0, 0.0, nullptr, D,
                                 missing, n, seed, T, alpha, nullptr, nullptr, score_out,
                                 di.cu_count, s));

    fbdt_model *m = new (std::nothrow) fbdt_model;
    if (!m) return fail(FBDT_E_DEVICE, "out of host memory");
    m->n_trees = T;
    m->depth = D;
    m->n_features = d;
    m->n_bins = n_bins;
    m->cut_feature.resize((size_t)T * nin);
    m->cut_bin.resize((size_t)T * nin);
    m->gain.resize((size_t)T * nin);
    // the boost weights of every node (missing values) or of the leaves
    std::vector<double> values((size_t)T * nslots);
    auto cleanup = [&](int code) {
        delete m;
        return code;
    };
    if (hipMemcpyAsync(m->cut_feature.data(), fb.cut_feature, (size_t)T * nin,
                       hipMemcpyDeviceToHost, s) != hipSuccess ||
        hipMemcpyAsync(m->cut_bin.data(), fb.cut_bin, (size_t)T * nin, hipMemcpyDeviceToHost,
                       s) != hipSuccess ||
        hipMemcpyAsync(m->gain.data(), fb.gain, (size_t)T * nin * sizeof(double),
                       hipMemcpyDeviceToHost, s) != hipSuccess ||
        hipMemcpyAsync(values.data(), fb.leaf, values.size() * sizeof(double),
                       hipMemcpyDeviceToHost, s) != hipSuccess ||
        hipMemcpyAsync(&m->f0, fb.f0, sizeof(double), hipMemcpyDeviceToHost, s) != hipSuccess ||
        hipMemcpyAsync(&h_err, fb.err, sizeof(int), hipMemcpyDeviceToHost, s) != hipSuccess) {
        return cleanup(fail(FBDT_E_DEVICE, "copying the model to the host failed: %s",
                            hipGetErrorString(hipGetLastError())));
    }
    hipError_t se = hipStreamSynchronize(s);
    if (se != hipSuccess)
        return cleanup(fail(FBDT_E_DEVICE, "fit failed: %s", hipGetErrorString(se)));
    if (h_err & kErrBin) return cleanup(fail(FBDT_E_INVAL, "a bin code is >= n_bins"));
    if (h_err & kErrRoute) return cleanup(fail(FBDT_E_DEVICE, "internal routing error"));
    if (timeline) {
        int rate = 0;
        HIP_TRY(hipDeviceGetAttribute(&rate, hipDeviceAttributeWallClockRate, dev));
        std::lock_guard<std::mutex> tlk(g_timeline.mu);
        g_timeline.stamps.resize(tl_count);
        HIP_TRY(hipMemcpy(g_timeline.stamps.data(), tl, tl_count * sizeof(uint64_t),
                          hipMemcpyDeviceToHost));
        g_timeline.launches = (int64_t)T * D;
        g_timeline.max_blocks = tl_blocks;
        g_timeline.rate_khz = rate;
        g_timeline.blocks.assign((size_t)T * D, 0);
        for (int t = 0; t < T; ++t)
            for (int l = 0; l < D; ++l) g_timeline.blocks[(size_t)t * D + l] = plans[l].blocks;
    }
    m->missing = missing;
    m->leaf.resize((size_t)T * nleaf);
    if (missing) m->inner.resize((size_t)T * nin);
    for (size_t t = 0; t < (size_t)T; ++t) {
        const double *row = values.data() + t * nslots;
        if (missing) {   // heap order: the inner nodes, then the leaves
            std::copy(row, row + nin, m->inner.begin() + t * nin);
            std::copy(row + nin, row + nin + nleaf, m->leaf.begin() + t * nleaf);
        } else {
            std::copy(row, row + nleaf, m->leaf.begin() + t * nleaf);
        }
    }
    *out = m;
    return FBDT_OK;
}

// ---- model ----------------------------------------------------------------
int fbdt_model_export(const fbdt_model *m, fbdt_model_view *v) {
    if (!m || !v) return fail(FBDT_E_INVAL, "NULL argument");
    v->n_trees = m->n_trees;
    v->depth = m->depth;
    v->n_features = m->n_features;
    v->n_bins = m->n_bins;
    v->f0 = m->f0;
    v->cut_feature = m->cut_feature.data();
    v->cut_bin = m->cut_bin.data();
    v->gain = m->gain.data();
    v->leaf = m->leaf.data();
    v->boundaries = m->boundaries.empty() ? nullptr : m->boundaries.data();
    v->inner = m->missing ? m->inner.data() : nullptr;
    return FBDT_OK;
}

int fbdt_model_import(const fbdt_model_view *v, fbdt_model **out) {
    if (!v || !out) return fail(FBDT_E_INVAL, "NULL argument");
    if (v->n_trees < 1 || v->depth < 1 || v->depth > 7 || v->n_features < 1 ||
        v->n_features > 255 || v->n_bins < 2 || v->n_bins > 256)
        return fail(FBDT_E_INVAL, "model dimensions out of range");
    if (!v->cut_feature || !v->cut_bin || !v->leaf)
        return fail(FBDT_E_INVAL, "cut_feature, cut_bin and leaf are required");
    if (v->inner && v->n_bins > kMissingCode)
        return fail(FBDT_E_INVAL, "inner boost weights (missing values) need n_bins <= %d",
                    kMissingCode);
    if (!std::isfinite(v->f0)) return fail(FBDT_E_INVAL, "f0 is not finite");
    const size_t T = v->n_trees, nin = ((size_t)1 << v->depth) - 1, nleaf = (size_t)1 << v->depth;
    for (size_t k = 0; k < T * nin; ++k) {
        if (v->cut_feature[k] >= v->n_features)
            return fail(FBDT_E_INVAL, "cut feature %d >= n_features", (int)v->cut_feature[k]);
        if (v->cut_bin[k] < 1 || v->cut_bin[k] >= v->n_bins)
            return fail(FBDT_E_INVAL, "cut bin %d not in [1, n_bins)", (int)v->cut_bin[k]);
    }
    if (v->boundaries) {
        const int rc = check_boundaries(v->boundaries, v->n_features, v->n_bins);
        if (rc) return rc;
    }
    fbdt_model *m = new (std::nothrow) fbdt_model;
    if (!m) return fail(FBDT_E_DEVICE, "out of host memory");
    m->n_trees = v->n_trees;
    m->depth = v->depth;
    m->n_features = v->n_features;
    m->n_bins = v->n_bins;
    m->f0 = v->f0;
    m->cut_feature.assign(v->cut_feature, v->cut_feature + T * nin);
    m->cut_bin.assign(v->cut_bin, v->cut_bin + T * nin);
    if (v->gain)
        m->gain.assign(v->gain, v->gain + T * nin);
    else
        m->gain.assign(T * nin, 0.0);
    m->leaf.assign(v->leaf, v->leaf + T * nleaf);
    if (v->boundaries)
        m->boundaries.assign(v->boundaries,
                             v->boundaries + (size_t)v->n_features * (v->n_bins - 1));
    if (v->inner) {
        m->missing = true;
        m->inner.assign(v->inner, v->inner + T * nin);
    }
    *out = m;
    return FBDT_OK;
}

int fbdt_model_set_boundaries(fbdt_model *m, const float *boundaries) {
    int rc;
    if (!m || !boundaries) return fail(FBDT_E_INVAL, "NULL argument");
    if ((rc = check_boundaries(boundaries, m->n_features, m->n_bins))) return rc;
    std::lock_guard<std::mutex> lk(m->mu);
    m->boundaries.assign(boundaries, boundaries + (size_t)m->n_features * (m->n_bins - 1));
    // the float-apply records hold thresholds: rebuilt on next use
    int cur = -1;
    (void)hipGetDevice(&cur);
    for (auto &c : m->copies)
        if (hipSetDevice(c.device) == hipSuccess) {
            if (c.frec) (void)hipFree(c.frec);
            if (c.ftab) (void)hipFree(c.ftab);
            if (c.fnodes) (void)hipFree(c.fnodes);
            c.frec = nullptr;
            c.ftab = nullptr;
            c.fnodes = nullptr;
            c.ftab_words = 0;
            c.fnodes_stride = 0;
        }
    if (cur >= 0) (void)hipSetDevice(cur);
    return FBDT_OK;
}

void fbdt_model_free(fbdt_model *m) {
    if (!m) return;
    int cur = -1;
    (void)hipGetDevice(&cur);
    for (auto &c : m->copies) {
        if (hipSetDevice(c.device) == hipSuccess) {
            (void)hipFree(c.cuts);
            (void)hipFree(c.leaves);
            if (c.nodes) (void)hipFree(c.nodes);
            if (c.frec) (void)hipFree(c.frec);
            if (c.gains) (void)hipFree(c.gains);
            if (c.ftab) (void)hipFree(c.ftab);
            if (c.fnodes) (void)hipFree(c.fnodes);
        }
    }
    if (cur >= 0) (void)hipSetDevice(cur);
    delete m;
}

// ---- apply ----------------------------------------------------------------
// The model's device copy on `dev`, created on first use: the packed cuts and
// the boost weights per tree (the leaves, or with missing values every node
// in heap order).  Call with m->mu held.
static int device_copy(fbdt_model *m, int dev, fbdt_model::DeviceCopy **out) {
    for (auto &c : m->copies)
        if (c.device == dev) {
            *out = &c;
            return FBDT_OK;
        }
    const size_t T = m->n_trees, nin = ((size_t)1 << m->depth) - 1;
    const size_t nleaf = (size_t)1 << m->depth;
    const size_t per_tree = m->missing ? nin + nleaf : nleaf;
    std::vector<uint16_t> packed(T * nin);
    for (size_t k = 0; k < packed.size(); ++k)
        packed[k] = (uint16_t)(m->cut_feature[k] | (m->cut_bin[k] << 8));
    std::vector<double> values(T * per_tree);
    for (size_t t = 0; t < T; ++t) {
        double *row = values.data() + t * per_tree;
        if (m->missing) {
            std::copy(m->inner.begin() + t * nin, m->inner.begin() + (t + 1) * nin, row);
            row += nin;
        }
        std::copy(m->leaf.begin() + t * nleaf, m->leaf.begin() + (t + 1) * nleaf, row);
    }
    fbdt_model::DeviceCopy c{dev, nullptr, nullptr, 0, nullptr, nullptr, nullptr};
    HIP_TRY(device_alloc(reinterpret_cast<void **>(&c.cuts), packed.size() * sizeof(uint16_t)));
    if (device_alloc(reinterpret_cast<void **>(&c.leaves), values.size() * sizeof(double)) !=
        hipSuccess) {
        (void)hipFree(c.cuts);
        return fail(FBDT_E_DEVICE, "out of device memory");
    }
    m->copies.push_back(c);
    fbdt_model::DeviceCopy *cp = &m->copies.back();
    HIP_TRY(hipMemcpy(cp->cuts, packed.data(), packed.size() * sizeof(uint16_t),
                      hipMemcpyHostToDevice));
    HIP_TRY(hipMemcpy(cp->leaves, values.data(), values.size() * sizeof(double),
                      hipMemcpyHostToDevice));
    *out = cp;
    return FBDT_OK;
}

int fbdt_apply(const fbdt_model *mc, const uint8_t *xb, int64_t n, int32_t d, int64_t ldb,
               float *prob, double *score, void *stream) {
    int rc;
    if (!mc) return fail(FBDT_E_INVAL, "model is NULL");
    if ((rc = check_codes(xb, n, d, ldb))) return rc;
    if (!prob) return fail(FBDT_E_INVAL, "prob is NULL");
    fbdt_model *m = const_cast<fbdt_model *>(mc);
    if (d < m->n_features)
        return fail(FBDT_E_SHAPE, "d = %d < the model's %d features", d, m->n_features);
    int dev;
    DeviceInfo di;
    if ((rc = current_device(&dev, &di))) return rc;
    hipStream_t s = static_cast<hipStream_t>(stream);
    const int T = m->n_trees, D = m->depth;
    const size_t nin = ((size_t)1 << D) - 1;
    ApplyShape as = plan_apply(n, m->n_features, T, D, m->missing, di.cu_count, di.max_lds,
                               (int)opt_apply_threads.load());
    if (as.lds_bytes + kHistStaticLdsReserve > di.max_lds)
        return fail(FBDT_E_INVAL, "apply needs %zu bytes of LDS, the device has %zu (fewer "
                    "apply_threads)", as.lds_bytes, di.max_lds);
    uint16_t *cuts = nullptr;
    uint32_t *nodes = nullptr;
    double *leaves = nullptr;
    {
        std::lock_guard<std::mutex> lk(m->mu);
        fbdt_model::DeviceCopy *copy = nullptr;
        if ((rc = device_copy(m, dev, &copy))) return rc;
        if (as.shallow && copy->nodes_stride != apply_node_stride(as)) {
            // node records for this launch's tile stride
            const int xs = apply_node_stride(as);
            std::vector<uint32_t> table((size_t)T * 16, 0u);
            for (size_t t = 0; t < (size_t)T; ++t)
                for (size_t k = 0; k < nin; ++k) {
                    table[t * 16 + k] = (uint32_t)m->cut_feature[t * nin + k] * (uint32_t)xs;
                    table[t * 16 + 8 + k] = (256u - m->cut_bin[t * nin + k]) * 0x10001u;
                }
            if (!copy->nodes)
                HIP_TRY(device_alloc(reinterpret_cast<void **>(&copy->nodes),
                                     table.size() * sizeof(uint32_t)));
            HIP_TRY(hipMemcpy(copy->nodes, table.data(), table.size() * sizeof(uint32_t),
                              hipMemcpyHostToDevice));
            copy->nodes_stride = xs;
        }
        cuts = copy->cuts;
        nodes = copy->nodes;
        leaves = copy->leaves;
    }
    Timed tm(FBDT_K_APPLY, s, (double)n * (m->n_features + 4));
    HIP_TRY(launch_apply(as, xb, ldb, n, cuts, nodes, leaves, T, D, m->f0, prob, score, s));
    tm.done();
    return FBDT_OK;
}

int fbdt_feature_importance(const fbdt_model *m, double *importance) {
    if (!m || !importance) return fail(FBDT_E_INVAL, "NULL argument");
    const size_t nin = ((size_t)1 << m->depth) - 1;
    std::vector<double> imp((size_t)m->n_features, 0.0);
    for (size_t k = 0; k < (size_t)m->n_trees * nin; ++k) imp[m->cut_feature[k]] += m->gain[k];
    std::memcpy(importance, imp.data(), imp.size() * sizeof(double));
    return FBDT_OK;
}

int fbdt_event_importance(const fbdt_model *mc, const uint8_t *xb, int64_t n, int32_t d,
                          int64_t ldb, double *importance, int64_t ldi, void *stream) {
    int rc;
    if (!mc) return fail(FBDT_E_INVAL, "model is NULL");
    if ((rc = check_codes(xb, n, d, ldb))) return rc;
    if (!importance) return fail(FBDT_E_INVAL, "importance is NULL");
    if (ldi < n) return fail(FBDT_E_INVAL, "ldi = %lld < n", (long long)ldi);
    fbdt_model *m = const_cast<fbdt_model *>(mc);
    if (d < m->n_features)
        return fail(FBDT_E_SHAPE, "d = %d < the model's %d features", d, m->n_features);
    int dev;
    DeviceInfo di;
    if ((rc = current_device(&dev, &di))) return rc;
    hipStream_t s = static_cast<hipStream_t>(stream);
    const int T = m->n_trees, D = m->depth;
    const size_t nin = ((size_t)1 << D) - 1;
    const ApplyShape as =
        plan_importance(n, m->n_features, T, D, m->missing, di.cu_count, di.max_lds);
    if (as.lds_bytes + kHistStaticLdsReserve > di.max_lds)
        return fail(FBDT_E_INVAL, "event importance needs %zu bytes of LDS, the device has %zu",
                    as.lds_bytes, di.max_lds);
    const uint16_t *cuts = nullptr;
    const double *gains = nullptr;
    {
        std::lock_guard<std::mutex> lk(m->mu);
        fbdt_model::DeviceCopy *copy = nullptr;
        if ((rc = device_copy(m, dev, &copy))) return rc;
        if (!copy->gains) {
            HIP_TRY(device_alloc(reinterpret_cast<void **>(&copy->gains),
                                 (size_t)T * nin * sizeof(double)));
            HIP_TRY(hipMemcpy(copy->gains, m->gain.data(), (size_t)T * nin * sizeof(double),
                              hipMemcpyHostToDevice));
        }
        cuts = copy->cuts;
        gains = copy->gains;
    }
    HIP_TRY(launch_importance(as, xb, ldb, n, cuts, gains, T, D, importance, ldi, d, s));
    return FBDT_OK;
}

int fbdt_apply_float(const fbdt_model *mc, const float *x, int64_t n, int32_t d, int64_t ldx,
                     float *prob, double *score, void *stream) {
    int rc;
    if (!mc) return fail(FBDT_E_INVAL, "model is NULL");
    if ((rc = check_float_input(x, n, d, ldx))) return rc;
    if (n < 1) return fail(FBDT_E_INVAL, "n = %lld must be >= 1", (long long)n);
    if (!prob) return fail(FBDT_E_INVAL, "prob is NULL");
    fbdt_model *m = const_cast<fbdt_model *>(mc);
    if (d < m->n_features)
        return fail(FBDT_E_SHAPE, "d = %d < the model's %d features", d, m->n_features);
    int dev;
    DeviceInfo di;
    if ((rc = current_device(&dev, &di))) return rc;
    hipStream_t s = static_cast<hipStream_t>(stream);
    const int T = m->n_trees, D = m->depth;
    const size_t nin = ((size_t)1 << D) - 1;
    const bool shallow = D <= kApplyShallowDepth && !m->missing;
    ApplyShape as{};
    const uint2 *rec = nullptr;
    const uint32_t *fnodes = nullptr, *ftab = nullptr;
    int ftab_words = 0;
    const double *leaves = nullptr;
    {
        std::lock_guard<std::mutex> lk(m->mu);
        if (m->boundaries.empty())
            return fail(FBDT_E_INVAL, "the model has no bin boundaries (fbdt_model_set_boundaries)");
        fbdt_model::DeviceCopy *copy = nullptr;
        if ((rc = device_copy(m, dev, &copy))) return rc;
        const size_t nb = (size_t)m->n_bins - 1;
        // cut "bin >= c" of feature j = "x >= boundary c of feature j"
        // (boundary index c - 1 of its row)
        auto threshold = [&](size_t k) {
            return m->boundaries[(size_t)m->cut_feature[k] * nb + m->cut_bin[k] - 1];
        };
        std::vector<uint32_t> rank;   // per node: rank of its threshold (shallow)
        if (shallow && !copy->ftab) {
            // per feature, the ascending distinct thresholds its cuts test
            // (equal values, +0 and -0 included, decide alike: one entry)
            const int d_used = m->n_features;
            std::vector<std::vector<float>> per(d_used);
            for (size_t k = 0; k < (size_t)T * nin; ++k)
                per[m->cut_feature[k]].push_back(threshold(k));
            std::vector<uint32_t> table(d_used + 1, 0u);
            for (int f = 0; f < d_used; ++f) {
                auto &v = per[f];
                std::sort(v.begin(), v.end());
                v.erase(std::unique(v.begin(), v.end(),
                                    [](float a, float b) { return a == b; }),
                        v.end());
                table[f + 1] = table[f] + (uint32_t)v.size();
            }
            for (int f = 0; f < d_used; ++f)
                for (float t : per[f]) {
                    uint32_t bits;
                    std::memcpy(&bits, &t, sizeof bits);
                    table.push_back(bits);
                }
            HIP_TRY(device_alloc(reinterpret_cast<void **>(&copy->ftab),
                                 table.size() * sizeof(uint32_t)));
            HIP_TRY(hipMemcpy(copy->ftab, table.data(), table.size() * sizeof(uint32_t),
                              hipMemcpyHostToDevice));
            copy->ftab_words = (int)table.size();
            copy->fnodes_stride = 0;
        }
        if (shallow) {
            as = plan_apply_float(n, m->n_features, T, D, false, di.cu_count, di.max_lds,
                                  (int)opt_apply_threads.load(),
                                  (size_t)copy->ftab_words * sizeof(uint32_t));
            if (copy->fnodes_stride != apply_node_stride(as)) {
                // node records for this launch's tile stride, with threshold ranks
                std::vector<uint32_t> ttab((size_t)copy->ftab_words);
                HIP_TRY(hipMemcpy(ttab.data(), copy->ftab, ttab.size() * sizeof(uint32_t),
                                  hipMemcpyDeviceToHost));
                const int xs = apply_node_stride(as);
                std::vector<uint32_t> table((size_t)T * 16, 0u);
                const uint32_t *off = ttab.data();
                const float *thr = reinterpret_cast<const float *>(ttab.data() + m->n_features + 1);
                for (size_t t = 0; t < (size_t)T; ++t)
                    for (size_t k = 0; k < nin; ++k) {
                        const size_t q = t * nin + k;
                        const uint32_t f = m->cut_feature[q];
                        const float v = threshold(q);
                        const float *lo = thr + off[f], *hi = thr + off[f + 1];
                        const uint32_t r = (uint32_t)(std::lower_bound(lo, hi, v) - lo) + 1u;
                        table[t * 16 + k] = f * (uint32_t)xs;
                        table[t * 16 + 8 + k] = (256u - r) * 0x10001u;
                    }
                if (!copy->fnodes)
                    HIP_TRY(device_alloc(reinterpret_cast<void **>(&copy->fnodes),
                                         table.size() * sizeof(uint32_t)));
                HIP_TRY(hipMemcpy(copy->fnodes, table.data(), table.size() * sizeof(uint32_t),
                                  hipMemcpyHostToDevice));
                copy->fnodes_stride = xs;
            }
            fnodes = copy->fnodes;
            ftab = copy->ftab;
            ftab_words = copy->ftab_words;
        } else {
            as = plan_apply_float(n, m->n_features, T, D, m->missing, di.cu_count, di.max_lds,
                                  (int)opt_apply_threads.load(), 0);
            if (!copy->frec) {
                std::vector<uint2> table((size_t)T * nin);
                for (size_t k = 0; k < table.size(); ++k) {
                    const float thr = threshold(k);
                    uint32_t bits;
                    std::memcpy(&bits, &thr, sizeof bits);
                    table[k] = make_uint2(m->cut_feature[k], bits);
                }
                HIP_TRY(device_alloc(reinterpret_cast<void **>(&copy->frec),
                                     table.size() * sizeof(uint2)));
                HIP_TRY(hipMemcpy(copy->frec, table.data(), table.size() * sizeof(uint2),
                                  hipMemcpyHostToDevice));
            }
            rec = copy->frec;
        }
        leaves = copy->leaves;
    }
    if (as.lds_bytes + kHistStaticLdsReserve > di.max_lds)
        return fail(FBDT_E_INVAL, "apply needs %zu bytes of LDS, the device has %zu (fewer "
                    "apply_threads)", as.lds_bytes, di.max_lds);
    Timed tm(FBDT_K_APPLY, s, (double)n * (4.0 * m->n_features + 4));
    HIP_TRY(launch_apply_float(as, x, ldx, n, rec, fnodes, ftab, ftab_words, leaves, T, D, m->f0,
                               prob, score, s));
    tm.done();
    return FBDT_OK;
}

// ---- single steps -----------------------------------------------------------
int fbdt_tree_weights(const int8_t *y, const float *v, const double *F, int64_t n, uint64_t seed,
                      int32_t tree, double alpha, float *w_out, void *stream) {
    if (!y || !F || !w_out) return fail(FBDT_E_INVAL, "NULL argument");
    if (n < 1) return fail(FBDT_E_INVAL, "n must be >= 1");
    if (tree < 0) return fail(FBDT_E_INVAL, "tree must be >= 0");
    if (!(alpha > 0.0 && alpha <= 1.0)) return fail(FBDT_E_INVAL, "alpha must be in (0, 1]");
    int rc, dev;
    DeviceInfo di;
    if ((rc = current_device(&dev, &di))) return rc;
    hipStream_t s = static_cast<hipStream_t>(stream);
    Timed tm(FBDT_K_TREE_PREP, s, (double)n * 17.0);
    HIP_TRY(launch_tree_prep(y, v, const_cast<double *>(F), nullptr, nullptr, nullptr, nullptr, 0,
                             0.0, nullptr, 1, false, n, seed, tree, alpha, w_out, nullptr, nullptr,
                             di.cu_count, s));
    tm.done();
    return FBDT_OK;
}

int fbdt_histogram(const uint8_t *xb, int64_t n, int32_t d, int64_t ldb, int32_t n_bins,
                   const uint8_t *node, const float *w, int32_t layer, double *hist,
                   void *stream) {
    int rc;
    if ((rc = check_codes(xb, n, d, ldb)) || (rc = check_bins(n_bins))) return rc;
    if (!node || !w || !hist) return fail(FBDT_E_INVAL, "NULL argument");
    if (!aligned16(node) || !aligned16(w))
        return fail(FBDT_E_INVAL, "node and w must be 16-byte aligned");
    if (layer < 0 || layer > 6) return fail(FBDT_E_INVAL, "layer %d not in [0, 6]", layer);
    int dev;
    DeviceInfo di;
    if ((rc = current_device(&dev, &di))) return rc;
    hipStream_t s = static_cast<hipStream_t>(stream);
    HistShape hs = plan_histogram(n, d, n_bins, layer, false, di.cu_count, di.max_lds,
                                  hist_overrides());
    if (hs.lds_bytes + kHistStaticLdsReserve > di.max_lds)
        return fail(FBDT_E_INVAL, "layer %d needs %zu bytes of LDS, the device has %zu", layer,
                    hs.lds_bytes, di.max_lds);
    const size_t count = ((size_t)1 << layer) * d * n_bins * 2;
    // the pass reads whole steps of events: node ids and weights are copied
    // into buffers padded with zero weights
    const int64_t npad = (n + 15) & ~(int64_t)15;
    Arena &a = g_arena[dev];
    std::lock_guard<std::mutex> lk(a.mu);
    Carver cv;
    uint64_t *partial;
    double *small, *bpart, *wsum;
    int *err;
    uint8_t *node_pad;
    float *w_pad;
    cv.add(&node_pad, (size_t)npad);
    cv.add(&w_pad, (size_t)npad);
    cv.add(&partial, (size_t)hs.chunks * count);
    cv.add(&small, count);
    cv.add(&bpart, kValidateBlocks);
    cv.add(&wsum, 1);
    cv.add(&err, 1);
    if ((rc = arena_reserve(a, cv.off))) return rc;
    cv.assign(a.ptr);
    HIP_TRY(launch_fill_u32(err, 0u, 1, s));
    HIP_TRY(launch_fill_u32(small, 0u, 2 * count, s));
    HIP_TRY(launch_fill_u32(node_pad, 0u, (size_t)npad / 4, s));
    HIP_TRY(launch_fill_u32(w_pad, 0u, (size_t)npad, s));
    HIP_TRY(hipMemcpyAsync(node_pad, node, (size_t)n, hipMemcpyDeviceToDevice, s));
    HIP_TRY(hipMemcpyAsync(w_pad, w, (size_t)n * sizeof(float), hipMemcpyDeviceToDevice, s));
    HIP_TRY(launch_abs_sum(w, n, bpart, wsum, s));
    double h_wsum = 0.0;
    HIP_TRY(hipMemcpyAsync(&h_wsum, wsum, sizeof h_wsum, hipMemcpyDeviceToHost, s));
    HIP_TRY(hipStreamSynchronize(s));
    if (!std::isfinite(h_wsum)) return fail(FBDT_E_WEIGHT, "weights must be finite");
    const int scale = histogram_scale(h_wsum * (1.0 + 1e-6));
    {
        Timed tm(FBDT_K_HISTOGRAM, s, hist_algorithmic_bytes(n, d, n_bins, layer, false, false));
        HIP_TRY(launch_histogram(hs, xb, ldb, n, d, n_bins, node_pad, nullptr, w_pad, nullptr,
                                 ParentCuts{}, layer, false, scale, partial, small, err, s));
        tm.done();
    }
    HIP_TRY(launch_merge_partials(partial, hs.chunks, count, scale, small, hist, s));
    int h_err = 0;
    if ((rc = read_err(err, s, &h_err))) return rc;
    if (h_err & kErrBin) return fail(FBDT_E_INVAL, "a bin code is >= n_bins");
    return FBDT_OK;
}

int fbdt_best_cuts(const double *hist, int32_t n_nodes, int32_t d, int32_t n_bins,
                   uint8_t *cut_feature, uint8_t *cut_bin, double *gain, void *stream) {
    int rc;
    if (!hist || !cut_feature || !cut_bin || !gain) return fail(FBDT_E_INVAL, "NULL argument");
    if (n_nodes < 1 || n_nodes > 64) return fail(FBDT_E_INVAL, "n_nodes not in [1, 64]");
    if (d < 1 || d > 255) return fail(FBDT_E_INVAL, "d not in [1, 255]");
    if ((rc = check_bins(n_bins))) return rc;
    if ((reinterpret_cast<uintptr_t>(hist) & 15u) != 0)
        return fail(FBDT_E_INVAL, "hist must be 16-byte aligned");
    int dev;
    DeviceInfo di;
    if ((rc = current_device(&dev, &di))) return rc;
    hipStream_t s = static_cast<hipStream_t>(stream);
    Arena &a = g_arena[dev];
    std::lock_guard<std::mutex> lk(a.mu);
    Carver cv;
    double *cg;
    int *cc;
    cv.add(&cg, (size_t)n_nodes * d);
    cv.add(&cc, (size_t)n_nodes * d);
    if ((rc = arena_reserve(a, cv.off))) return rc;
    cv.assign(a.ptr);
    Timed tm(FBDT_K_BEST_CUTS, s);
    HIP_TRY(launch_best_cuts_f64(hist, n_nodes, d, n_bins, cg, cc, s));
    HIP_TRY(launch_select_cuts(cg, cc, n_nodes, d, 1, cut_feature, cut_bin, gain, s));
    tm.done();
    HIP_TRY(hipStreamSynchronize(s));
    return FBDT_OK;
}

int fbdt_hist_timeline(int64_t *launches, int32_t *max_blocks, const int32_t **blocks,
                       const uint64_t **stamps, int64_t *rate_khz) {
    if (!launches || !max_blocks || !blocks || !stamps || !rate_khz)
        return fail(FBDT_E_INVAL, "NULL argument");
    std::lock_guard<std::mutex> lk(g_timeline.mu);
    *launches = g_timeline.launches;
    *max_blocks = g_timeline.max_blocks;
    *blocks = g_timeline.blocks.empty() ? nullptr : g_timeline.blocks.data();
    *stamps = g_timeline.stamps.empty() ? nullptr : g_timeline.stamps.data();
    *rate_khz = g_timeline.rate_khz;
    return FBDT_OK;
}

int fbdt_reference_pass(int32_t kind, const uint8_t *xb, int64_t n, int32_t d, int64_t ldb,
                        int32_t n_bins, int32_t layer, const uint8_t *node, const float *w,
                        void *stream) {
    int rc;
    if (kind < 0 || kind > 2) return fail(FBDT_E_INVAL, "reference kind %d not 0, 1 or 2", kind);
    if ((rc = check_codes(xb, n, d, ldb)) || (rc = check_bins(n_bins))) return rc;
    if (!w) return fail(FBDT_E_INVAL, "w is NULL");
    if (!aligned16(w) || (node && !aligned16(node)))
        return fail(FBDT_E_INVAL, "node and w must be 16-byte aligned");
    if (layer < 0 || layer > 6) return fail(FBDT_E_INVAL, "layer %d not in [0, 6]", layer);
    int dev;
    DeviceInfo di;
    if ((rc = current_device(&dev, &di))) return rc;
    hipStream_t s = static_cast<hipStream_t>(stream);
    const HistShape hs = plan_histogram(n, d, n_bins, layer, true, di.cu_count, di.max_lds,
                                        hist_overrides());
    Arena &a = g_arena[dev];
    std::lock_guard<std::mutex> lk(a.mu);
    Carver cv;
    uint32_t *sink;
    cv.add(&sink, (size_t)hs.blocks);
    if ((rc = arena_reserve(a, cv.off))) return rc;
    cv.assign(a.ptr);
    const double bytes = kind == 0 ? 0.0 : (double)n * d + 4.0 * n + (node ? (double)n : 0.0);
    Timed tm(FBDT_K_REFERENCE, s, bytes);
    HIP_TRY(launch_hist_reference(kind, hs, xb, ldb, n, d, node, w, sink, s));
    tm.done();
    return FBDT_OK;
}

int fbdt_best_cuts_noalloc(const double *hist, int32_t n_nodes, int32_t d, int32_t n_bins,
                           uint8_t *cut_feature, uint8_t *cut_bin, double *gain, void *stream) {
    int rc;
    if (!hist || !cut_feature || !cut_bin || !gain) return fail(FBDT_E_INVAL, "NULL argument");
    if (n_nodes < 1 || n_nodes > 64) return fail(FBDT_E_INVAL, "n_nodes not in [1, 64]");
    if (d < 1 || d > 255) return fail(FBDT_E_INVAL, "d not in [1, 255]");
    if ((rc = check_bins(n_bins))) return rc;
    if ((reinterpret_cast<uintptr_t>(hist) & 15u) != 0)
        return fail(FBDT_E_INVAL, "hist must be 16-byte aligned");
    if ((size_t)n_nodes * (size_t)d > kNoAllocCandidates)
        return fail(FBDT_E_INVAL, "%d nodes x %d features exceed the %zu candidates of the "
                    "no-allocation scratch", n_nodes, d, kNoAllocCandidates);
    int dev;
    DeviceInfo di;
    if ((rc = current_device(&dev, &di))) return rc;
    if (!di.scratch)
        return fail(FBDT_E_DEVICE, "hipGetSymbolAddress(scratch) failed on device %d: %s", dev,
                    hipGetErrorString(di.scratch_status));
    hipStream_t s = static_cast<hipStream_t>(stream);
    // every candidate entry [node][feature] is written before it is read:
    // nothing left in the scratch by an earlier call needs clearing
    double *cg = static_cast<double *>(di.scratch);
    int *cc = reinterpret_cast<int *>(static_cast<char *>(di.scratch) + kNoAllocGainBytes);
    HIP_TRY(launch_best_cuts_f64(hist, n_nodes, d, n_bins, cg, cc, s));
    HIP_TRY(launch_select_cuts(cg, cc, n_nodes, d, 1, cut_feature, cut_bin, gain, s));
    return FBDT_OK;
}

int fbdt_route(const uint8_t *xb, int64_t n, int32_t d, int64_t ldb, uint8_t *node,
               const uint8_t *cut_feature, const uint8_t *cut_bin, int32_t layer, void *stream) {
    int rc;
    if ((rc = check_codes(xb, n, d, ldb))) return rc;
    if (!node || !cut_feature || !cut_bin) return fail(FBDT_E_INVAL, "NULL argument");
    if (layer < 0 || layer > 6) return fail(FBDT_E_INVAL, "layer %d not in [0, 6]", layer);
    int dev;
    DeviceInfo di;
    if ((rc = current_device(&dev, &di))) return rc;
    hipStream_t s = static_cast<hipStream_t>(stream);
    Arena &a = g_arena[dev];
    std::lock_guard<std::mutex> lk(a.mu);
    Carver cv;
    int *err;
    cv.add(&err, 1);
    if ((rc = arena_reserve(a, cv.off))) return rc;
    cv.assign(a.ptr);
    HIP_TRY(launch_fill_u32(err, 0u, 1, s));
    {
        Timed tm(FBDT_K_ROUTE, s, 3.0 * (double)n);
        HIP_TRY(launch_route(xb, ldb, n, d, node, cut_feature, cut_bin, layer, err, s));
        tm.done();
    }
    int h_err = 0;
    if ((rc = read_err(err, s, &h_err))) return rc;
    if (h_err & kErrRoute)
        return fail(FBDT_E_INVAL, "a node id or cut feature is out of range (events skipped)");
    return FBDT_OK;
}

int fbdt_leaf_values(const uint8_t *node, const int8_t *y, const float *v, const double *F,
                     int64_t n, int32_t depth, uint64_t seed, int32_t tree, double alpha,
                     double eta, double *leaf, void *stream) {
    int rc;
    if (!node || !y || !F || !leaf) return fail(FBDT_E_INVAL, "NULL argument");
    if (n < 1) return fail(FBDT_E_INVAL, "n must be >= 1");
    if (depth < 1 || depth > 7) return fail(FBDT_E_INVAL, "depth not in [1, 7]");
    if (!(alpha > 0.0 && alpha <= 1.0)) return fail(FBDT_E_INVAL, "alpha must be in (0, 1]");
    int dev;
    DeviceInfo di;
    if ((rc = current_device(&dev, &di))) return rc;
    hipStream_t s = static_cast<hipStream_t>(stream);
    const int blocks = leaf_blocks(n, depth, false, di.cu_count);
    // the leaf pass reads whole steps of events: padded copies of the leaf
    // ids and weights, and y~ of the sampled events (0 beyond n) from the
    // re-weighting pass
    const int64_t npad = (n + 15) & ~(int64_t)15;
    Arena &a = g_arena[dev];
    std::lock_guard<std::mutex> lk(a.mu);
    Carver cv;
    double *lp, *yts;
    uint8_t *node_pad;
    float *v_pad = nullptr;
    int *err;
    cv.add(&lp, (size_t)blocks * 2 * (1 << depth));
    cv.add(&yts, (size_t)npad);
    cv.add(&node_pad, (size_t)npad);
    if (v) cv.add(&v_pad, (size_t)npad);
    cv.add(&err, 1);
    if ((rc = arena_reserve(a, cv.off))) return rc;
    cv.assign(a.ptr);
    HIP_TRY(launch_fill_u32(err, 0u, 1, s));
    HIP_TRY(launch_fill_u32(yts, 0u, 2 * (size_t)npad, s));
    HIP_TRY(launch_fill_u32(node_pad, 0u, (size_t)npad / 4, s));
    HIP_TRY(hipMemcpyAsync(node_pad, node, (size_t)n, hipMemcpyDeviceToDevice, s));
    if (v) {
        HIP_TRY(launch_fill_u32(v_pad, 0u, (size_t)npad, s));
        HIP_TRY(hipMemcpyAsync(v_pad, v, (size_t)n * sizeof(float), hipMemcpyDeviceToDevice, s));
    }
    HIP_TRY(launch_tree_prep(y, v, const_cast<double *>(F), nullptr, nullptr, nullptr, nullptr, 0,
                             0.0, nullptr, depth, false, n, seed, tree, alpha, nullptr, yts,
                             nullptr, di.cu_count, s));
    HIP_TRY(launch_leaf(nullptr, 0, n, 1, node_pad, nullptr, ParentCuts{}, depth, false, false,
                        v_pad, yts, blocks, lp, err, s));
    HIP_TRY(launch_leaf_finalize(lp, blocks, depth, false, eta, leaf, s));
    int h_err = 0;
    if ((rc = read_err(err, s, &h_err))) return rc;
    if (h_err & kErrRoute) return fail(FBDT_E_INVAL, "a node id is not a leaf id (skipped)");
    return FBDT_OK;
}

}  // extern "C"
