// C ABI of the rank-compensation hot path (declared in include/lrc.h).
//
// Every entry point validates its arguments on the host first, then
// enqueues kernels on the calling thread's stream.  Workspace is grow-only,
// one per (device, stream), so repeated calls allocate nothing after the
// first; lrc_shutdown releases it.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <map>
#include <mutex>
#include <string>
#include <utility>
#include <vector>

#include "../../include/lrc.h"
#include "lrc_internal.h"

using namespace lrc;

// Scratch of lrc_matrix_apply_noalloc: one array per device, held from the
// module's load until the process ends.  Host code never passes the array's
// name to a kernel (on the host it is only a stand-in for the symbol); the
// device address comes from hipGetSymbolAddress, taken once per device with
// that device current (noalloc_scratch), and every later use goes through it.
static __device__ __align__(256) char scratch[LRC_NOALLOC_SCRATCH_BYTES];

namespace {

thread_local std::string g_err;
thread_local hipStream_t g_stream = nullptr;
thread_local int g_force_path = LRC_PATH_AUTO;

int fail(int code, const char* fmt, ...) {
    char buf[512];
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(buf, sizeof(buf), fmt, ap);
    va_end(ap);
    g_err = buf;
    return code;
}

int fail_hip(hipError_t e, const char* what) {
    return fail(e == hipErrorOutOfMemory ? LRC_ENOMEM : LRC_EHIP, "%s: %s", what, hipGetErrorString(e));
}

bool valid_prec(int p) { return p == LRC_FP64 || p == LRC_FP32 || p == LRC_FP16; }

// a * b without overflow (both >= 0)
bool mul_ok(int64_t a, int64_t b, int64_t* out) {
    if (a != 0 && b > INT64_MAX / a) return false;
    *out = a * b;
    return true;
}

bool overlaps(const void* a, size_t na, const void* b, size_t nb) {
    const char* pa = static_cast<const char*>(a);
    const char* pb = static_cast<const char*>(b);
    return pa < pb + nb && pb < pa + na;
}

std::mutex g_mu;
std::map<std::pair<int, hipStream_t>, Workspace> g_ws;
std::map<int, std::pair<bool, size_t>> g_dev;   // device -> (is gfx950, max LDS per block)

int current_device(int* dev, size_t* max_lds) {
    hipError_t e = hipGetDevice(dev);
    if (e != hipSuccess) return fail(LRC_ENODEV, "no HIP device: %s", hipGetErrorString(e));
    std::lock_guard<std::mutex> lk(g_mu);
    auto it = g_dev.find(*dev);
    if (it == g_dev.end()) {
        hipDeviceProp_t prop;
        e = hipGetDeviceProperties(&prop, *dev);
        if (e != hipSuccess) return fail(LRC_ENODEV, "hipGetDeviceProperties: %s", hipGetErrorString(e));
        const bool ok = std::strncmp(prop.gcnArchName, "gfx950", 6) == 0;
        int lds = 0;
        if (hipDeviceGetAttribute(&lds, hipDeviceAttributeMaxSharedMemoryPerBlock, *dev) != hipSuccess || lds <= 0)
            lds = 65536;
        it = g_dev.emplace(*dev, std::make_pair(ok, (size_t)lds)).first;
    }
    if (!it->second.first) return fail(LRC_ENODEV, "device %d is not a gfx950 (MI355X) GPU", *dev);
    if (max_lds) *max_lds = it->second.second;
    return LRC_OK;
}

std::mutex g_scratch_mu;
std::map<int, void*> g_scratch;   // device -> device address of `scratch`

int noalloc_scratch(int dev, void** out) {
    std::lock_guard<std::mutex> lk(g_scratch_mu);
    auto it = g_scratch.find(dev);
    if (it == g_scratch.end()) {
        void* p = nullptr;
        hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess || !p)
            return fail(LRC_EHIP, "address of the scratch array on device %d: %s", dev,
                        e != hipSuccess ? hipGetErrorString(e) : "null");
        it = g_scratch.emplace(dev, p).first;
    }
    *out = it->second;
    return LRC_OK;
}

Workspace& workspace_for(int dev, hipStream_t s) {
    std::lock_guard<std::mutex> lk(g_mu);
    return g_ws[std::make_pair(dev, s)];
}

int64_t tt_count(const int64_t* dims, const int64_t* ranks, int d) {
    int64_t tot = 0;
    for (int l = 0; l < d; ++l) {
        int64_t a, b;
        if (!mul_ok(ranks[l], dims[l], &a) || !mul_ok(a, ranks[l + 1], &b) || tot > INT64_MAX - b) return -1;
        tot += b;
    }
    return tot;
}

int check_tt_shape(const int64_t* dims, const int64_t* ranks, int d, int64_t* total) {
    if (!dims || !ranks) return fail(LRC_EINVAL, "dims and ranks must not be NULL");
    if (d < 1 || d > LRC_TT_MAX_D) return fail(LRC_EINVAL, "d = %d outside [1, %d]", d, LRC_TT_MAX_D);
    if (ranks[0] != 1 || ranks[d] != 1) return fail(LRC_EINVAL, "boundary ranks must be 1 (got %lld, %lld)",
                                                    (long long)ranks[0], (long long)ranks[d]);
    int64_t n = 1;
    for (int l = 0; l < d; ++l) {
        if (dims[l] < 1) return fail(LRC_EINVAL, "dims[%d] = %lld < 1", l, (long long)dims[l]);
        if (!mul_ok(n, dims[l], &n)) return fail(LRC_EOVERFLOW, "number of tensor entries overflows");
    }
    for (int l = 0; l <= d; ++l) {
        if (ranks[l] < 1) return fail(LRC_EINVAL, "ranks[%d] = %lld < 1", l, (long long)ranks[l]);
        if (ranks[l] > LRC_TT_MAX_RANK)
            return fail(LRC_EINVAL, "ranks[%d] = %lld above %d", l, (long long)ranks[l], LRC_TT_MAX_RANK);
    }
    if (tt_count(dims, ranks, d) < 0) return fail(LRC_EOVERFLOW, "core sizes overflow");
    int64_t bytes;
    if (!mul_ok(n, 8, &bytes)) return fail(LRC_EOVERFLOW, "tensor byte count overflows");
    *total = n;
    return LRC_OK;
}

int tt_reconstruct_impl(const void* const* cores, const int64_t* dims, const int64_t* ranks, int d, void* out,
                        int prec) {
    int dev;
    size_t max_lds;
    int rc = current_device(&dev, &max_lds);
    if (rc) return rc;
    hipStream_t st = g_stream;
    const int64_t N = [&] {
        int64_t n = 1;
        for (int l = 0; l < d; ++l) n *= dims[l];
        return n;
    }();
    if (d == 1) {
        hipError_t e = hipMemcpyAsync(out, cores[0], (size_t)N * elem_bytes(prec), hipMemcpyDeviceToDevice, st);
        return e == hipSuccess ? LRC_OK : fail_hip(e, "copy of the single core");
    }
    TTPlan plan;
    const int64_t* rs[1] = {ranks};
    if (plan_tt(plan, dims, rs, 1, d, prec, max_lds) != 0)
        return fail(LRC_EINVAL, "TT ranks (%lld into the last core) exceed the on-chip buffers of the fused kernel",
                    (long long)ranks[d - 1]);
    Workspace& ws = workspace_for(dev, st);
    ws.reset();
    hipError_t e0 = ws.reserve(plan.stage_bytes, st);
    if (e0 != hipSuccess) return fail_hip(e0, "workspace");
    hipError_t e = launch_tt(plan, cores, out, ws, st);
    return e == hipSuccess ? LRC_OK : fail_hip(e, "TT reconstruction launch");
}

}  // namespace

// ------------------------------------------------------- kernel timing ---
namespace {
std::mutex g_pmu;
bool g_prof = false;
std::string g_prof_filter;   // empty: every label
struct PendingTime {
    std::string label;
    hipEvent_t a, b;
};
std::vector<PendingTime> g_pending;
std::vector<hipEvent_t> g_event_pool;
std::map<std::string, std::pair<int64_t, double>> g_times;

hipEvent_t pool_event() {
    if (!g_event_pool.empty()) {
        hipEvent_t e = g_event_pool.back();
        g_event_pool.pop_back();
        return e;
    }
    hipEvent_t e = nullptr;
    if (hipEventCreate(&e) != hipSuccess) return nullptr;
    return e;
}

int drain_times() {
    for (auto& p : g_pending) {
        float ms = 0.0f;
        hipError_t e = hipEventSynchronize(p.b);
        if (e == hipSuccess) e = hipEventElapsedTime(&ms, p.a, p.b);
        if (e != hipSuccess) return fail_hip(e, "kernel timing");
        auto& slot = g_times[p.label];
        slot.first += 1;
        slot.second += ms;
        g_event_pool.push_back(p.a);
        g_event_pool.push_back(p.b);
    }
    g_pending.clear();
    return LRC_OK;
}
}  // namespace

namespace lrc {
KernelTimer::KernelTimer(const char* lbl, hipStream_t s) : label(lbl), stream(s), start(nullptr) {
    std::lock_guard<std::mutex> lk(g_pmu);
    if (!g_prof) return;
    if (!g_prof_filter.empty() && g_prof_filter != lbl) return;
    hipEvent_t e = pool_event();
    if (e && hipEventRecord(e, s) == hipSuccess) start = e;
}

KernelTimer::~KernelTimer() {
    if (!start) return;
    std::lock_guard<std::mutex> lk(g_pmu);
    hipEvent_t e = pool_event();
    if (e && hipEventRecord(e, stream) == hipSuccess)
        g_pending.push_back(PendingTime{label, static_cast<hipEvent_t>(start), e});
}
}  // namespace lrc

// ------------------------------------------------------------- Workspace --
namespace lrc {
hipError_t Workspace::reserve(size_t bytes, hipStream_t stream) {
    bytes = (size_t)round_up((int64_t)bytes, 256) + 256;
    if (bytes > cap) {
        // grow by at least half the current size, so that a sequence of
        // slightly larger calls does not reallocate every time
        const size_t want = std::max(bytes, cap + cap / 2);
        if (base) {
            hipError_t e = hipStreamSynchronize(stream);
            if (e != hipSuccess) return e;
            (void)hipFree(base);
            base = nullptr;
            cap = 0;
        }
        hipError_t e = hipMalloc(reinterpret_cast<void**>(&base), want);
        if (e != hipSuccess) {
            base = nullptr;
            return e;
        }
        cap = want;
    }
    used = 0;
    return hipSuccess;
}

void* Workspace::take(size_t bytes) {
    size_t b = (size_t)round_up((int64_t)bytes, 256);
    if (b == 0) return nullptr;
    if (!base || used + b > cap) {
        overrun = true;
        return nullptr;
    }
    void* p = base + used;
    used += b;
    return p;
}

void Workspace::release() {
    if (base) (void)hipFree(base);
    base = nullptr;
    cap = used = 0;
}
}  // namespace lrc

// ------------------------------------------------------------------ ABI ---
extern "C" {

int lrc_version(void) { return LRC_VERSION; }

int lrc_mfma_ceiling(int prec, double* tflops) {
    if (!tflops) return fail(LRC_EINVAL, "NULL argument");
    if (!valid_prec(prec)) return fail(LRC_EINVAL, "unknown precision code %d", prec);
    int dev;
    int rc = current_device(&dev, nullptr);
    if (rc) return rc;
    int cus = 0;
    hipError_t e = hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev);
    if (e != hipSuccess || cus <= 0) return fail_hip(e != hipSuccess ? e : hipErrorInvalidValue, "compute unit count");
    hipStream_t st = g_stream;
    Workspace& ws = workspace_for(dev, st);
    ws.reset();
    e = ws.reserve(mfma_ceiling_workspace_bytes(cus), st);
    if (e != hipSuccess) return fail_hip(e, "workspace");
    e = launch_mfma_ceiling(prec, cus, tflops, ws, st);
    if (e != hipSuccess) return fail_hip(e, "matrix-core ceiling");
    return LRC_OK;
}

int lrc_set_stream(void* hip_stream) {
    g_stream = static_cast<hipStream_t>(hip_stream);
    return LRC_OK;
}

const char* lrc_last_error(void) { return g_err.c_str(); }

int lrc_set_apply_path(int path) {
    if (path != LRC_PATH_AUTO && path != LRC_PATH_STREAM && path != LRC_PATH_MFMA)
        return fail(LRC_EINVAL, "unknown apply path %d", path);
    g_force_path = path;
    return LRC_OK;
}

static int check_apply(int64_t m, int64_t n, int64_t k, int64_t batch, int prec) {
    if (!valid_prec(prec)) return fail(LRC_EINVAL, "unknown precision code %d", prec);
    if (m < 1 || n < 1 || k < 1 || batch < 1)
        return fail(LRC_EINVAL, "sizes must be >= 1 (m=%lld n=%lld k=%lld batch=%lld)", (long long)m,
                    (long long)n, (long long)k, (long long)batch);
    if (k > std::min(m, n)) return fail(LRC_EINVAL, "k = %lld exceeds min(m, n)", (long long)k);
    int64_t t;
    const int64_t e = elem_bytes(prec);
    if (!mul_ok(m, k, &t) || !mul_ok(t, e, &t) || !mul_ok(n, k, &t) || !mul_ok(t, e, &t) || !mul_ok(n, batch, &t) ||
        !mul_ok(t, e, &t) || !mul_ok(m, batch, &t) || !mul_ok(t, e, &t))
        return fail(LRC_EOVERFLOW, "array sizes overflow int64");
    return LRC_OK;
}

int lrc_matrix_apply_path(int64_t m, int64_t n, int64_t k, int64_t batch, int prec) {
    int rc = check_apply(m, n, k, batch, prec);
    if (rc) return rc;
    return plan_apply(m, n, k, batch, prec, LRC_PATH_AUTO).path;
}

static int check_apply_arrays(const void* U, const void* s, const void* V, const void* X, void* Y, int64_t m,
                              int64_t n, int64_t k, int64_t batch, int prec) {
    if (!U || !s || !V || !X || !Y) return fail(LRC_EINVAL, "NULL array argument");
    int rc = check_apply(m, n, k, batch, prec);
    if (rc) return rc;
    const size_t e = elem_bytes(prec);
    const size_t ny = (size_t)m * batch * e;
    if (overlaps(Y, ny, U, (size_t)m * k * e) || overlaps(Y, ny, s, (size_t)k * e) ||
        overlaps(Y, ny, V, (size_t)n * k * e) || overlaps(Y, ny, X, (size_t)n * batch * e))
        return fail(LRC_EINVAL, "output Y overlaps an input");
    return LRC_OK;
}

int lrc_matrix_apply_noalloc(const void* U, const void* s, const void* V, const void* X, void* Y, int64_t m,
                             int64_t n, int64_t k, int64_t batch, int prec) {
    int rc = check_apply_arrays(U, s, V, X, Y, m, n, k, batch, prec);
    if (rc) return rc;
    const ApplyPlan plan = plan_apply(m, n, k, batch, prec, g_force_path, U, V, X);
    const size_t need = apply_workspace_bytes(plan);
    if (need > (size_t)LRC_NOALLOC_SCRATCH_BYTES)
        return fail(LRC_EINVAL, "this apply needs %zu bytes of scratch, above the %lld of the allocation-free entry",
                    need, (long long)LRC_NOALLOC_SCRATCH_BYTES);
    int dev;
    rc = current_device(&dev, nullptr);
    if (rc) return rc;
    void* base = nullptr;
    rc = noalloc_scratch(dev, &base);
    if (rc) return rc;
    Workspace ws;   // a view of the device's scratch array: take() only, never reserve()
    ws.base = static_cast<char*>(base);
    ws.cap = (size_t)LRC_NOALLOC_SCRATCH_BYTES;
    hipError_t he = launch_apply(plan, U, s, V, X, Y, m, n, k, batch, prec, ws, g_stream);
    if (he != hipSuccess) return fail_hip(he, "apply launch");
    return LRC_OK;
}

int lrc_matrix_apply(const void* U, const void* s, const void* V, const void* X, void* Y, int64_t m, int64_t n,
                     int64_t k, int64_t batch, int prec) {
    int rc = check_apply_arrays(U, s, V, X, Y, m, n, k, batch, prec);
    if (rc) return rc;
    int dev;
    rc = current_device(&dev, nullptr);
    if (rc) return rc;
    hipStream_t st = g_stream;
    ApplyPlan plan = plan_apply(m, n, k, batch, prec, g_force_path, U, V, X);
    Workspace& ws = workspace_for(dev, st);
    ws.reset();
    hipError_t he = ws.reserve(apply_workspace_bytes(plan), st);
    if (he != hipSuccess) return fail_hip(he, "workspace");
    he = launch_apply(plan, U, s, V, X, Y, m, n, k, batch, prec, ws, st);
    if (he != hipSuccess) return fail_hip(he, "apply launch");
    return LRC_OK;
}

int lrc_tt_reconstruct(const void* const* cores, const int64_t* dims, const int64_t* ranks, int d, void* out,
                       int prec) {
    if (!cores || !out) return fail(LRC_EINVAL, "NULL array argument");
    if (!valid_prec(prec)) return fail(LRC_EINVAL, "unknown precision code %d", prec);
    int64_t N;
    int rc = check_tt_shape(dims, ranks, d, &N);
    if (rc) return rc;
    const size_t e = elem_bytes(prec);
    for (int l = 0; l < d; ++l) {
        if (!cores[l]) return fail(LRC_EINVAL, "cores[%d] is NULL", l);
        const size_t cb = (size_t)ranks[l] * dims[l] * ranks[l + 1] * e;
        if (overlaps(out, (size_t)N * e, cores[l], cb)) return fail(LRC_EINVAL, "output overlaps cores[%d]", l);
    }
    return tt_reconstruct_impl(cores, dims, ranks, d, out, prec);
}

int lrc_round(const void* x, void* y, int64_t count, int prec, int64_t* n_overflow) {
    if (count > 0 && (!x || !y)) return fail(LRC_EINVAL, "NULL array argument");
    if (!valid_prec(prec)) return fail(LRC_EINVAL, "unknown precision code %d", prec);
    if (count < 0) return fail(LRC_EINVAL, "count = %lld < 0", (long long)count);
    int64_t nx;
    if (!mul_ok(count, 8, &nx)) return fail(LRC_EOVERFLOW, "byte count overflows");
    const size_t ny = (size_t)count * elem_bytes(prec);
    if (count > 0 && overlaps(y, ny, x, (size_t)nx)) return fail(LRC_EINVAL, "output y overlaps the input x");
    int dev;
    int rc = current_device(&dev, nullptr);
    if (rc) return rc;
    hipStream_t st = g_stream;
    if (count == 0) {
        if (n_overflow) *n_overflow = 0;
        return LRC_OK;
    }
    if (prec == LRC_FP64) {
        hipError_t e = hipMemcpyAsync(y, x, (size_t)nx, hipMemcpyDeviceToDevice, st);
        if (e != hipSuccess) return fail_hip(e, "copy");
        if (n_overflow) *n_overflow = 0;
        return LRC_OK;
    }
    unsigned long long* ovf = nullptr;
    Workspace* ws = nullptr;
    if (n_overflow) {
        ws = &workspace_for(dev, st);
        ws->reset();
        hipError_t e = ws->reserve(256, st);
        if (e != hipSuccess) return fail_hip(e, "workspace");
        ovf = static_cast<unsigned long long*>(ws->take(sizeof(unsigned long long)));
    }
    hipError_t e = launch_round(static_cast<const double*>(x), y, count, prec, ovf, st);
    if (e != hipSuccess) return fail_hip(e, "rounding launch");
    if (n_overflow) {
        unsigned long long host = 0;
        e = hipMemcpyAsync(&host, ovf, sizeof(host), hipMemcpyDeviceToHost, st);
        if (e == hipSuccess) e = hipStreamSynchronize(st);
        if (e != hipSuccess) return fail_hip(e, "overflow count");
        *n_overflow = (int64_t)host;
    }
    return LRC_OK;
}

int lrc_tt_left_orthogonalize(void* const* cores, const int64_t* dims, const int64_t* ranks, int d) {
    if (!cores) return fail(LRC_EINVAL, "NULL array argument");
    int64_t N;
    int rc = check_tt_shape(dims, ranks, d, &N);
    if (rc) return rc;
    std::vector<size_t> bytes(d);
    for (int l = 0; l < d; ++l) {
        if (!cores[l]) return fail(LRC_EINVAL, "cores[%d] is NULL", l);
        bytes[l] = (size_t)ranks[l] * dims[l] * ranks[l + 1] * 8;
        for (int q = 0; q < l; ++q)
            if (overlaps(cores[l], bytes[l], cores[q], bytes[q]))
                return fail(LRC_EINVAL, "cores[%d] overlaps cores[%d]", l, q);
    }
    for (int l = 0; l + 1 < d; ++l) {
        if (ranks[l + 1] > LRC_GAUGE_MAX_RANK)
            return fail(LRC_EINVAL, "ranks[%d] = %lld above the gauge's limit %d", l + 1, (long long)ranks[l + 1],
                        LRC_GAUGE_MAX_RANK);
        if (ranks[l] * dims[l] < ranks[l + 1])
            return fail(LRC_EINVAL, "unfolding of core %d has %lld rows for rank %lld", l,
                        (long long)(ranks[l] * dims[l]), (long long)ranks[l + 1]);
    }
    if (d == 1) return LRC_OK;
    int dev;
    rc = current_device(&dev, nullptr);
    if (rc) return rc;
    hipStream_t st = g_stream;
    Workspace& ws = workspace_for(dev, st);
    ws.reset();
    hipError_t e = ws.reserve(gauge_workspace_bytes(dims, ranks, d), st);
    if (e != hipSuccess) return fail_hip(e, "workspace");
    int* flags = static_cast<int*>(ws.take(sizeof(int) * (size_t)d));
    std::vector<double*> cs(d);
    for (int l = 0; l < d; ++l) cs[l] = static_cast<double*>(cores[l]);
    e = launch_gauge(cs.data(), dims, ranks, d, flags, ws, st);
    if (e != hipSuccess) return fail_hip(e, "gauge launch");
    std::vector<int> hf(d, 0);
    e = hipMemcpyAsync(hf.data(), flags, sizeof(int) * (size_t)d, hipMemcpyDeviceToHost, st);
    if (e == hipSuccess) e = hipStreamSynchronize(st);
    if (e != hipSuccess) return fail_hip(e, "gauge status");
    for (int l = 0; l + 1 < d; ++l)
        if (hf[l])
            return fail(LRC_ENUMERIC,
                        "unfolding of core %d is numerically rank deficient (Cholesky pivot %d of its Gram matrix)",
                        l, hf[l] - 1);
    return LRC_OK;
}

int64_t lrc_storage_bytes(int64_t m, int64_t n, int64_t k, int prec) {
    if (!valid_prec(prec) || m < 1 || n < 1 || k < 0) return fail(LRC_EINVAL, "bad storage arguments");
    int64_t s, t;
    if (m > INT64_MAX - n - 1) return fail(LRC_EOVERFLOW, "m + n + 1 overflows");
    if (!mul_ok(k, m + n + 1, &s) || !mul_ok(s, elem_bytes(prec), &t)) return fail(LRC_EOVERFLOW, "overflow");
    return t;
}

int64_t lrc_tt_storage_bytes(const int64_t* dims, const int64_t* ranks, int d, int prec) {
    if (!valid_prec(prec)) return fail(LRC_EINVAL, "unknown precision code %d", prec);
    int64_t N;
    int rc = check_tt_shape(dims, ranks, d, &N);
    if (rc) return rc;
    int64_t c = tt_count(dims, ranks, d), t;
    if (c < 0 || !mul_ok(c, elem_bytes(prec), &t)) return fail(LRC_EOVERFLOW, "overflow");
    return t;
}

int lrc_profile_enable(int on) {
    std::lock_guard<std::mutex> lk(g_pmu);
    g_prof = on != 0;
    return LRC_OK;
}

int lrc_profile_filter(const char* label) {
    std::lock_guard<std::mutex> lk(g_pmu);
    g_prof_filter = label ? label : "";
    return LRC_OK;
}

void lrc_profile_reset(void) {
    std::lock_guard<std::mutex> lk(g_pmu);
    (void)drain_times();
    g_times.clear();
}

int lrc_profile_read(const char* label, int64_t* launches, double* total_ms) {
    if (!label || !launches || !total_ms) return fail(LRC_EINVAL, "NULL argument");
    std::lock_guard<std::mutex> lk(g_pmu);
    int rc = drain_times();
    if (rc) return rc;
    auto it = g_times.find(label);
    *launches = it == g_times.end() ? 0 : it->second.first;
    *total_ms = it == g_times.end() ? 0.0 : it->second.second;
    return LRC_OK;
}

int64_t lrc_profile_labels(char* buf, int64_t len) {
    std::lock_guard<std::mutex> lk(g_pmu);
    int rc = drain_times();
    if (rc) return rc;
    std::string all;
    for (auto& kv : g_times) {
        if (!all.empty()) all += ",";
        all += kv.first;
    }
    if (buf && len > 0) {
        std::strncpy(buf, all.c_str(), (size_t)len - 1);
        buf[len - 1] = 0;
    }
    return (int64_t)all.size();
}

void lrc_shutdown(void) {
    std::lock_guard<std::mutex> lk(g_mu);
    for (auto& kv : g_ws) kv.second.release();
    g_ws.clear();
}

// --------------------------------------------------------- certificates ---
static void finish_flags(lrc_cert_result* r, bool have_err) {
    r->margin = r->E_base - r->E_aug - r->eta;
    r->certified = (r->E_aug + r->eta <= r->E_base) ? 1 : 0;
    r->acc_nonincrease = (have_err && r->err_new <= r->E_base) ? 1 : 0;
    r->acc_win = (have_err && r->err_new < r->E_base) ? 1 : 0;
    r->mem_win = (r->bytes_aug < r->bytes_base) ? 1 : 0;
    r->practical_win = (r->acc_win && r->mem_win) ? 1 : 0;
    r->outcome = r->certified ? (r->mem_win ? LRC_OUTCOME_CERTIFIED_MEM : LRC_OUTCOME_CERTIFIED) : LRC_OUTCOME_FALLBACK;
}

static int certify_matrix(const lrc_cert_args* a, lrc_cert_result* res) {
    const int64_t m = a->m, n = a->n, k = a->k, r = k + 1;
    if (m < 1 || n < 1 || k < 1) return fail(LRC_EINVAL, "sizes must be >= 1");
    if (r > std::min(m, n)) return fail(LRC_EINVAL, "k + 1 = %lld exceeds min(m, n)", (long long)r);
    // E_k and E_{k+1} are Eckart-Young tails over the whole spectrum: a
    // truncated sigma would make both too small and could certify falsely
    if (!a->sigma || a->n_sigma != std::min(m, n))
        return fail(LRC_EINVAL, "sigma must hold all min(m, n) = %lld singular values (got %lld)",
                    (long long)std::min(m, n), (long long)a->n_sigma);
    if (!a->U || !a->s || !a->V || !a->Uh || !a->sh || !a->Vh) return fail(LRC_EINVAL, "NULL factor argument");
    for (int64_t j = 0; j < a->n_sigma; ++j) {
        if (!(a->sigma[j] >= 0.0)) return fail(LRC_EINVAL, "sigma[%lld] is negative or NaN", (long long)j);
        if (j > 0 && a->sigma[j] > a->sigma[j - 1]) return fail(LRC_EINVAL, "sigma is not non-increasing");
    }
    int64_t t;
    if (!mul_ok(m, n, &t) || !mul_ok(t, 8, &t) || !mul_ok(std::max(m, n), 2 * r, &t) || !mul_ok(t, 8, &t))
        return fail(LRC_EOVERFLOW, "sizes overflow");
    int dev;
    int rc = current_device(&dev, nullptr);
    if (rc) return rc;
    hipStream_t st = g_stream;

    // Eckart-Young tails from one reverse cumulative sum
    std::vector<double> E((size_t)a->n_sigma + 1, 0.0);
    double acc = 0.0;
    for (int64_t j = a->n_sigma - 1; j >= 0; --j) {
        const double sq = a->sigma[j] * a->sigma[j];   // separate statements: no fused multiply-add
        acc += sq;
        E[(size_t)j] = std::sqrt(acc);
    }
    res->E_base = E[(size_t)k];
    res->E_aug = E[(size_t)k + 1];
    res->norm_ref = E[0];
    res->gain = a->sigma[k] * a->sigma[k];  // sigma_{k+1}^2 (1-based)
    res->bytes_base = lrc_storage_bytes(m, n, k, LRC_FP64);
    res->bytes_aug = lrc_storage_bytes(m, n, r, a->prec);

    // workspace
    const int64_t w2 = 2 * r;
    const size_t gp1 = gram_workspace_bytes(m, w2);
    const size_t gp2 = gram_workspace_bytes(n, w2);
    size_t need = (size_t)(m + n) * w2 * 8 + 2 * (size_t)w2 * w2 * 8 + gp1 + gp2 + (size_t)w2 * 8 + 16 * 256;
    const bool have_A = a->A != nullptr;
    const int64_t rp = round_up(r, 2);   // pitch of the widened factors: 16-byte rows
    if (have_A) need += (size_t)(m + n) * rp * 8 + err_workspace_bytes(m, n) + 4 * 256;
    Workspace& ws = workspace_for(dev, st);
    ws.reset();
    hipError_t he = ws.reserve(need, st);
    if (he != hipSuccess) return fail_hip(he, "workspace");
    double* P = static_cast<double*>(ws.take((size_t)m * w2 * 8));
    double* Q = static_cast<double*>(ws.take((size_t)n * w2 * 8));
    double* Gu = static_cast<double*>(ws.take((size_t)w2 * w2 * 8));
    double* Gq = static_cast<double*>(ws.take((size_t)w2 * w2 * 8));
    if (ws.overrun) return fail(LRC_ENOMEM, "certificate workspace too small");
    he = launch_diff_factors(a->U, a->Uh, a->prec, m, r, P, st);
    if (he == hipSuccess) he = launch_diff_factors(a->V, a->Vh, a->prec, n, r, Q, st);
    if (he == hipSuccess) he = launch_gram(P, m, w2, Gu, ws, st);
    if (he == hipSuccess) he = launch_gram(Q, n, w2, Gq, ws, st);
    if (he != hipSuccess) return fail_hip(he, "certificate launch");
    double* errsum = nullptr;
    if (have_A) {
        double* W = static_cast<double*>(ws.take((size_t)m * rp * 8));
        double* Vw = static_cast<double*>(ws.take((size_t)n * rp * 8));
        double* part = static_cast<double*>(ws.take(err_workspace_bytes(m, n)));
        errsum = static_cast<double*>(ws.take(8));
        if (ws.overrun) return fail(LRC_ENOMEM, "certificate workspace too small");
        int64_t nparts = 0;
        he = launch_widen_scaled(a->Uh, a->sh, a->prec, m, r, rp, W, st);
        if (he == hipSuccess) he = launch_widen_scaled(a->Vh, nullptr, a->prec, n, r, rp, Vw, st);
        if (he == hipSuccess) he = launch_err_dense(a->A, W, Vw, m, n, r, rp, part, &nparts, st);
        if (he == hipSuccess) he = launch_reduce_rows(part, nparts, 1, errsum, st);
        if (he != hipSuccess) return fail_hip(he, "error-norm launch");
    }
    // eta^2 on the device; the host reads back two numbers
    double* eta_part = static_cast<double*>(ws.take((size_t)w2 * 8));
    double* sums = static_cast<double*>(ws.take(16));
    if (ws.overrun) return fail(LRC_ENOMEM, "certificate workspace too small");
    he = launch_eta2(Gu, Gq, a->s, a->sh, a->prec, r, eta_part, st);
    if (he == hipSuccess) he = launch_reduce_rows(eta_part, w2, 1, sums, st);
    if (he == hipSuccess && have_A) he = hipMemcpyAsync(sums + 1, errsum, 8, hipMemcpyDeviceToDevice, st);
    double hs[2] = {NAN, NAN};
    if (he == hipSuccess) he = hipMemcpyAsync(hs, sums, have_A ? 16 : 8, hipMemcpyDeviceToHost, st);
    if (he == hipSuccess) he = hipStreamSynchronize(st);
    if (he != hipSuccess) return fail_hip(he, "certificate readback");
    const double eta2 = hs[0], err2 = hs[1];
    res->eta = std::sqrt(std::max(eta2, 0.0));
    res->err_new = have_A ? std::sqrt(err2) : NAN;
    finish_flags(res, have_A);
    return LRC_OK;
}

// FP64 reconstruction into a caller-provided buffer on the calling thread's
// stream; its side interfaces (trains of four or more cores) take workspace
// that the caller reserved with tt_stage_need.  Used by the TT certificate
// and the dense quality path.
static int tt_into(const void* const* cores, const int64_t* dims, const int64_t* ranks, int d, double* out,
                   Workspace& ws, const char* label = "cert_tt_fused_f64") {
    hipStream_t st = g_stream;
    if (d == 1) {
        hipError_t e = hipMemcpyAsync(out, cores[0], (size_t)dims[0] * 8, hipMemcpyDeviceToDevice, st);
        return e == hipSuccess ? LRC_OK : fail_hip(e, "copy of the single core");
    }
    int dev;
    size_t max_lds;
    int rc = current_device(&dev, &max_lds);
    if (rc) return rc;
    TTPlan plan;
    const int64_t* rs[1] = {ranks};
    if (plan_tt(plan, dims, rs, 1, d, LRC_FP64, max_lds) != 0)
        return fail(LRC_EINVAL, "TT ranks exceed the on-chip buffers of the fused kernel");
    // the staged cores live only until this launch has run: the next
    // reconstruction on the stream reuses their workspace
    const size_t mark = ws.used;
    hipError_t e = launch_tt(plan, cores, out, ws, st, label);
    ws.used = mark;
    return e == hipSuccess ? LRC_OK : fail_hip(e, "TT reconstruction launch");
}

// workspace of the staged cores of one FP64 reconstruction (0 if it cannot be planned)
static size_t tt_stage_need(const int64_t* dims, const int64_t* ranks, int d) {
    if (d == 1) return 0;
    int dev;
    size_t max_lds;
    if (current_device(&dev, &max_lds)) return 0;
    TTPlan plan;
    const int64_t* rs[1] = {ranks};
    if (plan_tt(plan, dims, rs, 1, d, LRC_FP64, max_lds) != 0) return 0;
    return plan.stage_bytes;
}

// Result fields from the five sums ||T-T_R||^2, ||T-T_R+||^2, ||T_R+-T^||^2,
// ||T-T^||^2, ||T||^2.
static void tt_cert_result(const double* h, const lrc_cert_args* a, lrc_cert_result* res) {
    const int d = a->d;
    res->E_base = std::sqrt(h[0]);
    res->E_aug = std::sqrt(h[1]);
    res->eta = std::sqrt(h[2]);
    res->err_new = std::sqrt(h[3]);
    res->norm_ref = std::sqrt(h[4]);
    res->gain = h[0] - h[1];
    res->bytes_base = lrc_tt_storage_bytes(a->dims, a->ranks_base, d, LRC_FP64);
    res->bytes_aug = lrc_tt_storage_bytes(a->dims, a->ranks_aug, d, a->prec);
    finish_flags(res, true);
}

static int certify_tt(const lrc_cert_args* a, lrc_cert_result* res) {
    const int d = a->d;
    int64_t N, Nb;
    int rc = check_tt_shape(a->dims, a->ranks_base, d, &N);
    if (rc) return rc;
    rc = check_tt_shape(a->dims, a->ranks_aug, d, &Nb);
    if (rc) return rc;
    if (!a->T || !a->cores_base || !a->cores_aug || !a->cores_aug_h) return fail(LRC_EINVAL, "NULL TT argument");
    for (int l = 0; l < d; ++l)
        if (!a->cores_base[l] || !a->cores_aug[l] || !a->cores_aug_h[l])
            return fail(LRC_EINVAL, "core %d is NULL", l);
    int dev;
    size_t max_lds;
    rc = current_device(&dev, &max_lds);
    if (rc) return rc;
    hipStream_t st = g_stream;
    const int64_t cnt_aug = tt_count(a->dims, a->ranks_aug, d);

    // Fused path: the three FP64 reconstructions are formed tile by tile on
    // chip and compared with T there (no dense intermediate tensors).
    TTPlan cplan;
    const int64_t* rsets[3] = {a->ranks_base, a->ranks_aug, a->ranks_aug};
    if (d >= 2 && plan_tt(cplan, a->dims, rsets, 3, d, LRC_FP64, max_lds) == 0 && cplan.P <= 32) {
        const int64_t nparts = tt_cert_parts(cplan);
        const size_t need = (size_t)cnt_aug * 8 + cplan.stage_bytes + 5 * (size_t)nparts * 8 + 64 + (size_t)(8 + d) * 256;
        Workspace& ws = workspace_for(dev, st);
        ws.reset();
        hipError_t he = ws.reserve(need, st);
        if (he != hipSuccess) return fail_hip(he, "workspace");
        std::vector<const void*> wide(d);
        for (int l = 0; l < d; ++l) {
            const int64_t c = a->ranks_aug[l] * a->dims[l] * a->ranks_aug[l + 1];
            double* w = static_cast<double*>(ws.take((size_t)c * 8));
            if (ws.overrun || !w) return fail(LRC_ENOMEM, "certificate workspace too small");
            he = launch_widen(a->cores_aug_h[l], a->prec, c, w, st);
            if (he != hipSuccess) return fail_hip(he, "widen launch");
            wide[l] = w;
        }
        double* part = static_cast<double*>(ws.take(5 * (size_t)nparts * 8));
        double* sums = static_cast<double*>(ws.take(5 * 8));
        if (ws.overrun) return fail(LRC_ENOMEM, "certificate workspace too small");
        std::vector<const void*> cb(a->cores_base, a->cores_base + d), ca(a->cores_aug, a->cores_aug + d);
        const void* const* sets[3] = {cb.data(), ca.data(), wide.data()};
        he = launch_tt_cert(cplan, sets, static_cast<const double*>(a->T), part, ws, st);
        if (he == hipSuccess) he = launch_reduce_rows(part, nparts, 5, sums, st);
        double h[5];
        if (he == hipSuccess) he = hipMemcpyAsync(h, sums, sizeof(h), hipMemcpyDeviceToHost, st);
        if (he == hipSuccess) he = hipStreamSynchronize(st);
        if (he != hipSuccess) return fail_hip(he, "TT certificate");
        tt_cert_result(h, a, res);
        return LRC_OK;
    }

    // Otherwise: dense FP64 reconstructions, then one pass over the tensors.
    const int64_t groups = sumsq5_groups(N);
    size_t need = 3 * (size_t)N * 8 + (size_t)cnt_aug * 8 + 5 * (size_t)groups * 8 + 64 + (size_t)(8 + d) * 256;
    need += std::max(tt_stage_need(a->dims, a->ranks_base, d), tt_stage_need(a->dims, a->ranks_aug, d)) + 512;
    Workspace& ws = workspace_for(dev, st);
    ws.reset();
    hipError_t he = ws.reserve(need, st);
    if (he != hipSuccess) return fail_hip(he, "workspace");
    double* TR = static_cast<double*>(ws.take((size_t)N * 8));
    double* TRp = static_cast<double*>(ws.take((size_t)N * 8));
    double* Th = static_cast<double*>(ws.take((size_t)N * 8));
    std::vector<const void*> wide(d);
    for (int l = 0; l < d; ++l) {
        const int64_t c = a->ranks_aug[l] * a->dims[l] * a->ranks_aug[l + 1];
        double* w = static_cast<double*>(ws.take((size_t)c * 8));
        if (ws.overrun || !w) return fail(LRC_ENOMEM, "certificate workspace too small");
        he = launch_widen(a->cores_aug_h[l], a->prec, c, w, st);
        if (he != hipSuccess) return fail_hip(he, "widen launch");
        wide[l] = w;
    }
    double* part = static_cast<double*>(ws.take(5 * (size_t)groups * 8));
    double* sums = static_cast<double*>(ws.take(5 * 8));
    if (ws.overrun) return fail(LRC_ENOMEM, "certificate workspace too small");
    // FP64 reconstructions, one after the other on the stream
    std::vector<const void*> cb(a->cores_base, a->cores_base + d), ca(a->cores_aug, a->cores_aug + d);
    rc = tt_into(cb.data(), a->dims, a->ranks_base, d, TR, ws);
    if (rc) return rc;
    rc = tt_into(ca.data(), a->dims, a->ranks_aug, d, TRp, ws);
    if (rc) return rc;
    rc = tt_into(wide.data(), a->dims, a->ranks_aug, d, Th, ws);
    if (rc) return rc;
    he = launch_sumsq5(a->T, TR, TRp, Th, N, part, groups, st);
    if (he == hipSuccess) he = launch_reduce_rows(part, groups, 5, sums, st);
    double h[5];
    if (he == hipSuccess) he = hipMemcpyAsync(h, sums, sizeof(h), hipMemcpyDeviceToHost, st);
    if (he == hipSuccess) he = hipStreamSynchronize(st);
    if (he != hipSuccess) return fail_hip(he, "TT certificate");
    tt_cert_result(h, a, res);
    return LRC_OK;
}

int lrc_certify(const lrc_cert_args* args, lrc_cert_result* res) {
    if (!args || !res) return fail(LRC_EINVAL, "NULL args or result");
    if (!valid_prec(args->prec)) return fail(LRC_EINVAL, "unknown precision code %d", args->prec);
    std::memset(res, 0, sizeof(*res));
    if (args->kind == LRC_CERT_MATRIX) return certify_matrix(args, res);
    if (args->kind == LRC_CERT_TT) return certify_tt(args, res);
    return fail(LRC_EINVAL, "unknown certificate kind %d", args->kind);
}

}  // extern "C"

// ------------------------------------------------------ fixed-memory tools --
static void quality_result(const double* h, int64_t P, int64_t B, lrc_quality* q) {
    q->rel_err = h[0];
    q->psnr = h[1];
    q->ssim = h[2];
    q->sam = h[3];
    q->sam_pixels = (int64_t)h[4];
    q->pixels = P;
    q->bands = B;
}

int lrc_band_quality(const void* X, const void* Xh, int64_t pixels, int64_t bands, int prec, double scale,
                     lrc_quality* q) {
    if (!X || !Xh || !q) return fail(LRC_EINVAL, "NULL argument");
    if (!valid_prec(prec)) return fail(LRC_EINVAL, "unknown precision code %d", prec);
    if (pixels < 1 || bands < 1) return fail(LRC_EINVAL, "pixels and bands must be >= 1");
    int64_t N, nb;
    if (!mul_ok(pixels, bands, &N) || !mul_ok(N, 8, &nb)) return fail(LRC_EOVERFLOW, "entry count overflows");
    int dev;
    int rc = current_device(&dev, nullptr);
    if (rc) return rc;
    hipStream_t st = g_stream;
    Workspace& ws = workspace_for(dev, st);
    ws.reset();
    hipError_t e = ws.reserve(quality_workspace_bytes(pixels, bands) + 256, st);
    if (e != hipSuccess) return fail_hip(e, "workspace");
    double* out = static_cast<double*>(ws.take(5 * 8));
    e = launch_quality(static_cast<const double*>(X), Xh, prec, scale, pixels, bands, out, ws, st);
    double h[5];
    if (e == hipSuccess) e = hipMemcpyAsync(h, out, sizeof(h), hipMemcpyDeviceToHost, st);
    if (e == hipSuccess) e = hipStreamSynchronize(st);
    if (e != hipSuccess) return fail_hip(e, "quality");
    quality_result(h, pixels, bands, q);
    return LRC_OK;
}

int lrc_tt_quality(const void* const* cores, const int64_t* dims, const int64_t* ranks, int d, int prec,
                   const void* X, double scale, lrc_quality* q) {
    if (!cores || !X || !q) return fail(LRC_EINVAL, "NULL argument");
    if (!valid_prec(prec)) return fail(LRC_EINVAL, "unknown precision code %d", prec);
    int64_t N;
    int rc = check_tt_shape(dims, ranks, d, &N);
    if (rc) return rc;
    if (d < 2) return fail(LRC_EINVAL, "need d >= 2 (pixels and a band mode)");
    for (int l = 0; l < d; ++l)
        if (!cores[l]) return fail(LRC_EINVAL, "cores[%d] is NULL", l);
    const int64_t B = dims[d - 1], P = N / B;
    int dev;
    size_t max_lds;
    rc = current_device(&dev, &max_lds);
    if (rc) return rc;
    hipStream_t st = g_stream;
    const int64_t cnt = tt_count(dims, ranks, d);
    // Fused when the FP64 plan takes wave tiles: the measures are formed in
    // the reconstruction's epilogue, which reads only the cores and X.
    // Otherwise the FP64 reconstruction is written to the workspace and
    // measured densely.
    TTPlan plan;
    int64_t G = 0;
    if (d >= 3) {
        const int64_t* rs[1] = {ranks};
        if (plan_tt(plan, dims, rs, 1, d, LRC_FP64, max_lds, false) == 0) G = tt_quality_blocks(plan, max_lds);
    }
    size_t need = (size_t)cnt * 8 + (size_t)(d + 4) * 256 + 256;
    if (G > 0)
        need += plan.stage_bytes + 512 + round_up((size_t)G * QS_N * B * 8, 256) + round_up((size_t)G * 16, 256) +
                round_up((size_t)QS_N * B * 8, 256);
    else
        need += (size_t)N * 8 + quality_workspace_bytes(P, B) + tt_stage_need(dims, ranks, d) + 512;
    Workspace& ws = workspace_for(dev, st);
    ws.reset();
    hipError_t e = ws.reserve(need, st);
    if (e != hipSuccess) return fail_hip(e, "workspace");
    double* Xh = G > 0 ? nullptr : static_cast<double*>(ws.take((size_t)N * 8));
    // the stored cores, widened exactly to FP64 (Sec. 3.4: FP64 contraction of the rounded cores)
    std::vector<const void*> wide(d);
    for (int l = 0; l < d; ++l) {
        const int64_t c = ranks[l] * dims[l] * ranks[l + 1];
        if (prec == LRC_FP64) {
            wide[l] = cores[l];
            continue;
        }
        double* w = static_cast<double*>(ws.take((size_t)c * 8));
        if (ws.overrun || !w) return fail(LRC_ENOMEM, "quality workspace too small");
        e = launch_widen(cores[l], prec, c, w, st);
        if (e != hipSuccess) return fail_hip(e, "widen launch");
        wide[l] = w;
    }
    double* out = static_cast<double*>(ws.take(5 * 8));
    if (ws.overrun) return fail(LRC_ENOMEM, "quality workspace too small");
    if (G > 0) {
        double* part = static_cast<double*>(ws.take((size_t)G * QS_N * B * 8));
        double* part2 = static_cast<double*>(ws.take((size_t)G * 16));
        double* red = static_cast<double*>(ws.take((size_t)QS_N * B * 8));
        if (ws.overrun) return fail(LRC_ENOMEM, "quality workspace too small");
        e = launch_tt_quality(plan, wide.data(), static_cast<const double*>(X), scale, part, part2, max_lds, ws, st);
        if (e == hipSuccess)
            e = launch_quality_reduce(part, G, part2, G, static_cast<const double*>(X), P, B, red, out, st);
    } else {
        rc = tt_into(wide.data(), dims, ranks, d, Xh, ws, "quality_tt_f64");
        if (rc) return rc;
        e = launch_quality(static_cast<const double*>(X), Xh, LRC_FP64, scale, P, B, out, ws, st);
    }
    double h[5];
    if (e == hipSuccess) e = hipMemcpyAsync(h, out, sizeof(h), hipMemcpyDeviceToHost, st);
    if (e == hipSuccess) e = hipStreamSynchronize(st);
    if (e != hipSuccess) return fail_hip(e, "quality");
    quality_result(h, P, B, q);
    return LRC_OK;
}

int64_t lrc_tt_memory_matched_rank(const int64_t* dims, int d, int64_t budget_bytes, int64_t* ranks_out) {
    if (!dims || !ranks_out) return fail(LRC_EINVAL, "NULL argument");
    if (d < 1 || d > LRC_TT_MAX_D) return fail(LRC_EINVAL, "d = %d outside [1, %d]", d, LRC_TT_MAX_D);
    for (int l = 0; l < d; ++l)
        if (dims[l] < 1) return fail(LRC_EINVAL, "dims[%d] = %lld < 1", l, (long long)dims[l]);
    // ranks capped by the unfolding dimensions: r_l <= min(R, r_{l-1} n_l, prod_{i>l} n_i)
    auto sat_mul = [](int64_t a, int64_t b) { return a > INT64_MAX / b ? INT64_MAX : a * b; };
    auto capped = [&](int64_t R, std::vector<int64_t>& r) {
        r.assign(d + 1, 1);
        for (int l = 0; l + 1 < d; ++l) {
            int64_t right = 1;
            for (int i = l + 1; i < d; ++i) right = sat_mul(right, dims[i]);
            r[l + 1] = std::min(R, std::min(sat_mul(r[l], dims[l]), right));
        }
    };
    auto bytes = [&](const std::vector<int64_t>& r) {
        int64_t tot = 0;
        for (int l = 0; l < d; ++l) {
            int64_t a, b;
            if (!mul_ok(r[l], dims[l], &a) || !mul_ok(a, r[l + 1], &b) || tot > INT64_MAX / 8 - b) return INT64_MAX;
            tot += b;
        }
        return tot * 8;
    };
    std::vector<int64_t> r, next, best;
    int64_t R = 1, bestR = 0;
    for (;;) {
        capped(R, r);
        if (bytes(r) > budget_bytes) break;
        bestR = R;
        best = r;
        capped(R + 1, next);
        if (next == r) break;   // every rank capped: storage stops growing
        ++R;
    }
    for (int l = 0; l <= d; ++l) ranks_out[l] = bestR ? best[l] : 0;
    return bestR;
}

// ------------------------------------------------- randomized factorization
static int check_rsvd_sizes(int64_t rows, int64_t cols, int64_t l, int64_t k, const char* what) {
    if (l < 1 || l > LRC_RSVD_MAX_SAMPLES)
        return fail(LRC_EINVAL, "%s: %lld test vectors outside [1, %d]", what, (long long)l, LRC_RSVD_MAX_SAMPLES);
    if (k < 1 || k > l) return fail(LRC_EINVAL, "%s: rank %lld outside [1, l = %lld]", what, (long long)k, (long long)l);
    if (l > rows || l > cols)
        return fail(LRC_EINVAL, "%s: %lld test vectors exceed the matrix size %lld x %lld", what, (long long)l,
                    (long long)rows, (long long)cols);
    int64_t t;
    if (!mul_ok(rows, cols, &t) || !mul_ok(t, 16, &t)) return fail(LRC_EOVERFLOW, "%s: size overflows", what);
    return LRC_OK;
}

// Reads the device flags; *qr_broke tells whether only QR breakdowns (which
// shifted CholeskyQR3 may cure) were seen.
static int factor_status(const int* dflags, int nsteps, hipStream_t st, bool tt, bool* qr_broke = nullptr) {
    std::vector<int> hf(3 * (size_t)nsteps, 0);
    hipError_t e = hipMemcpyAsync(hf.data(), dflags, sizeof(int) * hf.size(), hipMemcpyDeviceToHost, st);
    if (e == hipSuccess) e = hipStreamSynchronize(st);
    if (e != hipSuccess) return fail_hip(e, "factorization status");
    if (qr_broke) {
        bool qr = false, jac = false;
        for (int s = 0; s < nsteps; ++s) {
            qr = qr || hf[3 * s] || hf[3 * s + 1];
            jac = jac || hf[3 * s + 2];
        }
        *qr_broke = qr && !jac;
    }
    static const char* what[3] = {"the range finder's sketch", "the projected matrix B^T", "the small Jacobi SVD"};
    for (int s = 0; s < nsteps; ++s)
        for (int q = 0; q < 3; ++q)
            if (hf[3 * s + q]) {
                if (tt)
                    return fail(LRC_ENUMERIC, "TT-SVD step %d: %s is numerically rank deficient or did not converge",
                                s, what[q]);
                return fail(LRC_ENUMERIC, "%s is numerically rank deficient or did not converge", what[q]);
            }
    return LRC_OK;
}

int lrc_rsvd(const double* A, int64_t m, int64_t n, const double* omega, int64_t l, int power_iters, int64_t k,
             double* U, double* s, double* V) {
    if (!A || !omega || !U || !s || !V) return fail(LRC_EINVAL, "NULL array argument");
    if (m < 1 || n < 1) return fail(LRC_EINVAL, "matrix size %lld x %lld", (long long)m, (long long)n);
    if (power_iters < 0 || power_iters > LRC_RSVD_MAX_POWER_ITERS)
        return fail(LRC_EINVAL, "power_iters = %d outside [0, %d]", power_iters, LRC_RSVD_MAX_POWER_ITERS);
    int rc = check_rsvd_sizes(m, n, l, k, "rsvd");
    if (rc) return rc;
    const size_t bA = (size_t)m * n * 8, bO = (size_t)l * n * 8;
    const size_t bU = (size_t)m * k * 8, bS = (size_t)k * 8, bV = (size_t)n * k * 8;
    const void* outs[3] = {U, s, V};
    const size_t nb[3] = {bU, bS, bV};
    for (int i = 0; i < 3; ++i) {
        if (overlaps(outs[i], nb[i], A, bA) || overlaps(outs[i], nb[i], omega, bO))
            return fail(LRC_EINVAL, "an output overlaps an input");
        for (int j = 0; j < i; ++j)
            if (overlaps(outs[i], nb[i], outs[j], nb[j])) return fail(LRC_EINVAL, "two outputs overlap");
    }
    int dev;
    rc = current_device(&dev, nullptr);
    if (rc) return rc;
    hipStream_t st = g_stream;
    Workspace& ws = workspace_for(dev, st);
    ws.reset();
    hipError_t e = ws.reserve(matrix_rsvd_workspace_bytes(m, n, (int)l, (int)k, power_iters), st);
    if (e != hipSuccess) return fail_hip(e, "workspace");
    int* flags = static_cast<int*>(ws.take(3 * sizeof(int)));
    const size_t mark = ws.used;
    e = launch_matrix_rsvd(A, m, n, omega, (int)l, power_iters, (int)k, U, s, V, flags, ws, st);
    if (e != hipSuccess) return fail_hip(e, "rsvd launch");
    bool qr_broke = false;
    rc = factor_status(flags, 1, st, false, &qr_broke);
    if (rc == LRC_ENUMERIC && qr_broke) {   // ill-conditioned sketch: once more with shifted CholeskyQR3
        ws.used = mark;
        e = launch_matrix_rsvd(A, m, n, omega, (int)l, power_iters, (int)k, U, s, V, flags, ws, st, true);
        if (e != hipSuccess) return fail_hip(e, "rsvd launch");
        rc = factor_status(flags, 1, st, false);
    }
    return rc;
}

int lrc_tt_rsvd(const double* T, const int64_t* dims, const int64_t* ranks, int d, const double* const* omegas,
                const int64_t* samples, int power_iters, double* const* cores, double* sigma) {
    if (!T || !omegas || !samples || !cores) return fail(LRC_EINVAL, "NULL array argument");
    int64_t N;
    int rc = check_tt_shape(dims, ranks, d, &N);
    if (rc) return rc;
    if (d < 2) return fail(LRC_EINVAL, "TT-SVD needs d >= 2 (got %d)", d);
    if (power_iters < 0 || power_iters > LRC_RSVD_MAX_POWER_ITERS)
        return fail(LRC_EINVAL, "power_iters = %d outside [0, %d]", power_iters, LRC_RSVD_MAX_POWER_ITERS);
    int64_t cols = N / dims[0], nsig = 0;
    std::vector<std::pair<const void*, size_t>> ins{{T, (size_t)N * 8}}, outs;
    for (int l = 0; l + 1 < d; ++l) {
        const int64_t rows = ranks[l] * dims[l];
        char what[48];
        snprintf(what, sizeof(what), "TT-SVD step %d", l);
        rc = check_rsvd_sizes(rows, cols, samples[l], ranks[l + 1], what);
        if (rc) return rc;
        if (!omegas[l]) return fail(LRC_EINVAL, "omegas[%d] is NULL", l);
        ins.emplace_back(omegas[l], (size_t)samples[l] * cols * 8);
        nsig += ranks[l + 1];
        cols /= dims[l + 1];
    }
    for (int l = 0; l < d; ++l) {
        if (!cores[l]) return fail(LRC_EINVAL, "cores[%d] is NULL", l);
        outs.emplace_back(cores[l], (size_t)ranks[l] * dims[l] * ranks[l + 1] * 8);
    }
    if (sigma) outs.emplace_back(sigma, (size_t)nsig * 8);
    for (size_t i = 0; i < outs.size(); ++i) {
        for (auto& in : ins)
            if (overlaps(outs[i].first, outs[i].second, in.first, in.second))
                return fail(LRC_EINVAL, "an output overlaps an input");
        for (size_t j = 0; j < i; ++j)
            if (overlaps(outs[i].first, outs[i].second, outs[j].first, outs[j].second))
                return fail(LRC_EINVAL, "two outputs overlap");
    }
    int dev;
    rc = current_device(&dev, nullptr);
    if (rc) return rc;
    hipStream_t st = g_stream;
    Workspace& ws = workspace_for(dev, st);
    ws.reset();
    hipError_t e = ws.reserve(tt_rsvd_workspace_bytes(dims, ranks, samples, d, power_iters), st);
    if (e != hipSuccess) return fail_hip(e, "workspace");
    int* flags = static_cast<int*>(ws.take(3 * sizeof(int) * (size_t)d));
    const size_t mark = ws.used;
    e = launch_tt_rsvd(T, dims, ranks, samples, d, omegas, power_iters, cores, sigma, flags, ws, st);
    if (e != hipSuccess) return fail_hip(e, "TT-SVD launch");
    bool qr_broke = false;
    rc = factor_status(flags, d - 1, st, true, &qr_broke);
    if (rc == LRC_ENUMERIC && qr_broke) {   // ill-conditioned sketch: once more with shifted CholeskyQR3
        ws.used = mark;
        e = launch_tt_rsvd(T, dims, ranks, samples, d, omegas, power_iters, cores, sigma, flags, ws, st, true);
        if (e != hipSuccess) return fail_hip(e, "TT-SVD launch");
        rc = factor_status(flags, d - 1, st, true);
    }
    return rc;
}
