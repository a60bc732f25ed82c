// C ABI of the routed-attention library: argument validation, workspace management and
// launch sequencing.  Validation runs entirely on the host and returns before any HIP call.
#include "../../include/sol_attn.h"

#include <algorithm>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <map>
#include <mutex>
#include <string>
#include <vector>

#include "sol_attn_internal.h"

namespace {

thread_local std::string g_err;

int fail(int code, const char* fmt, ...) {
    char buf[512];
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(buf, sizeof buf, fmt, ap);
    va_end(ap);
    g_err = buf;
    return code;
}

int ok() {
    g_err.clear();
    return SOL_OK;
}

int hip_fail(hipError_t e, const char* what) {
    return fail(SOL_ERR_HIP, "%s: %s", what, hipGetErrorString(e));
}

// Library-owned device buffers, one set per device, grown on demand.
struct DeviceBuffers {
    void* ws = nullptr;
    size_t ws_bytes = 0;
    uint32_t* counts = nullptr;
    size_t counts_n = 0;
};

std::mutex g_mu;
std::map<int, DeviceBuffers> g_bufs;

// What sol_attn_stats needs to turn a counts buffer into fractions: one record per counts
// buffer a forward wrote (keyed by its device address), with an event recorded on the
// forward's stream right after the counts were written.  Waiting on the event instead of the
// stream keeps the record valid after the caller destroys the stream.  Records are recycled
// first-in first-out beyond kMaxRecords buffers; their events are reused, never destroyed
// before sol_attn_release.
struct CountsRecord {
    int device = 0;
    int B = 0, H = 0;
    double routable_pairs = 0.0;   // (query block, routable key block) pairs of one head
    hipEvent_t done = nullptr;     // recorded on the forward's stream after its counts
    bool library = false;          // the library's own counts buffer (counts == NULL)
};
constexpr size_t kMaxRecords = 1024;
std::map<const uint32_t*, CountsRecord> g_records;
std::vector<const uint32_t*> g_record_order;        // insertion order, for recycling
std::map<int, std::vector<hipEvent_t>> g_free_events;  // per device: events of recycled records
std::map<int, std::vector<hipEvent_t>> g_all_events;   // per device: every event created

// The counts buffer of the last forward on this thread, for sol_attn_stats(..., NULL).
thread_local const uint32_t* t_last_counts = nullptr;

// Kernel timing: event pairs recorded around the fused attention kernel.
constexpr int kMaxTimed = 4096;
struct Timing {
    bool enabled = false;
    int device = -1;
    std::vector<hipEvent_t> start, stop;
    int used = 0;
};
Timing g_timing;

bool finite_or_inf(float x) { return !std::isnan(x); }

int check_common(int B, int H, int N, int d, int block_q, int block_k, int dtype) {
    if (B <= 0 || H <= 0 || N <= 0) return fail(SOL_ERR_INVALID_ARG, "B, H and N must be positive (got %d, %d, %d)", B, H, N);
    if (d <= 0 || block_q <= 0 || block_k <= 0)
        return fail(SOL_ERR_INVALID_ARG, "d, block_q and block_k must be positive (got %d, %d, %d)", d, block_q, block_k);
    if (dtype != SOL_BF16 && dtype != SOL_F32) return fail(SOL_ERR_INVALID_ARG, "dtype must be SOL_BF16 or SOL_F32 (got %d)", dtype);
    if (d != 64 && d != 128) return fail(SOL_ERR_UNSUPPORTED, "d must be 64 or 128 (got %d)", d);
    if ((long long)B * H > (1LL << 24)) return fail(SOL_ERR_UNSUPPORTED, "B*H too large");
    if ((long long)N * d * B * H > (1LL << 40)) return fail(SOL_ERR_UNSUPPORTED, "tensor too large");
    return SOL_OK;
}

int validate_forward(const void* q, const void* k, const void* v, const void* out, int B, int H, int N, int d,
                     int block_q, int block_k, float tau, int mode, int dtype, int keep_tail, int causal_granule = 0) {
    if (!q || !k || !v || !out) return fail(SOL_ERR_INVALID_ARG, "q, k, v and out must be non-null");
    int rc = check_common(B, H, N, d, block_q, block_k, dtype);
    if (rc) return rc;
    const int base = mode & ~SOL_THRESHOLD_DIAGONAL;
    if (base != SOL_DENSE && base != SOL_SPARSE && base != SOL_SPARSE_NO_CORRECTION)
        return fail(SOL_ERR_INVALID_ARG,
                    "mode must be SOL_DENSE, SOL_SPARSE or SOL_SPARSE_NO_CORRECTION, optionally | SOL_THRESHOLD_DIAGONAL "
                    "(got %d)", mode);
    if (!finite_or_inf(tau)) return fail(SOL_ERR_INVALID_ARG, "tau (standardised cutoff beta) is NaN");
    if (block_k != 64) return fail(SOL_ERR_UNSUPPORTED, "block_k must be 64 (got %d)", block_k);
    if (block_q != 64 && block_q != 128) return fail(SOL_ERR_UNSUPPORTED, "block_q must be 64 or 128 (got %d)", block_q);
    if (keep_tail < 0 || keep_tail % block_k) return fail(SOL_ERR_INVALID_ARG, "keep_tail_tokens must be a non-negative multiple of block_k (got %d)", keep_tail);
    if (keep_tail >= N && base != SOL_DENSE) return fail(SOL_ERR_INVALID_ARG, "keep_tail_tokens must leave at least one routable key block");
    if (keep_tail > N) return fail(SOL_ERR_INVALID_ARG, "keep_tail_tokens exceeds N");
    if (out == q || out == k || out == v) return fail(SOL_ERR_INVALID_ARG, "out must not alias q, k or v");
    if (causal_granule < 0) return fail(SOL_ERR_INVALID_ARG, "causal_granule must be >= 1 (got %d)", causal_granule);
    if (causal_granule > 0 && (mode & SOL_THRESHOLD_DIAGONAL))
        return fail(SOL_ERR_INVALID_ARG, "causal masks take their row statistics exactly; SOL_THRESHOLD_DIAGONAL is not supported");
    if (causal_granule > 0 && keep_tail != 0)
        return fail(SOL_ERR_INVALID_ARG, "causal masks take no forced tail");
    const sol::Shape s = sol::make_shape(B, H, N, d, block_q, block_k, mode, dtype, keep_tail, causal_granule);
    if (sol::attn_lds_bytes(s) > (size_t)sol::kMaxLds)
        return fail(SOL_ERR_UNSUPPORTED, "sequence too long: %d key blocks exceed the on-chip routing list", s.NK);
    return SOL_OK;
}

}  // namespace

extern "C" {

const char* sol_attn_last_error(void) { return g_err.c_str(); }

int sol_attn_pool_blocks(const void* q, const void* k, const void* v, float* qbar, float* kbar, float* vbar, int B, int H,
                         int N, int d, int block_q, int block_k, int dtype, void* stream) {
    int rc = check_common(B, H, N, d, block_q, block_k, dtype);
    if (rc) return rc;
    if (!qbar && !kbar && !vbar) return fail(SOL_ERR_INVALID_ARG, "at least one of qbar, kbar, vbar must be non-null");
    if ((qbar && !q) || (kbar && !k) || (vbar && !v))
        return fail(SOL_ERR_INVALID_ARG, "an input matching a non-null output is null");
    hipStream_t st = static_cast<hipStream_t>(stream);
    const int BH = B * H;
    hipError_t e;
    if (qbar && (e = sol::launch_pool_mean(q, qbar, dtype, BH, N, d, block_q, st)) != hipSuccess) return hip_fail(e, "pool q");
    if (kbar && (e = sol::launch_pool_mean(k, kbar, dtype, BH, N, d, block_k, st)) != hipSuccess) return hip_fail(e, "pool k");
    if (vbar && (e = sol::launch_pool_mean(v, vbar, dtype, BH, N, d, block_k, st)) != hipSuccess) return hip_fail(e, "pool v");
    return ok();
}

int sol_attn_thresholds(const float* qbar, const float* kbar, float* tau, float* mu, float* sigma, int B, int H, int NQ,
                        int NK, int nk_routable, int d, float beta, int threshold_mode, void* stream) {
    if (!qbar || !kbar || !tau) return fail(SOL_ERR_INVALID_ARG, "qbar, kbar and tau must be non-null");
    if (B <= 0 || H <= 0 || NQ <= 0 || NK <= 0) return fail(SOL_ERR_INVALID_ARG, "B, H, NQ and NK must be positive");
    if (nk_routable <= 0 || nk_routable > NK) return fail(SOL_ERR_INVALID_ARG, "nk_routable must be in [1, NK]");
    if (d != 64 && d != 128) return fail(SOL_ERR_UNSUPPORTED, "d must be 64 or 128 (got %d)", d);
    if (std::isnan(beta)) return fail(SOL_ERR_INVALID_ARG, "beta is NaN");
    if (threshold_mode != 0 && threshold_mode != SOL_THRESHOLD_DIAGONAL)
        return fail(SOL_ERR_INVALID_ARG, "threshold_mode must be 0 or SOL_THRESHOLD_DIAGONAL (got %d)", threshold_mode);
    hipStream_t st = static_cast<hipStream_t>(stream);
    const int BH = B * H;
    // Moment buffers are temporary: allocate, run, wait, free (this entry point synchronises).
    void* mom = nullptr;
    const size_t part = sol::moments_scratch_bytes(BH, nk_routable, d);
    hipError_t e = hipMalloc(&mom, part + ((size_t)BH * d * d + (size_t)BH * d) * sizeof(float));
    if (e != hipSuccess) return hip_fail(e, "hipMalloc(moments)");
    double* scratch = static_cast<double*>(mom);
    float* cov = reinterpret_cast<float*>(static_cast<char*>(mom) + part);
    float* muk = cov + (size_t)BH * d * d;
    e = sol::launch_moments(kbar, muk, cov, scratch, BH, NK, nk_routable, d, st);
    if (e == hipSuccess) e = sol::launch_tau(qbar, muk, cov, tau, mu, sigma, BH, NQ, d, beta,
                                                    threshold_mode == SOL_THRESHOLD_DIAGONAL ? 1 : 0, st);
    if (e == hipSuccess) e = hipStreamSynchronize(st);
    (void)hipFree(mom);
    if (e != hipSuccess) return hip_fail(e, "threshold kernels");
    return ok();
}

int sol_attn_route_materialized(const float* qbar, const float* kbar, float* proxies, uint32_t* mask_out, int B, int H,
                                int NQ, int NK, int nk_routable, int d, int rule, float param, void* stream) {
    if (!qbar || !kbar || !proxies || !mask_out)
        return fail(SOL_ERR_INVALID_ARG, "qbar, kbar, proxies and mask_out must be non-null");
    if (B <= 0 || H <= 0 || NQ <= 0 || NK <= 0) return fail(SOL_ERR_INVALID_ARG, "B, H, NQ and NK must be positive");
    if (nk_routable <= 0 || nk_routable > NK) return fail(SOL_ERR_INVALID_ARG, "nk_routable must be in [1, NK]");
    if (d != 64 && d != 128) return fail(SOL_ERR_UNSUPPORTED, "d must be 64 or 128 (got %d)", d);
    if ((long long)B * H > (1LL << 24) || (long long)NQ > (1 << 20))
        return fail(SOL_ERR_UNSUPPORTED, "too many (b, h) pairs or query blocks");
    if (rule == SOL_ROUTE_TOPK) {
        if (!(param >= 1.f && param <= (float)nk_routable) || param != std::floor(param))
            return fail(SOL_ERR_INVALID_ARG, "top-k needs an integer k in [1, nk_routable] (got %g)", (double)param);
        if (nk_routable > 8192) return fail(SOL_ERR_UNSUPPORTED, "top-k supports at most 8192 key blocks");
    } else if (rule == SOL_ROUTE_TOPP) {
        if (!(param > 0.f && param <= 1.f)) return fail(SOL_ERR_INVALID_ARG, "top-p needs p in (0, 1] (got %g)", (double)param);
        if (nk_routable > 4096) return fail(SOL_ERR_UNSUPPORTED, "top-p supports at most 4096 key blocks");
    } else {
        return fail(SOL_ERR_INVALID_ARG, "rule must be SOL_ROUTE_TOPK or SOL_ROUTE_TOPP (got %d)", rule);
    }
    hipError_t e = sol::launch_route_materialized(qbar, kbar, proxies, mask_out, B * H, NQ, NK, nk_routable, d, rule,
                                                  param, static_cast<hipStream_t>(stream));
    if (e != hipSuccess) return hip_fail(e, "materialised routing");
    return ok();
}

size_t sol_attn_workspace_bytes(int B, int H, int N, int d, int block_q, int block_k, int mode, int dtype,
                                int keep_tail_tokens) {
    static const char dummy = 0;
    if (validate_forward(&dummy, &dummy + 1, &dummy + 2, &dummy + 3, B, H, N, d, block_q, block_k, 0.f, mode, dtype,
                         keep_tail_tokens) != SOL_OK)
        return 0;
    const sol::Shape s = sol::make_shape(B, H, N, d, block_q, block_k, mode, dtype, keep_tail_tokens);
    return sol::workspace_layout(s, nullptr, nullptr);
}

}  // extern "C"

namespace {

// Routable (query block, key block) pairs of one head: NQ * NKr, or under a causal mask the
// sum over query blocks of the key blocks all their rows see.
double routable_pairs(const sol::Shape& s) {
    if (!s.causal) return (double)s.NQ * (double)s.NKr;
    double tot = 0.0;
    for (int i = 0; i < s.NQ; ++i) {
        const long long t0 = (long long)i * s.bq;
        const long long lo = std::min<long long>((t0 / s.causal + 1) * s.causal, s.N);
        tot += lo >= s.N ? s.NK : (double)(lo / s.bk);
    }
    return tot;
}

// Forgets the record of a counts buffer (its event goes back to its device's pool).  Caller
// holds g_mu.
void drop_record(const uint32_t* counts) {
    auto it = g_records.find(counts);
    if (it == g_records.end()) return;
    g_free_events[it->second.device].push_back(it->second.done);
    g_records.erase(it);
    auto pos = std::find(g_record_order.begin(), g_record_order.end(), counts);
    if (pos != g_record_order.end()) g_record_order.erase(pos);
}

// Creates or updates the record of a counts buffer and records its event on `st`.  Caller
// holds g_mu; device `dev` is current.
hipError_t note_counts(int dev, const uint32_t* counts, int B, int H, double pairs, bool library, hipStream_t st) {
    auto it = g_records.find(counts);
    if (it != g_records.end() && it->second.device != dev) {   // same address, another device's buffer
        drop_record(counts);
        it = g_records.end();
    }
    if (it == g_records.end()) {
        while (g_records.size() >= kMaxRecords && !g_record_order.empty()) drop_record(g_record_order.front());
        CountsRecord r;
        r.device = dev;
        auto& pool = g_free_events[dev];
        if (!pool.empty()) {
            r.done = pool.back();
            pool.pop_back();
        } else {
            hipError_t e = hipEventCreateWithFlags(&r.done, hipEventDisableTiming);
            if (e != hipSuccess) return e;
            g_all_events[dev].push_back(r.done);
        }
        it = g_records.emplace(counts, r).first;
        g_record_order.push_back(counts);
    }
    CountsRecord& r = it->second;
    r.B = B;
    r.H = H;
    r.routable_pairs = pairs;
    r.library = library;
    return hipEventRecord(r.done, st);
}

int forward_impl(const void* q, const void* k, const void* v, void* out, int B, int H, int N, int d, int block_q,
                 int block_k, float tau, int mode, int dtype, int keep_tail_tokens, int causal_granule,
                 void* workspace, size_t workspace_bytes, uint32_t* counts, uint32_t* mask_out, void* stream,
                 bool track_counts = true) {
    int rc = validate_forward(q, k, v, out, B, H, N, d, block_q, block_k, tau, mode, dtype, keep_tail_tokens,
                              causal_granule);
    if (rc) return rc;
    const sol::Shape s = sol::make_shape(B, H, N, d, block_q, block_k, mode, dtype, keep_tail_tokens, causal_granule);
    const size_t need = sol::workspace_layout(s, nullptr, nullptr);
    if (workspace && workspace_bytes < need)
        return fail(SOL_ERR_WORKSPACE, "workspace of %zu bytes is smaller than the %zu bytes required", workspace_bytes, need);
    hipStream_t st = static_cast<hipStream_t>(stream);
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return hip_fail(e, "hipGetDevice");

    std::lock_guard<std::mutex> lock(g_mu);
    DeviceBuffers& db = g_bufs[dev];
    if (!workspace) {
        if (db.ws_bytes < need) {
            if (db.ws) {
                e = hipDeviceSynchronize();
                if (e != hipSuccess) return hip_fail(e, "hipDeviceSynchronize");
                (void)hipFree(db.ws);
                db.ws = nullptr;
                db.ws_bytes = 0;
            }
            e = hipMalloc(&db.ws, need);
            if (e != hipSuccess) return hip_fail(e, "hipMalloc(workspace)");
            db.ws_bytes = need;
        }
        workspace = db.ws;
    }
    if (!counts) {
        const size_t n = (size_t)s.BH;
        if (db.counts_n < n) {
            if (db.counts) {
                e = hipDeviceSynchronize();
                if (e != hipSuccess) return hip_fail(e, "hipDeviceSynchronize");
                drop_record(db.counts);
                (void)hipFree(db.counts);
                db.counts = nullptr;
                db.counts_n = 0;
            }
            e = hipMalloc(reinterpret_cast<void**>(&db.counts), n * sizeof(uint32_t));
            if (e != hipSuccess) return hip_fail(e, "hipMalloc(counts)");
            db.counts_n = n;
        }
        counts = db.counts;
    }
    sol::Workspace ws;
    sol::workspace_layout(s, static_cast<char*>(workspace), &ws);
    hipEvent_t ev0 = nullptr, ev1 = nullptr;
    if (g_timing.enabled && g_timing.device == dev && g_timing.used < kMaxTimed) {
        ev0 = g_timing.start[g_timing.used];
        ev1 = g_timing.stop[g_timing.used];
        ++g_timing.used;
    }
    e = sol::launch_forward(s, q, k, v, out, tau, ws, counts, mask_out, st, ev0, ev1);
    if (e != hipSuccess) return hip_fail(e, "forward launch");
    if (track_counts) {
        // Record where these counts came from, and when they are complete (caller holds g_mu).
        e = note_counts(dev, counts, B, H, routable_pairs(s), counts == db.counts, st);
        if (e != hipSuccess) return hip_fail(e, "recording the counts event");
        t_last_counts = counts;
    }
    return ok();
}

}  // namespace

extern "C" {

int sol_attn_forward_ex(const void* q, const void* k, const void* v, void* out, int B, int H, int N, int d, int block_q,
                        int block_k, float tau, int mode, int dtype, int keep_tail_tokens, void* workspace,
                        size_t workspace_bytes, uint32_t* counts, uint32_t* mask_out, void* stream) {
    return forward_impl(q, k, v, out, B, H, N, d, block_q, block_k, tau, mode, dtype, keep_tail_tokens, 0, workspace,
                        workspace_bytes, counts, mask_out, stream);
}

int sol_attn_forward_causal(const void* q, const void* k, const void* v, void* out, int B, int H, int N, int d,
                            int block_q, int block_k, float tau, int mode, int dtype, int causal_granule,
                            void* workspace, size_t workspace_bytes, uint32_t* counts, uint32_t* mask_out,
                            void* stream) {
    if (causal_granule <= 0)
        return fail(SOL_ERR_INVALID_ARG, "causal_granule must be >= 1 (got %d)", causal_granule);
    return forward_impl(q, k, v, out, B, H, N, d, block_q, block_k, tau, mode, dtype, 0, causal_granule, workspace,
                        workspace_bytes, counts, mask_out, stream);
}

int sol_attn_forward_noalloc(const void* q, const void* k, const void* v, void* out, int B, int H, int N, int d,
                             int block_q, int block_k, float tau, int mode, int dtype, int keep_tail_tokens,
                             uint32_t* counts, uint32_t* mask_out, void* stream) {
    int rc = validate_forward(q, k, v, out, B, H, N, d, block_q, block_k, tau, mode, dtype, keep_tail_tokens);
    if (rc) return rc;
    if (!counts) return fail(SOL_ERR_INVALID_ARG, "counts must be given: this entry point allocates nothing");
    const sol::Shape s = sol::make_shape(B, H, N, d, block_q, block_k, mode, dtype, keep_tail_tokens);
    const size_t need = sol::workspace_layout(s, nullptr, nullptr);
    const size_t have = sol::noalloc_scratch_bytes();
    if (need > have)
        return fail(SOL_ERR_WORKSPACE,
                    "this shape needs %zu bytes of scratch; the built-in scratch of sol_attn_forward_noalloc holds "
                    "%zu bytes (use sol_attn_forward_ex with a workspace)", need, have);
    void* scratch = nullptr;
    hipError_t e = sol::noalloc_scratch(&scratch);
    if (e != hipSuccess) return hip_fail(e, "hipGetSymbolAddress(scratch)");
    return forward_impl(q, k, v, out, B, H, N, d, block_q, block_k, tau, mode, dtype, keep_tail_tokens, 0, scratch,
                        have, counts, mask_out, stream, /*track_counts=*/false);
}

int sol_attn_forward(const void* q, const void* k, const void* v, void* out, int B, int H, int N, int d, int block_q,
                     int block_k, float tau, int mode) {
    return sol_attn_forward_ex(q, k, v, out, B, H, N, d, block_q, block_k, tau, mode, SOL_BF16, 0, nullptr, 0, nullptr,
                               nullptr, nullptr);
}

int sol_attn_stats(float* frac_per_head, int B, int H, const uint32_t* counts) {
    if (!frac_per_head) return fail(SOL_ERR_INVALID_ARG, "frac_per_head must be non-null");
    if (B <= 0 || H <= 0) return fail(SOL_ERR_INVALID_ARG, "B and H must be positive (got %d, %d)", B, H);
    CountsRecord rec;
    const uint32_t* buf = counts;
    {
        std::lock_guard<std::mutex> lock(g_mu);
        if (!buf) {
            buf = t_last_counts;
            if (!buf) return fail(SOL_ERR_NO_DATA, "no forward call has been made on this thread");
        }
        auto it = g_records.find(buf);
        if (it == g_records.end())
            return fail(SOL_ERR_NO_DATA, counts ? "these counts were not written by a forward call of this library"
                                                : "no forward call has been made on this thread");
        rec = it->second;
        if (!counts && !rec.library)
            return fail(SOL_ERR_NO_DATA,
                        "the last forward on this thread wrote caller-owned counts: pass that buffer as `counts`");
    }
    if (rec.B != B || rec.H != H)
        return fail(SOL_ERR_NO_DATA, "B/H (%d, %d) differ from the forward that wrote these counts (%d, %d)", B, H,
                    rec.B, rec.H);
    int cur = 0;
    hipError_t e = hipGetDevice(&cur);
    if (e != hipSuccess) return hip_fail(e, "hipGetDevice");
    if (cur != rec.device && (e = hipSetDevice(rec.device)) != hipSuccess) return hip_fail(e, "hipSetDevice");
    const size_t n = (size_t)B * H;
    std::vector<uint32_t> host(n);
    e = hipEventSynchronize(rec.done);
    if (e == hipSuccess) e = hipMemcpy(host.data(), buf, n * sizeof(uint32_t), hipMemcpyDeviceToHost);
    if (cur != rec.device) (void)hipSetDevice(cur);
    if (e != hipSuccess) return hip_fail(e, "reading counts");
    const double denom = rec.routable_pairs > 0.0 ? rec.routable_pairs : 1.0;
    for (size_t i = 0; i < n; ++i) frac_per_head[i] = (float)((double)host[i] / denom);
    return ok();
}

int sol_attn_timing_enable(int enable) {
    std::lock_guard<std::mutex> lock(g_mu);
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return hip_fail(e, "hipGetDevice");
    if (enable && g_timing.start.empty()) {
        g_timing.start.resize(kMaxTimed);
        g_timing.stop.resize(kMaxTimed);
        for (int i = 0; i < kMaxTimed; ++i) {
            if ((e = hipEventCreate(&g_timing.start[i])) != hipSuccess) return hip_fail(e, "hipEventCreate");
            if ((e = hipEventCreate(&g_timing.stop[i])) != hipSuccess) return hip_fail(e, "hipEventCreate");
        }
        g_timing.device = dev;
    }
    if (enable && g_timing.device != dev) return fail(SOL_ERR_UNSUPPORTED, "timing events belong to device %d", g_timing.device);
    g_timing.enabled = enable != 0;
    g_timing.used = 0;
    return ok();
}

int sol_attn_kernel_timing(float* total_ms, int* launches) {
    if (!total_ms || !launches) return fail(SOL_ERR_INVALID_ARG, "total_ms and launches must be non-null");
    std::lock_guard<std::mutex> lock(g_mu);
    double total = 0.0;
    for (int i = 0; i < g_timing.used; ++i) {
        hipError_t e = hipEventSynchronize(g_timing.stop[i]);
        if (e != hipSuccess) return hip_fail(e, "hipEventSynchronize");
        float ms = 0.f;
        e = hipEventElapsedTime(&ms, g_timing.start[i], g_timing.stop[i]);
        if (e != hipSuccess) return hip_fail(e, "hipEventElapsedTime");
        total += ms;
    }
    *total_ms = (float)total;
    *launches = g_timing.used;
    g_timing.used = 0;
    return ok();
}

int sol_attn_release(void) {
    std::lock_guard<std::mutex> lock(g_mu);
    int cur = 0;
    (void)hipGetDevice(&cur);
    for (auto& kv : g_bufs) {
        (void)hipSetDevice(kv.first);
        (void)hipDeviceSynchronize();
        if (kv.second.ws) (void)hipFree(kv.second.ws);
        if (kv.second.counts) (void)hipFree(kv.second.counts);
        kv.second = DeviceBuffers{};
    }
    (void)hipSetDevice(cur);
    g_bufs.clear();
    for (auto& kv : g_all_events) {
        (void)hipSetDevice(kv.first);
        for (hipEvent_t ev : kv.second) (void)hipEventDestroy(ev);
    }
    (void)hipSetDevice(cur);
    g_all_events.clear();
    g_free_events.clear();
    g_records.clear();
    g_record_order.clear();
    t_last_counts = nullptr;
    return ok();
}

}  // extern "C"
