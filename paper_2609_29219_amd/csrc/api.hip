// C ABI of libattn.so: argument validation, per-thread stream and error
// state, plan cache, device description and the decode workspace.
#include <float.h>
#include <math.h>
#include <stdarg.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include <algorithm>
#include <atomic>
#include <map>
#include <memory>
#include <mutex>
#include <set>
#include <string>
#include <thread>
#include <tuple>
#include <vector>

#include "common.h"

namespace attn {
hipError_t launch_fwd_d64(const FwdPlan&, const FwdArgs&, hipStream_t);
hipError_t launch_fwd_d128(const FwdPlan&, const FwdArgs&, hipStream_t);

bool fwd_resources_d64(int bn, int waves, int pipe, int causal, KernelRes* r);
bool fwd_resources_d128(int bn, int waves, int pipe, int causal, KernelRes* r);

bool fwd_resources(int d, int bn, int waves, int pipe, int causal, KernelRes* r) {
    if (d == 64) return fwd_resources_d64(bn, waves, pipe, causal, r);
    if (d == 128) return fwd_resources_d128(bn, waves, pipe, causal, r);
    return false;
}

// Forced tiles (ablation only) may run a variant that spills: slow, not wrong.
bool fwd_resources_forced(int d, int bn, int waves, int pipe, int causal, KernelRes* r) {
    if (!fwd_resources(d, bn, waves, pipe, causal, r)) return false;
    r->scratch_bytes = 0;
    return true;
}

hipError_t launch_fwd(const FwdPlan& p, const void* q, const void* k, const void* v, void* o,
                      float* lse, int group, int out_bf16, long long rows, int Sq, int Skv,
                      float scale, int num_xcds, float* workspace, hipStream_t stream) {
    // softmax in base 2: exp(x) = 2^(x*log2 e); a negative scale is applied
    // as an exact sign flip of Q.  The kernel needs a factor > 0 (masked
    // scores are -inf); a zero scale becomes the smallest normal float, with
    // which every exponent rounds to 0 and the weights are exactly equal.
    double s = fabs((double)scale) * 1.4426950408889634;
    if (s < (double)FLT_MIN) s = (double)FLT_MIN;
    FwdArgs a;
    a.q = static_cast<const uint16_t*>(q);
    a.k = static_cast<const uint16_t*>(k);
    a.v = static_cast<const uint16_t*>(v);
    a.o = o;
    a.lse = lse;
    a.Sq = Sq;
    a.Skv = Skv;
    a.n_qtiles = p.n_qtiles;
    a.n_wg = (int)p.grid;
    a.num_xcds = num_xcds;
    a.group = group;
    a.out_bf16 = out_bf16;
    a.scale_log2 = (float)s;
    a.q_sign = scale < 0.f ? 0x80008000u : 0u;
    const int n = p.kv_splits;
    a.kv_splits = n;
    a.kv_chunk = n > 1 ? p.kv_chunk : Skv;
    // partial outputs first: their rows of d floats stay 16-byte aligned
    a.ws_o = n > 1 ? workspace : nullptr;
    a.ws_m = n > 1 ? workspace + rows * n * p.d : nullptr;
    a.ws_l = n > 1 ? a.ws_m + rows * n : nullptr;
    if (n > 1 && (p.causal || p.pipe == 2 || !workspace || p.kv_chunk % p.block_n != 0 ||
                  (long long)(n - 1) * p.kv_chunk >= Skv))
        return hipErrorInvalidValue;
    hipError_t e = hipErrorInvalidValue;
    if (p.d == 64) e = launch_fwd_d64(p, a, stream);
    if (p.d == 128) e = launch_fwd_d128(p, a, stream);
    if (e != hipSuccess || n == 1) return e;
    return launch_split_combine(p.d, a.ws_m, a.ws_l, a.ws_o, o, out_bf16, lse, rows, n, stream);
}
}  // namespace attn

using namespace attn;

namespace {

thread_local hipStream_t t_stream = nullptr;
thread_local std::string t_error;

int fail(int code, const char* fmt, ...) {
    char buf[512];
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(buf, sizeof buf, fmt, ap);
    va_end(ap);
    t_error = buf;
    return code;
}

int fail_hip(hipError_t e, const char* what) {
    return fail(ATTN_EHIP, "%s: %s", what, hipGetErrorString(e));
}

bool aligned16(const void* p) { return ((uintptr_t)p & 15u) == 0; }

// ---- library-owned workspace ------------------------------------------
// One buffer per stream, reused by every later call on that stream (stream
// order serialises them) and grown to the next power of two when a call
// needs more.  The stream's entry lock is held from the moment a call takes
// the buffer until that call has enqueued its kernels: a call on another
// host thread that grows the buffer therefore releases the old one only
// after every kernel that uses it has been enqueued, and the release is
// stream-ordered (it takes effect once the stream has passed those
// kernels), so growth never waits for the device.  (hipFree synchronises
// the whole device, so it is never called on this path.)  The map's own
// lock guards only the map and is never held across an allocation.
class WorkspaceMap {
public:
    // Stream-ordered allocation and release: HIP's, or a host-only double
    // in the self-test.  Both return 0 or an ATTN_E* code.
    struct Ops {
        int (*alloc)(void* ctx, void* stream, size_t bytes, void** out);
        int (*release)(void* ctx, void* stream, void* ptr);
        void* ctx;
    };
    // On success *lk holds the stream's entry (keep it until the kernels
    // that use *out are enqueued) and *out is its buffer of at least bytes.
    int acquire(void* stream, size_t bytes, const Ops& ops, std::unique_lock<std::mutex>* lk,
                void** out) {
        Entry* e = nullptr;
        {
            std::lock_guard<std::mutex> g(mu_);
            std::unique_ptr<Entry>& slot = entries_[stream];
            if (!slot) slot.reset(new Entry);
            e = slot.get();
        }
        std::unique_lock<std::mutex> l(e->mu);
        if (e->bytes < bytes) {
            size_t want = 4096;
            while (want < bytes) want *= 2;
            void* fresh = nullptr;
            const int rc = ops.alloc(ops.ctx, stream, want, &fresh);
            if (rc) return rc;
            void* old = e->ptr;
            e->ptr = fresh;
            e->bytes = want;
            // work already enqueued on the stream still reads the old buffer:
            // released behind it, in stream order
            if (old) {
                const int rr = ops.release(ops.ctx, stream, old);
                if (rr) return rr;
            }
        }
        *out = e->ptr;
        *lk = std::move(l);
        return ATTN_OK;
    }

private:
    struct Entry {
        std::mutex mu;
        void* ptr = nullptr;
        size_t bytes = 0;
    };
    std::mutex mu_;
    std::map<void*, std::unique_ptr<Entry>> entries_;
};

int hip_ws_alloc(void*, void* stream, size_t bytes, void** out) {
    const hipError_t e = hipMallocAsync(out, bytes, static_cast<hipStream_t>(stream));
    if (e != hipSuccess || !*out) {
        (void)hipGetLastError();
        return fail(ATTN_ENOMEM, "workspace of %zu bytes: %s", bytes, hipGetErrorString(e));
    }
    return ATTN_OK;
}

int hip_ws_release(void*, void* stream, void* ptr) {
    const hipError_t e = hipFreeAsync(ptr, static_cast<hipStream_t>(stream));
    return e == hipSuccess ? ATTN_OK : fail_hip(e, "workspace release");
}

const WorkspaceMap::Ops kHipWorkspaceOps = {hip_ws_alloc, hip_ws_release, nullptr};

// ---- static decode scratch ---------------------------------------------
// Device memory for attn_decode_noalloc, the entry point for callers that
// cannot allocate: a file-scope array that every device the library runs on
// holds (its own copy, at its own address) until the process ends.  Host
// code never names it except to look up that address: the name is only a
// host-side stand-in, and a kernel given it would fault.
static __device__ __align__(256) float scratch[ATTN_NOALLOC_SCRATCH_BYTES / sizeof(float)];

// ---- per-device state --------------------------------------------------
// Set up once per device, on the first call made with it current.
struct DeviceState {
    std::once_flag once;
    hipError_t init_err = hipSuccess;
    bool is_gfx950 = false;
    attn_device_desc desc{};
    WorkspaceMap ws;
    void* scratch_ptr = nullptr;  // this device's copy of `scratch`
    hipError_t scratch_err = hipSuccess;
};
std::mutex g_mu;  // guards the maps below; never held across a HIP call
std::map<int, DeviceState> g_devices;  // nodes never move
std::map<std::tuple<int, int, int, int, int, int, int, int>, FwdPlan> g_fwd_cache;
std::map<std::tuple<int, int, int, int, int, int, int>, DecodePlan> g_dec_cache;
std::map<std::tuple<int, int, int, int, int>, GemmPlan> g_gemm_cache;

// Structural properties from the runtime; performance properties from the
// built-in gfx950 description.
hipError_t fill_desc(int dev, attn_device_desc* d) {
    default_desc(d);
    hipDeviceProp_t prop;
    hipError_t e = hipGetDeviceProperties(&prop, dev);
    if (e != hipSuccess) return e;
    snprintf(d->arch, sizeof d->arch, "%s", prop.gcnArchName);
    char* colon = strchr(d->arch, ':');
    if (colon) *colon = 0;
    d->num_cus = prop.multiProcessorCount;
    if (prop.maxSharedMemoryPerMultiProcessor > 0)
        d->lds_bytes_per_cu = (int)prop.maxSharedMemoryPerMultiProcessor;
    if (prop.clockRate > 0) d->clock_ghz = prop.clockRate / 1e6;
    return hipSuccess;
}

int device_state(DeviceState** out) {
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return fail_hip(e, "hipGetDevice");
    DeviceState* st = nullptr;
    {
        std::lock_guard<std::mutex> lk(g_mu);
        st = &g_devices[dev];
    }
    std::call_once(st->once, [&] {
        st->init_err = fill_desc(dev, &st->desc);
        st->is_gfx950 = st->init_err == hipSuccess && strcmp(st->desc.arch, "gfx950") == 0;
        // the device address of this device's scratch array, looked up once
        // with the device current (it differs per device)
        if (st->is_gfx950) {
            st->scratch_err = hipGetSymbolAddress(&st->scratch_ptr, HIP_SYMBOL(scratch));
            if (st->scratch_err != hipSuccess) {
                st->scratch_ptr = nullptr;
                (void)hipGetLastError();
            }
        }
    });
    if (st->init_err != hipSuccess) return fail_hip(st->init_err, "hipGetDeviceProperties");
    if (!st->is_gfx950)
        return fail(ATTN_EUNSUPPORTED, "device %d is %s; this library is built for gfx950", dev,
                    st->desc.arch);
    *out = st;
    return ATTN_OK;
}

// Optional fixed tile choice for the block-size ablation only:
// ATTN_FORCE_PLAN="bn=64,waves=8,pipe=2" (optionally ",splits=4").  Never
// used to select tiles.
bool forced_fwd(int* bn, int* waves, int* pipe, int* splits) {
    const char* s = getenv("ATTN_FORCE_PLAN");
    if (!s || !*s) return false;
    *splits = 1;
    const int n = sscanf(s, "bn=%d,waves=%d,pipe=%d,splits=%d", bn, waves, pipe, splits);
    return n == 3 || n == 4;
}

// The per-stream workspace (decode partials, split-key prefill partials) of
// at least bytes bytes; *lk holds the stream's entry until the caller has
// enqueued the kernels that use it.
int stream_workspace(DeviceState* st, size_t bytes, std::unique_lock<std::mutex>* lk,
                     void** out) {
    return st->ws.acquire(t_stream, bytes, kHipWorkspaceOps, lk, out);
}

// Optional fixed GEMM tile for the block-size ablation only:
// ATTN_FORCE_GEMM="bm=256,bn=256,bk=64,wm=2,wn=4,pipe=1[,splits=4]".  Never
// used to select tiles.
bool forced_gemm(int* bm, int* bn, int* bk, int* wm, int* wn, int* pipe, int* splits) {
    const char* s = getenv("ATTN_FORCE_GEMM");
    if (!s || !*s) return false;
    *splits = 1;
    const int n =
        sscanf(s, "bm=%d,bn=%d,bk=%d,wm=%d,wn=%d,pipe=%d,splits=%d", bm, bn, bk, wm, wn, pipe, splits);
    return n == 6 || n == 7;
}

// Forced tiles (ablation only) may run a variant that spills: slow, not wrong.
bool gemm_resources_forced(const GemmPlan& p, KernelRes* r) {
    if (!gemm_resources(p, r)) return false;
    r->scratch_bytes = 0;
    return true;
}

int validate_common(const void* q, const void* k, const void* v, const void* o, int B, int H,
                    int Skv, int d) {
    if (!q || !k || !v || !o) return fail(ATTN_EINVAL, "null tensor pointer");
    if (!aligned16(q) || !aligned16(k) || !aligned16(v) || !aligned16(o))
        return fail(ATTN_EINVAL, "tensor pointers must be 16-byte aligned");
    if (B <= 0 || H <= 0 || Skv <= 0 || d <= 0)
        return fail(ATTN_EINVAL, "dimensions must be positive (B=%d H=%d Skv=%d d=%d)", B, H,
                    Skv, d);
    if (d != 64 && d != 128) return fail(ATTN_EUNSUPPORTED, "head dim %d not in {64, 128}", d);
    return ATTN_OK;
}

}  // namespace

extern "C" {

int attn_set_stream(void* hip_stream) {
    t_stream = static_cast<hipStream_t>(hip_stream);
    return ATTN_OK;
}

void* attn_get_stream(void) { return t_stream; }

const char* attn_last_error(void) { return t_error.c_str(); }

int attn_query_device(attn_device_desc* out) {
    if (!out) return fail(ATTN_EINVAL, "null descriptor");
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e == hipSuccess) e = fill_desc(dev, out);
    if (e != hipSuccess) {
        default_desc(out);
        return fail_hip(e, "no usable HIP device (MI355X specification values returned)");
    }
    return ATTN_OK;
}

int attn_measure_device(attn_device_desc* out) {
    if (!out) return fail(ATTN_EINVAL, "null descriptor");
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e == hipSuccess) e = fill_desc(dev, out);
    if (e != hipSuccess) return fail_hip(e, "no usable HIP device");
    e = measure_device(out);
    if (e != hipSuccess) return fail_hip(e, "device microbenchmarks");
    return ATTN_OK;
}

int attn_get_plan_for(const attn_device_desc* desc, int kind, int B, int H, int Sq, int Skv,
                      int d, int causal, int n_splits, char* buf, int buflen) {
    attn_device_desc local;
    FwdResFn res = nullptr;
    if (!desc) {
        // the current device (compiled kernels' real footprint), else the
        // specification values
        if (attn_query_device(&local) == ATTN_OK && strcmp(local.arch, "gfx950") == 0)
            res = fwd_resources;
        desc = &local;
    }
    if (buflen < 0 || (buflen > 0 && !buf)) return fail(ATTN_EINVAL, "bad output buffer");
    if (B <= 0 || H <= 0 || Skv <= 0 || d <= 0 || (kind == ATTN_KIND_FWD && Sq <= 0))
        return fail(ATTN_EINVAL, "dimensions must be positive");
    if (d != 64 && d != 128) return fail(ATTN_EUNSUPPORTED, "head dim %d not in {64, 128}", d);
    if (desc->num_cus <= 0 || desc->num_xcds <= 0 || desc->clock_ghz <= 0.0 ||
        desc->lds_bytes_per_cu <= 0 || desc->hbm_bytes_per_s <= 0.0 ||
        desc->mfma_bf16_flops_per_clk_cu <= 0.0 || desc->lds_bytes_per_clk_cu <= 0.0 ||
        desc->l2_bytes_per_clk_xcd <= 0.0 || desc->valu_lanes_per_clk_simd <= 0.0 ||
        desc->simds_per_cu <= 0 || desc->wave_size <= 0 || desc->vgprs_per_simd_lane <= 0 ||
        desc->max_waves_per_simd <= 0 || desc->issue_cycles_per_score < 0.0 ||
        desc->valu_mfma_overlap < 0.0 || desc->valu_mfma_overlap >= 1.0 ||
        desc->tile_sync_cycles < 0.0 || desc->tile_latency_cycles < 0.0)
        return fail(ATTN_EINVAL, "device description has out-of-range fields");
    if (kind == ATTN_KIND_FWD) {
        if (causal && Sq > Skv) return fail(ATTN_EUNSUPPORTED, "causal needs Sq <= Skv");
        FwdPlan p;
        if (!plan_fwd(*desc, B, H, Sq, Skv, d, causal ? 1 : 0, &p, res))
            return fail(ATTN_EUNSUPPORTED, "no feasible prefill plan");
        return format_fwd_plan(p, buf, buflen);
    }
    if (kind == ATTN_KIND_DECODE) {
        DecodePlan p;
        if (!plan_decode(*desc, B, H, H, Skv, d, n_splits, &p))
            return fail(ATTN_EUNSUPPORTED, "no feasible decode plan");
        return format_decode_plan(p, buf, buflen);
    }
    return fail(ATTN_EINVAL, "unknown plan kind %d", kind);
}

// Not part of the ABI: every feasible prefill candidate with its modelled
// time, one plan line each (newline-separated), for the block-size ablation
// that validates the model (plan_ablation.py).  Returns the full length.
// device_footprint != 0: with a gfx950 device present, use the compiled
// kernels' real register and occupancy footprint (always so for desc NULL);
// otherwise the estimate, as attn_get_plan_for does for an explicit desc.
int attn__fwd_candidates(const attn_device_desc* desc, int B, int H, int Sq, int Skv, int d,
                         int causal, int device_footprint, char* buf, int buflen) {
    attn_device_desc local;
    FwdResFn res = nullptr;
    const bool have = attn_query_device(&local) == ATTN_OK && strcmp(local.arch, "gfx950") == 0;
    // bit 0: the compiled kernels' real footprint; bit 1: the analytic model
    // without the measured per-variant tile costs
    if (have && ((device_footprint & 1) || !desc)) res = fwd_resources;
    struct Scales {
        explicit Scales(bool on) { use_fwd_primitive_costs(on); }
        ~Scales() { use_fwd_primitive_costs(true); }
    } scales(!(device_footprint & 2));
    if (!desc) desc = &local;
    if (buflen < 0 || (buflen > 0 && !buf)) return fail(ATTN_EINVAL, "bad output buffer");
    if (B <= 0 || H <= 0 || Sq <= 0 || Skv <= 0) return fail(ATTN_EINVAL, "bad dimensions");
    if (d != 64 && d != 128) return fail(ATTN_EUNSUPPORTED, "head dim %d not in {64, 128}", d);
    constexpr int kCap = 512;
    std::vector<FwdPlan> plans(kCap);
    const int n = std::min(kCap, plan_fwd_all(*desc, B, H, Sq, Skv, d, causal ? 1 : 0,
                                              plans.data(), kCap, res));
    int len = 0;
    for (int i = 0; i < n; ++i) {
        char line[512];
        const int l = format_fwd_plan(plans[i], line, sizeof line);
        if (buf && len + l + 1 < buflen) {
            memcpy(buf + len, line, l);
            buf[len + l] = '\n';
            buf[len + l + 1] = '\0';
        }
        len += l + 1;
    }
    if (buf && buflen > 0 && len >= buflen) buf[buflen - 1] = '\0';
    return len;
}

// Not part of the ABI: a host-only check of the workspace locking, with no
// device.  threads host threads share simulated streams; for each of rounds
// streams every thread makes calls that need a workspace twice as large as
// its previous call (so most calls grow the buffer), and "enqueues" a job
// naming the buffer it was given.  Allocation hands out fresh addresses and
// release is enqueued on the simulated stream, like the HIP calls.  The
// stream log is then replayed in order: a job that runs after its buffer's
// release is a use after free.  hold_lock != 0 enqueues while holding the
// entry lock (what the library does); hold_lock == 0 drops the lock first
// and yields, the order in which a growth on another thread can release the
// buffer before the job is enqueued.  Returns the number of such jobs.
int attn__workspace_selftest(int threads, int rounds, int hold_lock) {
    struct Sim {
        std::mutex mu;
        std::vector<std::pair<int, uintptr_t>> log;  // (0 job | 1 release, buffer)
        std::atomic<uintptr_t> next{4096};
    } sim;
    auto alloc = [](void* ctx, void*, size_t bytes, void** out) -> int {
        Sim* s = static_cast<Sim*>(ctx);
        *out = reinterpret_cast<void*>(s->next.fetch_add((bytes + 4095) / 4096 * 4096));
        return ATTN_OK;
    };
    auto release = [](void* ctx, void*, void* ptr) -> int {
        Sim* s = static_cast<Sim*>(ctx);
        std::lock_guard<std::mutex> g(s->mu);
        s->log.emplace_back(1, reinterpret_cast<uintptr_t>(ptr));
        return ATTN_OK;
    };
    const WorkspaceMap::Ops ops = {alloc, release, &sim};
    WorkspaceMap map;
    std::vector<std::thread> pool;
    for (int t = 0; t < threads; ++t)
        pool.emplace_back([&, t] {
            for (int r = 0; r < rounds; ++r) {
                void* stream = reinterpret_cast<void*>((uintptr_t)(r + 1) * 64);
                for (int i = 0; i < 12; ++i) {
                    std::unique_lock<std::mutex> lk;
                    void* buf = nullptr;
                    if (map.acquire(stream, ((size_t)2048 << i) + (size_t)t, ops, &lk, &buf))
                        continue;
                    if (!hold_lock) {
                        lk.unlock();
                        std::this_thread::yield();
                    }
                    std::lock_guard<std::mutex> g(sim.mu);
                    sim.log.emplace_back(0, reinterpret_cast<uintptr_t>(buf));
                }
            }
        });
    for (auto& th : pool) th.join();
    std::set<uintptr_t> released;
    int bad = 0;
    for (const auto& rec : sim.log) {
        if (rec.first == 1) released.insert(rec.second);
        else if (released.count(rec.second)) ++bad;
    }
    return bad;
}

int attn_get_plan(int kind, int B, int H, int Sq, int Skv, int d, int causal, int n_splits,
                  char* buf, int buflen) {
    return attn_get_plan_for(nullptr, kind, B, H, Sq, Skv, d, causal, n_splits, buf, buflen);
}

int attn_fwd_ex(const void* q, const void* k, const void* v, void* o, float* lse, int B, int Hq,
                int Hkv, int Sq, int Skv, int d, float scale, int causal, int flags) {
    int rc = validate_common(q, k, v, o, B, Hq, Skv, d);
    if (rc) return rc;
    if (Sq <= 0) return fail(ATTN_EINVAL, "Sq must be positive (got %d)", Sq);
    if (Hkv <= 0 || Hq % Hkv != 0)
        return fail(ATTN_EINVAL, "Hkv (%d) must be positive and divide Hq (%d)", Hkv, Hq);
    if (flags & ~ATTN_OUT_BF16) return fail(ATTN_EINVAL, "unknown flags 0x%x", flags);
    if (lse && ((uintptr_t)lse & 3u)) return fail(ATTN_EINVAL, "lse must be 4-byte aligned");
    if (!isfinite(scale)) return fail(ATTN_EINVAL, "scale must be finite");
    if (causal && Sq > Skv)
        return fail(ATTN_EUNSUPPORTED, "causal attention needs Sq <= Skv (Sq=%d Skv=%d)", Sq, Skv);
    if ((long long)Skv * d * 2 > 0x7fffffffLL)
        return fail(ATTN_EUNSUPPORTED, "one head's K or V (%lld bytes) exceeds 2 GiB",
                    (long long)Skv * d * 2);
    DeviceState* st = nullptr;
    rc = device_state(&st);
    if (rc) return rc;

    const int c = causal ? 1 : 0;
    FwdPlan plan;
    int fbn, fw, fpipe, fsplits;
    if (forced_fwd(&fbn, &fw, &fpipe, &fsplits)) {
        if (!plan_fwd_fixed(st->desc, B, Hq, Sq, Skv, d, c, fbn, fw, fpipe, &plan,
                            fwd_resources_forced, fsplits))
            return fail(ATTN_EINVAL, "ATTN_FORCE_PLAN names an infeasible or unknown tile");
    } else {
        // looked up under the lock; planned (which queries the runtime for the
        // compiled kernels' footprint) outside it
        const auto key = std::make_tuple(B, Hq, Sq, Skv, d, c, st->desc.num_cus, 0);
        bool hit = false;
        {
            std::lock_guard<std::mutex> lk(g_mu);
            auto it = g_fwd_cache.find(key);
            if ((hit = it != g_fwd_cache.end())) plan = it->second;
        }
        if (!hit) {
            if (!plan_fwd(st->desc, B, Hq, Sq, Skv, d, c, &plan, fwd_resources))
                return fail(ATTN_EUNSUPPORTED, "no feasible prefill plan for this shape");
            std::lock_guard<std::mutex> lk(g_mu);
            g_fwd_cache[key] = plan;
        }
    }
    const long long rows = (long long)B * Hq * Sq;
    void* ws = nullptr;
    std::unique_lock<std::mutex> ws_lock;  // held until the kernels are enqueued
    if (plan.kv_splits > 1) {
        rc = stream_workspace(st, (size_t)fwd_workspace_bytes(plan, rows), &ws_lock, &ws);
        if (rc) return rc;
    }
    hipError_t e = launch_fwd(plan, q, k, v, o, lse, Hq / Hkv, (flags & ATTN_OUT_BF16) ? 1 : 0,
                              rows, Sq, Skv, scale, st->desc.num_xcds, static_cast<float*>(ws),
                              t_stream);
    if (e != hipSuccess) return fail_hip(e, "prefill launch");
    return ATTN_OK;
}

int attn_fwd(const void* q, const void* k, const void* v, float* o, int B, int H, int Sq,
             int Skv, int d, float scale, int causal) {
    return attn_fwd_ex(q, k, v, o, nullptr, B, H, H, Sq, Skv, d, scale, causal, 0);
}

// Plan of one decode call (cached per shape).
static int decode_plan(DeviceState* st, int B, int Hq, int Hkv, int Skv, int d, int n_splits,
                       DecodePlan* plan) {
    const auto key = std::make_tuple(B, Hq, Hkv, Skv, d, n_splits, st->desc.num_cus);
    {
        std::lock_guard<std::mutex> lk(g_mu);
        auto it = g_dec_cache.find(key);
        if (it != g_dec_cache.end()) {
            *plan = it->second;
            return ATTN_OK;
        }
    }
    if (!plan_decode(st->desc, B, Hq, Hkv, Skv, d, n_splits, plan))
        return fail(ATTN_EUNSUPPORTED, "no feasible decode plan for this shape");
    std::lock_guard<std::mutex> lk(g_mu);
    g_dec_cache[key] = *plan;
    return ATTN_OK;
}

static int validate_decode(const void* q, const void* k, const void* v, const void* o, int B,
                           int Hq, int Hkv, int Skv, int d) {
    int rc = validate_common(q, k, v, o, B, Hq, Skv, d);
    if (rc) return rc;
    if (Hkv <= 0 || Hq % Hkv != 0)
        return fail(ATTN_EINVAL, "Hkv (%d) must be positive and divide Hq (%d)", Hkv, Hq);
    return ATTN_OK;
}

long long attn_decode_workspace_bytes(int B, int Hq, int Hkv, int Skv, int d, int n_splits) {
    if (B <= 0 || Hq <= 0 || Hkv <= 0 || Hq % Hkv != 0 || Skv <= 0)
        return fail(ATTN_EINVAL, "bad dimensions");
    if (d != 64 && d != 128) return fail(ATTN_EUNSUPPORTED, "head dim %d not in {64, 128}", d);
    DeviceState* st = nullptr;
    int rc = device_state(&st);
    if (rc) return rc;
    DecodePlan plan;
    rc = decode_plan(st, B, Hq, Hkv, Skv, d, n_splits, &plan);
    if (rc) return rc;
    return (long long)B * Hq * plan.n_splits * (d + 2) * (long long)sizeof(float);
}

int attn_decode_ex(const void* q, const void* k, const void* v, float* o, float* lse, int B,
                   int Hq, int Hkv, int Skv, int d, int n_splits, void* workspace,
                   size_t workspace_bytes) {
    int rc = validate_decode(q, k, v, o, B, Hq, Hkv, Skv, d);
    if (rc) return rc;
    if (lse && ((uintptr_t)lse & 3u)) return fail(ATTN_EINVAL, "lse must be 4-byte aligned");
    if (workspace && !aligned16(workspace))
        return fail(ATTN_EINVAL, "workspace must be 16-byte aligned");
    DeviceState* st = nullptr;
    rc = device_state(&st);
    if (rc) return rc;
    DecodePlan plan;
    rc = decode_plan(st, B, Hq, Hkv, Skv, d, n_splits, &plan);
    if (rc) return rc;
    const size_t ws_bytes = (size_t)B * Hq * plan.n_splits * (d + 2) * sizeof(float);
    void* ws = workspace;
    std::unique_lock<std::mutex> ws_lock;  // held until the kernels are enqueued
    if (ws) {
        if (workspace_bytes < ws_bytes)
            return fail(ATTN_EINVAL, "workspace of %zu bytes, %zu needed", workspace_bytes,
                        ws_bytes);
    } else {
        rc = stream_workspace(st, ws_bytes, &ws_lock, &ws);
        if (rc) return rc;
    }
    const float scale = (float)(1.0 / sqrt((double)d));
    const hipError_t e = launch_decode(plan, q, k, v, o, lse, static_cast<float*>(ws), B, Hq,
                                       Hkv, Skv, scale, st->desc.num_xcds, t_stream);
    if (e != hipSuccess) return fail_hip(e, "decode launch");
    return ATTN_OK;
}

int attn_decode(const void* q, const void* k, const void* v, float* o, int B, int H, int Skv,
                int d, int n_splits) {
    return attn_decode_ex(q, k, v, o, nullptr, B, H, H, Skv, d, n_splits, nullptr, 0);
}

int attn_decode_noalloc(const void* q, const void* k, const void* v, float* o, float* lse, int B,
                        int Hq, int Hkv, int Skv, int d, int n_splits) {
    int rc = validate_decode(q, k, v, o, B, Hq, Hkv, Skv, d);
    if (rc) return rc;
    if (lse && ((uintptr_t)lse & 3u)) return fail(ATTN_EINVAL, "lse must be 4-byte aligned");
    DeviceState* st = nullptr;
    rc = device_state(&st);
    if (rc) return rc;
    if (!st->scratch_ptr) return fail_hip(st->scratch_err, "static scratch address");
    DecodePlan plan;
    rc = decode_plan(st, B, Hq, Hkv, Skv, d, n_splits, &plan);
    if (rc) return rc;
    const size_t ws_bytes = (size_t)B * Hq * plan.n_splits * (d + 2) * sizeof(float);
    if (ws_bytes > (size_t)ATTN_NOALLOC_SCRATCH_BYTES)
        return fail(ATTN_ENOMEM,
                    "this call's decode partials need %zu bytes (%lld rows x %d splits); the "
                    "static scratch holds %zu",
                    ws_bytes, (long long)B * Hq, plan.n_splits,
                    (size_t)ATTN_NOALLOC_SCRATCH_BYTES);
    // every partial the combine reads is written by the partial kernel first,
    // so nothing in the scratch needs clearing
    const float scale = (float)(1.0 / sqrt((double)d));
    const hipError_t e = launch_decode(plan, q, k, v, o, lse, static_cast<float*>(st->scratch_ptr),
                                       B, Hq, Hkv, Skv, scale, st->desc.num_xcds, t_stream);
    if (e != hipSuccess) return fail_hip(e, "decode launch");
    return ATTN_OK;
}

// ---------------------------------------------------------------- GEMM --
static int validate_gemm_dims(int M, int N, int K, int flags) {
    if (M <= 0 || N <= 0 || K <= 0)
        return fail(ATTN_EINVAL, "dimensions must be positive (M=%d N=%d K=%d)", M, N, K);
    if (flags & ~(ATTN_OUT_BF16 | ATTN_GEMM_B_NK))
        return fail(ATTN_EINVAL, "unknown flags 0x%x", flags);
    if (K % 8 != 0 || N % 8 != 0)
        return fail(ATTN_EUNSUPPORTED, "K (%d) and N (%d) must be multiples of 8", K, N);
    if ((long long)M * K * 2 > 0x7fffffffLL || (long long)N * K * 2 > 0x7fffffffLL)
        return fail(ATTN_EUNSUPPORTED, "A or B exceeds 2 GiB");
    return ATTN_OK;
}

int attn_gemm_plan(const attn_device_desc* desc, int M, int N, int K, int flags, char* buf,
                   int buflen) {
    attn_device_desc local;
    GemmResFn res = nullptr;
    if (!desc) {
        const int q = attn_query_device(&local);
        if (q == ATTN_OK && strcmp(local.arch, "gfx950") == 0) res = gemm_resources;
        desc = &local;
    }
    if (buflen < 0 || (buflen > 0 && !buf)) return fail(ATTN_EINVAL, "bad output buffer");
    int rc = validate_gemm_dims(M, N, K, flags);
    if (rc) return rc;
    GemmPlan p;
    if (!plan_gemm(*desc, M, N, K, (flags & ATTN_GEMM_B_NK) ? 1 : 0, &p, res))
        return fail(ATTN_EUNSUPPORTED, "no feasible GEMM plan");
    return format_gemm_plan(p, buf, buflen);
}

// Not part of the ABI: every feasible GEMM candidate with its modelled time,
// one plan line each (for the block-size ablation).  Returns the full length.
int attn__gemm_candidates(const attn_device_desc* desc, int M, int N, int K, int flags,
                          int device_footprint, char* buf, int buflen) {
    attn_device_desc local;
    GemmResFn res = nullptr;
    const bool have = attn_query_device(&local) == ATTN_OK && strcmp(local.arch, "gfx950") == 0;
    // bit 0: the compiled kernels' real footprint; bit 1: the analytic model
    // without the measured per-variant costs
    if (have && ((device_footprint & 1) || !desc)) res = gemm_resources;
    struct Scales {
        explicit Scales(bool on) { use_fwd_primitive_costs(on); }
        ~Scales() { use_fwd_primitive_costs(true); }
    } scales(!(device_footprint & 2));
    if (!desc) desc = &local;
    if (buflen < 0 || (buflen > 0 && !buf)) return fail(ATTN_EINVAL, "bad output buffer");
    int rc = validate_gemm_dims(M, N, K, flags);
    if (rc) return rc;
    GemmPlan plans[64];
    const int n = std::min(64, plan_gemm_all(*desc, M, N, K, (flags & ATTN_GEMM_B_NK) ? 1 : 0,
                                             plans, 64, res));
    int len = 0;
    for (int i = 0; i < n; ++i) {
        char line[512];
        const int l = format_gemm_plan(plans[i], line, sizeof line);
        if (buf && len + l + 1 < buflen) {
            memcpy(buf + len, line, l);
            buf[len + l] = '\n';
            buf[len + l + 1] = '\0';
        }
        len += l + 1;
    }
    if (buf && buflen > 0 && len >= buflen) buf[buflen - 1] = '\0';
    return len;
}

int attn_gemm(const void* a, const void* b, void* c, int M, int N, int K, int flags) {
    if (!a || !b || !c) return fail(ATTN_EINVAL, "null matrix pointer");
    if (!aligned16(a) || !aligned16(b) || !aligned16(c))
        return fail(ATTN_EINVAL, "matrix pointers must be 16-byte aligned");
    int rc = validate_gemm_dims(M, N, K, flags);
    if (rc) return rc;
    DeviceState* st = nullptr;
    rc = device_state(&st);
    if (rc) return rc;
    const int b_nk = (flags & ATTN_GEMM_B_NK) ? 1 : 0;
    GemmPlan plan;
    int bm, bn, bk, wm, wn, pipe, splits;
    if (forced_gemm(&bm, &bn, &bk, &wm, &wn, &pipe, &splits)) {
        if (!plan_gemm_fixed(st->desc, M, N, K, b_nk, bm, bn, bk, wm, wn, pipe, &plan,
                             gemm_resources_forced, splits))
            return fail(ATTN_EINVAL, "ATTN_FORCE_GEMM names an infeasible or unknown tile");
    } else {
        const auto key = std::make_tuple(M, N, K, b_nk, st->desc.num_cus);
        bool hit = false;
        {
            std::lock_guard<std::mutex> lk(g_mu);
            auto it = g_gemm_cache.find(key);
            if ((hit = it != g_gemm_cache.end())) plan = it->second;
        }
        if (!hit) {
            if (!plan_gemm(st->desc, M, N, K, b_nk, &plan, gemm_resources))
                return fail(ATTN_EUNSUPPORTED, "no feasible GEMM plan for this shape");
            std::lock_guard<std::mutex> lk(g_mu);
            g_gemm_cache[key] = plan;
        }
    }
    void* ws = nullptr;
    std::unique_lock<std::mutex> ws_lock;  // held until the kernels are enqueued
    if (plan.k_splits > 1) {
        rc = stream_workspace(st, (size_t)gemm_workspace_bytes(plan, M, N), &ws_lock, &ws);
        if (rc) return rc;
    }
    const hipError_t e = launch_gemm(plan, a, b, c, M, N, K, (flags & ATTN_OUT_BF16) ? 1 : 0,
                                     st->desc.num_xcds, static_cast<float*>(ws), t_stream);
    if (e != hipSuccess) return fail_hip(e, "GEMM launch");
    return ATTN_OK;
}

}  // extern "C"
