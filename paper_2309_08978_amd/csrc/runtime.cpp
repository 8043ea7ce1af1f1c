// Runtime of libnnjit: argument validation, lazy HIP initialisation,
// dispatch, split-K scratch, the just-in-time tuner and its per-shape cache,
// and the extern "C" entry points declared in include/nnjit.h.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <chrono>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <map>
#include <memory>
#include <mutex>
#include <string>
#include <tuple>
#include <vector>

#include "space.h"

namespace nnjit {
namespace {

thread_local std::string t_err;
thread_local nnjit_tune_stats t_stats{};
thread_local std::vector<std::tuple<int, double, double>> t_trace;

int fail(int code, const char *fmt, ...) {
    char buf[512];
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(buf, sizeof buf, fmt, ap);
    va_end(ap);
    t_err = buf;
    return code;
}

int hip_fail(hipError_t e, const char *what) {
    return fail(NNJIT_EHIP, "%s: %s (%d)", what, hipGetErrorString(e), (int)e);
}

bool env_flag(const char *name) {
    const char *v = getenv(name);
    return v && *v && strcmp(v, "0") != 0;
}
int env_int(const char *name, int dflt) {
    const char *v = getenv(name);
    return (v && *v) ? atoi(v) : dflt;
}

// Environment overrides, read once when the library first initialises a
// device and again by nnjit_cache_clear(), never on the dispatch path.
struct Settings {
    int tune_budget_ms = 900;
    int tune_reps = 3;
    bool tune_runoff = true;
    bool tune_graph = true;
    bool retune = false;
    bool log = false;
    bool trace = false;
    int force_config = -1;
    int fault_config = -1;
    int group_m = 0;
};

Settings read_settings() {
    Settings s;
    s.tune_budget_ms = env_int("NNJIT_TUNE_BUDGET_MS", 900);
    s.tune_reps = std::max(1, env_int("NNJIT_TUNE_REPS", 3));
    s.tune_runoff = env_int("NNJIT_TUNE_RUNOFF", 1) != 0;
    s.tune_graph = env_int("NNJIT_TUNE_GRAPH", 1) != 0;
    s.retune = env_flag("NNJIT_RETUNE");
    s.log = env_flag("NNJIT_LOG");
    s.trace = env_flag("NNJIT_TRACE");
    s.force_config = env_int("NNJIT_FORCE_CONFIG", -1);
    s.fault_config = env_flag("NNJIT_FAULT_CONFIG") ? env_int("NNJIT_FAULT_CONFIG", -1) : -1;
    s.group_m = env_int("NNJIT_GROUP_M", 0);
    return s;
}

// ------------------------------------------------------------ device state

// Split-K partials of the calls on one (device, stream).  A buffer that is
// outgrown is retired, not freed: a HIP graph captured earlier on the stream
// keeps its address and may still be replayed.  Retired buffers are released
// by nnjit_cache_clear() (after a device synchronisation) or at exit.
struct Workspace {
    float *ws = nullptr;
    int64_t ws_floats = 0;
};

struct Device {
    bool ready = false;
    int ordinal = -1;
    nnjit_device_limits limits{};
    std::string arch;
    std::vector<int> regs;    // measured VGPR+AGPR per lane, per variant
    std::vector<int> spills;  // private segment (scratch) > 0, per variant
    void *zero = nullptr;     // 256 zero bytes: load address of out-of-range GEMM elements
    float *fixed_ws = nullptr;  // the allocation-free entry point's split-K scratch (a static device array)
    std::map<hipStream_t, Workspace> workspaces;
    std::vector<float *> retired;   // outgrown split-K buffers (see Workspace)
};

std::mutex g_mu;                  // guards everything below
Settings g_set;                   // valid once any device is ready
bool g_set_loaded = false;
std::map<int, Device> g_devices;
// tuned and default configurations: key (device, kind, dtype, batch, M, N, K)
typedef std::tuple<int, int, int, int64_t, int64_t, int64_t, int64_t> ShapeKey;
struct Tuned {
    int cfg;
    double us;
    std::vector<std::pair<int, double>> ranked;   // up to kRanked (config, us): the registered one, then the fastest others
};
constexpr int kRanked = 5;
constexpr int kRunoff = 6;   // candidates re-timed in the tuner's run-off
std::map<ShapeKey, Tuned> g_tuned;
std::map<ShapeKey, int> g_default;

// Online just-in-time tuning (Sec. 3: a candidate is measured between
// inferences and re-registered when significantly faster).  Per untuned shape:
// the lite space in evaluation order, the configuration serving calls, and at
// most one measurement in flight (its events are read back by a later call).
struct OnlineShape {
    std::vector<int> ids;
    size_t next = 0;
    int registered = -1;
    double registered_us = 1e300;
    int pending = -1;
    hipEvent_t ev[2] = {nullptr, nullptr};
    std::vector<std::pair<int, double>> times;
};
std::map<ShapeKey, OnlineShape> g_online;
bool g_online_on = false;

void online_drop(OnlineShape &o) {
    for (auto &e : o.ev)
        if (e) (void)hipEventDestroy(e);
    o.ev[0] = o.ev[1] = nullptr;
}

int current_device(int *dev) {
    int n = 0;
    hipError_t e = hipGetDeviceCount(&n);
    if (e != hipSuccess || n <= 0) {
        (void)hipGetLastError();
        return fail(NNJIT_EHIP, "no HIP device available (%s)", e == hipSuccess ? "0 devices" : hipGetErrorString(e));
    }
    e = hipGetDevice(dev);
    if (e != hipSuccess) return hip_fail(e, "hipGetDevice");
    return NNJIT_OK;
}

// Initialise the calling thread's current device (under g_mu).
int device_ready(Device **out) {
    int ord = -1;
    int rc = current_device(&ord);
    if (rc != NNJIT_OK) return rc;
    if (!g_set_loaded) {
        g_set = read_settings();
        g_set_loaded = true;
    }
    Device &d = g_devices[ord];
    if (!d.ready) {
        hipDeviceProp_t prop;
        hipError_t e = hipGetDeviceProperties(&prop, ord);
        if (e != hipSuccess) return hip_fail(e, "hipGetDeviceProperties");
        d.ordinal = ord;
        d.arch = prop.gcnArchName;
        d.limits = mi355x_limits();
        d.limits.num_cus = prop.multiProcessorCount;
        d.limits.wave_size = prop.warpSize > 0 ? prop.warpSize : 64;
        if (prop.maxSharedMemoryPerMultiProcessor > 0) d.limits.lds_per_cu = (int64_t)prop.maxSharedMemoryPerMultiProcessor;
        if (prop.sharedMemPerBlock > 0) d.limits.lds_per_wg = (int64_t)prop.sharedMemPerBlock;
        if (prop.maxThreadsPerBlock > 0) d.limits.max_threads_per_wg = prop.maxThreadsPerBlock;
        if (prop.maxThreadsPerMultiProcessor > 0)
            d.limits.max_waves_per_simd =
                std::max(1, prop.maxThreadsPerMultiProcessor / d.limits.wave_size / d.limits.simds_per_cu);
        const int nv = total_variants();
        d.regs.assign(nv, -1);
        d.spills.assign(nv, 0);
        for (const Config &c : configs()) {
            const int gi = variant_index(c.v);
            if (d.regs[gi] >= 0) continue;
            hipFuncAttributes attr;
            e = hipFuncGetAttributes(&attr, c.v->kernel);
            if (e != hipSuccess) return hip_fail(e, "hipFuncGetAttributes");
            d.regs[gi] = attr.numRegs;
            d.spills[gi] = attr.localSizeBytes > 0 ? 1 : 0;
        }
        // the zero block and the fixed scratch are static device arrays:
        // their addresses on this device, taken once (nothing is allocated)
        void *fixed = nullptr;
        e = static_buffer_addresses(&fixed, &d.zero);
        if (e != hipSuccess) return hip_fail(e, "hipGetSymbolAddress");
        d.fixed_ws = (float *)fixed;
        d.ready = true;
    }
    *out = &d;
    return NNJIT_OK;
}

// Split-K scratch for (device, stream); grown on demand (under g_mu).  The
// outgrown buffer is retired, not freed: launches still queued on the stream
// and graphs captured on it keep using it, so growing needs no wait.
int workspace_for(Device &d, hipStream_t stream, int64_t ws_floats, float **out) {
    Workspace &w = d.workspaces[stream];
    if (w.ws_floats < ws_floats) {
        // allocating is not allowed while the stream is being captured:
        // refuse instead of breaking the capture
        hipStreamCaptureStatus cap = hipStreamCaptureStatusNone;
        if (hipStreamIsCapturing(stream, &cap) != hipSuccess) (void)hipGetLastError();
        if (cap != hipStreamCaptureStatusNone)
            return fail(NNJIT_EHIP, "split-K scratch of %lld floats needed while the stream is being captured; "
                                    "run this shape once on the stream outside capture first", (long long)ws_floats);
        const int64_t nf = std::max(w.ws_floats, ws_floats + ws_floats / 4);
        float *fresh = nullptr;
        hipError_t e = hipMalloc((void **)&fresh, (size_t)std::max<int64_t>(nf, 1) * sizeof(float));
        if (e != hipSuccess) {
            (void)hipGetLastError();
            return fail(NNJIT_ENOMEM, "split-K scratch of %lld floats", (long long)nf);
        }
        if (w.ws) d.retired.push_back(w.ws);
        w.ws = fresh;
        w.ws_floats = nf;
    }
    *out = w.ws;
    return NNJIT_OK;
}

// --------------------------------------------------------------- validation

struct Call {
    int64_t batch, M, N, K;
    const void *A;
    int64_t lda, sA;
    const void *B;
    int64_t ldb, sB;
    void *C;
    int64_t ldc, sC;
    int dtype;
    hipStream_t stream;
    // 4-bit GEMV (q4 = true): A = x, B = the code words [N][ldq] (ldb = ldq),
    // Sc = the scales [N][lds], batch = the group size, M = 1
    bool q4 = false;
    const void *Sc = nullptr;
    int64_t lds = 0;
};

int validate_q4(const Call &c) {
    if (c.N < 0 || c.K < 0) return fail(NNJIT_EINVAL, "negative dimension (N=%lld K=%lld)", (long long)c.N, (long long)c.K);
    if (c.N > INT32_MAX || c.K > INT32_MAX) return fail(NNJIT_EINVAL, "dimension above 2^31-1");
    if (c.batch < 1 || c.batch > INT32_MAX) return fail(NNJIT_EINVAL, "group=%lld must be in [1, 2^31)", (long long)c.batch);
    if (c.ldb < (c.K + 7) / 8) return fail(NNJIT_EINVAL, "ldq=%lld < ceil(K/8)=%lld", (long long)c.ldb, (long long)((c.K + 7) / 8));
    if (c.lds < (c.K + c.batch - 1) / c.batch)
        return fail(NNJIT_EINVAL, "lds=%lld < ceil(K/group)=%lld", (long long)c.lds, (long long)((c.K + c.batch - 1) / c.batch));
    if (c.N > 0) {
        if (c.K > 0 && (!c.A || !c.B || !c.Sc)) return fail(NNJIT_EINVAL, "x, Wq or scales is NULL");
        if (!c.C) return fail(NNJIT_EINVAL, "y is NULL");
    }
    return NNJIT_OK;
}

int validate(const Call &c) {
    if (c.q4) return validate_q4(c);
    if (c.dtype != NNJIT_F32 && c.dtype != NNJIT_F16) return fail(NNJIT_EDTYPE, "unknown dtype %d", c.dtype);
    if (c.batch < 0 || c.M < 0 || c.N < 0 || c.K < 0)
        return fail(NNJIT_EINVAL, "negative dimension (batch=%lld M=%lld N=%lld K=%lld)", (long long)c.batch,
                    (long long)c.M, (long long)c.N, (long long)c.K);
    if (c.M > INT32_MAX || c.N > INT32_MAX || c.K > INT32_MAX || c.batch > INT32_MAX)
        return fail(NNJIT_EINVAL, "dimension above 2^31-1");
    if (c.lda < std::max<int64_t>(1, c.K)) return fail(NNJIT_EINVAL, "lda=%lld < max(1,K=%lld)", (long long)c.lda, (long long)c.K);
    if (c.ldb < std::max<int64_t>(1, c.N)) return fail(NNJIT_EINVAL, "ldb=%lld < max(1,N=%lld)", (long long)c.ldb, (long long)c.N);
    if (c.ldc < std::max<int64_t>(1, c.N)) return fail(NNJIT_EINVAL, "ldc=%lld < max(1,N=%lld)", (long long)c.ldc, (long long)c.N);
    if (c.sA < 0 || c.sB < 0 || c.sC < 0) return fail(NNJIT_EINVAL, "negative batch stride");
    if (c.batch > 0) {
        if (c.M * c.K > 0 && !c.A) return fail(NNJIT_EINVAL, "A is NULL");
        if (c.K * c.N > 0 && !c.B) return fail(NNJIT_EINVAL, "B is NULL");
        if (c.M * c.N > 0 && !c.C) return fail(NNJIT_EINVAL, "C is NULL");
    }
    return NNJIT_OK;
}

bool is_noop(const Call &c) { return c.batch == 0 || c.M == 0 || c.N == 0; }

int kind_of(const Call &c) {
    if (c.q4) return NNJIT_KIND_GEMV_Q4;
    if (c.batch == 1 && c.M == 1) return NNJIT_KIND_GEMV;
    return c.batch == 1 ? NNJIT_KIND_GEMM : NNJIT_KIND_BATCHED;
}

// Can a vector-load (16-byte) configuration run these operands?
bool vec_aligned(const Call &c, bool gemv) {
    const int V = vec_elems(c.dtype);
    const int elt = c.dtype == NNJIT_F16 ? 2 : 4;
    auto al = [](const void *p) { return ((uintptr_t)p & 15u) == 0; };
    if (c.N % V || c.ldb % V || !al(c.B) || (c.batch > 1 && c.sB % V)) return false;
    if (gemv) return true;  // x is read element by element
    (void)elt;
    return c.K % V == 0 && c.lda % V == 0 && al(c.A) && (c.batch <= 1 || c.sA % V == 0);
}

// Can a 16-byte-load 4-bit GEMV configuration run these operands?
bool vec_aligned_q4(const Call &c) {
    auto al = [](const void *p) { return ((uintptr_t)p & 15u) == 0; };
    return c.batch % 32 == 0 && c.ldb % 4 == 0 && al(c.B) && al(c.A);
}

// vector-load eligibility for the family a call runs on
bool aligned_for(int kind, const Call &c) {
    if (kind == NNJIT_KIND_GEMV_Q4) return vec_aligned_q4(c);
    return vec_aligned(c, kind == NNJIT_KIND_GEMV);
}

// ------------------------------------------------------------------ launch

// Tile rows per group of a GEMM's tile order (see tile_of in kcommon.h): the
// ~tiles/8 consecutive tiles that one XCD holds form a block of G rows by
// about tiles/(8 G) columns; G is the largest power of two with G^2 <= that
// run, so the block is near square and its A rows plus B columns are fewest.
int tile_group_rows(int tiles_m, int tiles_n, int override_rows) {
    const int ov = override_rows;
    if (ov > 0) return std::min(ov, std::max(tiles_m, 1));
    const int64_t run = ((int64_t)tiles_m * tiles_n + 7) / 8;
    int G = 1;
    while ((int64_t)(2 * G) * (2 * G) <= run) G *= 2;
    return std::max(1, std::min(G, tiles_m));
}

// Launch geometry of a configuration on this device (a stream-K
// configuration launches one workgroup per resident slot).
Geometry geom(const Device &d, const Config &cfg, int64_t batch, int64_t M, int64_t N, int64_t K) {
    int64_t sk = 0;
    if (cfg.split == kStreamK && !family_is_gemv(cfg.v->family) && !family_is_q4(cfg.v->family)) {
        const int gi = variant_index(cfg.v);
        const int regs = gi < (int)d.regs.size() ? d.regs[gi] : -1;
        sk = (int64_t)d.limits.num_cus * std::max(1, resources_of(*cfg.v, d.limits, regs).wg_per_cu);
    }
    return geometry_of(cfg, batch, M, N, K, sk);
}

// Launch one configuration on c.stream.  ws: split-K partial storage of at
// least the geometry's ws_floats floats (unused when the split is 1).  Needs
// no lock: it reads only the device's constant zero buffer.
int launch(const Device &d, const Config &cfg, const Call &c, float *ws, const Settings &s) {
    if (s.fault_config >= 0 && s.fault_config == cfg.id)
        return fail(NNJIT_EHIP, "config %d: launch failure injected by NNJIT_FAULT_CONFIG", cfg.id);
    const Variant &v = *cfg.v;
    const Geometry g = geom(d, cfg, c.batch, c.M, c.N, c.K);
    if (g.ws_floats > 0 && !ws) return fail(NNJIT_EINVAL, "config %d needs split-K scratch", cfg.id);
    hipError_t e = hipSuccess;
    if (family_is_q4(v.family)) {
        GemvQ4Params p{};
        p.x = c.A;
        p.Wq = c.B;
        p.S = c.Sc;
        p.y = (float *)c.C;
        p.ldq = c.ldb;
        p.lds = c.lds;
        p.K = (int)c.K;
        p.N = (int)c.N;
        p.G = (int)g.group;
        e = v.launch(&p, dim3((unsigned)g.wgs), c.stream);
    } else if (!family_is_gemv(v.family)) {
        GemmParams p{};
        p.lda = c.lda;
        p.ldb = c.ldb;
        p.ldc = c.ldc;
        p.sA = c.sA;
        p.sB = c.sB;
        p.sC = c.sC;
        p.M = (int)c.M;
        p.N = (int)c.N;
        p.K = (int)c.K;
        p.S = g.split;
        p.kchunk = g.kchunk;
        p.tiles_m = g.tiles_m;
        p.tiles_n = g.tiles_n;
        p.group_m = tile_group_rows(g.tiles_m, g.tiles_n, s.group_m);
        p.ws = ws;
        p.zero = d.zero;
        if (g.stream_k) {
            p.A = c.A;
            p.B = c.B;
            p.C = (float *)c.C;
            p.batch = 1;
            p.sk_wgs = (int)g.wgs;
            p.nslab = g.nslab;
            p.units = g.units;
            e = v.launch(&p, dim3((unsigned)g.wgs), c.stream);
            if (e == hipSuccess) e = launch_streamk_fixup(p, v.mt, v.nt, c.stream);
            if (e != hipSuccess) return hip_fail(e, v.name);
            return NNJIT_OK;
        }
        const int64_t gx = (int64_t)g.tiles_m * g.tiles_n * g.split;
        // the kernels number workgroups (x + gx * z) in 32-bit integers
        if (gx * std::min<int64_t>(c.batch, 65535) > INT32_MAX)
            return fail(NNJIT_EINVAL, "%lld workgroups per launch exceed 2^31-1; split the batch or the matrix",
                        (long long)(gx * std::min<int64_t>(c.batch, 65535)));
        const int elt = c.dtype == NNJIT_F16 ? 2 : 4;
        for (int64_t b0 = 0; b0 < c.batch && e == hipSuccess; b0 += 65535) {
            const int64_t nb = std::min<int64_t>(65535, c.batch - b0);
            p.A = (const char *)c.A + b0 * c.sA * elt;
            p.B = (const char *)c.B + b0 * c.sB * elt;
            p.C = (float *)c.C + b0 * c.sC;
            p.batch = (int)nb;
            e = v.launch(&p, dim3((unsigned)gx, 1, (unsigned)nb), c.stream);
            if (e == hipSuccess && g.split > 1)
                e = launch_splitk_reduce(p.ws, g.split, (int)nb, p.M, p.N, p.C, c.ldc, c.sC, c.stream);
        }
    } else {
        GemvParams p{};
        p.x = c.A;
        p.W = c.B;
        p.y = (float *)c.C;
        p.ldw = c.ldb;
        p.K = (int)c.K;
        p.N = (int)c.N;
        p.S = cfg.split;
        p.kchunk = g.kchunk;
        p.segs = g.tiles_n;
        p.ws = ws;
        e = v.launch(&p, dim3((unsigned)g.wgs), c.stream);
        if (e == hipSuccess && cfg.split > 1) e = launch_splitk_reduce(p.ws, cfg.split, 1, 1, p.N, p.y, p.N, 0, c.stream);
    }
    if (e != hipSuccess) return hip_fail(e, v.name);
    return NNJIT_OK;
}

// Launch on the caller's stream with that stream's split-K scratch (under g_mu).
int launch_on_stream(Device &d, const Config &cfg, const Call &c) {
    const Geometry g = geom(d, cfg, c.batch, c.M, c.N, c.K);
    float *ws = nullptr;
    if (g.ws_floats > 0) {
        const int rc = workspace_for(d, c.stream, g.ws_floats, &ws);
        if (rc != NNJIT_OK) return rc;
    }
    return launch(d, cfg, c, ws, g_set);
}

// First non-vector configuration of a family with split 1 (GEMM) or the split
// that best fills the chip (GEMV): serves operands that are not 16-byte aligned.
const Config *fallback_config(int family, const Call &c, const Device &d) {
    const Config *best = nullptr;
    for (const Config &cfg : configs()) {
        if (cfg.v->family != family || cfg.v->vec_bytes == 16) continue;
        if (family_is_q4(family)) {
            // the word-load configuration with the most workgroups that still
            // fill at most two per CU (else the one with the most)
            const Geometry g = geometry_of(cfg, c.batch, c.M, c.N, c.K);
            if (!best || g.wgs >= 2LL * d.limits.num_cus) best = &cfg;
            continue;
        }
        if (!family_is_gemv(family)) {
            if (cfg.split == 1) return &cfg;
            continue;
        }
        const Geometry g = geometry_of(cfg, c.batch, c.M, c.N, c.K);
        if (g.kchunk < cfg.v->kt && cfg.split > 1) continue;
        if (!best || g.wgs <= 2LL * d.limits.num_cus) best = &cfg;
    }
    return best;
}

ShapeKey key_of(int dev, int kind, const Call &c) {
    return ShapeKey(dev, kind, c.dtype, c.batch, c.M, c.N, c.K);
}

Shape shape_of(int kind, const Call &c) { return Shape{kind, c.dtype, c.batch, c.M, c.N, c.K}; }

// Default configuration of a shape: first of its lite space (memoised).
int default_config(Device &d, int kind, const Call &c) {
    const ShapeKey k = key_of(d.ordinal, kind, c);
    auto it = g_default.find(k);
    if (it != g_default.end()) return it->second;
    LiteResult lr = lite_space(shape_of(kind, c), d.limits, &d.regs, &d.spills);
    if (lr.ids.empty()) return fail(NNJIT_ENOCFG, "no configuration fits this shape");
    g_default[k] = lr.ids[0];
    return lr.ids[0];
}

// One call on a shape that is being tuned online (caller holds g_mu).
int online_call(Device &d, int kind, const ShapeKey &key, const Call &c) {
    auto it = g_online.find(key);
    if (it == g_online.end()) {
        LiteResult lr = lite_space(shape_of(kind, c), d.limits, &d.regs, &d.spills);
        if (lr.ids.empty()) return fail(NNJIT_ENOCFG, "no configuration fits this shape");
        OnlineShape o;
        o.ids = lr.ids;
        o.registered = lr.ids[0];
        it = g_online.emplace(key, std::move(o)).first;
    }
    OnlineShape &o = it->second;
    hipError_t e;
    // collect the measurement in flight, if its events have completed
    if (o.pending >= 0) {
        e = hipEventQuery(o.ev[1]);
        if (e == hipSuccess) {
            float ms = 0.f;
            if (hipEventElapsedTime(&ms, o.ev[0], o.ev[1]) == hipSuccess) {
                const double us = ms * 1e3;
                o.times.emplace_back(o.pending, us);
                if (o.pending == o.registered) {
                    o.registered_us = us;
                } else if (us < o.registered_us / 1.03) {   // significantly faster: re-register
                    o.registered = o.pending;
                    o.registered_us = us;
                }
            }
            o.pending = -1;
        } else if (e != hipErrorNotReady) {
            (void)hipGetLastError();
            o.pending = -1;
        }
    }
    // every candidate measured: the shape becomes a tuned shape
    if (o.pending < 0 && o.next >= o.ids.size()) {
        Tuned tu{o.registered, o.registered_us, {{o.registered, o.registered_us}}};
        std::vector<std::pair<double, int>> by_time;
        for (const auto &t : o.times)
            if (t.first != o.registered && t.second < 1e299) by_time.emplace_back(t.second, t.first);
        std::sort(by_time.begin(), by_time.end());
        for (const auto &bt : by_time)
            if ((int)tu.ranked.size() < kRanked) tu.ranked.emplace_back(bt.second, bt.first);
        const int id = o.registered;
        online_drop(o);
        g_online.erase(it);
        g_tuned[key] = tu;
        const Config &cfg = configs()[id];
        if (cfg.v->vec_bytes == 16 && !aligned_for(kind, c)) {
            const Config *fb = fallback_config(family_of(kind, c.dtype), c, d);
            if (!fb) return fail(NNJIT_ENOCFG, "no element-load fallback configuration");
            return launch_on_stream(d, *fb, c);
        }
        return launch_on_stream(d, cfg, c);
    }
    // measure the next candidate on this call, unless measuring is off, one is
    // still in flight, the stream is being captured or the operands need the
    // element-load path
    hipStreamCaptureStatus cap = hipStreamCaptureStatusNone;
    (void)hipStreamIsCapturing(c.stream, &cap);
    const bool aligned = aligned_for(kind, c);
    if (g_online_on && o.pending < 0 && cap == hipStreamCaptureStatusNone && aligned) {
        if (!o.ev[0]) {
            if ((e = hipEventCreate(&o.ev[0])) != hipSuccess || (e = hipEventCreate(&o.ev[1])) != hipSuccess)
                return hip_fail(e, "hipEventCreate");
        }
        const int cand = o.ids[o.next++];
        (void)hipEventRecord(o.ev[0], c.stream);
        const int rc = launch_on_stream(d, configs()[cand], c);
        if (rc == NNJIT_OK) {
            (void)hipEventRecord(o.ev[1], c.stream);
            o.pending = cand;
            return NNJIT_OK;
        }
        // a candidate that cannot launch is recorded as failed (never timed,
        // never registered) and this call's product is computed by the
        // registered configuration below
        (void)hipGetLastError();
        o.times.emplace_back(cand, 1e300);
    }
    const Config *cfg = &configs()[o.registered];
    if (cfg->v->vec_bytes == 16 && !aligned) {
        cfg = fallback_config(family_of(kind, c.dtype), c, d);
        if (!cfg) return fail(NNJIT_ENOCFG, "no element-load fallback configuration");
    }
    t_err.clear();
    return launch_on_stream(d, *cfg, c);
}

int run(const Call &c, int forced) {
    int rc = validate(c);
    if (rc != NNJIT_OK) return rc;
    if (forced >= 0) {
        if (forced >= (int)configs().size()) return fail(NNJIT_EINVAL, "config id %d out of range", forced);
        const Config &cfg = configs()[forced];
        if (family_is_q4(cfg.v->family) != c.q4)
            return fail(NNJIT_EINVAL, "config %d is %s, %s", forced, family_name(cfg.v->family),
                        c.q4 ? "not a 4-bit GEMV configuration" : "a 4-bit GEMV configuration");
        if (family_dtype(cfg.v->family) != c.dtype)
            return fail(NNJIT_EINVAL, "config %d is %s, not dtype %d", forced, family_name(cfg.v->family), c.dtype);
        if (family_is_gemv(cfg.v->family) && !(c.batch <= 1 && c.M <= 1))
            return fail(NNJIT_EINVAL, "config %d is a GEMV configuration (needs batch == 1, M == 1)", forced);
        const bool al = c.q4 ? vec_aligned_q4(c) : vec_aligned(c, family_is_gemv(cfg.v->family));
        if (cfg.v->vec_bytes == 16 && !is_noop(c) && !al)
            return fail(NNJIT_EINVAL, "config %d needs 16-byte aligned operands", forced);
    }
    if (is_noop(c)) return NNJIT_OK;
    std::lock_guard<std::mutex> lk(g_mu);
    Device *d = nullptr;
    rc = device_ready(&d);
    if (rc != NNJIT_OK) return rc;
    const Config *cfg = nullptr;
    if (forced >= 0) {
        cfg = &configs()[forced];
    } else {
        const int kind = kind_of(c);
        int id = -1;
        const int env_force = g_set.force_config;
        if (env_force >= 0 && env_force < (int)configs().size() &&
            configs()[env_force].v->family == family_of(kind, c.dtype))
            id = env_force;
        if (id < 0) {
            const ShapeKey key = key_of(d->ordinal, kind, c);
            auto it = g_tuned.find(key);
            if (it != g_tuned.end()) {
                id = it->second.cfg;
            } else if (g_online_on || g_online.count(key)) {
                return online_call(*d, kind, key, c);
            } else {
                id = default_config(*d, kind, c);
                if (id < 0) return id;
            }
        }
        cfg = &configs()[id];
        if (cfg->v->vec_bytes == 16 && !aligned_for(kind, c)) {
            cfg = fallback_config(family_of(kind, c.dtype), c, *d);
            if (!cfg) return fail(NNJIT_ENOCFG, "no element-load fallback configuration");
        }
    }
    return launch_on_stream(*d, *cfg, c);
}

// The allocation-free variant of run(): the configuration nnjit_matmul /
// nnjit_batched_matmul would use (online shapes are served by their
// registered configuration without measuring), with split-K partials in the
// device's fixed static scratch.  Makes no allocating call once the device
// is initialised (initialisation itself only takes the static arrays'
// addresses).
int run_noalloc(const Call &c) {
    int rc = validate(c);
    if (rc != NNJIT_OK) return rc;
    if (is_noop(c)) return NNJIT_OK;
    std::lock_guard<std::mutex> lk(g_mu);
    Device *d = nullptr;
    rc = device_ready(&d);
    if (rc != NNJIT_OK) return rc;
    const int kind = kind_of(c);
    int id = -1;
    const int env_force = g_set.force_config;
    if (env_force >= 0 && env_force < (int)configs().size() && configs()[env_force].v->family == family_of(kind, c.dtype))
        id = env_force;
    if (id < 0) {
        const ShapeKey key = key_of(d->ordinal, kind, c);
        auto it = g_tuned.find(key);
        auto on = g_online.find(key);
        if (it != g_tuned.end()) id = it->second.cfg;
        else if (on != g_online.end()) id = on->second.registered;
        else id = default_config(*d, kind, c);
        if (id < 0) return id;
    }
    const Config *cfg = &configs()[id];
    if (cfg->v->vec_bytes == 16 && !aligned_for(kind, c)) {
        cfg = fallback_config(family_of(kind, c.dtype), c, *d);
        if (!cfg) return fail(NNJIT_ENOCFG, "no element-load fallback configuration");
    }
    const Geometry g = geom(*d, *cfg, c.batch, c.M, c.N, c.K);
    if ((size_t)g.ws_floats * sizeof(float) > kNoAllocScratchBytes)
        return fail(NNJIT_ENOMEM, "configuration %d (%s, split %d) needs %lld bytes of split-K scratch, above the "
                                  "%zu bytes of the fixed scratch; use nnjit_batched_matmul",
                    cfg->id, cfg->v->name, cfg->split, (long long)g.ws_floats * (long long)sizeof(float),
                    kNoAllocScratchBytes);
    return launch(*d, *cfg, c, d->fixed_ws, g_set);
}

// -------------------------------------------------------------------- tuner

double median(std::vector<float> v) {
    std::sort(v.begin(), v.end());
    const size_t n = v.size();
    return n % 2 ? v[n / 2] : 0.5 * (v[n / 2 - 1] + v[n / 2]);
}

// Device resources that one tune call owns -- its stream, the operand scratch
// of the tuned shape and the split-K scratch of its candidates -- released
// before the call returns.
struct TuneResources {
    hipStream_t stream = nullptr;
    void *scratch = nullptr;
    float *ws = nullptr;
    std::vector<hipEvent_t> events;
    ~TuneResources() {
        if (stream) (void)hipStreamSynchronize(stream);
        for (hipEvent_t e : events) (void)hipEventDestroy(e);
        if (scratch) (void)hipFree(scratch);
        if (ws) (void)hipFree(ws);
        if (stream) (void)hipStreamDestroy(stream);
        (void)hipGetLastError();
    }
    hipError_t event(hipEvent_t *out) {
        hipError_t e = hipEventCreate(out);
        if (e == hipSuccess) events.push_back(*out);
        return e;
    }
};

// The tuner's operand values follow the workloads' recipe (activations
// N(0, 1), weights N(0, 0.02)): matrix-core time depends somewhat on the data.
constexpr float kActScale = 1.0f, kWeightScale = 0.02f;

int tune(int kind, int dtype, int64_t batch, int64_t M, int64_t N, int64_t K) {
    using clock = std::chrono::steady_clock;
    auto ms_since = [&](clock::time_point t) {
        return std::chrono::duration<double, std::milli>(clock::now() - t).count();
    };
    t_stats = nnjit_tune_stats{};
    t_stats.chosen = -1;
    t_trace.clear();
    const int elt = dtype == NNJIT_F16 ? 2 : 4;
    const bool q4 = kind == NNJIT_KIND_GEMV_Q4;
    Call c{batch, M, N, K, nullptr, std::max<int64_t>(1, K), M * K, nullptr, std::max<int64_t>(1, N), K * N,
           nullptr, std::max<int64_t>(1, N), M * N, dtype, nullptr};
    if (q4) {
        // 4-bit GEMV scratch layout: rows of ceil(K/8) words padded to 16
        // bytes, rows of ceil(K/G) scales
        c.q4 = true;
        c.ldb = ((K + 7) / 8 + 3) / 4 * 4;
        c.lds = std::max<int64_t>(1, (K + batch - 1) / batch);
    }
    if (dtype != NNJIT_F32 && dtype != NNJIT_F16) return fail(NNJIT_EDTYPE, "unknown dtype %d", dtype);
    if (batch < 1 || M < 1 || N < 1 || K < 0) return fail(NNJIT_EINVAL, "tune needs batch, M, N >= 1 and K >= 0");
    if (M > INT32_MAX || N > INT32_MAX || K > INT32_MAX || batch > INT32_MAX)
        return fail(NNJIT_EINVAL, "dimension above 2^31-1");

    // Under the lock: the device, the settings, the cache lookup and the lite
    // space.  Candidates are then timed without it (on this call's own stream
    // and scratch), so calls on other threads and streams are not held up;
    // the lock is taken again only to register the result.
    Device *d = nullptr;
    Settings set;
    clock::time_point t0;
    ShapeKey key;
    LiteResult lr;
    int cached = -1;
    {
        std::lock_guard<std::mutex> lk(g_mu);
        int rc = device_ready(&d);
        if (rc != NNJIT_OK) return rc;
        set = g_set;
        t0 = clock::now();  // one-time library initialisation is not tune time
        key = key_of(d->ordinal, kind, c);
        auto hit = g_tuned.find(key);
        if (hit != g_tuned.end() && !set.retune) {
            t_stats.cache_hit = 1;
            t_stats.chosen = hit->second.cfg;
            t_stats.best_us = hit->second.us;
            t_stats.wall_ms = ms_since(t0);
            return hit->second.cfg;
        }
        if (hit != g_tuned.end()) cached = hit->second.cfg;
        lr = lite_space(shape_of(kind, c), d->limits, &d->regs, &d->spills);
    }
    t_stats.n_enumerated = lr.n_enumerated;
    t_stats.n_lite = (int)lr.ids.size();
    if (lr.ids.empty()) return fail(NNJIT_ENOCFG, "no configuration fits this shape");
    const int limit = std::min<int>((int)lr.ids.size(), kMaxTimed);
    // the registered kernel this tune competes with: the cached one, else the default
    const int incumbent = cached >= 0 ? cached : lr.ids[0];

    // scratch operands of this exact shape, filled on the device.  A GEMV is
    // bandwidth bound and runs on weights streamed from HBM, so it is timed
    // that way: its weight operand rotates over enough copies (>= 512 MiB
    // together) that the 256 MB last-level cache cannot hold them.
    // (4-bit GEMV: x [K] fp16; per copy the code words [N][ldq] followed by
    // the scales [N][lds]; y [N])
    const size_t q4_codes = q4 ? (size_t)(N * c.ldb) * 4 : 0;
    const size_t a_bytes = q4 ? (size_t)K * 2 : (size_t)(batch * M * K) * elt;
    const size_t b_bytes = q4 ? ((q4_codes + 255) & ~(size_t)255) + (size_t)(N * c.lds) * 2
                              : (size_t)(batch * K * N) * elt;
    const size_t c_bytes = q4 ? (size_t)N * 4 : (size_t)(batch * M * N) * 4;
    auto up = [](size_t x) { return (x + 255) & ~(size_t)255; };
    const size_t kColdBytes = (size_t)512 << 20;
    const int b_copies = (kind == NNJIT_KIND_GEMV || q4)
                             ? (int)std::min<size_t>(16, std::max<size_t>(1, (kColdBytes + up(b_bytes) - 1) / up(b_bytes)))
                             : 1;
    const size_t need = up(a_bytes) + (size_t)b_copies * up(b_bytes) + up(c_bytes);
    int64_t ws_floats = 0;
    for (int i = 0; i < limit; ++i)
        ws_floats = std::max(ws_floats, geom(*d, configs()[lr.ids[i]], batch, M, N, K).ws_floats);

    TuneResources res;
    hipError_t e = hipStreamCreateWithFlags(&res.stream, hipStreamNonBlocking);
    if (e != hipSuccess) return hip_fail(e, "hipStreamCreate");
    if ((e = hipMalloc(&res.scratch, need)) != hipSuccess) {
        (void)hipGetLastError();
        return fail(NNJIT_ENOMEM, "tuner scratch of %zu bytes", need);
    }
    if (ws_floats > 0 && (e = hipMalloc((void **)&res.ws, (size_t)ws_floats * sizeof(float))) != hipSuccess) {
        (void)hipGetLastError();
        return fail(NNJIT_ENOMEM, "tuner split-K scratch of %lld floats", (long long)ws_floats);
    }
    char *base = (char *)res.scratch;
    char *b0 = base + up(a_bytes);
    c.A = base;
    c.B = b0;
    c.C = b0 + (size_t)b_copies * up(b_bytes);
    c.stream = res.stream;
    if ((e = launch_fill((void *)c.A, q4 ? K : batch * M * K, dtype == NNJIT_F16 ? FILL_F16 : FILL_F32, kActScale,
                         1234u, c.stream)) != hipSuccess)
        return hip_fail(e, "scratch fill");
    for (int i = 0; i < b_copies; ++i) {
        char *dst = b0 + (size_t)i * up(b_bytes);
        // 4-bit codes: any word is valid, so they are random words; the
        // scales follow as fp16 (their sign does not matter to the timing)
        e = q4 ? launch_fill(dst, N * c.ldb, FILL_WORDS, 0.f, 5678u + i, c.stream)
               : launch_fill(dst, batch * K * N, dtype == NNJIT_F16 ? FILL_F16 : FILL_F32, kWeightScale, 5678u + i,
                             c.stream);
        if (e == hipSuccess && q4) e = launch_fill(dst + up(q4_codes), N * c.lds, FILL_F16, 0.006f, 9012u + i, c.stream);
        if (e != hipSuccess) return hip_fail(e, "scratch fill");
    }
    int rot = 0;
    auto launch_next = [&](const Config &cfg) {   // next weight copy, then launch
        c.B = b0 + (size_t)(rot % b_copies) * up(b_bytes);
        if (q4) c.Sc = (const char *)c.B + up(q4_codes);
        ++rot;
        return launch(*d, cfg, c, res.ws, set);
    };

    // A burst of n launches captured as a graph on the tuner's stream, so that
    // its replay measures device time per launch even when one launch takes
    // less time on the device than on the host (a few-microsecond kernel
    // launched eagerly measures the host's launch rate).  nullptr when the
    // capture fails; the caller then launches eagerly.
    auto capture_burst = [&](const Config &cfg, int n) -> hipGraphExec_t {
        if (!set.tune_graph) return nullptr;
        if (hipStreamBeginCapture(c.stream, hipStreamCaptureModeThreadLocal) != hipSuccess) {
            (void)hipGetLastError();
            return nullptr;
        }
        bool ok = true;
        for (int b = 0; b < n && ok; ++b) ok = launch_next(cfg) == NNJIT_OK;
        hipGraph_t g = nullptr;
        const hipError_t ee = hipStreamEndCapture(c.stream, &g);
        hipGraphExec_t x = nullptr;
        if (!(ok && ee == hipSuccess && g && hipGraphInstantiate(&x, g, nullptr, nullptr, 0) == hipSuccess &&
              hipGraphUpload(x, c.stream) == hipSuccess)) {
            if (x) (void)hipGraphExecDestroy(x);
            x = nullptr;
            (void)hipGetLastError();
        }
        if (g) (void)hipGraphDestroy(g);
        return x;
    };

    const int reps = set.tune_reps;
    const double budget_ms = (double)set.tune_budget_ms;
    const bool trace = set.trace;
    std::vector<hipEvent_t> ev(2 * (reps + 1));
    for (auto &x : ev)
        if ((e = res.event(&x)) != hipSuccess) return hip_fail(e, "hipEventCreate");

    // A candidate's cost is the device time per launch of a burst of
    // back-to-back launches (what a stream or a graph of dependent products
    // pays), not the host-visible latency of one launch. The burst length is
    // fixed per shape from the first candidate's single launch so that all
    // candidates are compared on the same measure.
    int burst = 0;
    const auto te = clock::now();
    int best = -1;
    double best_us = 1e300, best_first_us = 1e300;
    std::map<int, double> timed;
    for (int i = 0; i < limit; ++i) {
        if (ms_since(te) > budget_ms) break;
        const Config &cfg = configs()[lr.ids[i]];
        // warm-up launch (untimed: the first launch of a kernel pays one-time
        // costs), then one single timed launch that decides the early abort
        int rc = launch_next(cfg);
        if (rc == NNJIT_OK) {
            (void)hipEventRecord(ev[0], c.stream);
            rc = launch_next(cfg);
            (void)hipEventRecord(ev[1], c.stream);
        }
        if (rc != NNJIT_OK) {
            ++t_stats.n_failed;
            t_trace.emplace_back(cfg.id, -1.0, ms_since(t0));
            (void)hipGetLastError();
            continue;
        }
        if ((e = hipEventSynchronize(ev[1])) != hipSuccess) return hip_fail(e, "candidate warm-up");
        float first_ms = 0.f;
        (void)hipEventElapsedTime(&first_ms, ev[0], ev[1]);
        const double first_us = first_ms * 1e3;
        // ~500 us of device work per burst (1 .. 64 launches), so that the
        // fixed cost of launching the burst's graph is a small share of it
        if (burst == 0) burst = std::min(64, std::max(1, (int)std::ceil(500.0 / std::max(first_us, 0.5))));
        if (best >= 0 && first_us > 1.5 * best_first_us) {
            ++t_stats.n_aborted;
            t_trace.emplace_back(cfg.id, -1.0, ms_since(t0));
            if (trace) fprintf(stderr, "[nnjit] tune cand %d %s S=%d first %.1f us > 1.5x best, dropped\n", cfg.id, cfg.v->name, cfg.split, first_us);
            continue;
        }
        // one graph per repetition, so each replays a fresh run of the
        // rotating weight copies (cold, as eager launches would be)
        std::vector<hipGraphExec_t> gx(reps, nullptr);
        for (int r = 0; r < reps; ++r) gx[r] = capture_burst(cfg, burst);
        const bool graphs = std::all_of(gx.begin(), gx.end(), [](hipGraphExec_t x) { return x != nullptr; });
        auto drop_graphs = [&]() {
            for (auto &x : gx)
                if (x) (void)hipGraphExecDestroy(x);
        };
        bool ok = true;
        for (int r = 0; r < reps && ok; ++r) {
            (void)hipEventRecord(ev[2 + 2 * r], c.stream);
            if (graphs) ok = hipGraphLaunch(gx[r], c.stream) == hipSuccess;
            else
                for (int b = 0; b < burst && ok; ++b) ok = launch_next(cfg) == NNJIT_OK;
            (void)hipEventRecord(ev[3 + 2 * r], c.stream);
        }
        if (!ok) {
            ++t_stats.n_failed;
            t_trace.emplace_back(cfg.id, -1.0, ms_since(t0));
            (void)hipGetLastError();
            (void)hipStreamSynchronize(c.stream);
            drop_graphs();
            continue;
        }
        if ((e = hipEventSynchronize(ev[1 + 2 * reps])) != hipSuccess) {
            drop_graphs();
            return hip_fail(e, "candidate timing");
        }
        drop_graphs();
        std::vector<float> ts(reps);
        for (int r = 0; r < reps; ++r) (void)hipEventElapsedTime(&ts[r], ev[2 + 2 * r], ev[3 + 2 * r]);
        const double us = median(ts) * 1e3 / burst;
        ++t_stats.n_timed;
        timed[cfg.id] = us;
        if (i == 0) t_stats.default_us = us;
        t_trace.emplace_back(cfg.id, us, ms_since(t0));
        if (trace) fprintf(stderr, "[nnjit] tune cand %d %s S=%d %.2f us (single %.2f us)\n", cfg.id, cfg.v->name, cfg.split, us, first_us);
        if (us < best_us) {
            best_us = us;
            best = cfg.id;
        }
        best_first_us = std::min(best_first_us, first_us);
    }
    if (best < 0) return fail(NNJIT_ENOCFG, "every candidate failed");

    // Run-off: the candidates within 15% of the best (at most kRunoff) are
    // timed again with bursts of >= ~500 us, taking turns over several
    // rounds so that clock drift reaches them alike; each keeps the median
    // of its rounds.  Short bursts of a few-microsecond kernel cannot tell
    // such candidates apart.
    if (set.tune_runoff && ms_since(te) < budget_ms) {
        std::vector<std::pair<double, int>> close;
        for (const auto &kv : timed)
            if (kv.second <= best_us * 1.15) close.emplace_back(kv.second, kv.first);
        std::sort(close.begin(), close.end());
        if ((int)close.size() > kRunoff) {
            // the incumbent keeps its place, so the 3% rule below compares
            // run-off times with run-off times
            auto it = std::find_if(close.begin(), close.end(),
                                   [&](const std::pair<double, int> &x) { return x.second == incumbent; });
            if (it != close.end() && it - close.begin() >= kRunoff) std::swap(*it, close[kRunoff - 1]);
            close.resize(kRunoff);
        }
        if (close.size() >= 2) {
            const int rounds = 5;
            const int burst2 = std::min(64, std::max(burst, (int)std::ceil(500.0 / std::max(best_us, 0.1))));
            const int nc = (int)close.size();
            std::vector<hipEvent_t> rev(2 * nc * rounds);
            bool ok = true;
            for (auto &x : rev)
                if (res.event(&x) != hipSuccess) ok = false;
            std::vector<hipGraphExec_t> rg(nc * rounds, nullptr);
            for (int r = 0; r < rounds && ok; ++r)
                for (int j = 0; j < nc; ++j) rg[r * nc + j] = capture_burst(configs()[close[j].second], burst2);
            const bool graphs = std::all_of(rg.begin(), rg.end(), [](hipGraphExec_t x) { return x != nullptr; });
            for (int r = 0; r < rounds && ok; ++r)
                for (int j = 0; j < nc && ok; ++j) {
                    const Config &cfg = configs()[close[j].second];
                    (void)hipEventRecord(rev[2 * (r * nc + j)], c.stream);
                    if (graphs) ok = hipGraphLaunch(rg[r * nc + j], c.stream) == hipSuccess;
                    else
                        for (int b = 0; b < burst2 && ok; ++b) ok = launch_next(cfg) == NNJIT_OK;
                    (void)hipEventRecord(rev[2 * (r * nc + j) + 1], c.stream);
                }
            if (ok && hipEventSynchronize(rev.back()) == hipSuccess) {
                best_us = 1e300;
                for (int j = 0; j < nc; ++j) {
                    std::vector<float> ts(rounds);
                    for (int r = 0; r < rounds; ++r)
                        (void)hipEventElapsedTime(&ts[r], rev[2 * (r * nc + j)], rev[2 * (r * nc + j) + 1]);
                    const double us = median(ts) * 1e3 / burst2;
                    timed[close[j].second] = us;
                    if (trace)
                        fprintf(stderr, "[nnjit] tune run-off %d %s S=%d %.2f us (was %.2f)\n", close[j].second,
                                configs()[close[j].second].v->name, configs()[close[j].second].split, us, close[j].first);
                }
                // the best of the re-timed candidates: the others were timed
                // only in the first pass, whose back-to-back bursts of one
                // candidate read lower than the run-off's interleaved ones
                for (const auto &cj : close) {
                    if (timed[cj.second] < best_us) {
                        best_us = timed[cj.second];
                        best = cj.second;
                    }
                    // the default's time is reported on the same measure as the pick
                    if (cj.second == lr.ids[0]) t_stats.default_us = timed[cj.second];
                }
            } else {
                (void)hipGetLastError();
                (void)hipStreamSynchronize(c.stream);
            }
            for (auto &x : rg)
                if (x) (void)hipGraphExecDestroy(x);
        }
    }
    t_stats.eval_ms = ms_since(te);
    // the registered kernel (cached, else the default) is replaced only by one
    // that is significantly (>= 3%) faster
    auto inc = timed.find(incumbent);
    if (inc != timed.end() && best != incumbent && best_us > inc->second / 1.03) {
        best = incumbent;
        best_us = inc->second;
    }
    Tuned tu{best, best_us, {}};
    tu.ranked.emplace_back(best, best_us);
    {
        std::vector<std::pair<double, int>> by_time;
        for (const auto &kv : timed)
            if (kv.first != best) by_time.emplace_back(kv.second, kv.first);
        std::sort(by_time.begin(), by_time.end());
        for (const auto &bt : by_time) {
            if ((int)tu.ranked.size() >= kRanked) break;
            tu.ranked.emplace_back(bt.second, bt.first);
        }
    }
    {
        std::lock_guard<std::mutex> lk(g_mu);
        // another thread may have registered this shape meanwhile: its entry
        // stays unless this result is significantly faster
        auto now = g_tuned.find(key);
        if (now != g_tuned.end() && now->second.cfg != cached && !(best_us < now->second.us / 1.03)) {
            best = now->second.cfg;
            best_us = now->second.us;
        } else {
            g_tuned[key] = tu;
        }
    }
    t_stats.chosen = best;
    t_stats.best_us = best_us;
    t_stats.wall_ms = ms_since(t0);
    if (set.log)
        fprintf(stderr, "[nnjit] tuned kind=%d dtype=%d batch=%lld M=%lld N=%lld K=%lld -> %d (%s S=%d) %.2f us, lite %d, timed %d, %.1f ms\n",
                kind, dtype, (long long)batch, (long long)M, (long long)N, (long long)K, best,
                configs()[best].v->name, configs()[best].split, best_us, t_stats.n_lite, t_stats.n_timed, t_stats.wall_ms);
    return best;
}

}  // namespace
}  // namespace nnjit

using namespace nnjit;

extern "C" {

int nnjit_matmul(int64_t M, int64_t N, int64_t K, const void *A, int64_t lda, const void *B, int64_t ldb, void *C,
                 int64_t ldc, int dtype, void *stream) {
    t_err.clear();
    Call c{1, M, N, K, A, lda, 0, B, ldb, 0, C, ldc, 0, dtype, (hipStream_t)stream};
    return run(c, -1);
}

int nnjit_batched_matmul(int64_t batch, int64_t M, int64_t N, int64_t K, const void *A, int64_t lda, int64_t strideA,
                         const void *B, int64_t ldb, int64_t strideB, void *C, int64_t ldc, int64_t strideC, int dtype,
                         void *stream) {
    t_err.clear();
    Call c{batch, M, N, K, A, lda, strideA, B, ldb, strideB, C, ldc, strideC, dtype, (hipStream_t)stream};
    return run(c, -1);
}

int nnjit_batched_matmul_noalloc(int64_t batch, int64_t M, int64_t N, int64_t K, const void *A, int64_t lda,
                                 int64_t strideA, const void *B, int64_t ldb, int64_t strideB, void *C, int64_t ldc,
                                 int64_t strideC, int dtype, void *stream) {
    t_err.clear();
    Call c{batch, M, N, K, A, lda, strideA, B, ldb, strideB, C, ldc, strideC, dtype, (hipStream_t)stream};
    return run_noalloc(c);
}

int nnjit_matmul_config(int cfg, int64_t batch, int64_t M, int64_t N, int64_t K, const void *A, int64_t lda,
                        int64_t strideA, const void *B, int64_t ldb, int64_t strideB, void *C, int64_t ldc,
                        int64_t strideC, int dtype, void *stream) {
    t_err.clear();
    if (cfg < 0) return fail(NNJIT_EINVAL, "config id %d out of range", cfg);
    Call c{batch, M, N, K, A, lda, strideA, B, ldb, strideB, C, ldc, strideC, dtype, (hipStream_t)stream};
    return run(c, cfg);
}

int nnjit_tune(int64_t M, int64_t N, int64_t K, int dtype) {
    t_err.clear();
    return tune(M == 1 ? NNJIT_KIND_GEMV : NNJIT_KIND_GEMM, dtype, 1, M, N, K);
}

int nnjit_tune_batched(int64_t batch, int64_t M, int64_t N, int64_t K, int dtype) {
    t_err.clear();
    if (batch == 1) return nnjit_tune(M, N, K, dtype);
    return tune(NNJIT_KIND_BATCHED, dtype, batch, M, N, K);
}

int nnjit_gemv_q4(int64_t N, int64_t K, int64_t group, const void *x, const void *Wq, int64_t ldq,
                  const void *scales, int64_t lds, void *y, void *stream) {
    t_err.clear();
    Call c{group, 1, N, K, x, std::max<int64_t>(1, K), 0, Wq, ldq, 0, y, std::max<int64_t>(1, N), 0, NNJIT_F16,
           (hipStream_t)stream, true, scales, lds};
    return run(c, -1);
}

int nnjit_gemv_q4_config(int cfg, int64_t N, int64_t K, int64_t group, const void *x, const void *Wq, int64_t ldq,
                         const void *scales, int64_t lds, void *y, void *stream) {
    t_err.clear();
    if (cfg < 0) return fail(NNJIT_EINVAL, "config id %d out of range", cfg);
    Call c{group, 1, N, K, x, std::max<int64_t>(1, K), 0, Wq, ldq, 0, y, std::max<int64_t>(1, N), 0, NNJIT_F16,
           (hipStream_t)stream, true, scales, lds};
    return run(c, cfg);
}

int nnjit_tune_gemv_q4(int64_t N, int64_t K, int64_t group) {
    t_err.clear();
    if (group < 1 || group > INT32_MAX) return fail(NNJIT_EINVAL, "group=%lld must be in [1, 2^31)", (long long)group);
    return tune(NNJIT_KIND_GEMV_Q4, NNJIT_F16, group, 1, N, K);
}

int nnjit_num_configs(void) { return (int)configs().size(); }

int nnjit_config_info(int cfg, char *buf, int64_t len) {
    t_err.clear();
    if (cfg < 0 || cfg >= (int)configs().size()) return fail(NNJIT_EINVAL, "config id %d out of range", cfg);
    const Config &c = configs()[cfg];
    const Variant &v = *c.v;
    char tmp[512];
    int n;
    if (family_is_q4(v.family))
        n = snprintf(tmp, sizeof tmp,
                     "id=%d family=%s name=%s rows_per_wave=%d rows_per_wg=%d kslices=%d unroll=%d vec=%d split=%d "
                     "threads=%d lds=%d est_regs=%d",
                     c.id, family_name(v.family), v.name, v.mt, v.nt, v.kslices, v.unroll, v.vec_bytes, c.split,
                     v.threads, v.lds_bytes, v.est_regs);
    else if (!family_is_gemv(v.family))
        n = snprintf(tmp, sizeof tmp,
                     "id=%d family=%s name=%s mfma=%dx%dx%d Mt=%d Nt=%d Kt=%d waves=%dx%d stages=%d prefetch=%d kslices=%d "
                     "vec=%d split=%d threads=%d lds=%d est_regs=%d direct=%d layout=%s unroll=%s",
                     c.id, family_name(v.family), v.name, v.mfma_m, v.mfma_m, v.mfma_k, v.mt, v.nt, v.kt, v.wm, v.wn,
                     v.stages, v.prefetch, v.kslices, v.vec_bytes, c.split, v.threads, v.lds_bytes, v.est_regs,
                     v.direct_copy, v.lds_layout == LAYOUT_PAD ? "pad" : v.lds_layout == LAYOUT_PLAIN ? "plain" : "swz",
                     v.rolled ? "rolled" : "full");
    else
        n = snprintf(tmp, sizeof tmp,
                     "id=%d family=%s name=%s cols=%d rows_per_pass=%d lanes_per_seg=%d unroll=%d vec=%d split=%d "
                     "threads=%d lds=%d est_regs=%d",
                     c.id, family_name(v.family), v.name, v.nt, v.kt, v.lanes_seg, v.unroll, v.vec_bytes, c.split,
                     v.threads, v.lds_bytes, v.est_regs);
    if (buf && len > 0) {
        strncpy(buf, tmp, (size_t)len - 1);
        buf[len - 1] = '\0';
    }
    return n;
}

int nnjit_config_resources(int cfg, const nnjit_device_limits *dev, nnjit_resources *out) {
    t_err.clear();
    if (cfg < 0 || cfg >= (int)configs().size() || !out) return fail(NNJIT_EINVAL, "bad config id or NULL output");
    const Config &c = configs()[cfg];
    if (dev) {
        *out = resources_of(*c.v, *dev, -1);
        return NNJIT_OK;
    }
    std::lock_guard<std::mutex> lk(g_mu);
    Device *d = nullptr;
    int rc = device_ready(&d);
    if (rc != NNJIT_OK) return rc;
    *out = resources_of(*c.v, d->limits, d->regs[variant_index(c.v)]);
    return NNJIT_OK;
}

int nnjit_lite_space(int kind, int dtype, int64_t batch, int64_t M, int64_t N, int64_t K,
                     const nnjit_device_limits *dev, int *ids, int cap, int *n_enumerated, int64_t *n_naive) {
    t_err.clear();
    if (kind < NNJIT_KIND_GEMM || kind > NNJIT_KIND_GEMV_Q4) return fail(NNJIT_EINVAL, "unknown kind %d", kind);
    if (dtype != NNJIT_F32 && dtype != NNJIT_F16) return fail(NNJIT_EDTYPE, "unknown dtype %d", dtype);
    if (kind == NNJIT_KIND_GEMV_Q4 && (dtype != NNJIT_F16 || M != 1))
        return fail(NNJIT_EINVAL, "a 4-bit GEMV shape is (NNJIT_F16, group, 1, N, K)");
    if (batch < 1 || M < 1 || N < 1 || K < 0 || cap < 0) return fail(NNJIT_EINVAL, "bad shape");
    Shape s{kind, dtype, batch, M, N, K};
    LiteResult lr;
    if (dev) {
        lr = lite_space(s, *dev, nullptr, nullptr);
    } else {
        std::lock_guard<std::mutex> lk(g_mu);
        Device *d = nullptr;
        int rc = device_ready(&d);
        if (rc != NNJIT_OK) return rc;
        lr = lite_space(s, d->limits, &d->regs, &d->spills);
    }
    for (int i = 0; i < cap && i < (int)lr.ids.size(); ++i) ids[i] = lr.ids[i];
    if (n_enumerated) *n_enumerated = lr.n_enumerated;
    if (n_naive) *n_naive = lr.n_naive;
    return (int)lr.ids.size();
}

int nnjit_last_tune_stats(double *wall_ms, int *n_enum, int *n_pruned, int *n_timed) {
    if (wall_ms) *wall_ms = t_stats.wall_ms;
    if (n_enum) *n_enum = t_stats.n_enumerated;
    if (n_pruned) *n_pruned = t_stats.n_lite;
    if (n_timed) *n_timed = t_stats.n_timed;
    return NNJIT_OK;
}

int nnjit_last_tune_stats_ex(nnjit_tune_stats *out) {
    if (!out) return fail(NNJIT_EINVAL, "NULL output");
    *out = t_stats;
    return NNJIT_OK;
}

int nnjit_last_tune_trace(int *ids, double *us, double *at_ms, int cap) {
    for (int i = 0; i < cap && i < (int)t_trace.size(); ++i) {
        if (ids) ids[i] = std::get<0>(t_trace[i]);
        if (us) us[i] = std::get<1>(t_trace[i]);
        if (at_ms) at_ms[i] = std::get<2>(t_trace[i]);
    }
    return (int)t_trace.size();
}

int nnjit_cached_config(int kind, int dtype, int64_t batch, int64_t M, int64_t N, int64_t K) {
    t_err.clear();
    std::lock_guard<std::mutex> lk(g_mu);
    int ord = -1;
    int rc = current_device(&ord);
    if (rc != NNJIT_OK) return rc;
    auto it = g_tuned.find(ShapeKey(ord, kind, dtype, batch, M, N, K));
    if (it == g_tuned.end()) return fail(NNJIT_ENOCFG, "shape not tuned");
    return it->second.cfg;
}

int nnjit_cached_ranked(int kind, int dtype, int64_t batch, int64_t M, int64_t N, int64_t K, int *ids, double *us,
                        int cap) {
    t_err.clear();
    std::lock_guard<std::mutex> lk(g_mu);
    int ord = -1;
    int rc = current_device(&ord);
    if (rc != NNJIT_OK) return rc;
    auto it = g_tuned.find(ShapeKey(ord, kind, dtype, batch, M, N, K));
    if (it == g_tuned.end()) return fail(NNJIT_ENOCFG, "shape not tuned");
    const auto &r = it->second.ranked;
    for (int i = 0; i < (int)r.size() && i < cap; ++i) {
        if (ids) ids[i] = r[i].first;
        if (us) us[i] = r[i].second;
    }
    return (int)r.size();
}

int nnjit_set_online(int enable) {
    t_err.clear();
    std::lock_guard<std::mutex> lk(g_mu);
    const int prev = g_online_on ? 1 : 0;
    g_online_on = enable != 0;
    return prev;
}

int nnjit_online_status(int kind, int dtype, int64_t batch, int64_t M, int64_t N, int64_t K, int *measured,
                        int *total, int *registered) {
    t_err.clear();
    std::lock_guard<std::mutex> lk(g_mu);
    int ord = -1;
    int rc = current_device(&ord);
    if (rc != NNJIT_OK) return rc;
    const ShapeKey key(ord, kind, dtype, batch, M, N, K);
    auto it = g_online.find(key);
    if (it != g_online.end()) {
        if (measured) *measured = (int)it->second.times.size();
        if (total) *total = (int)it->second.ids.size();
        if (registered) *registered = it->second.registered;
        return 0;
    }
    auto tt = g_tuned.find(key);
    if (tt == g_tuned.end()) return fail(NNJIT_ENOCFG, "shape neither tuned nor being tuned online");
    if (registered) *registered = tt->second.cfg;
    return 1;
}

int nnjit_cache_clear(void) {
    t_err.clear();
    std::lock_guard<std::mutex> lk(g_mu);
    for (auto &kv : g_online) online_drop(kv.second);
    g_online.clear();
    g_tuned.clear();
    g_default.clear();
    // outgrown split-K buffers: no launch may still be using them once the
    // device is idle
    int cur = -1;
    (void)hipGetDevice(&cur);
    for (auto &kv : g_devices) {
        if (kv.second.retired.empty()) continue;
        (void)hipSetDevice(kv.first);
        (void)hipDeviceSynchronize();
        for (float *p : kv.second.retired) (void)hipFree(p);
        kv.second.retired.clear();
    }
    if (cur >= 0) (void)hipSetDevice(cur);
    (void)hipGetLastError();
    g_set = read_settings();
    g_set_loaded = true;
    return NNJIT_OK;
}

int nnjit_cache_save(const char *path) {
    t_err.clear();
    if (!path) return fail(NNJIT_EINVAL, "NULL path");
    std::lock_guard<std::mutex> lk(g_mu);
    FILE *f = fopen(path, "w");
    if (!f) return fail(NNJIT_EINVAL, "cannot write %s", path);
    fprintf(f, "# nnjit kernel database v2: signature kind dtype batch M N K, then up to %d ranked (config split us), "
               "the registered one first\n", kRanked);
    int n = 0;
    for (const auto &kv : g_tuned) {
        const int dev = std::get<0>(kv.first);
        auto di = g_devices.find(dev);
        if (di == g_devices.end() || !di->second.ready) continue;
        fprintf(f, "%s:%d %d %d %lld %lld %lld %lld", di->second.arch.c_str(), di->second.limits.num_cus,
                std::get<1>(kv.first), std::get<2>(kv.first), (long long)std::get<3>(kv.first),
                (long long)std::get<4>(kv.first), (long long)std::get<5>(kv.first), (long long)std::get<6>(kv.first));
        std::vector<std::pair<int, double>> ranked = kv.second.ranked;
        if (ranked.empty()) ranked.emplace_back(kv.second.cfg, kv.second.us);
        for (const auto &r : ranked) fprintf(f, " %s %d %.4f", configs()[r.first].v->name, configs()[r.first].split, r.second);
        fprintf(f, "\n");
        ++n;
    }
    fclose(f);
    return n;
}

int nnjit_cache_load(const char *path) {
    t_err.clear();
    if (!path) return fail(NNJIT_EINVAL, "NULL path");
    std::lock_guard<std::mutex> lk(g_mu);
    Device *d = nullptr;
    int rc = device_ready(&d);
    if (rc != NNJIT_OK) return rc;
    FILE *f = fopen(path, "r");
    if (!f) return fail(NNJIT_EINVAL, "cannot read %s", path);
    char sig_want[160];
    snprintf(sig_want, sizeof sig_want, "%s:%d", d->arch.c_str(), d->limits.num_cus);
    char line[4096];
    int n = 0;
    auto find_id = [](const char *name, int split) {
        for (const Config &c : configs())
            if (c.split == split && strcmp(c.v->name, name) == 0) return c.id;
        return -1;
    };
    while (fgets(line, sizeof line, f)) {
        if (line[0] == '#') continue;
        char sig[160], name[160];
        int kind, dtype, split, used = 0;
        long long batch, M, N, K;
        double us;
        if (sscanf(line, "%159s %d %d %lld %lld %lld %lld %159s %d %lf%n", sig, &kind, &dtype, &batch, &M, &N, &K, name,
                   &split, &us, &used) != 10)
            continue;
        if (strcmp(sig, sig_want) != 0) continue;
        if (kind < NNJIT_KIND_GEMM || kind > NNJIT_KIND_GEMV_Q4 || (dtype != NNJIT_F32 && dtype != NNJIT_F16)) continue;
        if (batch < 1 || M < 1 || N < 1 || K < 0) continue;
        const int id = find_id(name, split);
        if (id < 0 || configs()[id].v->family != family_of(kind, dtype)) continue;
        Tuned tu{id, us, {{id, us}}};
        // the other ranked candidates (v2 lines); unknown names are skipped
        const char *rest = line + used;
        int more = 0;
        while ((int)tu.ranked.size() < kRanked && sscanf(rest, "%159s %d %lf%n", name, &split, &us, &more) == 3) {
            rest += more;
            const int rid = find_id(name, split);
            if (rid >= 0 && configs()[rid].v->family == family_of(kind, dtype)) tu.ranked.emplace_back(rid, us);
        }
        // merging databases: a shape already known keeps the faster measurement
        const ShapeKey key(d->ordinal, kind, dtype, batch, M, N, K);
        auto it = g_tuned.find(key);
        if (it == g_tuned.end() || tu.us < it->second.us) g_tuned[key] = tu;
        ++n;
    }
    fclose(f);
    return n;
}

int nnjit_stream_read(const void *src, int64_t bytes, void *sink, int workgroups, void *stream) {
    t_err.clear();
    if (bytes < 0 || bytes % 16) return fail(NNJIT_EINVAL, "bytes=%lld must be a non-negative multiple of 16", (long long)bytes);
    if (workgroups < 1 || workgroups > (1 << 20)) return fail(NNJIT_EINVAL, "workgroups=%d out of [1, 2^20]", workgroups);
    if (bytes > 0 && (!src || ((uintptr_t)src & 15u))) return fail(NNJIT_EINVAL, "src is NULL or not 16-byte aligned");
    if (!sink) return fail(NNJIT_EINVAL, "sink is NULL");
    if (bytes == 0) return NNJIT_OK;
    {
        std::lock_guard<std::mutex> lk(g_mu);
        Device *d = nullptr;
        const int rc = device_ready(&d);
        if (rc != NNJIT_OK) return rc;
    }
    const hipError_t e = launch_stream_read(src, bytes, (unsigned *)sink, workgroups, (hipStream_t)stream);
    return e == hipSuccess ? NNJIT_OK : hip_fail(e, "stream_read");
}

const char *nnjit_last_error(void) { return t_err.c_str(); }

int nnjit_version(void) { return (0 << 16) | 2; }

}  // extern "C"
