// Host runtime behind include/dash.h: argument checks, model and paged-KV
// handles (page free list, reference counts, group fork with copy of a partial
// last page), workspace planning, the prefill / decode-step sequencing of the
// kernels, and the native rollout driver (reservation one page ahead, ragged
// retirement, optional HIP-graph replay of the fixed-batch decode step).
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <map>
#include <mutex>
#include <tuple>
#include <string>
#include <vector>

#include "../../include/dash.h"
#include "common.h"
#include "kernels.h"
#include "kv_pages.h"

using namespace dash;

// ---------------------------------------------------------------- errors ----

namespace {

thread_local std::string g_last_error;

int fail(int status, const char* fmt, ...) {
    char buf[512];
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(buf, sizeof buf, fmt, ap);
    va_end(ap);
    g_last_error = buf;
    return status;
}

#define DASH_HIP(call)                                                                              \
    do {                                                                                            \
        hipError_t e_ = (call);                                                                     \
        if (e_ != hipSuccess) return fail(DASH_EDEVICE, "%s: %s", #call, hipGetErrorString(e_));   \
    } while (0)

size_t align_up(size_t x, size_t a) { return (x + a - 1) / a * a; }

constexpr int kMaxGroupRows = 8;  // rows per prefix-shared group the grouped kernel serves

// ------------------------------------------------------------- profiler ----
// Event pairs around launches, by kernel class; a ring of pairs is harvested
// lazily (a pair is read back only when its slot is reused or on read-out).
// Under stream capture the pairs become event-record nodes of the graph (a set
// per captured graph, re-armed by every replay and harvested before the next).

struct GraphProf;

// The profiler's events only time launches, so they are created without the
// system-scope fence: recording one then neither writes back nor invalidates the
// caches, which would slow the launch that follows it and lengthen the very
// interval being measured.
hipError_t create_timing_event(hipEvent_t* ev) { return hipEventCreateWithFlags(ev, hipEventDisableSystemFence); }

struct Profiler {
    struct Pair {
        hipEvent_t a = nullptr, b = nullptr;
        int cls = 0;
        bool live = false;
    };
    uint32_t mask = 0;
    bool capturing = false;
    std::vector<Pair> ring;
    size_t next = 0;
    GraphProf* capture_set = nullptr;  // hands out the pairs recorded while capturing
    double ms[DASH_K_COUNT] = {};
    int64_t n[DASH_K_COUNT] = {};
    std::string err;  // first timing failure since the last read-out
    int layer = -1;   // >= 0: per-layer classes are timed in this layer only
};
Profiler g_prof;

void prof_error(const char* what, hipError_t e, int cls = -1, int idx = -1) {
    if (g_prof.err.empty()) {
        char buf[256];
        snprintf(buf, sizeof buf, "%s (class %d, pair %d): %s", what, cls, idx, hipGetErrorString(e));
        g_prof.err = buf;
    }
    (void)hipGetLastError();
}

void prof_harvest(Profiler::Pair& p) {
    if (!p.live) return;
    p.live = false;
    float ms = 0.f;
    hipError_t e = hipEventSynchronize(p.b);
    if (e != hipSuccess) return prof_error("hipEventSynchronize", e);
    if ((e = hipEventElapsedTime(&ms, p.a, p.b)) != hipSuccess) return prof_error("hipEventElapsedTime", e);
    g_prof.ms[p.cls] += ms;
    g_prof.n[p.cls] += 1;
}

// Append an event-record node to the capture in progress on `st` (after the
// nodes captured so far; later captured work depends on it).  Explicit nodes
// rather than hipEventRecordWithFlags(hipEventRecordExternal), which some HIP
// runtime builds reject during capture.
hipError_t capture_event_record(hipStream_t st, hipEvent_t ev) {
    hipStreamCaptureStatus cs;
    unsigned long long id;
    hipGraph_t g;
    const hipGraphNode_t* deps;
    size_t nd;
    hipError_t e = hipStreamGetCaptureInfo_v2(st, &cs, &id, &g, &deps, &nd);
    if (e != hipSuccess) return e;
    if (cs != hipStreamCaptureStatusActive) return hipErrorIllegalState;
    hipGraphNode_t node;
    if ((e = hipGraphAddEventRecordNode(&node, g, deps, nd, ev)) != hipSuccess) return e;
    return hipStreamUpdateCaptureDependencies(st, &node, 1, hipStreamSetCaptureDependencies);
}

// Timed pairs of one captured graph.  Events cannot be created during capture,
// so the pairs are created beforehand (reserve) and handed out by ProfScope.
struct GraphProf {
    std::vector<Profiler::Pair> pairs;
    size_t used = 0;
    bool reserve(size_t n) {
        while (pairs.size() < n) {
            Profiler::Pair p;
            if (create_timing_event(&p.a) != hipSuccess) return false;
            if (create_timing_event(&p.b) != hipSuccess) {
                (void)hipEventDestroy(p.a);
                return false;
            }
            pairs.push_back(p);
        }
        return true;
    }
    void armed() {  // after a replay was launched
        for (size_t i = 0; i < used; ++i) pairs[i].live = true;
    }
    void harvest() {
        for (auto& p : pairs) prof_harvest(p);
    }
    ~GraphProf() {
        harvest();
        for (auto& p : pairs) {
            (void)hipEventDestroy(p.a);
            (void)hipEventDestroy(p.b);
        }
    }
};

// Times the launches made during its lifetime if class `cls` is enabled (cls < 0: never).
struct ProfScope {
    int slot = -1;
    hipStream_t st;
    Profiler::Pair* gp = nullptr;  // capture mode: a pair of the graph's set
    ProfScope(int cls, hipStream_t s) : st(s) {
        if (cls < 0 || !(g_prof.mask & (1u << cls))) return;
        if (g_prof.capturing) {
            GraphProf* set = g_prof.capture_set;
            if (!set || set->used >= set->pairs.size()) return;
            Profiler::Pair& p = set->pairs[set->used];
            const hipError_t e = capture_event_record(st, p.a);
            if (e != hipSuccess) {
                prof_error("start record under capture", e, cls, (int)set->used);
                return;
            }
            p.cls = cls;
            gp = &p;
            return;
        }
        if (g_prof.ring.empty()) return;
        Profiler::Pair& p = g_prof.ring[g_prof.next];
        prof_harvest(p);
        if (hipEventRecord(p.a, st) != hipSuccess) return;
        p.cls = cls;
        slot = (int)g_prof.next;
        g_prof.next = (g_prof.next + 1) % g_prof.ring.size();
    }
    ~ProfScope() {
        if (gp) {
            const hipError_t e = capture_event_record(st, gp->b);
            if (e == hipSuccess) g_prof.capture_set->used++;
            else prof_error("end record under capture", e, gp->cls, (int)g_prof.capture_set->used);
            return;
        }
        if (slot < 0) return;
        Profiler::Pair& p = g_prof.ring[slot];
        p.live = hipEventRecord(p.b, st) == hipSuccess;
    }
};

}  // namespace

// ----------------------------------------------------------------- model ----

struct dash_model {
    dash_model_desc d;
    std::vector<const void*> w;
    size_t esz;
    int qkv_rows() const { return (d.n_heads + 2 * d.n_kv_heads) * d.head_dim; }
    const void* embed() const { return w[0]; }
    const void* final_norm() const { return w[1]; }
    const void* lw(int l, int i) const { return w[3 + 7 * l + i]; }
};

// -------------------------------------------------------------------- kv ----

struct dash_kv {
    const dash_model* m;
    void* pool;
    int32_t* d_table;
    uint32_t* d_status;
    KVGeom g;
    int max_ctx;
    PageBook pb;  // host mirror of the page table, reference counts, free list
    // pinned staging ring for uploads (two halves, each guarded by an event)
    char* stage = nullptr;
    size_t stage_half = 0;
    int stage_cur = 0;
    size_t stage_off = 0;
    hipEvent_t stage_ev[2] = {nullptr, nullptr};
    bool stage_ev_live[2] = {false, false};
};

namespace {

size_t table_entries(int max_seqs, int max_ctx, int ps) {
    return (size_t)max_seqs * (size_t)((max_ctx + ps - 1) / ps);
}

// Copy host bytes to device memory on `st` through the pinned ring.
int kv_upload(dash_kv* kv, void* dst, const void* src, size_t bytes, hipStream_t st) {
    if (bytes == 0) return DASH_OK;
    size_t done = 0;
    while (done < bytes) {
        if (kv->stage_off >= kv->stage_half) {  // switch halves
            DASH_HIP(hipEventRecord(kv->stage_ev[kv->stage_cur], st));
            kv->stage_ev_live[kv->stage_cur] = true;
            kv->stage_cur ^= 1;
            kv->stage_off = 0;
            if (kv->stage_ev_live[kv->stage_cur]) DASH_HIP(hipEventSynchronize(kv->stage_ev[kv->stage_cur]));
        }
        const size_t n = std::min(bytes - done, kv->stage_half - kv->stage_off);
        char* p = kv->stage + kv->stage_cur * kv->stage_half + kv->stage_off;
        memcpy(p, (const char*)src + done, n);
        DASH_HIP(hipMemcpyAsync((char*)dst + done, p, n, hipMemcpyHostToDevice, st));
        kv->stage_off = align_up(kv->stage_off + n, 256);
        done += n;
    }
    return DASH_OK;
}

// Upload page-table rows [s0, s1] of the host mirror.
int kv_push_rows(dash_kv* kv, int s0, int s1, hipStream_t st) {
    if (s1 < s0) return DASH_OK;
    const size_t mp = kv->g.max_pages;
    return kv_upload(kv, kv->d_table + s0 * mp, kv->pb.table.data() + s0 * mp, (size_t)(s1 - s0 + 1) * mp * 4, st);
}

// Returns the listed slots' pages to the pool unless disarmed: a call that fails
// after mapping pages (a failed launch) leaves the cache as it found it.  Work
// already enqueued may still write those pages; they are reused only by later
// stream-ordered work.
struct ReleaseOnError {
    dash_kv* kv;
    const int32_t* slots;
    int n;
    bool armed = true;
    ~ReleaseOnError() {
        if (armed)
            for (int i = 0; i < n; ++i) kv->pb.release(slots[i]);
    }
};

}  // namespace

// ------------------------------------------------------------- workspace ----

namespace {

struct Ws {
    float* x;
    void* y;
    float* qkv;
    void* q;
    void* o;
    float* delta;
    void* h;
    float* cs;
    float* attn_part;
    int32_t* pos;    // prefill rows
    int32_t* slot;   // prefill rows
    int32_t* pslot;  // prefill prompt -> slot
    int32_t* gather; // prefill last rows
    int32_t* pairs;  // fork copies
    size_t bytes;
};

// max_ctx bounds the decode attention's context splits (0: no decode use).
// decode_rows (default max_rows) sizes the decode-attention partials: a rollout's step
// workspace also serves the prefill's larger row count, which needs none.
Ws plan_ws(const dash_model* m, int max_rows, char* base, int max_ctx, int decode_rows = -1) {
    const auto& d = m->d;
    const size_t e = m->esz;
    size_t off = 0;
    auto take = [&](size_t bytes) {
        char* p = base ? base + off : nullptr;
        off = align_up(off + bytes, 256);
        return p;
    };
    Ws w{};
    const size_t R = (size_t)max_rows;
    const int qr = m->qkv_rows();
    w.x = (float*)take(R * d.d_model * 4);
    w.y = take(R * d.d_model * e);
    w.qkv = (float*)take((size_t)gemm_pick_splits(d.dtype, EPI_STORE_F32, qr, d.d_model) * R * qr * 4);
    w.q = take(R * d.n_heads * d.head_dim * e);
    w.o = take(R * d.n_heads * d.head_dim * e);
    const int so = gemm_pick_splits(d.dtype, EPI_STORE_F32, d.d_model, d.n_heads * d.head_dim);
    const int sd = gemm_pick_splits(d.dtype, EPI_STORE_F32, d.d_model, d.d_ff);
    w.delta = (float*)take((size_t)std::max(so, sd) * R * d.d_model * 4);
    w.h = take(R * d.d_ff * e);
    w.cs = (float*)take(R * d.head_dim * 4);
    w.attn_part = (float*)take(
        attention_partial_floats(decode_rows < 0 ? max_rows : decode_rows, d.n_heads, d.head_dim, max_ctx) * 4);
    w.pos = (int32_t*)take(R * 4);
    w.slot = (int32_t*)take(R * 4);
    w.pslot = (int32_t*)take(R * 4);
    w.gather = (int32_t*)take(R * 4);
    w.pairs = (int32_t*)take(R * 8);
    w.bytes = off;
    return w;
}

}  // namespace

// ------------------------------------------------------------------- ABI ----

extern "C" {

int dash_abi_version(void) { return DASH_ABI_VERSION; }

const char* dash_status_str(int s) {
    switch (s) {
        case DASH_OK: return "ok";
        case DASH_EINVAL: return "invalid argument";
        case DASH_ENOMEM: return "out of host memory";
        case DASH_ECAPACITY: return "capacity exceeded (pool, page table or workspace)";
        case DASH_EDEVICE: return "HIP runtime error";
        case DASH_ENOTSUP: return "shape not supported by the kernels";
        default: return "unknown status";
    }
}

const char* dash_last_error(void) { return g_last_error.c_str(); }

int32_t dash_weight_count(const dash_model_desc* d) { return d && d->n_layers > 0 ? 3 + 7 * d->n_layers : -1; }

int dash_model_create(const dash_model_desc* d, const void* const* w, int32_t n_w, dash_model** out) {
    if (!d || !w || !out) return fail(DASH_EINVAL, "dash_model_create: NULL argument");
    *out = nullptr;
    if (d->n_layers < 1 || d->d_model < 1 || d->n_heads < 1 || d->n_kv_heads < 1 || d->head_dim < 2 ||
        d->d_ff < 1 || d->vocab < 1)
        return fail(DASH_EINVAL, "dash_model_create: non-positive dimension");
    if (d->vocab > (1 << 28)) return fail(DASH_EINVAL, "vocab %d exceeds 2^28", d->vocab);
    if (d->n_heads % d->n_kv_heads) return fail(DASH_EINVAL, "n_heads %% n_kv_heads != 0");
    if (d->head_dim % 2) return fail(DASH_EINVAL, "head_dim must be even (RoPE pairs)");
    if (d->dtype != DASH_F32 && d->dtype != DASH_BF16) return fail(DASH_EINVAL, "dtype must be DASH_F32 or DASH_BF16");
    if (!(d->rope_theta > 0.f) || !(d->rms_eps >= 0.f)) return fail(DASH_EINVAL, "bad rope_theta or rms_eps");
    if (n_w != dash_weight_count(d)) return fail(DASH_EINVAL, "expected %d weight pointers, got %d", dash_weight_count(d), n_w);
    if (d->d_model > 4096) return fail(DASH_ENOTSUP, "d_model > 4096");
    if (d->dtype == DASH_BF16) {
        if (d->head_dim != 64 && d->head_dim != 128) return fail(DASH_ENOTSUP, "bf16 head_dim must be 64 or 128");
        if (d->d_model % 64 || d->d_ff % 64) return fail(DASH_ENOTSUP, "bf16 d_model and d_ff must be multiples of 64");
        if (d->n_heads / d->n_kv_heads > 16) return fail(DASH_ENOTSUP, "GQA group larger than 16");
    } else {
        if (d->head_dim > 128) return fail(DASH_ENOTSUP, "fp32 head_dim must be <= 128");
        if (d->d_model % 4 || d->d_ff % 4) return fail(DASH_ENOTSUP, "fp32 d_model and d_ff must be multiples of 4");
    }
    for (int i = 0; i < n_w; ++i) {
        if (i == 2) {
            if (w[i]) return fail(DASH_ENOTSUP, "untied lm_head is not supported (pass NULL)");
            continue;
        }
        if (!w[i]) return fail(DASH_EINVAL, "weight %d is NULL", i);
        if ((uintptr_t)w[i] & 15) return fail(DASH_EINVAL, "weight %d is not 16-byte aligned", i);
    }
    dash_model* m = new (std::nothrow) dash_model;
    if (!m) return fail(DASH_ENOMEM, "out of host memory");
    m->d = *d;
    m->w.assign(w, w + n_w);
    m->esz = d->dtype == DASH_BF16 ? 2 : 4;
    *out = m;
    return DASH_OK;
}

void dash_model_destroy(dash_model* m) { delete m; }

size_t dash_kv_page_bytes(const dash_model* m, int32_t ps) {
    if (!m || ps < 1) return 0;
    return (size_t)m->d.n_layers * m->d.n_kv_heads * 2 * (size_t)ps * m->d.head_dim * m->esz;
}

size_t dash_kv_table_bytes(int32_t max_seqs, int32_t max_ctx, int32_t ps) {
    if (max_seqs < 1 || max_ctx < 1 || ps < 1) return 0;
    return align_up(table_entries(max_seqs, max_ctx, ps) * 4, 256) + 256;
}

int dash_kv_create(const dash_model* m, void* pool, size_t pool_bytes, int32_t ps, int32_t max_seqs, int32_t max_ctx,
                   void* d_table, void* stream, dash_kv** out) {
    if (!m || !pool || !d_table || !out) return fail(DASH_EINVAL, "dash_kv_create: NULL argument");
    *out = nullptr;
    if (ps < 1 || ps > 1024 || max_seqs < 1 || max_ctx < 1) return fail(DASH_EINVAL, "dash_kv_create: bad sizes");
    if (m->d.dtype == DASH_BF16 && ps % 32) return fail(DASH_ENOTSUP, "bf16 page_size must be a multiple of 32");
    if ((uintptr_t)pool & 255) return fail(DASH_EINVAL, "pool must be 256-byte aligned");
    const size_t pb = dash_kv_page_bytes(m, ps);
    const size_t pages = pool_bytes / pb;
    if (pages < 1) return fail(DASH_ECAPACITY, "pool holds no page (%zu bytes per page)", pb);
    if (pages > 0x7FFFFFFF) return fail(DASH_EINVAL, "too many pages");
    dash_kv* kv = new (std::nothrow) dash_kv;
    if (!kv) return fail(DASH_ENOMEM, "out of host memory");
    kv->m = m;
    kv->pool = pool;
    kv->max_ctx = max_ctx;
    const int max_pages = (max_ctx + ps - 1) / ps;
    kv->g = KVGeom{m->d.n_layers, (int)pages, m->d.n_kv_heads, m->d.head_dim, ps, max_pages, max_seqs,
                   attention_split_keys(max_seqs, m->d.n_kv_heads, max_ctx, m->d.head_dim), 0};
    const size_t ent = table_entries(max_seqs, max_ctx, ps);
    kv->d_table = (int32_t*)d_table;
    kv->d_status = (uint32_t*)((char*)d_table + align_up(ent * 4, 256));
    kv->pb.init((int)pages, max_seqs, max_pages, ps);
    kv->stage_half = std::max<size_t>(align_up(ent * 4, 256), 1 << 16);
    hipError_t e = hipHostMalloc((void**)&kv->stage, 2 * kv->stage_half, hipHostMallocDefault);
    if (e != hipSuccess) {
        delete kv;
        return fail(DASH_EDEVICE, "hipHostMalloc of the staging ring: %s", hipGetErrorString(e));
    }
    for (int i = 0; i < 2; ++i) {
        e = hipEventCreateWithFlags(&kv->stage_ev[i], hipEventDisableTiming);
        if (e != hipSuccess) {
            dash_kv_destroy(kv);
            return fail(DASH_EDEVICE, "hipEventCreate: %s", hipGetErrorString(e));
        }
    }
    hipStream_t st = (hipStream_t)stream;
    e = launch_fill_i32(kv->d_table, -1, ent, st);
    if (e == hipSuccess) e = launch_fill_i32((int32_t*)kv->d_status, 0, 1, st);
    if (e != hipSuccess) {
        dash_kv_destroy(kv);
        return fail(DASH_EDEVICE, "clearing the page table: %s", hipGetErrorString(e));
    }
    *out = kv;
    return DASH_OK;
}

void dash_kv_destroy(dash_kv* kv) {
    if (!kv) return;
    for (int i = 0; i < 2; ++i) {
        if (kv->stage_ev[i]) {
            if (kv->stage_ev_live[i]) (void)hipEventSynchronize(kv->stage_ev[i]);
            (void)hipEventDestroy(kv->stage_ev[i]);
        }
    }
    if (kv->stage) {
        (void)hipDeviceSynchronize();  // uploads still in flight read the ring
        (void)hipHostFree(kv->stage);
    }
    delete kv;
}

int dash_kv_free_pages(const dash_kv* kv, int32_t* out) {
    if (!kv || !out) return fail(DASH_EINVAL, "NULL argument");
    *out = (int32_t)kv->pb.free_pages();
    return DASH_OK;
}

int dash_kv_slot_len(const dash_kv* kv, int32_t slot, int32_t* out) {
    if (!kv || !out) return fail(DASH_EINVAL, "NULL argument");
    if (slot < 0 || slot >= kv->g.max_seqs) return fail(DASH_EINVAL, "slot %d out of range", slot);
    *out = kv->pb.len[slot];
    return DASH_OK;
}

int dash_kv_split_keys(const dash_kv* kv, int32_t* out) {
    if (!kv || !out) return fail(DASH_EINVAL, "NULL argument");
    *out = kv->g.split_keys;
    return DASH_OK;
}

int dash_kv_reserve(dash_kv* kv, const int32_t* h_slots, int32_t n, int32_t new_len, void* stream) {
    if (!kv || (n > 0 && !h_slots)) return fail(DASH_EINVAL, "NULL argument");
    if (n < 0 || new_len < 0) return fail(DASH_EINVAL, "negative count or length");
    if (new_len > kv->max_ctx) return fail(DASH_ECAPACITY, "new_len %d exceeds max_ctx %d", new_len, kv->max_ctx);
    for (int i = 0; i < n; ++i) {
        const int s = h_slots[i];
        if (s < 0 || s >= kv->g.max_seqs) return fail(DASH_EINVAL, "slot %d out of range", s);
    }
    // duplicates in h_slots would double count: harmless (over-estimate)
    const size_t need = kv->pb.grow_need(h_slots, n, new_len);
    if (need > kv->pb.free_pages())
        return fail(DASH_ECAPACITY, "pool exhausted: need %zu pages, %zu free", need, kv->pb.free_pages());
    int lo = kv->g.max_seqs, hi = -1;
    for (int i = 0; i < n; ++i) {
        const int s = h_slots[i];
        if (kv->pb.grow(s, new_len)) {
            lo = std::min(lo, s);
            hi = std::max(hi, s);
        }
    }
    return kv_push_rows(kv, lo, hi, (hipStream_t)stream);
}

int dash_kv_release(dash_kv* kv, const int32_t* h_slots, int32_t n) {
    if (!kv || (n > 0 && !h_slots)) return fail(DASH_EINVAL, "NULL argument");
    for (int i = 0; i < n; ++i) {
        const int s = h_slots[i];
        if (s < 0 || s >= kv->g.max_seqs) return fail(DASH_EINVAL, "slot %d out of range", s);
    }
    for (int i = 0; i < n; ++i) kv->pb.release(h_slots[i]);
    // The device rows keep stale page ids until the slot is reused (the next
    // reserve / prefill of the slot uploads its row); nothing reads a released slot.
    return DASH_OK;
}

int dash_kv_device_status(dash_kv* kv, uint32_t* out, void* stream) {
    if (!kv || !out) return fail(DASH_EINVAL, "NULL argument");
    hipStream_t st = (hipStream_t)stream;
    DASH_HIP(hipMemcpyAsync(out, kv->d_status, 4, hipMemcpyDeviceToHost, st));
    DASH_HIP(hipStreamSynchronize(st));
    DASH_HIP(launch_fill_i32((int32_t*)kv->d_status, 0, 1, st));
    return DASH_OK;
}

size_t dash_workspace_bytes(const dash_model* m, int32_t max_rows, int32_t max_ctx) {
    if (!m || max_rows < 1) return 0;
    if (max_ctx < 0) return 0;
    return plan_ws(m, max_rows, nullptr, max_ctx).bytes;
}

int dash_profile_enable(uint32_t class_mask) {
    if (class_mask && g_prof.ring.empty()) {
        g_prof.ring.resize(8192);
        for (auto& p : g_prof.ring) {
            if (create_timing_event(&p.a) != hipSuccess || create_timing_event(&p.b) != hipSuccess) {
                g_prof.ring.clear();
                return fail(DASH_EDEVICE, "hipEventCreate failed");
            }
        }
    }
    g_prof.mask = class_mask & ((1u << DASH_K_COUNT) - 1u);
    return DASH_OK;
}

int dash_profile_layer(int32_t layer) {
    if (layer < -1) return fail(DASH_EINVAL, "layer must be >= -1");
    g_prof.layer = layer;
    return DASH_OK;
}

int dash_profile_read(double* ms_out, int64_t* launches_out, int32_t reset) {
    for (auto& p : g_prof.ring) prof_harvest(p);
    for (int i = 0; i < DASH_K_COUNT; ++i) {
        if (ms_out) ms_out[i] = g_prof.ms[i];
        if (launches_out) launches_out[i] = g_prof.n[i];
        if (reset) {
            g_prof.ms[i] = 0;
            g_prof.n[i] = 0;
        }
    }
    if (!g_prof.err.empty()) {
        const std::string e = g_prof.err;
        g_prof.err.clear();
        return fail(DASH_EDEVICE, "kernel timing failed: %s", e.c_str());
    }
    return DASH_OK;
}

}  // extern "C"

// ------------------------------------------------------- forward passes ----

namespace {

// Most token rows one forward pass may hold: the bf16 GEMMs address their left
// operand [rows, K] with 32-bit byte offsets, so rows * K * 2 must stay below 2^31
// for every K of the layer (d_model, the attention width and d_ff).
int max_forward_rows(const dash_model* m) {
    const int64_t k = std::max({(int64_t)m->d.d_model, (int64_t)m->d.n_heads * m->d.head_dim, (int64_t)m->d.d_ff});
    return (int)std::min<int64_t>(((int64_t)1 << 31) / (2 * k) - 1, 0x7FFFFFFF);
}

int ws_rows_for(const dash_model* m, size_t ws_bytes, int want) {
    // largest row count <= want (and <= max_forward_rows) whose plan fits (plans grow
    // monotonically in rows)
    want = std::min(want, max_forward_rows(m));
    if (plan_ws(m, want, nullptr, 0).bytes <= ws_bytes) return want;
    int lo = 0, hi = want;
    while (lo < hi) {
        const int mid = (lo + hi + 1) / 2;
        if (plan_ws(m, mid, nullptr, 0).bytes <= ws_bytes) lo = mid;
        else hi = mid - 1;
    }
    return lo;
}

// Rows grouped by shared prefix (decode only): rows [off[i], off[i+1]) share
// their first shared_len positions; group_size bounds the rows per group.
struct GroupInfo {
    const int32_t* off;
    int n_groups, group_size, shared_len;
};

// Transformer body over `rows` rows whose x/y are already set (x fp32, y = RMSNorm(x) * attn_norm[0]).
// prefill: attention via the generic causal kernel over the rows' own slots; decode: MFMA paged kernel.
// Leaves x updated by the last layer's down projection in (x, delta split partials) and
// returns the split count of the last delta via *last_split.
int run_layers(dash_model* m, dash_kv* kv, const Ws& w, int rows, const int32_t* pos, const int32_t* slot,
               bool prefill, int prefill_len, hipStream_t st, int* last_split, const GroupInfo* gi) {
    const auto& d = m->d;
    const int dt = d.dtype;
    const int qr = m->qkv_rows();
    const int hq = d.n_heads * d.head_dim;
    const int sq = gemm_pick_splits(dt, EPI_STORE_F32, qr, d.d_model);
    const int so = gemm_pick_splits(dt, EPI_STORE_F32, d.d_model, hq);
    const int sd = gemm_pick_splits(dt, EPI_STORE_F32, d.d_model, d.d_ff);
    const bool fuse_qkv = gemm_qkv_fusable(dt, d.n_heads, d.n_kv_heads, d.head_dim) && gemm_qkv_fuse_pays(rows, qr);
    // Prefix-shared decode attention keeps its per-row states in the fp32 QKV buffer, dead
    // while attention runs (the fused projection never writes it; the unfused one's output
    // is consumed by the RoPE / append kernel first).  It always fits: n_heads (hd + 8)
    // <= (n_heads + 2 n_kv) hd whenever hd >= 4 rep, which the prefix kernel's shapes
    // satisfy.  For shapes the prefix kernel does not cover, the per-row kernel alone gives
    // the same bits.
    float* prefix_state = nullptr;
    if (gi && !prefill && dt == DASH_BF16 &&
        decode_attention_prefix_ok(kv->g, d.n_heads, gi->group_size, gi->shared_len) &&
        decode_attention_prefix_state_bytes(rows, d.n_heads, d.head_dim) <= (size_t)rows * qr * 4)
        prefix_state = w.qkv;
    // prefill is timed as one class by its caller; per-layer classes may be limited to one layer
    int cur_layer = -1;
    auto cls = [&](int c) {
        return prefill || (g_prof.layer >= 0 && cur_layer >= 0 && cur_layer != g_prof.layer) ? -1 : c;
    };
    {
        ProfScope ps(cls(DASH_K_ROPE), st);
        DASH_HIP(launch_rope_table(pos, w.cs, rows, d.head_dim, d.rope_theta, st));
    }
    for (int l = 0; l < d.n_layers; ++l) {
        cur_layer = l;
        if (l > 0) {
            ProfScope ps(cls(DASH_K_NORM), st);
            DASH_HIP(launch_add_rmsnorm(dt, w.x, w.delta, sd, (size_t)rows * d.d_model, m->lw(l, 0), w.y, nullptr, rows,
                                        d.d_model, d.rms_eps, 1, st));
        }
        if (fuse_qkv) {  // projection, bias, RoPE and the KV append in one kernel
            ProfScope ps(cls(DASH_K_GEMM_QKV), st);
            const QkvRopeArgs qa{(const bf16_t*)m->lw(l, 2), w.cs, pos, slot, kv->d_table, (bf16_t*)kv->pool,
                                 kv->g, l, (bf16_t*)w.q, d.n_heads, kv->d_status};
            DASH_HIP(launch_gemm_qkv_rope(w.y, m->lw(l, 1), rows, qr, d.d_model, qa, st));
        } else {
            {
                ProfScope ps(cls(DASH_K_GEMM_QKV), st);
                DASH_HIP(launch_gemm(dt, EPI_STORE_F32, w.y, m->lw(l, 1), w.qkv, rows, qr, d.d_model, qr, sq,
                                     (size_t)rows * qr, st));
            }
            ProfScope ps(cls(DASH_K_ROPE), st);
            DASH_HIP(launch_qkv_rope_append(dt, w.qkv, sq, (size_t)rows * qr, m->lw(l, 2), w.cs, pos, slot,
                                            kv->d_table, kv->pool, kv->g, l, w.q, rows, d.n_heads, kv->d_status, st));
        }
        if (prefill) {
            DASH_HIP(launch_prefill_attention(dt, w.q, pos, slot, kv->d_table, kv->pool, kv->g, l, d.n_heads, w.o, rows,
                                              prefill_len, st));
        } else {
            {
                ProfScope ps(cls(DASH_K_ATTN), st);
                if (prefix_state)
                    DASH_HIP(launch_decode_attention_grouped(w.q, pos, slot, kv->d_table, kv->pool, kv->g, l, d.n_heads,
                                                             gi->off, gi->n_groups, gi->group_size, gi->shared_len,
                                                             w.o, rows, kv->max_ctx, w.attn_part, prefix_state, st));
                else
                    DASH_HIP(launch_decode_attention(dt, w.q, pos, slot, kv->d_table, kv->pool, kv->g, l, d.n_heads,
                                                     w.o, rows, kv->max_ctx, w.attn_part, st));
            }
            if (dt == DASH_BF16 && kv->max_ctx > kv->g.split_keys) {  // the combine launches only for several splits
                ProfScope ps(cls(DASH_K_ATTN_COMBINE), st);
                DASH_HIP(launch_attention_combine(dt, pos, rows, d.n_heads, d.head_dim, kv->max_ctx, kv->g.split_keys,
                                                  w.attn_part, w.o, st));
            }
        }
        {
            ProfScope ps(cls(DASH_K_GEMM_O), st);
            DASH_HIP(launch_gemm(dt, EPI_STORE_F32, w.o, m->lw(l, 3), w.delta, rows, d.d_model, hq, d.d_model, so,
                                 (size_t)rows * d.d_model, st));
        }
        {
            ProfScope ps(cls(DASH_K_NORM), st);
            DASH_HIP(launch_add_rmsnorm(dt, w.x, w.delta, so, (size_t)rows * d.d_model, m->lw(l, 4), w.y, nullptr, rows,
                                        d.d_model, d.rms_eps, 1, st));
        }
        {
            ProfScope ps(cls(DASH_K_GEMM_GATE_UP), st);
            DASH_HIP(launch_gemm(dt, EPI_SWIGLU, w.y, m->lw(l, 5), w.h, rows, 2 * d.d_ff, d.d_model, d.d_ff, 1, 0, st));
        }
        {
            ProfScope ps(cls(DASH_K_GEMM_DOWN), st);
            DASH_HIP(launch_gemm(dt, EPI_STORE_F32, w.h, m->lw(l, 6), w.delta, rows, d.d_model, d.d_ff, d.d_model, sd,
                                 (size_t)rows * d.d_model, st));
        }
    }
    *last_split = sd;
    return DASH_OK;
}

int check_ws(const dash_model* m, void* ws, size_t ws_bytes, int rows, int max_ctx) {
    if (rows > max_forward_rows(m))
        return fail(DASH_ENOTSUP, "%d rows exceed the %d one forward pass may hold", rows, max_forward_rows(m));
    if (!ws) return fail(DASH_EINVAL, "workspace is NULL");
    if ((uintptr_t)ws & 255) return fail(DASH_EINVAL, "workspace must be 256-byte aligned");
    const size_t need = plan_ws(m, rows, nullptr, max_ctx).bytes;
    if (ws_bytes < need) return fail(DASH_ECAPACITY, "workspace too small: %zu < %zu bytes for %d rows", ws_bytes, need, rows);
    return DASH_OK;
}

int decode_step_impl(dash_model* m, dash_kv* kv, const int32_t* tok, const int32_t* slot, const int32_t* pos, int rows,
                     float* logits, void* ws, hipStream_t st, const GroupInfo* gi = nullptr) {
    const auto& d = m->d;
    Ws w = plan_ws(m, rows, (char*)ws, kv->max_ctx);
    {
        ProfScope ps(DASH_K_EMBED, st);
        DASH_HIP(launch_embed_rmsnorm(d.dtype, tok, m->embed(), m->lw(0, 0), w.x, w.y, rows, d.d_model, d.vocab,
                                      d.rms_eps, kv->d_status, st));
    }
    int sd = 1;
    int rc = run_layers(m, kv, w, rows, pos, slot, false, 0, st, &sd, gi);
    if (rc) return rc;
    {
        ProfScope ps(DASH_K_NORM, st);
        DASH_HIP(launch_add_rmsnorm(d.dtype, w.x, w.delta, sd, (size_t)rows * d.d_model, m->final_norm(), w.y, nullptr,
                                    rows, d.d_model, d.rms_eps, 1, st));
    }
    ProfScope ps(DASH_K_GEMM_LM_HEAD, st);
    DASH_HIP(launch_gemm(d.dtype, EPI_STORE_F32, w.y, m->embed(), logits, rows, d.vocab, d.d_model, d.vocab, 1, 0, st));
    return DASH_OK;
}

int prefill_impl(dash_model* m, dash_kv* kv, const int32_t* d_tokens, int n_prompts, int P, int G,
                 const int32_t* h_slots, float* d_logits, void* ws, size_t ws_bytes, hipStream_t st) {
    const auto& d = m->d;
    // capacity: full prompt pages once per prompt, one private partial page per sample
    const size_t need = kv->pb.fork_need(n_prompts, P, G);
    if (need > kv->pb.free_pages())
        return fail(DASH_ECAPACITY, "pool exhausted: prefill needs %zu pages, %zu free", need, kv->pb.free_pages());
    const int rows_fit = ws_rows_for(m, ws_bytes, (int)std::min<int64_t>((int64_t)n_prompts * P, 0x7FFFFFFF));
    int chunk = rows_fit / P;
    if (chunk < 1)
        return fail(P > max_forward_rows(m) ? DASH_ENOTSUP : DASH_ECAPACITY,
                    "workspace cannot hold one prompt of %d tokens", P);
    const int n_chunks = (n_prompts + chunk - 1) / chunk;
    chunk = (n_prompts + n_chunks - 1) / n_chunks;  // as many chunks, of equal size (the last may be smaller)
    // host bookkeeping: pages of every sample's slot
    std::vector<int32_t> pairs;
    kv->pb.fork(h_slots, n_prompts, P, G, pairs);
    ReleaseOnError guard{kv, h_slots, n_prompts * G};
    int lo = kv->g.max_seqs, hi = -1;
    for (int i = 0; i < n_prompts * G; ++i) {
        lo = std::min(lo, h_slots[i]);
        hi = std::max(hi, h_slots[i]);
    }
    int rc = kv_push_rows(kv, lo, hi, st);
    if (rc) return rc;

    Ws w = plan_ws(m, chunk * P, (char*)ws, 0);
    for (int p0 = 0; p0 < n_prompts; p0 += chunk) {
        const int np = std::min(chunk, n_prompts - p0);
        const int rows = np * P;
        std::vector<int32_t> pos(rows), slot(rows), gather(np);
        for (int i = 0; i < rows; ++i) {
            pos[i] = i % P;
            slot[i] = h_slots[(p0 + i / P) * G];
        }
        for (int i = 0; i < np; ++i) gather[i] = i * P + P - 1;
        if ((rc = kv_upload(kv, w.pos, pos.data(), rows * 4, st))) return rc;
        if ((rc = kv_upload(kv, w.slot, slot.data(), rows * 4, st))) return rc;
        if ((rc = kv_upload(kv, w.gather, gather.data(), np * 4, st))) return rc;
        DASH_HIP(launch_embed_rmsnorm(d.dtype, d_tokens + (size_t)p0 * P, m->embed(), m->lw(0, 0), w.x, w.y, rows,
                                      d.d_model, d.vocab, d.rms_eps, kv->d_status, st));
        int sd = 1;
        if ((rc = run_layers(m, kv, w, rows, w.pos, w.slot, true, P, st, &sd, nullptr))) return rc;
        // final norm of the last position of every prompt only
        DASH_HIP(launch_add_rmsnorm(d.dtype, w.x, w.delta, sd, (size_t)rows * d.d_model, m->final_norm(), w.y, w.gather,
                                    np, d.d_model, d.rms_eps, 0, st));
        DASH_HIP(launch_gemm(d.dtype, EPI_STORE_F32, w.y, m->embed(), d_logits + (size_t)p0 * d.vocab, np, d.vocab,
                             d.d_model, d.vocab, 1, 0, st));
    }
    if (!pairs.empty()) {
        const int n = (int)pairs.size() / 2;
        for (int i0 = 0; i0 < n; i0 += chunk * P) {  // the pairs buffer holds rows-many pairs
            const int c = std::min(n - i0, chunk * P);
            if ((rc = kv_upload(kv, w.pairs, pairs.data() + 2 * i0, (size_t)c * 8, st))) return rc;
            DASH_HIP(launch_copy_pages(d.dtype, kv->pool, kv->g, w.pairs, c, st));
        }
    }
    guard.armed = false;
    return DASH_OK;
}

}  // namespace

extern "C" {

int dash_prefill(dash_model* m, dash_kv* kv, const int32_t* d_tokens, int32_t n_prompts, int32_t P, int32_t G,
                 const int32_t* h_slots, float* d_logits, void* ws, size_t ws_bytes, void* stream) {
    if (!m || !kv || !d_tokens || !h_slots || !d_logits) return fail(DASH_EINVAL, "dash_prefill: NULL argument");
    if (kv->m != m) return fail(DASH_EINVAL, "kv handle belongs to another model");
    if (n_prompts < 1 || P < 1 || G < 1) return fail(DASH_EINVAL, "n_prompts, prompt_len and group must be >= 1");
    if (P > kv->max_ctx) return fail(DASH_ECAPACITY, "prompt_len %d exceeds max_ctx %d", P, kv->max_ctx);
    if ((int64_t)n_prompts * G > kv->g.max_seqs) return fail(DASH_ECAPACITY, "more samples than slots");
    std::vector<char> seen(kv->g.max_seqs, 0);
    for (int i = 0; i < n_prompts * G; ++i) {
        const int s = h_slots[i];
        if (s < 0 || s >= kv->g.max_seqs) return fail(DASH_EINVAL, "slot %d out of range", s);
        if (seen[s]) return fail(DASH_EINVAL, "slot %d listed twice", s);
        seen[s] = 1;
        if (!kv->pb.empty(s)) return fail(DASH_EINVAL, "slot %d is not empty", s);
    }
    if (!ws) return fail(DASH_EINVAL, "workspace is NULL");
    if ((uintptr_t)ws & 255) return fail(DASH_EINVAL, "workspace must be 256-byte aligned");
    ProfScope ps(DASH_K_PREFILL, (hipStream_t)stream);
    return prefill_impl(m, kv, d_tokens, n_prompts, P, G, h_slots, d_logits, ws, ws_bytes, (hipStream_t)stream);
}

int dash_decode_step(dash_model* m, dash_kv* kv, const int32_t* tok, const int32_t* slot, const int32_t* pos,
                     int32_t rows, float* logits, void* ws, size_t ws_bytes, void* stream) {
    if (!m || !kv || !tok || !slot || !pos || !logits) return fail(DASH_EINVAL, "dash_decode_step: NULL argument");
    if (kv->m != m) return fail(DASH_EINVAL, "kv handle belongs to another model");
    if (rows < 1) return fail(DASH_EINVAL, "n_rows must be >= 1");
    int rc = check_ws(m, ws, ws_bytes, rows, kv->max_ctx);
    if (rc) return rc;
    return decode_step_impl(m, kv, tok, slot, pos, rows, logits, ws, (hipStream_t)stream);
}

}  // extern "C"

// ------------------------------------------- allocation-free decode step ----
// dash_decode_step_noalloc runs the decode step with its workspace in `scratch`,
// a device array of this file (one copy per device, held until the process ends).
// In host code `scratch` names a host-side stand-in, never a device address: the
// device address comes from hipGetSymbolAddress, once per device, and only that
// address is handed to kernels.  No kernel of the decode step needs any of the
// scratch to start at zero (every buffer is written before it is read in the same
// call), so nothing is cleared between calls.

namespace {

constexpr size_t kScratchBytes = (size_t)64 << 20;
constexpr int kMaxDevices = 64;
static __device__ __align__(256) char scratch[kScratchBytes];

std::mutex g_scratch_mu;
void* g_scratch_dev[kMaxDevices] = {};

// Device address of the current device's scratch (looked up on the first call per device).
int scratch_address(void** out) {
    int dev = -1;
    DASH_HIP(hipGetDevice(&dev));
    if (dev < 0 || dev >= kMaxDevices) return fail(DASH_ENOTSUP, "device %d beyond the %d supported", dev, kMaxDevices);
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    if (!g_scratch_dev[dev]) {
        void* p = nullptr;
        const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess || !p) return fail(DASH_EDEVICE, "hipGetSymbolAddress(scratch): %s", hipGetErrorString(e));
        g_scratch_dev[dev] = p;
    }
    *out = g_scratch_dev[dev];
    return DASH_OK;
}

}  // namespace

extern "C" {

int dash_decode_step_noalloc(dash_model* m, dash_kv* kv, const int32_t* tok, const int32_t* slot, const int32_t* pos,
                             int32_t rows, float* logits, void* stream) {
    if (!m || !kv || !tok || !slot || !pos || !logits) return fail(DASH_EINVAL, "dash_decode_step_noalloc: NULL argument");
    if (kv->m != m) return fail(DASH_EINVAL, "kv handle belongs to another model");
    if (rows < 1) return fail(DASH_EINVAL, "n_rows must be >= 1");
    if (rows > max_forward_rows(m))
        return fail(DASH_ENOTSUP, "%d rows exceed the %d one forward pass may hold", rows, max_forward_rows(m));
    const size_t need = plan_ws(m, rows, nullptr, kv->max_ctx).bytes;
    if (need > kScratchBytes)
        return fail(DASH_ECAPACITY, "%d rows need %zu bytes of workspace; the allocation-free decode step has %zu",
                    rows, need, kScratchBytes);
    void* ws = nullptr;
    const int rc = scratch_address(&ws);
    if (rc) return rc;
    return decode_step_impl(m, kv, tok, slot, pos, rows, logits, ws, (hipStream_t)stream);
}

int dash_decode_step_grouped(dash_model* m, dash_kv* kv, const int32_t* tok, const int32_t* slot, const int32_t* pos,
                             int32_t rows, const int32_t* d_group_off, int32_t n_groups, int32_t group_size,
                             int32_t shared_len, float* logits, void* ws, size_t ws_bytes, void* stream) {
    if (!m || !kv || !tok || !slot || !pos || !logits || !d_group_off)
        return fail(DASH_EINVAL, "dash_decode_step_grouped: NULL argument");
    if (kv->m != m) return fail(DASH_EINVAL, "kv handle belongs to another model");
    if (rows < 1 || n_groups < 1 || n_groups > rows) return fail(DASH_EINVAL, "bad n_rows / n_groups");
    if (group_size < 1 || group_size > kMaxGroupRows) return fail(DASH_ENOTSUP, "group_size must be in [1, %d]", kMaxGroupRows);
    if (shared_len < 0 || shared_len % kv->g.page_size || shared_len > kv->max_ctx)
        return fail(DASH_EINVAL, "shared_len must be a multiple of page_size, at most max_ctx");
    int rc = check_ws(m, ws, ws_bytes, rows, kv->max_ctx);
    if (rc) return rc;
    if (m->d.dtype != DASH_BF16)  // the fp32 path has no grouped kernel: same results without it
        return decode_step_impl(m, kv, tok, slot, pos, rows, logits, ws, (hipStream_t)stream);
    GroupInfo gi{d_group_off, n_groups, group_size, shared_len};
    return decode_step_impl(m, kv, tok, slot, pos, rows, logits, ws, (hipStream_t)stream, &gi);
}

int dash_sample(const float* logits, int64_t ld, int32_t rows, int32_t vocab, const int32_t* row_of,
                const int32_t* uid, const int32_t* step, float temperature, uint64_t seed, int32_t* tok_out,
                float* lp_out, float* row_max_lse, uint32_t* d_status, void* stream) {
    if (!logits || !uid || !step || !tok_out) return fail(DASH_EINVAL, "dash_sample: NULL argument");
    if (rows < 0 || vocab < 1 || vocab > (1 << 28) || ld < vocab) return fail(DASH_EINVAL, "dash_sample: bad sizes");
    if (!(temperature > 0.f) || !std::isfinite(temperature)) return fail(DASH_EINVAL, "temperature must be > 0 and finite");
    if (rows == 0) return DASH_OK;
    ProfScope ps(DASH_K_SAMPLE, (hipStream_t)stream);
    DASH_HIP(launch_sample(logits, ld, rows, vocab, row_of, uid, step, temperature, seed, tok_out, lp_out, row_max_lse,
                           d_status, nullptr, nullptr, 0, (hipStream_t)stream));
    return DASH_OK;
}

int dash_sampler_check(double* h_max_err, double* h_tol) {
    if (!h_max_err || !h_tol) return fail(DASH_EINVAL, "dash_sampler_check: NULL argument");
    float f = 0.f;
    const hipError_t e = sampler_screen_check(&f);
    if (e != hipSuccess) return fail(DASH_EDEVICE, "sampler check: %s", hipGetErrorString(e));
    *h_max_err = f;
    *h_tol = sampler_screen_tol();
    return DASH_OK;
}

int dash_bf16_round_check(uint64_t* h_mismatches) {
    if (!h_mismatches) return fail(DASH_EINVAL, "dash_bf16_round_check: NULL argument");
    unsigned long long n = 0;
    const hipError_t e = bf16_round_check(&n);
    if (e != hipSuccess) return fail(DASH_EDEVICE, "bf16 rounding check: %s", hipGetErrorString(e));
    *h_mismatches = n;
    return DASH_OK;
}

int dash_group_advantage_filter(const float* r, int32_t n_groups, int32_t group, int32_t mode, float eps, float tau,
                                float* adv, int32_t* kept, int32_t* count, void* stream) {
    if (!r || !adv || !kept || !count) return fail(DASH_EINVAL, "dash_group_advantage_filter: NULL argument");
    if (n_groups < 1 || group < 1) return fail(DASH_EINVAL, "n_groups and group must be >= 1");
    if (mode < DASH_ADV_MEAN_ONLY || mode > DASH_ADV_LOO) return fail(DASH_EINVAL, "bad mode %d", mode);
    if (mode == DASH_ADV_LOO && group < 2) return fail(DASH_EINVAL, "the leave-one-out baseline needs group >= 2");
    if (!(eps >= 0.f) || !(tau >= 0.f)) return fail(DASH_EINVAL, "eps and tau must be >= 0 (and not NaN)");
    if (group > 65536) return fail(DASH_ENOTSUP, "group > 65536");
    if ((int64_t)n_groups * group > (1 << 24)) return fail(DASH_ENOTSUP, "more than 2^24 samples");
    ProfScope ps(DASH_K_ADVANTAGE, (hipStream_t)stream);
    DASH_HIP(launch_group_advantage_filter(r, n_groups, group, mode, eps, tau, adv, kept, count, (hipStream_t)stream));
    return DASH_OK;
}

int dash_live_compact(const int32_t* tok, const int32_t* slot, const int32_t* pos, const int32_t* step,
                      const int32_t* uid, const int32_t* budget, int32_t eos_id, int32_t n, int32_t* tok_o,
                      int32_t* slot_o, int32_t* pos_o, int32_t* step_o, int32_t* uid_o, int32_t* count, void* stream) {
    if (!tok || !slot || !pos || !step || !uid || !budget || !tok_o || !slot_o || !pos_o || !step_o || !uid_o || !count)
        return fail(DASH_EINVAL, "dash_live_compact: NULL argument");
    if (n < 0) return fail(DASH_EINVAL, "n_rows must be >= 0");
    DASH_HIP(launch_live_compact(tok, slot, pos, step, uid, budget, eos_id, n, tok_o, slot_o, pos_o, step_o, uid_o,
                                 count, (hipStream_t)stream));
    return DASH_OK;
}

// ------------------------------------------------------ rollout driver ----

namespace {

struct RolloutWs {
    Ws step;
    float* logits;
    int32_t* st[2][5];  // tok, slot, pos, step, uid
    int32_t* row_of;
    int32_t* budget;
    int32_t* count;
    size_t bytes;
};

RolloutWs plan_rollout(const dash_model* m, int n_prompts, int P, int G, int max_ctx, char* base) {
    const int N = n_prompts * G;
    // prefill chunks of up to 64 prompts (rows = 64 P) unless the batch is smaller
    const int prefill_rows = std::min(n_prompts, std::max(1, 16384 / std::max(1, P))) * P;
    const int rows = std::max(N, prefill_rows);
    RolloutWs r{};
    r.step = plan_ws(m, rows, base, max_ctx, N);
    size_t off = r.step.bytes;
    auto take = [&](size_t bytes) {
        char* p = base ? base + off : nullptr;
        off = align_up(off + bytes, 256);
        return p;
    };
    r.logits = (float*)take((size_t)std::max(N, n_prompts) * m->d.vocab * 4);
    for (int b = 0; b < 2; ++b)
        for (int i = 0; i < 5; ++i) r.st[b][i] = (int32_t*)take((size_t)N * 4);
    r.row_of = (int32_t*)take((size_t)N * 4);
    r.budget = (int32_t*)take((size_t)N * 4);
    r.count = (int32_t*)take(256);
    r.bytes = off;
    return r;
}

}  // namespace

namespace {

// Teacher-forced log-probs: the prefill plan for c sequences of L tokens, then
// the fp32 logits of their c * (L - P) scored positions.
struct TfWs {
    Ws step;
    float* logits;
    size_t bytes;
};

TfWs plan_tf(const dash_model* m, int c, int L, int P, char* base) {
    TfWs t{};
    t.step = plan_ws(m, c * L, base, 0);
    size_t off = t.step.bytes;
    t.logits = base ? (float*)(base + off) : nullptr;
    off = align_up(off + (size_t)c * (L - P) * m->d.vocab * 4, 256);
    t.bytes = off;
    return t;
}

// Forward of a chunk of whole sequences (rows = sequences x L tokens, positions,
// slots and gather rows already uploaded to w, pages mapped) through model m on
// kv's pages; the LM head writes the logits of the rows_lm gathered positions.
int tf_forward(dash_model* m, dash_kv* kv, const Ws& w, const int32_t* tok, int rows, int rows_lm, int L,
               float* logits, hipStream_t st) {
    const auto& d = m->d;
    DASH_HIP(launch_embed_rmsnorm(d.dtype, tok, m->embed(), m->lw(0, 0), w.x, w.y, rows, d.d_model, d.vocab, d.rms_eps,
                                  kv->d_status, st));
    int sd = 1, rc;
    if ((rc = run_layers(m, kv, w, rows, w.pos, w.slot, true, L, st, &sd, nullptr))) return rc;
    // final norm of the positions that predict a completion token, then the LM head
    DASH_HIP(launch_add_rmsnorm(d.dtype, w.x, w.delta, sd, (size_t)rows * d.d_model, m->final_norm(), w.y, w.gather,
                                rows_lm, d.d_model, d.rms_eps, 0, st));
    DASH_HIP(launch_gemm(d.dtype, EPI_STORE_F32, w.y, m->embed(), logits, rows_lm, d.vocab, d.d_model, d.vocab, 1, 0,
                         st));
    return DASH_OK;
}

// Teacher-forced KL workspace: the step buffers plus logits of both models.
struct TfKlWs {
    Ws step;
    float* logits;
    float* logits_base;
    size_t bytes;
};

TfKlWs plan_tf_kl(const dash_model* m, int c, int L, int P, char* base) {
    TfKlWs t{};
    t.step = plan_ws(m, c * L, base, 0);
    const size_t lb = (size_t)c * (L - P) * m->d.vocab * 4;
    size_t off = t.step.bytes;
    t.logits = base ? (float*)(base + off) : nullptr;
    off = align_up(off + lb, 256);
    t.logits_base = base ? (float*)(base + off) : nullptr;
    t.bytes = align_up(off + lb, 256);
    return t;
}

bool same_architecture(const dash_model_desc& a, const dash_model_desc& b) {
    return a.n_layers == b.n_layers && a.d_model == b.d_model && a.n_heads == b.n_heads &&
           a.n_kv_heads == b.n_kv_heads && a.head_dim == b.head_dim && a.d_ff == b.d_ff && a.vocab == b.vocab &&
           a.dtype == b.dtype && a.rope_theta == b.rope_theta && a.rms_eps == b.rms_eps;
}

}  // namespace

size_t dash_teacher_forced_workspace_bytes(const dash_model* m, int32_t seqs_per_chunk, int32_t L, int32_t P) {
    if (!m || seqs_per_chunk < 1 || P < 1 || L <= P) return 0;
    return plan_tf(m, seqs_per_chunk, L, P, nullptr).bytes;
}

int dash_teacher_forced_logprobs(dash_model* m, dash_kv* kv, const int32_t* d_tokens, int32_t n_seqs, int32_t L,
                                 int32_t P, float* d_lp, void* ws, size_t ws_bytes, void* stream) {
    if (!m || !kv || !d_tokens || !d_lp || !ws) return fail(DASH_EINVAL, "dash_teacher_forced_logprobs: NULL argument");
    if (kv->m != m) return fail(DASH_EINVAL, "kv handle belongs to another model");
    if (n_seqs < 1 || P < 1 || L <= P) return fail(DASH_EINVAL, "need n_seqs >= 1 and 1 <= prompt_len < seq_len");
    if (L > kv->max_ctx) return fail(DASH_ECAPACITY, "seq_len %d exceeds max_ctx %d", L, kv->max_ctx);
    if ((uintptr_t)ws & 255) return fail(DASH_EINVAL, "workspace must be 256-byte aligned");
    const hipStream_t st = (hipStream_t)stream;
    const auto& d = m->d;
    const int ps = kv->g.page_size;
    const int pps = (L + ps - 1) / ps;  // private pages per sequence
    const int Tg = L - P;
    // chunk: the most sequences that fit the workspace, the slots and the free pages
    int cmax = std::min<int>(n_seqs, kv->g.max_seqs);
    cmax = std::min<int>(cmax, (int)(kv->pb.free_pages() / pps));
    if (cmax < 1) return fail(DASH_ECAPACITY, "the pool cannot hold one sequence of %d tokens", L);
    cmax = std::min(cmax, max_forward_rows(m) / L);  // every row of a chunk goes through the GEMMs
    if (cmax < 1) return fail(DASH_ENOTSUP, "seq_len %d exceeds the rows one forward pass may hold", L);
    int lo = 0, hi = cmax;
    while (lo < hi) {
        const int mid = (lo + hi + 1) / 2;
        if (plan_tf(m, mid, L, P, nullptr).bytes <= ws_bytes) lo = mid;
        else hi = mid - 1;
    }
    const int c = lo;
    if (c < 1)
        return fail(DASH_ECAPACITY, "workspace too small: %zu < %zu bytes for one sequence", ws_bytes,
                    plan_tf(m, 1, L, P, nullptr).bytes);
    for (int j = 0; j < c; ++j)
        if (!kv->pb.empty(j)) return fail(DASH_EINVAL, "kv slot %d is not empty", j);
    const TfWs t = plan_tf(m, c, L, P, (char*)ws);
    const Ws& w = t.step;
    std::vector<int32_t> pos, slot, gather, slots(c);
    for (int j = 0; j < c; ++j) slots[j] = j;
    int rc;
    for (int s0 = 0; s0 < n_seqs; s0 += c) {
        const int nc = std::min(c, n_seqs - s0);
        for (int j = 0; j < nc; ++j) kv->pb.grow(j, L);
        ReleaseOnError guard{kv, slots.data(), nc};
        if ((rc = kv_push_rows(kv, 0, nc - 1, st))) return rc;
        const int rows = nc * L, rows_lm = nc * Tg;
        pos.resize(rows);
        slot.resize(rows);
        gather.resize(rows_lm);
        for (int i = 0; i < rows; ++i) {
            pos[i] = i % L;
            slot[i] = i / L;
        }
        for (int i = 0; i < rows_lm; ++i) gather[i] = (i / Tg) * L + P - 1 + i % Tg;
        if ((rc = kv_upload(kv, w.pos, pos.data(), (size_t)rows * 4, st))) return rc;
        if ((rc = kv_upload(kv, w.slot, slot.data(), (size_t)rows * 4, st))) return rc;
        if ((rc = kv_upload(kv, w.gather, gather.data(), (size_t)rows_lm * 4, st))) return rc;
        const int32_t* tok = d_tokens + (size_t)s0 * L;
        if ((rc = tf_forward(m, kv, w, tok, rows, rows_lm, L, t.logits, st))) return rc;
        DASH_HIP(launch_logprob_gather(t.logits, d.vocab, rows_lm, d.vocab, tok, Tg, L, P, d_lp + (size_t)s0 * Tg, st));
        guard.armed = false;
        if ((rc = dash_kv_release(kv, slots.data(), nc))) return rc;
    }
    return DASH_OK;
}

int dash_pg_loss(const float* d_lp, int64_t ld, int32_t T, const int32_t* d_len, const float* d_adv,
                 const int32_t* d_kept, const int32_t* d_kept_count, int32_t n_total, double* d_loss,
                 double* d_seq_lp, void* stream) {
    if (!d_lp || !d_adv || !d_kept || !d_kept_count || !d_loss) return fail(DASH_EINVAL, "dash_pg_loss: NULL argument");
    if (T < 1 || ld < T || n_total < 1) return fail(DASH_EINVAL, "dash_pg_loss: bad sizes");
    DASH_HIP(launch_pg_loss(d_lp, ld, T, d_len, d_adv, d_kept, d_kept_count, n_total, d_loss, d_seq_lp,
                            (hipStream_t)stream));
    return DASH_OK;
}

int dash_policy_loss(const float* d_lp, const float* d_lp_old, const float* d_kl, int64_t ld, int32_t T,
                     const int32_t* d_len, const float* d_adv, const int32_t* d_kept, const int32_t* d_kept_count,
                     int32_t n_total, double clip_eps, double beta, double* d_loss, double* d_stats, void* stream) {
    if (!d_lp || !d_adv || !d_kept || !d_kept_count || !d_loss)
        return fail(DASH_EINVAL, "dash_policy_loss: NULL argument");
    if (T < 1 || ld < T || n_total < 1) return fail(DASH_EINVAL, "dash_policy_loss: bad sizes");
    if (d_lp_old && !(clip_eps >= 0.0 && clip_eps < 1.0))
        return fail(DASH_EINVAL, "dash_policy_loss: clip_eps must lie in [0, 1)");
    if (!std::isfinite(beta)) return fail(DASH_EINVAL, "dash_policy_loss: beta must be finite");
    DASH_HIP(launch_policy_loss(d_lp, d_lp_old, d_kl, ld, T, d_len, d_adv, d_kept, d_kept_count, n_total, clip_eps,
                                beta, d_loss, nullptr, d_stats, (hipStream_t)stream));
    return DASH_OK;
}

int dash_logits_kl(const float* d_theta, const float* d_base, int64_t ld, int32_t rows, int32_t vocab, float* d_kl,
                   float* d_kl_rev, void* stream) {
    if (!d_theta || !d_base || !d_kl) return fail(DASH_EINVAL, "dash_logits_kl: NULL argument");
    if (rows < 0 || vocab < 1 || ld < vocab) return fail(DASH_EINVAL, "dash_logits_kl: bad sizes");
    DASH_HIP(launch_logits_kl(d_theta, d_base, ld, rows, vocab, d_kl, d_kl_rev, (hipStream_t)stream));
    return DASH_OK;
}

size_t dash_teacher_forced_kl_workspace_bytes(const dash_model* m, int32_t seqs_per_chunk, int32_t L, int32_t P) {
    if (!m || seqs_per_chunk < 1 || P < 1 || L <= P) return 0;
    return plan_tf_kl(m, seqs_per_chunk, L, P, nullptr).bytes;
}

int dash_teacher_forced_kl(dash_model* m, dash_model* base, dash_kv* kv, const int32_t* d_tokens, int32_t n_seqs,
                           int32_t L, int32_t P, float* d_lp, float* d_kl, float* d_kl_rev, void* ws, size_t ws_bytes,
                           void* stream) {
    if (!m || !base || !kv || !d_tokens || !d_kl || !ws) return fail(DASH_EINVAL, "dash_teacher_forced_kl: NULL argument");
    if (kv->m != m) return fail(DASH_EINVAL, "kv handle belongs to another model");
    if (!same_architecture(m->d, base->d))
        return fail(DASH_EINVAL, "the base model must have the policy model's architecture");
    if (n_seqs < 1 || P < 1 || L <= P) return fail(DASH_EINVAL, "need n_seqs >= 1 and 1 <= prompt_len < seq_len");
    if (L > kv->max_ctx) return fail(DASH_ECAPACITY, "seq_len %d exceeds max_ctx %d", L, kv->max_ctx);
    if ((uintptr_t)ws & 255) return fail(DASH_EINVAL, "workspace must be 256-byte aligned");
    const hipStream_t st = (hipStream_t)stream;
    const auto& d = m->d;
    const int ps = kv->g.page_size;
    const int pps = (L + ps - 1) / ps;
    const int Tg = L - P;
    int cmax = std::min<int>(n_seqs, kv->g.max_seqs);
    cmax = std::min<int>(cmax, (int)(kv->pb.free_pages() / pps));
    if (cmax < 1) return fail(DASH_ECAPACITY, "the pool cannot hold one sequence of %d tokens", L);
    cmax = std::min(cmax, max_forward_rows(m) / L);
    if (cmax < 1) return fail(DASH_ENOTSUP, "seq_len %d exceeds the rows one forward pass may hold", L);
    int lo = 0, hi = cmax;
    while (lo < hi) {
        const int mid = (lo + hi + 1) / 2;
        if (plan_tf_kl(m, mid, L, P, nullptr).bytes <= ws_bytes) lo = mid;
        else hi = mid - 1;
    }
    const int c = lo;
    if (c < 1)
        return fail(DASH_ECAPACITY, "workspace too small: %zu < %zu bytes for one sequence", ws_bytes,
                    plan_tf_kl(m, 1, L, P, nullptr).bytes);
    for (int j = 0; j < c; ++j)
        if (!kv->pb.empty(j)) return fail(DASH_EINVAL, "kv slot %d is not empty", j);
    const TfKlWs t = plan_tf_kl(m, c, L, P, (char*)ws);
    const Ws& w = t.step;
    std::vector<int32_t> pos, slot, gather, slots(c);
    for (int j = 0; j < c; ++j) slots[j] = j;
    int rc;
    for (int s0 = 0; s0 < n_seqs; s0 += c) {
        const int nc = std::min(c, n_seqs - s0);
        for (int j = 0; j < nc; ++j) kv->pb.grow(j, L);
        ReleaseOnError guard{kv, slots.data(), nc};
        if ((rc = kv_push_rows(kv, 0, nc - 1, st))) return rc;
        const int rows = nc * L, rows_lm = nc * Tg;
        pos.resize(rows);
        slot.resize(rows);
        gather.resize(rows_lm);
        for (int i = 0; i < rows; ++i) {
            pos[i] = i % L;
            slot[i] = i / L;
        }
        for (int i = 0; i < rows_lm; ++i) gather[i] = (i / Tg) * L + P - 1 + i % Tg;
        if ((rc = kv_upload(kv, w.pos, pos.data(), (size_t)rows * 4, st))) return rc;
        if ((rc = kv_upload(kv, w.slot, slot.data(), (size_t)rows * 4, st))) return rc;
        if ((rc = kv_upload(kv, w.gather, gather.data(), (size_t)rows_lm * 4, st))) return rc;
        const int32_t* tok = d_tokens + (size_t)s0 * L;
        // the base model first: its cache entries are then overwritten by the policy's
        if ((rc = tf_forward(base, kv, w, tok, rows, rows_lm, L, t.logits_base, st))) return rc;
        if ((rc = tf_forward(m, kv, w, tok, rows, rows_lm, L, t.logits, st))) return rc;
        if (d_lp)
            DASH_HIP(launch_logprob_gather(t.logits, d.vocab, rows_lm, d.vocab, tok, Tg, L, P, d_lp + (size_t)s0 * Tg,
                                           st));
        DASH_HIP(launch_logits_kl(t.logits, t.logits_base, d.vocab, rows_lm, d.vocab, d_kl + (size_t)s0 * Tg,
                                  d_kl_rev ? d_kl_rev + (size_t)s0 * Tg : nullptr, st));
        guard.armed = false;
        if ((rc = dash_kv_release(kv, slots.data(), nc))) return rc;
    }
    return DASH_OK;
}

size_t dash_rollout_workspace_bytes(const dash_model* m, int32_t n_prompts, int32_t P, int32_t G, int32_t max_ctx) {
    if (!m || n_prompts < 1 || P < 1 || G < 1 || max_ctx < 1) return 0;
    return plan_rollout(m, n_prompts, P, G, max_ctx, nullptr).bytes;
}

int dash_rollout(dash_model* m, dash_kv* kv, const int32_t* d_prompts, int32_t n_prompts, int32_t P, int32_t G,
                 int32_t T, const int32_t* h_budget, float temperature, uint64_t seed, int32_t* d_out_tokens,
                 float* d_out_lp, int32_t use_graph, void* ws, size_t ws_bytes, void* stream) {
    if (!m || !kv || !d_prompts || !d_out_tokens || !ws) return fail(DASH_EINVAL, "dash_rollout: NULL argument");
    if (kv->m != m) return fail(DASH_EINVAL, "kv handle belongs to another model");
    if (n_prompts < 1 || P < 1 || G < 1 || T < 1) return fail(DASH_EINVAL, "sizes must be >= 1");
    if (!(temperature > 0.f) || !std::isfinite(temperature)) return fail(DASH_EINVAL, "temperature must be > 0 and finite");
    if ((int64_t)n_prompts * G > kv->g.max_seqs)
        return fail(DASH_ECAPACITY, "kv has %d slots, rollout needs %lld", kv->g.max_seqs, (long long)n_prompts * G);
    const int N = n_prompts * G;
    if (N > max_forward_rows(m)) return fail(DASH_ENOTSUP, "%d rows exceed the rows one forward pass may hold", N);
    if (P + T > kv->max_ctx) return fail(DASH_ECAPACITY, "prompt_len + gen_len exceeds max_ctx");
    for (int s = 0; s < N; ++s)
        if (!kv->pb.empty(s)) return fail(DASH_EINVAL, "kv slot %d is not empty", s);
    std::vector<int32_t> budget(N, T);
    if (h_budget)
        for (int i = 0; i < N; ++i) {
            if (h_budget[i] < 1 || h_budget[i] > T) return fail(DASH_EINVAL, "budget[%d] = %d outside [1, %d]", i, h_budget[i], T);
            budget[i] = h_budget[i];
        }
    if ((uintptr_t)ws & 255) return fail(DASH_EINVAL, "workspace must be 256-byte aligned");
    RolloutWs rw = plan_rollout(m, n_prompts, P, G, kv->max_ctx, (char*)ws);
    if (ws_bytes < rw.bytes) return fail(DASH_ECAPACITY, "rollout workspace too small: %zu < %zu", ws_bytes, rw.bytes);
    // page budget: worst case with every page private except shared full prompt pages
    {
        const int ps = kv->g.page_size;
        size_t need = (size_t)n_prompts * (P / ps);
        for (int i = 0; i < N; ++i) need += (size_t)(P + budget[i] + ps - 1) / ps - P / ps;
        if (need > kv->pb.free_pages())
            return fail(DASH_ECAPACITY, "pool too small for this rollout: %zu pages needed, %zu free", need,
                        kv->pb.free_pages());
    }
    hipStream_t st = (hipStream_t)stream;
    const auto& d = m->d;
    const int V = d.vocab;
    const bool ragged = std::any_of(budget.begin(), budget.end(), [&](int b) { return b != T; });
    const size_t step_ws_bytes = rw.step.bytes;
    // the prompt's full pages are shared by the group's G rows for the whole rollout
    // (decode attention keeps them cached); restored on every way out
    struct SharedKeys {
        KVGeom& g;
        int saved;
        ~SharedKeys() { g.shared_keys = saved; }
    } shared_keys_scope{kv->g, kv->g.shared_keys};
    kv->g.shared_keys = G > 1 ? P / kv->g.page_size * kv->g.page_size : 0;

    DASH_HIP(launch_fill_i32(d_out_tokens, -1, (size_t)N * T, st));
    int rc;
    if ((rc = kv_upload(kv, rw.budget, budget.data(), (size_t)N * 4, st))) return rc;
    std::vector<int32_t> slots(N);
    for (int i = 0; i < N; ++i) slots[i] = i;
    // 1. prefill
    {
        ProfScope ps(DASH_K_PREFILL, st);
        if ((rc = prefill_impl(m, kv, d_prompts, n_prompts, P, G, slots.data(), rw.logits, ws, step_ws_bytes, st)))
            return rc;
    }
    // 2. first token of every sample from its prompt's logits row
    int cur = 0;
    int32_t** S = rw.st[cur];  // tok, slot, pos, step, uid
    DASH_HIP(launch_rows_init(S[1], S[4], S[2], S[3], N, P - 1, 0, st));
    DASH_HIP(launch_iota_div(rw.row_of, N, G, st));
    DASH_HIP(launch_sample(rw.logits, V, N, V, rw.row_of, S[4], S[3], temperature, seed, S[0], nullptr, nullptr,
                           kv->d_status, d_out_tokens, d_out_lp, T, st));
    // live rows after each step are known on the host from the budgets
    std::vector<int> live_after(T + 1, 0);  // rows live for step t (t >= 1): budget > t
    for (int i = 0; i < N; ++i)
        for (int t = 1; t < budget[i] && t <= T; ++t) live_after[t]++;
    std::vector<std::vector<int32_t>> done_at(T + 1);  // samples whose last token is step t
    for (int i = 0; i < N; ++i) done_at[budget[i] - 1].push_back(i);

    auto advance = [&](int n_rows) -> int {
        if (!ragged) {
            DASH_HIP(launch_rows_advance(S[2], S[3], n_rows, st));
            return DASH_OK;
        }
        int32_t** O = rw.st[cur ^ 1];
        DASH_HIP(launch_live_compact(S[0], S[1], S[2], S[3], S[4], rw.budget, -1, n_rows, O[0], O[1], O[2], O[3], O[4],
                                     rw.count, st));
        cur ^= 1;
        S = rw.st[cur];
        return DASH_OK;
    };
    if ((rc = advance(N))) return rc;
    if ((rc = dash_kv_release(kv, done_at[0].data(), (int)done_at[0].size()))) return rc;

    // Decode attention runs per row here.  The prefix-shared form (dash_decode_step_grouped:
    // the group's prompt pages once per group and kv head, then every row continued from
    // that state, bit-identical) was measured slower on the 1.5B, 1024-sequence rollout:
    // its prefix kernel takes 23.6 us per launch while skipping the 8 shared blocks saves
    // the per-row kernel 12.5-16 us (those blocks come from L2 and overlap its streaming).

    // Decode steps.  With graphs, one step (decode + sample + advance) is captured
    // once and replayed; when kernel classes are being timed, two copies are
    // captured, each with its own events, and replayed alternately so that one
    // copy's timings are read back while the other runs.
    const bool graphs = use_graph && !ragged && st != nullptr;
    const int n_exec = graphs && g_prof.mask ? 2 : 1;
    hipGraphExec_t exec[2] = {nullptr, nullptr};
    GraphProf gprof[2];
    int64_t replays = 0;
    auto destroy_graphs = [&]() {
        for (int i = 0; i < 2; ++i)
            if (exec[i]) {
                gprof[i].harvest();
                (void)hipGraphExecDestroy(exec[i]);
                exec[i] = nullptr;
            }
    };
    auto one_step = [&](int B) -> int {
        int rc2 = decode_step_impl(m, kv, S[0], S[1], S[2], B, rw.logits, ws, st);
        if (rc2) return rc2;
        {
            ProfScope ps(DASH_K_SAMPLE, st);
            DASH_HIP(launch_sample(rw.logits, V, B, V, nullptr, S[4], S[3], temperature, seed, S[0], nullptr, nullptr,
                                   kv->d_status, d_out_tokens, d_out_lp, T, st));
        }
        ProfScope ps(DASH_K_OTHER, st);
        return advance(B);
    };
    auto capture = [&](int i, int B) -> int {
        // timed launches per step: at most 12 per layer plus a few outside the layers
        if (g_prof.mask && !gprof[i].reserve(12 * (size_t)d.n_layers + 16))
            return fail(DASH_EDEVICE, "hipEventCreate failed");
        DASH_HIP(hipStreamBeginCapture(st, hipStreamCaptureModeThreadLocal));
        g_prof.capturing = true;
        g_prof.capture_set = &gprof[i];
        const int rc2 = one_step(B);
        g_prof.capturing = false;
        g_prof.capture_set = nullptr;
        hipGraph_t graph = nullptr;
        hipError_t e = hipStreamEndCapture(st, &graph);
        if (rc2) {
            if (graph) (void)hipGraphDestroy(graph);
            return rc2;
        }
        if (e != hipSuccess) return fail(DASH_EDEVICE, "hipStreamEndCapture: %s", hipGetErrorString(e));
        e = hipGraphInstantiate(&exec[i], graph, nullptr, nullptr, 0);
        (void)hipGraphDestroy(graph);
        if (e != hipSuccess) return fail(DASH_EDEVICE, "hipGraphInstantiate: %s", hipGetErrorString(e));
        return DASH_OK;
    };
    std::vector<int32_t> live_slots;
    for (int t = 1; t < T; ++t) {
        const int B = ragged ? live_after[t] : N;
        if (B == 0) break;
        // rows live at step t feed position P + t - 1: reserve pages covering it
        const int need_len = P + t;
        if ((need_len - 1) % kv->g.page_size == 0) {
            live_slots.clear();
            for (int i = 0; i < N; ++i)
                if (budget[i] > t) live_slots.push_back(i);
            // one page ahead, capped at the last position the sample will feed (P + budget - 2)
            const int ahead = (need_len + kv->g.page_size - 1) / kv->g.page_size * kv->g.page_size;
            for (int s : live_slots) kv->pb.grow(s, std::min(P + budget[s] - 1, ahead));
            if ((rc = kv_push_rows(kv, live_slots.front(), live_slots.back(), st))) {
                destroy_graphs();
                return rc;
            }
        }
        if (graphs) {
            const int i = (int)(replays % n_exec);
            if (!exec[i] && (rc = capture(i, B))) {
                destroy_graphs();
                return rc;
            }
            gprof[i].harvest();  // the timings of this copy's previous replay
            const hipError_t e = hipGraphLaunch(exec[i], st);
            if (e != hipSuccess) {
                destroy_graphs();
                return fail(DASH_EDEVICE, "hipGraphLaunch: %s", hipGetErrorString(e));
            }
            gprof[i].armed();
            ++replays;
            continue;
        }
        if ((rc = one_step(B))) return rc;
        if (ragged && (rc = dash_kv_release(kv, done_at[t].data(), (int)done_at[t].size()))) return rc;
    }
    destroy_graphs();
    // release whatever is still held (fixed-length rollouts end with every slot live)
    std::vector<int32_t> held;
    for (int i = 0; i < N; ++i)
        if (kv->pb.npages[i]) held.push_back(i);
    return dash_kv_release(kv, held.data(), (int)held.size());
}

}  // extern "C"
