// Host side of the C ABI declared in include/lora.h: adapter registry,
// argument validation, the rank-bucketed planner and the launches.
//
// Everything a call needs is checked here before anything is enqueued, so a
// bad argument never reaches a kernel.  The planner turns the step's
// segments into (a) the rows grouped by adapter and (b) a flat list of work
// items sized by bytes, then the plan is copied into the caller's workspace
// in stream order and the kernels read it from there.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstdio>
#include <cstring>
#include <mutex>
#include <new>
#include <string>
#include <vector>

#include "lora.h"
#include "lora_internal.h"

namespace lora {
hipError_t launch_shrink(const KernelArgs& a, int dtype, hipStream_t s);
hipError_t launch_expand(const KernelArgs& a, int dtype, hipStream_t s);
}  // namespace lora

using namespace lora;

namespace {

thread_local std::string g_err;

int fail(int code, const std::string& msg) {
    g_err = msg;
    return code;
}

#define LORA_HIP_TRY(expr)                                                                    \
    do {                                                                                      \
        hipError_t e_ = (expr);                                                               \
        if (e_ != hipSuccess)                                                                 \
            return fail(LORA_E_HIP, std::string(#expr) + ": " + hipGetErrorString(e_));       \
    } while (0)

constexpr size_t kAlign = 256;
inline size_t align_up(size_t v, size_t a = kAlign) { return (v + a - 1) / a * a; }
inline bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

bool fast_rank(int r) {
    return r == 8 || r == 16 || r == 32 || r == 64 || r == 128 || r == 256;
}

// Rows of A_g per shrink item and columns of B_g per expand item.  Fast
// ranks move kChunkElems elements per item; other ranks use a smaller chunk
// so the generic body's LDS staging fits.
int shrink_klen(int r) {
    if (fast_rank(r)) return kChunkElems / r;
    int k = (8192 / r) & ~7;
    return std::max(8, k);
}
int expand_nlen(int r) {
    if (fast_rank(r)) return kChunkElems / r;
    int n = (kChunkElems / r) & ~7;
    return std::max(8, n);
}

struct DeviceGuard {
    int prev = -1;
    bool ok = true;
    explicit DeviceGuard(int d) {
        if (hipGetDevice(&prev) != hipSuccess) prev = -1;
        if (prev != d) ok = hipSetDevice(d) == hipSuccess;
    }
    ~DeviceGuard() {
        int cur = -1;
        if (prev >= 0 && hipGetDevice(&cur) == hipSuccess && cur != prev) (void)hipSetDevice(prev);
    }
};

}  // namespace

// ---------------------------------------------------------------------------
// adapter table
// ---------------------------------------------------------------------------
struct lora_table_s {
    int device = 0;
    int h_in = 0, h_out = 0, dtype = 0, n = 0;
    std::vector<DevAdapter> host;
    DevAdapter* dev = nullptr;
};

// ---------------------------------------------------------------------------
// plan
// ---------------------------------------------------------------------------
namespace {

struct HostPlan {
    int n_active = 0;
    int n_groups = 0;
    int r_max = 0;
    int vld = 0;
    std::vector<int32_t> perm, group_off, group_adapter;
    std::vector<DevItem> shrink, expand;
    std::vector<int64_t> part_off;
    int64_t n_partials = 0;
    size_t off_shrink = 0, off_expand = 0, off_perm = 0, off_partoff = 0, off_counters = 0;
    size_t plan_bytes = 0, off_v = 0, off_partials = 0, total_bytes = 0;
    std::vector<unsigned char> blob;
};

int validate_batch(const lora_batch_t* b, int n_adapters) {
    if (!b) return fail(LORA_E_ARG, "batch is NULL");
    if (b->n_rows < 0 || b->n_segments < 0) return fail(LORA_E_ARG, "negative n_rows or n_segments");
    if (!b->seg_offset) return fail(LORA_E_ARG, "seg_offset is NULL");
    if (b->n_segments > 0 && !b->seg_adapter) return fail(LORA_E_ARG, "seg_adapter is NULL");
    if (b->seg_offset[0] != 0) return fail(LORA_E_SHAPE, "seg_offset[0] must be 0");
    for (int s = 0; s < b->n_segments; ++s) {
        if (b->seg_offset[s + 1] < b->seg_offset[s])
            return fail(LORA_E_SHAPE, "seg_offset decreases at segment " + std::to_string(s));
        const int a = b->seg_adapter[s];
        if (a < -1 || a >= n_adapters)
            return fail(LORA_E_INDEX, "segment " + std::to_string(s) + " has adapter index " +
                                          std::to_string(a) + " outside [-1, " +
                                          std::to_string(n_adapters) + ")");
    }
    if (b->seg_offset[b->n_segments] != b->n_rows)
        return fail(LORA_E_SHAPE, "seg_offset[n_segments] != n_rows");
    return LORA_OK;
}

// Stable grouping: groups in order of the first row that uses the adapter,
// rows ascending inside a group, adapter -1 dropped.  O(n_rows + n_adapters).
void group_rows(const lora_batch_t* b, int n_adapters, std::vector<int32_t>& perm,
                std::vector<int32_t>& group_off, std::vector<int32_t>& group_adapter) {
    std::vector<int32_t> gid(n_adapters, -1);
    std::vector<int32_t> count;
    group_adapter.clear();
    for (int s = 0; s < b->n_segments; ++s) {
        const int a = b->seg_adapter[s];
        const int len = b->seg_offset[s + 1] - b->seg_offset[s];
        if (a < 0 || len == 0) continue;
        if (gid[a] < 0) {
            gid[a] = (int32_t)group_adapter.size();
            group_adapter.push_back(a);
            count.push_back(0);
        }
        count[gid[a]] += len;
    }
    const int G = (int)group_adapter.size();
    group_off.assign(G + 1, 0);
    for (int g = 0; g < G; ++g) group_off[g + 1] = group_off[g] + count[g];
    perm.assign(group_off[G], 0);
    std::vector<int32_t> fill(group_off.begin(), group_off.end() - 1);
    for (int s = 0; s < b->n_segments; ++s) {
        const int a = b->seg_adapter[s];
        if (a < 0) continue;
        int32_t& f = fill[gid[a]];
        for (int t = b->seg_offset[s]; t < b->seg_offset[s + 1]; ++t) perm[f++] = t;
    }
}

int build_plan(const lora_table_s* t, const lora_batch_t* b, HostPlan& p) {
    int rc = validate_batch(b, t->n);
    if (rc) return rc;
    group_rows(b, t->n, p.perm, p.group_off, p.group_adapter);
    p.n_groups = (int)p.group_adapter.size();
    p.n_active = p.n_groups ? p.group_off[p.n_groups] : 0;
    p.r_max = 0;
    p.shrink.clear();
    p.expand.clear();
    p.part_off.assign(p.n_groups, 0);
    p.n_partials = 0;
    for (int g = 0; g < p.n_groups; ++g) {
        const int a = p.group_adapter[g];
        const int r = t->host[a].rank;
        const int n = p.group_off[g + 1] - p.group_off[g];
        const int p0 = p.group_off[g];
        p.r_max = std::max(p.r_max, r);
        const int klen = shrink_klen(r);
        const int nsplit = (t->h_in + klen - 1) / klen;
        if (nsplit > 0xffff) return fail(LORA_E_SHAPE, "h_in too large for the chunking");
        for (int c = 0; c < nsplit; ++c) {
            DevItem it{};
            it.kind = kItemShrink;
            it.adapter = a;
            it.p0 = p0;
            it.nrows = n;
            it.lo = c * klen;
            it.len = std::min(klen, t->h_in - c * klen);
            it.group = g;
            it.split = (c << 16) | nsplit;
            p.shrink.push_back(it);
        }
        p.part_off[g] = p.n_partials;
        if (nsplit > 1) p.n_partials += (int64_t)nsplit * n * r;
        const int nlen = expand_nlen(r);
        const int ntiles = (t->h_out + nlen - 1) / nlen;
        for (int c = 0; c < ntiles; ++c) {
            DevItem it{};
            it.kind = kItemExpand;
            it.adapter = a;
            it.p0 = p0;
            it.nrows = n;
            it.lo = c * nlen;
            it.len = std::min(nlen, t->h_out - c * nlen);
            it.group = g;
            it.split = 0;
            p.expand.push_back(it);
        }
    }
    p.vld = std::max(4, (p.r_max + 3) / 4 * 4);

    // device layout: [shrink items][expand items][perm][part_off][counters] | [v][partials]
    size_t off = 0;
    p.off_shrink = off;
    off = align_up(off + p.shrink.size() * sizeof(DevItem));
    p.off_expand = off;
    off = align_up(off + p.expand.size() * sizeof(DevItem));
    p.off_perm = off;
    off = align_up(off + p.perm.size() * sizeof(int32_t));
    p.off_partoff = off;
    off = align_up(off + p.part_off.size() * sizeof(int64_t));
    p.off_counters = off;
    off = align_up(off + (size_t)p.n_groups * sizeof(int32_t));
    p.plan_bytes = off;
    p.off_v = off;
    off = align_up(off + (size_t)p.n_active * p.vld * sizeof(float));
    p.off_partials = off;
    off = align_up(off + (size_t)p.n_partials * sizeof(float));
    p.total_bytes = std::max<size_t>(off, kAlign);

    p.blob.assign(p.plan_bytes, 0);   // counters start at zero
    auto put = [&](size_t at, const void* src, size_t n) {
        if (n) std::memcpy(p.blob.data() + at, src, n);
    };
    put(p.off_shrink, p.shrink.data(), p.shrink.size() * sizeof(DevItem));
    put(p.off_expand, p.expand.data(), p.expand.size() * sizeof(DevItem));
    put(p.off_perm, p.perm.data(), p.perm.size() * sizeof(int32_t));
    put(p.off_partoff, p.part_off.data(), p.part_off.size() * sizeof(int64_t));
    return LORA_OK;
}

// Pinned staging ring per device for plan uploads: a slot is reused only
// after the copy that last read it has completed.
struct StageSlot {
    void* host = nullptr;
    size_t cap = 0;
    hipEvent_t ev = nullptr;
    bool pending = false;
};
constexpr int kStageSlots = 16;
struct StageRing {
    StageSlot slot[kStageSlots];
    unsigned next = 0;
};
std::mutex g_stage_mu;
std::vector<StageRing*> g_rings;

int stage_upload(int device, const void* src, size_t bytes, void* dst, hipStream_t s) {
    if (bytes == 0) return LORA_OK;
    std::lock_guard<std::mutex> lk(g_stage_mu);
    if ((int)g_rings.size() <= device) g_rings.resize(device + 1, nullptr);
    if (!g_rings[device]) g_rings[device] = new (std::nothrow) StageRing();
    if (!g_rings[device]) return fail(LORA_E_NOMEM, "staging ring allocation failed");
    StageRing& ring = *g_rings[device];
    StageSlot& sl = ring.slot[ring.next++ % kStageSlots];
    if (sl.pending) {
        LORA_HIP_TRY(hipEventSynchronize(sl.ev));
        sl.pending = false;
    }
    if (!sl.ev) LORA_HIP_TRY(hipEventCreateWithFlags(&sl.ev, hipEventDisableTiming));
    if (sl.cap < bytes) {
        if (sl.host) (void)hipHostFree(sl.host);
        sl.host = nullptr;
        sl.cap = 0;
        const size_t cap = std::max<size_t>(align_up(bytes, 65536), 65536);
        LORA_HIP_TRY(hipHostMalloc(&sl.host, cap, hipHostMallocDefault));
        sl.cap = cap;
    }
    std::memcpy(sl.host, src, bytes);
    LORA_HIP_TRY(hipMemcpyAsync(dst, sl.host, bytes, hipMemcpyHostToDevice, s));
    LORA_HIP_TRY(hipEventRecord(sl.ev, s));
    sl.pending = true;
    return LORA_OK;
}

KernelArgs base_args(const lora_table_s* t, const HostPlan& p, unsigned char* ws) {
    KernelArgs a{};
    a.table = t->dev;
    a.perm = (const int32_t*)(ws + p.off_perm);
    a.counters = (int32_t*)(ws + p.off_counters);
    a.partials = (float*)(ws + p.off_partials);
    a.part_off = (const int64_t*)(ws + p.off_partoff);
    a.h_in = t->h_in;
    a.h_out = t->h_out;
    return a;
}

int check_table(const lora_table_s* t) {
    if (!t || !t->dev) return fail(LORA_E_ARG, "table is NULL or released");
    return LORA_OK;
}

int check_ld(const char* name, int64_t ld, int h) {
    if (ld < h || ld % 8 != 0)
        return fail(LORA_E_SHAPE, std::string(name) + " must be a multiple of 8 and >= " +
                                      std::to_string(h));
    return LORA_OK;
}

int check_overlap(const void* x, int64_t ldx, int h_in, const void* y, int64_t ldy, int h_out,
                  int n_rows) {
    if (n_rows <= 0) return LORA_OK;
    const uintptr_t xs = (uintptr_t)x, ys = (uintptr_t)y;
    const uintptr_t xe = xs + ((uintptr_t)(n_rows - 1) * ldx + h_in) * 2;
    const uintptr_t ye = ys + ((uintptr_t)(n_rows - 1) * ldy + h_out) * 2;
    if (xs < ye && ys < xe) return fail(LORA_E_OVERLAP, "x and y overlap");
    return LORA_OK;
}

int check_ws(const HostPlan& p, const void* ws, size_t ws_bytes) {
    if (!ws) return fail(LORA_E_ARG, "workspace is NULL");
    if (!aligned16(ws)) return fail(LORA_E_ALIGN, "workspace not 16-byte aligned");
    if (ws_bytes < p.total_bytes)
        return fail(LORA_E_WORKSPACE, "workspace has " + std::to_string(ws_bytes) +
                                          " bytes, needs " + std::to_string(p.total_bytes));
    return LORA_OK;
}

}  // namespace

// ---------------------------------------------------------------------------
// plan handle
// ---------------------------------------------------------------------------
struct lora_plan_s {
    const lora_table_s* table = nullptr;
    int n_rows = 0;
    HostPlan plan;
    unsigned char* dmem = nullptr;
};

// ---------------------------------------------------------------------------
// C ABI
// ---------------------------------------------------------------------------
extern "C" {

int lora_abi_version(void) { return LORA_ABI_VERSION; }

const char* lora_last_error(void) { return g_err.c_str(); }

int lora_register_adapters(lora_table_t* out, int device, int h_in, int h_out, int dtype,
                           int n_adapters, const void* const* A_ptrs, const void* const* B_ptrs,
                           const int32_t* ranks, const float* scales, void* stream) {
    if (!out) return fail(LORA_E_ARG, "out is NULL");
    *out = nullptr;
    if (dtype != LORA_F16 && dtype != LORA_BF16) return fail(LORA_E_ARG, "dtype must be LORA_F16 or LORA_BF16");
    if (device < 0) return fail(LORA_E_ARG, "negative device");
    if (n_adapters < 0) return fail(LORA_E_ARG, "negative n_adapters");
    if (h_in <= 0 || h_out <= 0 || h_in % 8 || h_out % 8)
        return fail(LORA_E_SHAPE, "h_in and h_out must be positive multiples of 8");
    if (n_adapters > 0 && (!A_ptrs || !B_ptrs || !ranks || !scales))
        return fail(LORA_E_ARG, "adapter arrays must not be NULL");
    std::vector<DevAdapter> host(n_adapters);
    for (int i = 0; i < n_adapters; ++i) {
        if (ranks[i] < 1 || ranks[i] > kMaxRank)
            return fail(LORA_E_RANK, "adapter " + std::to_string(i) + " has rank " +
                                         std::to_string(ranks[i]) + " outside [1, 256]");
        if (!A_ptrs[i] || !B_ptrs[i])
            return fail(LORA_E_ARG, "adapter " + std::to_string(i) + " has a NULL factor");
        if (!aligned16(A_ptrs[i]) || !aligned16(B_ptrs[i]))
            return fail(LORA_E_ALIGN, "adapter " + std::to_string(i) + " factor not 16-byte aligned");
        host[i].A = A_ptrs[i];
        host[i].B = B_ptrs[i];
        host[i].rank = ranks[i];
        host[i].scale = scales[i];
    }
    DeviceGuard dg(device);
    if (!dg.ok) return fail(LORA_E_HIP, "hipSetDevice failed");
    auto* t = new (std::nothrow) lora_table_s();
    if (!t) return fail(LORA_E_NOMEM, "table allocation failed");
    t->device = device;
    t->h_in = h_in;
    t->h_out = h_out;
    t->dtype = dtype;
    t->n = n_adapters;
    t->host = std::move(host);
    const size_t bytes = std::max<size_t>(1, (size_t)n_adapters) * sizeof(DevAdapter);
    hipError_t e = hipMalloc((void**)&t->dev, bytes);
    if (e != hipSuccess) {
        delete t;
        return fail(LORA_E_NOMEM, std::string("hipMalloc of the adapter table: ") + hipGetErrorString(e));
    }
    if (n_adapters > 0) {
        hipStream_t s = (hipStream_t)stream;
        e = hipMemcpyAsync(t->dev, t->host.data(), n_adapters * sizeof(DevAdapter),
                           hipMemcpyHostToDevice, s);
        if (e == hipSuccess) e = hipStreamSynchronize(s);
        if (e != hipSuccess) {
            (void)hipFree(t->dev);
            delete t;
            return fail(LORA_E_HIP, std::string("adapter table upload: ") + hipGetErrorString(e));
        }
    }
    *out = t;
    return LORA_OK;
}

int lora_release_adapters(lora_table_t t) {
    if (!t) return fail(LORA_E_ARG, "table is NULL");
    if (t->dev) {
        DeviceGuard dg(t->device);
        (void)hipFree(t->dev);
    }
    delete t;
    return LORA_OK;
}

int lora_workspace_bytes(lora_table_t t, const lora_batch_t* b, size_t* bytes) {
    if (int rc = check_table(t)) return rc;
    if (!bytes) return fail(LORA_E_ARG, "bytes is NULL");
    HostPlan p;
    if (int rc = build_plan(t, b, p)) return rc;
    *bytes = p.total_bytes;
    return LORA_OK;
}

int lora_group_rows(const lora_batch_t* b, int32_t n_adapters, int32_t* perm, int32_t* group_off,
                    int32_t* group_adapter, int32_t* n_groups) {
    if (!perm || !group_off || !group_adapter || !n_groups) return fail(LORA_E_ARG, "output is NULL");
    if (n_adapters < 0) return fail(LORA_E_ARG, "negative n_adapters");
    if (int rc = validate_batch(b, n_adapters)) return rc;
    std::vector<int32_t> pv, go, ga;
    group_rows(b, n_adapters, pv, go, ga);
    std::copy(pv.begin(), pv.end(), perm);
    std::copy(go.begin(), go.end(), group_off);
    std::copy(ga.begin(), ga.end(), group_adapter);
    *n_groups = (int32_t)ga.size();
    return LORA_OK;
}

int lora_shrink(lora_table_t t, const lora_batch_t* b, const void* x, int64_t ldx, float* v,
                int64_t ldv, void* ws, size_t ws_bytes, void* stream) {
    if (int rc = check_table(t)) return rc;
    HostPlan p;
    if (int rc = build_plan(t, b, p)) return rc;
    if (p.n_active == 0) return LORA_OK;
    if (!x || !v) return fail(LORA_E_ARG, "x or v is NULL");
    if (!aligned16(x) || !aligned16(v)) return fail(LORA_E_ALIGN, "x or v not 16-byte aligned");
    if (int rc = check_ld("ldx", ldx, t->h_in)) return rc;
    if (ldv < p.r_max || ldv % 4) return fail(LORA_E_SHAPE, "ldv must be a multiple of 4 and >= the largest rank used");
    if (int rc = check_ws(p, ws, ws_bytes)) return rc;
    DeviceGuard dg(t->device);
    hipStream_t s = (hipStream_t)stream;
    unsigned char* w = (unsigned char*)ws;
    if (int rc = stage_upload(t->device, p.blob.data(), p.plan_bytes, w, s)) return rc;
    KernelArgs a = base_args(t, p, w);
    a.items = (const DevItem*)(w + p.off_shrink);
    a.n_items = (int32_t)p.shrink.size();
    a.x = x;
    a.ldx = ldx;
    a.v = v;
    a.ldv = ldv;
    a.v_by_row = 1;
    LORA_HIP_TRY(launch_shrink(a, t->dtype, s));
    return LORA_OK;
}

int lora_expand(lora_table_t t, const lora_batch_t* b, const float* v, int64_t ldv, void* y,
                int64_t ldy, void* ws, size_t ws_bytes, void* stream) {
    if (int rc = check_table(t)) return rc;
    HostPlan p;
    if (int rc = build_plan(t, b, p)) return rc;
    if (p.n_active == 0) return LORA_OK;
    if (!v || !y) return fail(LORA_E_ARG, "v or y is NULL");
    if (!aligned16(v) || !aligned16(y)) return fail(LORA_E_ALIGN, "v or y not 16-byte aligned");
    if (int rc = check_ld("ldy", ldy, t->h_out)) return rc;
    if (ldv < p.r_max || ldv % 4) return fail(LORA_E_SHAPE, "ldv must be a multiple of 4 and >= the largest rank used");
    if (int rc = check_ws(p, ws, ws_bytes)) return rc;
    DeviceGuard dg(t->device);
    hipStream_t s = (hipStream_t)stream;
    unsigned char* w = (unsigned char*)ws;
    if (int rc = stage_upload(t->device, p.blob.data(), p.plan_bytes, w, s)) return rc;
    KernelArgs a = base_args(t, p, w);
    a.items = (const DevItem*)(w + p.off_expand);
    a.n_items = (int32_t)p.expand.size();
    a.v = const_cast<float*>(v);
    a.ldv = ldv;
    a.v_by_row = 1;
    a.y = y;
    a.ldy = ldy;
    LORA_HIP_TRY(launch_expand(a, t->dtype, s));
    return LORA_OK;
}

// Launch the shrink (x != NULL) and/or the expand (y != NULL) of a plan whose
// float32 intermediate lives in the workspace w.
static int enqueue_apply(const lora_table_s* t, const HostPlan& p, unsigned char* w, const void* x,
                         int64_t ldx, void* y, int64_t ldy, hipStream_t s) {
    KernelArgs a = base_args(t, p, w);
    a.x = x;
    a.ldx = ldx;
    a.v = (float*)(w + p.off_v);
    a.ldv = p.vld;
    a.v_by_row = 0;
    a.y = y;
    a.ldy = ldy;
    if (x) {
        a.items = (const DevItem*)(w + p.off_shrink);
        a.n_items = (int32_t)p.shrink.size();
        LORA_HIP_TRY(launch_shrink(a, t->dtype, s));
    }
    if (y) {
        a.items = (const DevItem*)(w + p.off_expand);
        a.n_items = (int32_t)p.expand.size();
        LORA_HIP_TRY(launch_expand(a, t->dtype, s));
    }
    return LORA_OK;
}

static int check_xy(const lora_table_s* t, int n_rows, const void* x, int64_t ldx, const void* y,
                    int64_t ldy) {
    if (!x || !y) return fail(LORA_E_ARG, "x or y is NULL");
    if (!aligned16(x) || !aligned16(y)) return fail(LORA_E_ALIGN, "x or y not 16-byte aligned");
    if (int rc = check_ld("ldx", ldx, t->h_in)) return rc;
    if (int rc = check_ld("ldy", ldy, t->h_out)) return rc;
    return check_overlap(x, ldx, t->h_in, y, ldy, t->h_out, n_rows);
}

int lora_apply_fused(lora_table_t t, const lora_batch_t* b, const void* x, int64_t ldx, void* y,
                     int64_t ldy, void* ws, size_t ws_bytes, void* stream) {
    if (int rc = check_table(t)) return rc;
    HostPlan p;
    if (int rc = build_plan(t, b, p)) return rc;
    if (p.n_active == 0) return LORA_OK;
    if (int rc = check_xy(t, b->n_rows, x, ldx, y, ldy)) return rc;
    if (int rc = check_ws(p, ws, ws_bytes)) return rc;
    DeviceGuard dg(t->device);
    hipStream_t s = (hipStream_t)stream;
    unsigned char* w = (unsigned char*)ws;
    if (int rc = stage_upload(t->device, p.blob.data(), p.plan_bytes, w, s)) return rc;
    return enqueue_apply(t, p, w, x, ldx, y, ldy, s);
}

int lora_plan_create(lora_plan_t* out, lora_table_t t, const lora_batch_t* b, void* stream) {
    if (!out) return fail(LORA_E_ARG, "out is NULL");
    *out = nullptr;
    if (int rc = check_table(t)) return rc;
    auto* pl = new (std::nothrow) lora_plan_s();
    if (!pl) return fail(LORA_E_NOMEM, "plan allocation failed");
    pl->table = t;
    pl->n_rows = b ? b->n_rows : 0;
    if (int rc = build_plan(t, b, pl->plan)) {
        delete pl;
        return rc;
    }
    DeviceGuard dg(t->device);
    hipError_t e = hipMalloc((void**)&pl->dmem, pl->plan.total_bytes);
    if (e != hipSuccess) {
        delete pl;
        return fail(LORA_E_NOMEM, std::string("hipMalloc of the plan: ") + hipGetErrorString(e));
    }
    hipStream_t s = (hipStream_t)stream;
    e = hipMemcpyAsync(pl->dmem, pl->plan.blob.data(), pl->plan.plan_bytes, hipMemcpyHostToDevice, s);
    if (e == hipSuccess) e = hipStreamSynchronize(s);
    if (e != hipSuccess) {
        (void)hipFree(pl->dmem);
        delete pl;
        return fail(LORA_E_HIP, std::string("plan upload: ") + hipGetErrorString(e));
    }
    *out = pl;
    return LORA_OK;
}

int lora_plan_apply(lora_plan_t pl, const void* x, int64_t ldx, void* y, int64_t ldy, void* stream) {
    if (!pl || !pl->dmem) return fail(LORA_E_ARG, "plan is NULL");
    const lora_table_s* t = pl->table;
    if (pl->plan.n_active == 0) return LORA_OK;
    if (int rc = check_xy(t, pl->n_rows, x, ldx, y, ldy)) return rc;
    DeviceGuard dg(t->device);
    return enqueue_apply(t, pl->plan, pl->dmem, x, ldx, y, ldy, (hipStream_t)stream);
}

int lora_plan_shrink(lora_plan_t pl, const void* x, int64_t ldx, void* stream) {
    if (!pl || !pl->dmem) return fail(LORA_E_ARG, "plan is NULL");
    const lora_table_s* t = pl->table;
    if (pl->plan.n_active == 0) return LORA_OK;
    if (!x) return fail(LORA_E_ARG, "x is NULL");
    if (!aligned16(x)) return fail(LORA_E_ALIGN, "x not 16-byte aligned");
    if (int rc = check_ld("ldx", ldx, t->h_in)) return rc;
    DeviceGuard dg(t->device);
    return enqueue_apply(t, pl->plan, pl->dmem, x, ldx, nullptr, 0, (hipStream_t)stream);
}

int lora_plan_expand(lora_plan_t pl, void* y, int64_t ldy, void* stream) {
    if (!pl || !pl->dmem) return fail(LORA_E_ARG, "plan is NULL");
    const lora_table_s* t = pl->table;
    if (pl->plan.n_active == 0) return LORA_OK;
    if (!y) return fail(LORA_E_ARG, "y is NULL");
    if (!aligned16(y)) return fail(LORA_E_ALIGN, "y not 16-byte aligned");
    if (int rc = check_ld("ldy", ldy, t->h_out)) return rc;
    DeviceGuard dg(t->device);
    return enqueue_apply(t, pl->plan, pl->dmem, nullptr, 0, y, ldy, (hipStream_t)stream);
}

int lora_plan_destroy(lora_plan_t pl) {
    if (!pl) return fail(LORA_E_ARG, "plan is NULL");
    if (pl->dmem) {
        DeviceGuard dg(pl->table->device);
        (void)hipFree(pl->dmem);
    }
    delete pl;
    return LORA_OK;
}

}  // extern "C"
