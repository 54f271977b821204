// Host side of the C ABI declared in include/lora.h: adapter registry,
// argument validation, the rank-bucketed planner and the launches.
//
// Everything a call needs is checked here before anything is enqueued, so a
// bad argument never reaches a kernel.  The planner turns the step's segments
// into (a) the rows grouped by adapter and (b) flat lists of work items sized
// by bytes.  A plan depends on the batch, the ranks and the shapes only; each
// launch carries the weight pointers and scales of the table it is applied
// to, so one plan serves every compatible table.
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
hipError_t launch_shrink(const KernelArgs& a, const uint32_t* hdr, int dtype, hipStream_t s);
hipError_t launch_expand(const KernelArgs& a, const uint32_t* hdr, int dtype, hipStream_t s);
hipError_t launch_reduce(const KernelArgs& a, const uint32_t* hdr, hipStream_t s);
hipError_t launch_step(const KernelArgs& a, const uint32_t* hdr, int dtype, hipStream_t s);
hipError_t launch_fill(uint32_t* p, uint32_t v, uint64_t n_words, hipStream_t s);
hipError_t launch_base(const BaseArgs& a, int dtype, hipStream_t s);
int set_error(int code, const std::string& msg);
}  // namespace lora

using namespace lora;

namespace {

thread_local std::string g_err;

int fail(int code, const std::string& msg) {
    g_err = msg;
    return code;
}

}  // namespace

// the same thread-local message for the library's other host sources
int lora::set_error(int code, const std::string& msg) { return fail(code, msg); }

namespace {

#define LORA_HIP_TRY(expr)                                                                    \
    do {                                                                                      \
        hipError_t e_ = (expr);                                                               \
        if (e_ != hipSuccess)                                                                 \
            return fail(LORA_E_HIP, std::string(#expr) + ": " + hipGetErrorString(e_));       \
    } while (0)

constexpr size_t kAlign = 256;
inline size_t align_up(size_t v, size_t a = kAlign) { return (v + a - 1) / a * a; }
inline bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

// Workgroups the planner aims for when it sizes the K ranges of prompt-sized
// row blocks (two per CU on a 256-CU device).
constexpr int kTargetItems = 512;

// Polling rounds a step launch's thread may spend waiting before it gives up
// (each round is a device-coherent load, about a microsecond under load), in
// all: a quarter of a second, against waits of microseconds.
constexpr int kSpinLimit = 1 << 18;

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
    int n_xcd = 1;                      // XCDs of the device (workgroup p of a launch runs on XCD p % n_xcd)
    int n_cu = 0;                       // compute units of the device
    int h_in = 0, h_out = 0, dtype = 0, n = 0;
    std::vector<DevAdapter> host;
    DevAdapter* dev = nullptr;
};

// ---------------------------------------------------------------------------
// plan
// ---------------------------------------------------------------------------
namespace {

struct HostPlan {
    int h_in = 0, h_out = 0, dtype = 0, n_adapters = 0;
    int n_active = 0;
    int n_groups = 0;
    int r_max = 0;
    int n_rb = 0;                       // row blocks
    int n_proj = 1;                     // projections sharing x that one launch runs (copies of the lists)
    std::vector<int> proj_h_out;        // their h_out (n_proj > 1)
    std::vector<int64_t> rb_bytes;      // bytes each row block streams
    std::vector<int32_t> perm, group_off, group_adapter, group_rank;
    std::vector<DevItem> shrink, expand, reduce, reduce_all, step;
    int n_rows = 0;
    int64_t n_partials = 0;
    size_t off_shrink = 0, off_expand = 0, off_reduce = 0, off_reduce_all = 0, off_step = 0, off_perm = 0;
    size_t plan_bytes = 0, off_partials = 0, off_sync = 0, sync_bytes = 0, total_bytes = 0;
    size_t off_step_partials = 0, step_partials_bytes = 0, plan_total_bytes = 0;
    uint32_t generation = 0;            // header word 0 of the uploaded work list
    std::vector<unsigned char> blob;    // [header][item lists][perm], as uploaded
    void set_generation(uint32_t g) {
        generation = g;
        std::memcpy(blob.data(), &g, sizeof g);
    }
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
        // an empty segment may name an adapter that no row uses (no group)
        if (a < 0 || b->seg_offset[s + 1] == b->seg_offset[s]) continue;
        int32_t& f = fill[gid[a]];
        for (int t = b->seg_offset[s]; t < b->seg_offset[s + 1]; ++t) perm[f++] = t;
    }
}

int plan_lists(const lora_table_s* t, const lora_batch_t* b, HostPlan& p) {
    int rc = validate_batch(b, t->n);
    if (rc) return rc;
    p.h_in = t->h_in;
    p.h_out = t->h_out;
    p.dtype = t->dtype;
    p.n_adapters = t->n;
    group_rows(b, t->n, p.perm, p.group_off, p.group_adapter);
    p.n_groups = (int)p.group_adapter.size();
    p.n_active = p.n_groups ? p.group_off[p.n_groups] : 0;
    p.group_rank.assign(p.n_groups, 0);
    p.r_max = 0;
    p.shrink.clear();
    p.expand.clear();
    p.reduce.clear();
    p.reduce_all.clear();
    p.n_rows = b->n_rows;
    p.step.clear();
    std::vector<int64_t>& rb_bytes = p.rb_bytes;
    rb_bytes.clear();
    p.n_proj = 1;
    p.n_partials = 0;
    p.n_rb = 0;

    // Row blocks of more than 16 rows (prompt segments, popular adapters) are
    // cut into about kTargetItems / (number of such blocks) K ranges: few
    // such blocks get one pass per item (as the small blocks do), many get
    // fewer, longer items that stream their range in several passes.
    int big_blocks = 0;
    for (int g = 0; g < p.n_groups; ++g) {
        const int r = t->host[p.group_adapter[g]].rank;
        const int rb = row_block(r);
        const int n = p.group_off[g + 1] - p.group_off[g];
        for (int q0 = 0; q0 < n; q0 += rb)
            if (std::min(rb, n - q0) > kInlineRows) ++big_blocks;
    }
    const int big_split = big_blocks ? std::max(1, (kTargetItems + big_blocks - 1) / big_blocks) : 1;
    // K ranges and column tiles of a row block of nb rows at rank r
    auto splits = [&](int r, int nb, int& sub, int& krange, int& nsplit, int& nlen, int& ntiles) {
        sub = shrink_sub(r, nb);
        krange = sub;
        if (nb > kInlineRows) {
            const int per = (t->h_in + big_split - 1) / big_split;
            krange = round_up_i(std::max(per, sub), sub);
        }
        nsplit = (t->h_in + krange - 1) / krange;
        nlen = expand_nlen(r, nb);
        ntiles = (t->h_out + nlen - 1) / nlen;
    };
    // A step whose shrink and expand items fit one round of workgroups
    // (decode) lets expand items add small partial blocks themselves, one hop
    // fewer on its critical path; larger steps add them in reduce items,
    // which leaves each expand item one v block to read (measured: 13B layer
    // 115.5 -> 110 us, decode step +0.1 us had it done so too).
    int64_t step_items = 0;
    for (int g = 0; g < p.n_groups; ++g) {
        const int r = t->host[p.group_adapter[g]].rank;
        const int rb = row_block(r);
        const int n = p.group_off[g + 1] - p.group_off[g];
        for (int q0 = 0; q0 < n; q0 += rb) {
            int sub, krange, nsplit, nlen, ntiles;
            splits(r, std::min(rb, n - q0), sub, krange, nsplit, nlen, ntiles);
            step_items += nsplit + ntiles;
        }
    }
    const bool small_step = step_items <= kTargetItems;

    for (int g = 0; g < p.n_groups; ++g) {
        const DevAdapter& ad = t->host[p.group_adapter[g]];
        const int r = ad.rank;
        const int rv = rank_stride(r);
        p.group_rank[g] = r;
        p.r_max = std::max(p.r_max, r);
        const int rb = row_block(r);
        for (int p0 = p.group_off[g]; p0 < p.group_off[g + 1]; p0 += rb) {
            const int nb = std::min(rb, p.group_off[g + 1] - p0);
            int sub, krange, nsplit, nlen, ntiles;
            splits(r, nb, sub, krange, nsplit, nlen, ntiles);
            const int pstride = nb * rv;              // one partial (or v) block: [nb][rv] floats
            DevItem base{};
            base.rb = p.n_rb++;
            rb_bytes.push_back((int64_t)(r + nb) * t->h_in * 2 + (int64_t)(r + 2 * nb) * t->h_out * 2);
            base.nexp = ntiles;
            base.group = g;
            base.adapter = p.group_adapter[g];
            base.rank = r;
            base.nrows = nb;
            base.nsplit = nsplit;
            base.p0 = p0;
            base.pstride = pstride;
            if (nb <= kInlineRows)
                for (int i = 0; i < nb; ++i) base.rows[i] = p.perm[p0 + i];
            base.row0 = p.perm[p0];
            for (int i = 1; i < nb; ++i)
                if (p.perm[p0 + i] != p.perm[p0] + i) {
                    base.row0 = -1;
                    break;
                }
            // the row block's nsplit partial blocks, then its v block
            const int64_t part0 = p.n_partials;
            p.n_partials += (int64_t)(nsplit + 1) * pstride;
            // small partial blocks of a small step are added up by the expand items themselves
            const bool direct =
                small_step && nsplit <= kDirectSplits && (int64_t)nsplit * pstride * 4 <= kDirectBytes;
            for (int c = 0; c < nsplit; ++c) {
                DevItem it = base;
                it.kind = kItemShrink;
                it.part = part0 + (int64_t)c * pstride;
                it.lo = c * krange;
                it.len = std::min(krange, t->h_in - c * krange);
                it.sub = shrink_uses_dma(r, nb) ? shrink_stage_sub(r, nb) : sub;
                if (!shrink_uses_dma(r, nb) && shrink_lds_bytes(r, sub, nb) > kShrinkLds)
                    return fail(LORA_E_SHAPE, "internal: shrink tile exceeds LDS");
                p.shrink.push_back(it);
            }
            // reduce slices: at most kReduceBytes of partial values each; G
            // split groups share a float4 position (G * positions <= threads),
            // each thread adding at most kMaxSplitLoads blocks
            int gmin = 1;
            while (gmin * kMaxSplitLoads < nsplit) gmin *= 2;
            const int64_t pbytes = (int64_t)nsplit * pstride * 4;
            int nslice = (int)std::max<int64_t>(1, (pbytes + kReduceBytes - 1) / kReduceBytes);
            int slen = round_up_i((pstride + nslice - 1) / nslice, 4);
            slen = std::min(slen, 4 * (kThreads / gmin));
            nslice = (pstride + slen - 1) / slen;
            for (int c = 0; c < nslice; ++c) {
                DevItem it = base;
                it.kind = kItemReduce;
                it.part = part0;
                it.lo = c * slen;
                it.len = std::min(slen, pstride - c * slen);
                const int np = it.len / 4;
                int G = 1;
                // a row block whose expand items add the partial blocks up
                // themselves adds them in order 0..nsplit-1: one group here too
                while (!direct && 2 * G <= nsplit && 2 * G * np <= kThreads) G *= 2;
                if (G * kMaxSplitLoads < nsplit) return fail(LORA_E_SHAPE, "internal: reduce slice too wide");
                it.sub = G;
                p.reduce_all.push_back(it);         // lora_shrink's reduce into the caller's v
                if (!direct) p.reduce.push_back(it);
            }
            for (int c = 0; c < ntiles; ++c) {
                DevItem it = base;
                it.kind = kItemExpand;
                it.part = part0;
                it.sub = direct ? 1 : 0;
                it.lo = c * nlen;
                it.len = std::min(nlen, t->h_out - c * nlen);
                if (!expand_fits_lds(r, nb))
                    return fail(LORA_E_SHAPE, "internal: expand tile exceeds LDS");
                p.expand.push_back(it);
            }
        }
    }

    return LORA_OK;
}

// The lists of n projections that share x, one after the other: projection c
// carries c in its kind, its own partial and v blocks and its own row block
// counters (offsets past the projections before it).  Each projection's
// items wait only on items of the same projection.
void append_lists(HostPlan& p, const HostPlan& q, int c) {
    const int64_t np = p.n_partials;
    const int nrb = p.n_rb;
    auto app = [&](std::vector<DevItem>& dst, const std::vector<DevItem>& src) {
        for (DevItem it : src) {
            it.kind |= c << kProjShift;
            it.part += np;
            it.rb += nrb;
            dst.push_back(it);
        }
    };
    app(p.shrink, q.shrink);
    app(p.reduce, q.reduce);
    app(p.expand, q.expand);
    app(p.reduce_all, q.reduce_all);
    p.rb_bytes.insert(p.rb_bytes.end(), q.rb_bytes.begin(), q.rb_bytes.end());
    p.n_partials += q.n_partials;
    p.n_rb += q.n_rb;
}

// The grid layout and the device layout of the lists, and the upload image.
int plan_layout(const lora_table_s* t, HostPlan& p) {
    const std::vector<int64_t>& rb_bytes = p.rb_bytes;
    if ((uint64_t)p.n_partials * 4 > kMaxSpan)
        return fail(LORA_E_SHAPE, "batch too large: its partial results exceed 2 GiB");

    // A step small enough to run in one round of workgroups (decode) gets a
    // grid laid out per XCD: workgroup p of a launch runs on XCD p % n_xcd (the
    // order in which the hardware hands workgroups to the XCDs), every row
    // block gets one XCD (largest first, each to the XCD with the fewest bytes
    // so far), and on each XCD its shrink, reduce and expand items follow in
    // that order, slots it does not need holding items of no kind.  A row
    // block's partial and v blocks then stay in one L2 and one fabric path.
    // Larger steps keep the list order: there the balance of the whole grid
    // matters more (measured: the decode step 12.9 -> 12.2 us, the 13B-layer,
    // 70B and prompt steps 2-5% slower with the layout), and so do steps whose
    // row blocks cannot be spread evenly (the busiest XCD above 1.25 times the
    // average).  Every item still waits only on items earlier in the grid,
    // whatever the hardware does.
    const size_t n_step = p.shrink.size() + p.reduce.size() + p.expand.size();
    if (t->n_xcd > 1 && n_step <= (size_t)kTargetItems) {
        const int nx = t->n_xcd;
        std::vector<int> home(p.n_rb, 0), order(p.n_rb);
        for (int i = 0; i < p.n_rb; ++i) order[i] = i;
        std::stable_sort(order.begin(), order.end(), [&](int u, int v) { return rb_bytes[u] > rb_bytes[v]; });
        std::vector<int64_t> load(nx, 0);
        for (int i : order) {
            const int x = (int)(std::min_element(load.begin(), load.end()) - load.begin());
            home[i] = x;
            load[x] += rb_bytes[i];
        }
        // only when the XCDs come out balanced: a step of few row blocks
        // (few adapters) would otherwise leave XCDs idle
        int64_t total = 0, most = 0;
        for (int64_t v : load) {
            total += v;
            most = std::max(most, v);
        }
        if (4 * most * nx <= 5 * total) {
            std::vector<std::vector<DevItem>> q(nx);
            for (const auto* list : {&p.shrink, &p.reduce, &p.expand})
                for (const DevItem& it : *list) q[home[it.rb]].push_back(it);
            size_t len = 0;
            for (const auto& v : q) len = std::max(len, v.size());
            const DevItem none{};            // kind 0: does nothing
            p.step.assign(len * nx, none);
            for (int x = 0; x < nx; ++x)
                for (size_t i = 0; i < q[x].size(); ++i) p.step[i * nx + x] = q[x][i];
        }
    }

    // device layout: [header][shrink items][reduce items][expand items][all reduce
    // items][step grid laid out per XCD, small steps only][perm] | [partial and v blocks][row block counters, status] (a
    // workspace ends here) | [step partial and v blocks x 2] (plans only: the
    // step launch's blocks in two buffers used by alternate launches, each
    // armed with the sentinel before the launch that reads it).  The first
    // three lists are contiguous: the step launch runs them as one grid (or the
    // fifth, the same items laid out per XCD); the separate launches run one
    // each, lora_shrink the fourth.
    size_t off = kHeaderBytes;                // the header (generation, status) comes first
    p.off_shrink = off;
    off += p.shrink.size() * sizeof(DevItem);
    p.off_reduce = off;
    off += p.reduce.size() * sizeof(DevItem);
    p.off_expand = off;
    off += p.expand.size() * sizeof(DevItem);
    p.off_reduce_all = off;
    off += p.reduce_all.size() * sizeof(DevItem);
    p.off_step = off;
    off = align_up(off + p.step.size() * sizeof(DevItem));
    p.off_perm = off;
    off = align_up(off + p.perm.size() * sizeof(int32_t));
    p.plan_bytes = off;
    p.off_partials = off;
    off = align_up(off + (size_t)p.n_partials * sizeof(float));
    p.off_sync = off;
    p.sync_bytes = align_up(std::max<size_t>(1, (size_t)p.n_rb) * kSyncStride * sizeof(uint32_t));
    off += p.sync_bytes;
    p.total_bytes = std::max<size_t>(off, kAlign);
    p.off_step_partials = off;
    p.step_partials_bytes = 2 * align_up((size_t)p.n_partials * sizeof(float));   // two buffers
    p.plan_total_bytes = std::max<size_t>(off + p.step_partials_bytes, kAlign);

    p.blob.assign(p.plan_bytes, 0);
    auto put = [&](size_t at, const void* src, size_t n) {
        if (n) std::memcpy(p.blob.data() + at, src, n);
    };
    put(p.off_shrink, p.shrink.data(), p.shrink.size() * sizeof(DevItem));
    put(p.off_reduce, p.reduce.data(), p.reduce.size() * sizeof(DevItem));
    put(p.off_expand, p.expand.data(), p.expand.size() * sizeof(DevItem));
    put(p.off_reduce_all, p.reduce_all.data(), p.reduce_all.size() * sizeof(DevItem));
    put(p.off_step, p.step.data(), p.step.size() * sizeof(DevItem));
    put(p.off_perm, p.perm.data(), p.perm.size() * sizeof(int32_t));
    return LORA_OK;
}

int build_plan(const lora_table_s* t, const lora_batch_t* b, HostPlan& p) {
    if (int rc = plan_lists(t, b, p)) return rc;
    return plan_layout(t, p);
}

// One plan for n projections that share x (the same h_in and dtype, the
// batch's adapters of the same ranks in every table; h_out may differ).
int build_plan_multi(const lora_table_s* const* t, int n, const lora_batch_t* b, HostPlan& p) {
    if (int rc = plan_lists(t[0], b, p)) return rc;
    p.proj_h_out.assign(1, t[0]->h_out);
    for (int c = 1; c < n; ++c) {
        if (t[c]->h_in != t[0]->h_in || t[c]->dtype != t[0]->dtype)
            return fail(LORA_E_SHAPE, "the projections differ in h_in or dtype");
        HostPlan q;
        if (int rc = plan_lists(t[c], b, q)) return rc;
        append_lists(p, q, c);
        p.proj_h_out.push_back(t[c]->h_out);
    }
    p.n_proj = n;
    return plan_layout(t[0], p);
}

int check_compatible(const HostPlan& p, const lora_table_s* t);

// Projection i of a plan of several projections: its table must agree with
// the plan in h_in, dtype, its projection's h_out and the referenced ranks.
int check_compatible_proj(const HostPlan& p, const lora_table_s* t, int i) {
    if (!t || !t->dev) return fail(LORA_E_ARG, "table is NULL or released");
    if (p.n_proj > 1 && t->h_out != p.proj_h_out[i])
        return fail(LORA_E_SHAPE, "table " + std::to_string(i) + " has another h_out than its projection in the plan");
    if (p.n_proj <= 1) return check_compatible(p, t);
    if (t->h_in != p.h_in || t->dtype != p.dtype) return fail(LORA_E_SHAPE, "table shape or dtype differs from the plan's");
    for (int g = 0; g < p.n_groups; ++g) {
        const int a = p.group_adapter[g];
        if (a >= t->n) return fail(LORA_E_INDEX, "table has fewer adapters than the plan references");
        if (t->host[a].rank != p.group_rank[g])
            return fail(LORA_E_RANK, "adapter " + std::to_string(a) + " has another rank than in the plan");
    }
    return LORA_OK;
}

// A table may run a plan made with another table when shapes, dtype and the
// ranks of every adapter the plan references agree.
int check_compatible(const HostPlan& p, const lora_table_s* t) {
    if (!t || !t->dev) return fail(LORA_E_ARG, "table is NULL or released");
    if (t->h_in != p.h_in || t->h_out != p.h_out || t->dtype != p.dtype)
        return fail(LORA_E_SHAPE, "table shape or dtype differs from the plan's");
    for (int g = 0; g < p.n_groups; ++g) {
        const int a = p.group_adapter[g];
        if (a >= t->n) return fail(LORA_E_INDEX, "table has fewer adapters than the plan references");
        if (t->host[a].rank != p.group_rank[g])
            return fail(LORA_E_RANK, "adapter " + std::to_string(a) + " has another rank than in the plan");
    }
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

// The calls that upload their work list through the shared ring below cannot
// be recorded in a graph: a replay would copy whatever the ring slot holds by
// then.  They refuse a capturing stream before enqueuing anything.
int check_not_capturing(hipStream_t s, const char* what) {
    hipStreamCaptureStatus cs = hipStreamCaptureStatusNone;
    LORA_HIP_TRY(hipStreamIsCapturing(s, &cs));
    if (cs != hipStreamCaptureStatusNone)
        return fail(LORA_E_CAPTURE, std::string(what) +
                                        " cannot be recorded in a graph (it uploads its work list from a reused "
                                        "host buffer); record lora_plan_apply / _shrink / _expand instead");
    return LORA_OK;
}

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

// The allocation-free entry point's workspace: one array per device, set up
// by the HIP runtime when the library's code object is loaded there and kept
// until the process ends.  Host code never takes its address directly (that
// would be a host-side stand-in, not device memory): the first call on each
// device looks the device address up and keeps it.
constexpr size_t kScratchBytes = size_t(16) << 20;
constexpr int kMaxDevices = 64;
static __device__ __align__(256) unsigned char scratch[kScratchBytes];
std::mutex g_scratch_mu;
unsigned char* g_scratch_ptr[kMaxDevices] = {};

// Device address of `scratch` on `device` (which must be current).
int scratch_address(int device, unsigned char** out) {
    if (device < 0 || device >= kMaxDevices) return fail(LORA_E_ARG, "device index beyond the static scratch table");
    std::lock_guard<std::mutex> lk(g_scratch_mu);
    if (!g_scratch_ptr[device]) {
        void* ptr = nullptr;
        const hipError_t e = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch));
        if (e != hipSuccess || !ptr)
            return fail(LORA_E_HIP, std::string("hipGetSymbolAddress(scratch): ") + hipGetErrorString(e));
        g_scratch_ptr[device] = (unsigned char*)ptr;
    }
    *out = g_scratch_ptr[device];
    return LORA_OK;
}

// Launch arguments of one plan on one table: the plan's buffers in workspace
// w and the factor pointers and scales of its groups.
KernelArgs make_args(const lora_table_s* t, const HostPlan& p, unsigned char* w, int spin_limit) {
    KernelArgs a{};
    a.perm = (const int32_t*)(w + p.off_perm);
    a.table = t->dev;
    a.partials = (float*)(w + p.off_partials);
    a.sync = (uint32_t*)(w + p.off_sync);
    a.status = (int32_t*)(w + sizeof(uint32_t));   // header word 1
    a.generation = p.generation;
    a.pbuf = (int64_t)(p.step_partials_bytes / 2 / sizeof(float));
    a.spin_limit = spin_limit;
    a.h_in = t->h_in;
    a.h_out = t->h_out;
    a.n_groups = p.n_groups;
    const int ng = std::min(p.n_groups, kKargGroups);
    for (int g = 0; g < ng; ++g) {
        const DevAdapter& ad = t->host[p.group_adapter[g]];
        a.gfac[2 * g] = ad.A;
        a.gfac[2 * g + 1] = ad.B;
        a.gscale[g] = ad.scale;
    }
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

// Bytes from the first element of a [n_rows, ld] matrix to the end of its
// last row of h elements.
uint64_t span_bytes(int n_rows, int64_t ld, int h) {
    return n_rows > 0 ? ((uint64_t)(n_rows - 1) * (uint64_t)ld + (uint64_t)h) * 2 : 0;
}

int check_x(const lora_table_s* t, const void* x, int64_t ldx, int n_rows) {
    if (!x) return fail(LORA_E_ARG, "x is NULL");
    if (!aligned16(x)) return fail(LORA_E_ALIGN, "x not 16-byte aligned");
    if (int rc = check_ld("ldx", ldx, t->h_in)) return rc;
    if (span_bytes(n_rows, ldx, t->h_in) > kMaxSpan) return fail(LORA_E_SHAPE, "x spans more than 2 GiB");
    return LORA_OK;
}

int check_y(const lora_table_s* t, const void* y, int64_t ldy, int n_rows) {
    if (!y) return fail(LORA_E_ARG, "y is NULL");
    if (!aligned16(y)) return fail(LORA_E_ALIGN, "y not 16-byte aligned");
    if (int rc = check_ld("ldy", ldy, t->h_out)) return rc;
    if (span_bytes(n_rows, ldy, t->h_out) > kMaxSpan) return fail(LORA_E_SHAPE, "y spans more than 2 GiB");
    return LORA_OK;
}

int check_v(const HostPlan& p, const void* v, int64_t ldv) {
    if (!v) return fail(LORA_E_ARG, "v is NULL");
    if (!aligned16(v)) return fail(LORA_E_ALIGN, "v not 16-byte aligned");
    if (ldv < p.r_max || ldv % 4)
        return fail(LORA_E_SHAPE, "ldv must be a multiple of 4 and >= the largest rank used");
    return LORA_OK;
}

// Enqueue the shrink (x != NULL) and/or the expand (y != NULL) of plan p on
// table t with its workspace at w, as separate launches: shrink, then (unless
// the caller reduces into its own v) reduce into the v blocks; expand.
int enqueue(const lora_table_s* t, const HostPlan& p, unsigned char* w, const void* x, int64_t ldx,
            void* y, int64_t ldy, hipStream_t s, bool v_out = false) {
    if (x) {
        KernelArgs a = make_args(t, p, w, kSpinLimit);
        a.items = (const DevItem*)(w + p.off_shrink);
        a.n_items = (int32_t)p.shrink.size();
        a.x = x;
        a.ldx = ldx;
        a.x_bytes = (uint32_t)span_bytes(p.n_rows, ldx, t->h_in);
        LORA_HIP_TRY(launch_shrink(a, (const uint32_t*)w, t->dtype, s));
        if (!v_out) {
            a.items = (const DevItem*)(w + p.off_reduce);
            a.n_items = (int32_t)p.reduce.size();
            LORA_HIP_TRY(launch_reduce(a, (const uint32_t*)w, s));
        }
    }
    if (y) {
        KernelArgs a = make_args(t, p, w, kSpinLimit);
        a.items = (const DevItem*)(w + p.off_expand);
        a.n_items = (int32_t)p.expand.size();
        a.y = y;
        a.ldy = ldy;
        a.y_bytes = (uint32_t)span_bytes(p.n_rows, ldy, t->h_out);
        LORA_HIP_TRY(launch_expand(a, (const uint32_t*)w, t->dtype, s));
    }
    return LORA_OK;
}

// Enqueue the whole step of plan p as one launch (shrink and expand items in
// one grid).  The row block counters at w + off_sync must be zero and the
// step partial blocks armed.
// The arguments of the step launch of plan p (one projection).
int step_args(const lora_table_s* t, const HostPlan& p, unsigned char* w, const void* x, int64_t ldx, void* y,
              int64_t ldy, int spin_limit, KernelArgs& out) {
    KernelArgs a = make_args(t, p, w, spin_limit);
    a.partials = (float*)(w + p.off_step_partials);
    if (!p.step.empty()) {                    // the grid laid out per XCD
        a.items = (const DevItem*)(w + p.off_step);
        a.n_items = (int32_t)p.step.size();
    } else {
        a.items = (const DevItem*)(w + p.off_shrink);
        a.n_items = (int32_t)(p.shrink.size() + p.reduce.size() + p.expand.size());
    }
    a.x = x;
    a.ldx = ldx;
    a.x_bytes = (uint32_t)span_bytes(p.n_rows, ldx, t->h_in);
    a.y = y;
    a.ldy = ldy;
    a.y_bytes = (uint32_t)span_bytes(p.n_rows, ldy, t->h_out);
    out = a;
    return LORA_OK;
}

int enqueue_step(const lora_table_s* t, const HostPlan& p, unsigned char* w, const void* x,
                 int64_t ldx, void* y, int64_t ldy, int spin_limit, hipStream_t s) {
    KernelArgs a = make_args(t, p, w, spin_limit);
    a.partials = (float*)(w + p.off_step_partials);
    if (!p.step.empty()) {                    // the grid laid out per XCD
        a.items = (const DevItem*)(w + p.off_step);
        a.n_items = (int32_t)p.step.size();
    } else {
        a.items = (const DevItem*)(w + p.off_shrink);
        a.n_items = (int32_t)(p.shrink.size() + p.reduce.size() + p.expand.size());
    }
    a.x = x;
    a.ldx = ldx;
    a.x_bytes = (uint32_t)span_bytes(p.n_rows, ldx, t->h_in);
    a.y = y;
    a.ldy = ldy;
    a.y_bytes = (uint32_t)span_bytes(p.n_rows, ldy, t->h_out);
    LORA_HIP_TRY(launch_step(a, (const uint32_t*)w, t->dtype, s));
    return LORA_OK;
}

// Status and row block counters to zero, both step partial buffers to the
// sentinel (all-ones words): fill kernels, no memset.  Plan creation,
// re-planning and the status reset.
hipError_t arm_step(const HostPlan& p, unsigned char* w, hipStream_t s) {
    hipError_t e = launch_fill((uint32_t*)(w + sizeof(uint32_t)), 0u, 1, s);
    if (e == hipSuccess) e = launch_fill((uint32_t*)(w + p.off_sync), 0u, p.sync_bytes / sizeof(uint32_t), s);
    if (e == hipSuccess && p.step_partials_bytes)
        e = launch_fill((uint32_t*)(w + p.off_step_partials), 0xffffffffu, p.step_partials_bytes / sizeof(uint32_t), s);
    return e;
}

}  // namespace

// ---------------------------------------------------------------------------
// plan handle
// ---------------------------------------------------------------------------
struct lora_plan_s {
    const lora_table_s* table = nullptr;
    int device = 0;
    int n_rows = 0;
    int spin_limit = kSpinLimit;
    HostPlan plan;
    unsigned char* dmem = nullptr;
    size_t capacity = 0;                // device bytes at dmem, fixed at creation
    uint32_t generation = 0;            // of the work list last uploaded
    // two pinned staging buffers of `capacity` bytes for the uploads of
    // lora_plan_update, used in turn; each is rewritten only after the copy
    // that last read it has run
    struct Stage {
        void* host = nullptr;
        hipEvent_t ev = nullptr;
        bool pending = false;
    } stage[2];
    unsigned next_stage = 0;
};

namespace {

void plan_free(lora_plan_s* pl) {
    DeviceGuard dg(pl->device);
    for (auto& st : pl->stage) {
        if (st.pending && st.ev) (void)hipEventSynchronize(st.ev);
        if (st.ev) (void)hipEventDestroy(st.ev);
        if (st.host) (void)hipHostFree(st.host);
        st = lora_plan_s::Stage{};
    }
    if (pl->dmem) (void)hipFree(pl->dmem);
    pl->dmem = nullptr;
    delete pl;
}

// Upload the plan's work list (header with a new generation, item lists,
// grouped row order) from the next staging buffer and arm its step buffers,
// all on stream s.  No allocation; the host waits only if the staging buffer
// it takes is still being read by the copy enqueued two uploads before.
int plan_upload(lora_plan_s* pl, hipStream_t s) {
    if (++pl->generation == 0) pl->generation = 1;
    pl->plan.set_generation(pl->generation);
    auto& st = pl->stage[pl->next_stage++ & 1u];
    if (st.pending) {
        LORA_HIP_TRY(hipEventSynchronize(st.ev));
        st.pending = false;
    }
    std::memcpy(st.host, pl->plan.blob.data(), pl->plan.plan_bytes);
    LORA_HIP_TRY(hipMemcpyAsync(pl->dmem, st.host, pl->plan.plan_bytes, hipMemcpyHostToDevice, s));
    LORA_HIP_TRY(hipEventRecord(st.ev, s));
    st.pending = true;
    LORA_HIP_TRY(arm_step(pl->plan, pl->dmem, s));
    return LORA_OK;
}

}  // namespace

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
    if ((uint64_t)std::max(h_in, h_out) * kMaxRank * 2 > kMaxSpan)
        return fail(LORA_E_SHAPE, "h_in and h_out must be at most 4 Mi elements (factors below 2 GiB)");
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
    {
        int nx = 1;
        if (hipDeviceGetAttribute(&nx, hipDeviceAttributeNumberOfXccs, device) != hipSuccess || nx < 1) nx = 1;
        t->n_xcd = std::min(nx, 64);
        int nc = 0;
        if (hipDeviceGetAttribute(&nc, hipDeviceAttributeMultiprocessorCount, device) != hipSuccess) nc = 0;
        t->n_cu = std::max(nc, 0);
    }
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

int lora_plan_inspect(const lora_batch_t* b, int32_t h_in, int32_t h_out, int32_t n_adapters,
                      const int32_t* ranks, int32_t n_xcd, lora_item_info_t* items, int32_t capacity,
                      int32_t* n_items) {
    if (!n_items) return fail(LORA_E_ARG, "n_items is NULL");
    *n_items = 0;
    if (h_in <= 0 || h_out <= 0 || h_in % 8 || h_out % 8)
        return fail(LORA_E_SHAPE, "h_in and h_out must be positive multiples of 8");
    if ((uint64_t)std::max(h_in, h_out) * kMaxRank * 2 > kMaxSpan)
        return fail(LORA_E_SHAPE, "h_in and h_out must be at most 4 Mi elements (factors below 2 GiB)");
    if (n_adapters < 0 || (n_adapters > 0 && !ranks)) return fail(LORA_E_ARG, "bad adapter ranks");
    if (capacity < 0) return fail(LORA_E_ARG, "negative capacity");
    lora_table_s t;                           // host-side table: ranks and shapes only
    t.h_in = h_in;
    t.h_out = h_out;
    t.n = n_adapters;
    t.n_xcd = std::max(1, std::min(n_xcd, 64));
    t.host.assign(n_adapters, DevAdapter{});
    for (int i = 0; i < n_adapters; ++i) {
        if (ranks[i] < 1 || ranks[i] > kMaxRank)
            return fail(LORA_E_RANK, "adapter " + std::to_string(i) + " has rank " + std::to_string(ranks[i]) +
                                         " outside [1, 256]");
        t.host[i].rank = ranks[i];
        t.host[i].scale = 1.f;
    }
    HostPlan p;
    if (int rc = build_plan(&t, b, p)) return rc;
    std::vector<const DevItem*> grid;
    if (!p.step.empty()) {
        for (const DevItem& it : p.step) grid.push_back(&it);
    } else {
        for (const auto* list : {&p.shrink, &p.reduce, &p.expand})
            for (const DevItem& it : *list) grid.push_back(&it);
    }
    const size_t total = grid.size() + p.reduce_all.size();
    if (total > (size_t)INT32_MAX) return fail(LORA_E_SHAPE, "plan too large to list");
    *n_items = (int32_t)total;
    if (!items) return LORA_OK;               // size query
    if ((size_t)capacity < total) return fail(LORA_E_ARG, "capacity smaller than the plan's item count (see n_items)");
    auto put = [&](int32_t at, const DevItem& it, int32_t pos) {
        lora_item_info_t& o = items[at];
        o.kind = it.kind;
        o.row_block = it.rb;
        o.rank = it.rank;
        o.nrows = it.nrows;
        o.lo = it.lo;
        o.len = it.len;
        o.sub = it.sub;
        o.nsplit = it.nsplit;
        o.pstride = it.pstride;
        o.grid_pos = pos;
    };
    int32_t k = 0;
    for (size_t i = 0; i < grid.size(); ++i, ++k) put(k, *grid[i], (int32_t)i);
    for (const DevItem& it : p.reduce_all) put(k++, it, -1);
    return LORA_OK;
}

int lora_shrink(lora_table_t t, const lora_batch_t* b, const void* x, int64_t ldx, float* v,
                int64_t ldv, void* ws, size_t ws_bytes, void* stream) {
    if (int rc = check_table(t)) return rc;
    HostPlan p;
    if (int rc = build_plan(t, b, p)) return rc;
    if (p.n_active == 0) return LORA_OK;
    if (int rc = check_x(t, x, ldx, b->n_rows)) return rc;
    if (int rc = check_v(p, v, ldv)) return rc;
    if (int rc = check_ws(p, ws, ws_bytes)) return rc;
    DeviceGuard dg(t->device);
    hipStream_t s = (hipStream_t)stream;
    if (int rc = check_not_capturing(s, "lora_shrink")) return rc;
    unsigned char* w = (unsigned char*)ws;
    if (int rc = stage_upload(t->device, p.blob.data(), p.plan_bytes, w, s)) return rc;
    if (int rc = enqueue(t, p, w, x, ldx, nullptr, 0, s, true)) return rc;
    KernelArgs a = make_args(t, p, w, kSpinLimit);
    a.items = (const DevItem*)(w + p.off_reduce_all);
    a.n_items = (int32_t)p.reduce_all.size();
    a.v = v;
    a.ldv = ldv;
    LORA_HIP_TRY(launch_reduce(a, (const uint32_t*)w, s));
    return LORA_OK;
}

int lora_expand(lora_table_t t, const lora_batch_t* b, const float* v, int64_t ldv, void* y,
                int64_t ldy, void* ws, size_t ws_bytes, void* stream) {
    if (int rc = check_table(t)) return rc;
    HostPlan p;
    if (int rc = build_plan(t, b, p)) return rc;
    if (p.n_active == 0) return LORA_OK;
    if (int rc = check_v(p, v, ldv)) return rc;
    if (int rc = check_y(t, y, ldy, b->n_rows)) return rc;
    if (int rc = check_ws(p, ws, ws_bytes)) return rc;
    DeviceGuard dg(t->device);
    hipStream_t s = (hipStream_t)stream;
    if (int rc = check_not_capturing(s, "lora_expand")) return rc;
    unsigned char* w = (unsigned char*)ws;
    if (int rc = stage_upload(t->device, p.blob.data(), p.plan_bytes, w, s)) return rc;
    KernelArgs a = make_args(t, p, w, kSpinLimit);
    a.items = (const DevItem*)(w + p.off_expand);
    a.n_items = (int32_t)p.expand.size();
    a.v = const_cast<float*>(v);
    a.ldv = ldv;
    a.y = y;
    a.ldy = ldy;
    a.y_bytes = (uint32_t)span_bytes(p.n_rows, ldy, t->h_out);
    LORA_HIP_TRY(launch_expand(a, (const uint32_t*)w, t->dtype, s));
    return LORA_OK;
}

int lora_apply_fused(lora_table_t t, const lora_batch_t* b, const void* x, int64_t ldx, void* y,
                     int64_t ldy, void* ws, size_t ws_bytes, void* stream) {
    if (int rc = check_table(t)) return rc;
    HostPlan p;
    if (int rc = build_plan(t, b, p)) return rc;
    if (p.n_active == 0) return LORA_OK;
    if (int rc = check_x(t, x, ldx, b->n_rows)) return rc;
    if (int rc = check_y(t, y, ldy, b->n_rows)) return rc;
    if (int rc = check_overlap(x, ldx, t->h_in, y, ldy, t->h_out, b->n_rows)) return rc;
    if (int rc = check_ws(p, ws, ws_bytes)) return rc;
    DeviceGuard dg(t->device);
    hipStream_t s = (hipStream_t)stream;
    if (int rc = check_not_capturing(s, "lora_apply_fused")) return rc;
    unsigned char* w = (unsigned char*)ws;
    if (int rc = stage_upload(t->device, p.blob.data(), p.plan_bytes, w, s)) return rc;
    return enqueue(t, p, w, x, ldx, y, ldy, s);
}

// ---------------------------------------------------------------------------
// fused base projection (Eq. 1 whole)
// ---------------------------------------------------------------------------
namespace {

// Workspace of lora_base_apply: [plan (header, items, grouped rows) | partial
// and v blocks | counters] [dense float32 v: n_rows x ldv] [per row tile:
// offsets into the runs, then the runs of rows that share an adapter]
// [float32 partial tiles of the split tiles].
struct BaseLayout {
    HostPlan p;
    int ldv = 8;
    int tile = kBaseBig;
    int n_mt = 0, n_nt = 0;
    int n_whole = 0, split = 1, chunk = 0;
    size_t off_v = 0, v_bytes = 0, off_pieces = 0, off_part = 0, part_bytes = 0, total = 0;
    std::vector<unsigned char> pieces_blob;
    size_t off_piece_list = 0;           // within pieces_blob
};

// Work of one launch: whole rounds of tiles over the compute units run whole;
// the tiles of a last, partial round are split along K into ranges of at
// least kBaseMinSplitStages stages (an even number of them), as many as fill
// the compute units, their partial tiles added by a second kernel.
void choose_split(int n_tiles, int h_in, int n_cu, BaseLayout& L) {
    const int bk = base_bk(L.tile);
    const int nk = ((h_in + 2 * bk - 1) / (2 * bk)) * 2;
    L.n_whole = n_tiles;
    L.split = 1;
    L.chunk = nk;
    if (n_cu <= 0 || n_tiles == 0) return;
    const int rounds = n_tiles / n_cu;
    const int rem = n_tiles - rounds * n_cu;
    if (rem == 0) return;
    const int s = std::min(n_cu / rem, nk / kBaseMinSplitStages);
    if (s < 2) return;
    const int chunk = round_up_i((nk + s - 1) / s, 2);
    const int split = (nk + chunk - 1) / chunk;
    if (split < 2) return;
    L.n_whole = rounds * n_cu;
    L.split = split;
    L.chunk = chunk;
}

int build_base(const lora_table_s* t, const lora_batch_t* b, BaseLayout& L) {
    if (int rc = build_plan(t, b, L.p)) return rc;
    L.ldv = round_up_i(std::max(L.p.r_max, 1), 8);
    L.off_v = align_up(L.p.total_bytes);
    L.v_bytes = (size_t)b->n_rows * L.ldv * sizeof(float);
    if (L.v_bytes > kMaxSpan) return fail(LORA_E_SHAPE, "batch too large: its float32 intermediate exceeds 2 GiB");
    // the big tile while its whole tiles fill the compute units; else the
    // small one, which has four times as many tiles to spread (a 1024-token
    // prompt at 4096 columns: 256 whole tiles instead of 64 split four ways)
    const int64_t big_tiles = (int64_t)((b->n_rows + kBaseBig - 1) / kBaseBig) * ((t->h_out + kBaseBig - 1) / kBaseBig);
    L.tile = big_tiles >= t->n_cu ? kBaseBig : kBaseSmall;
    L.n_mt = (b->n_rows + L.tile - 1) / L.tile;
    L.n_nt = (t->h_out + L.tile - 1) / L.tile;
    // runs of rows sharing an adapter, per row tile; neighbouring segments of
    // one adapter inside a tile make one run
    std::vector<std::vector<BasePiece>> per(L.n_mt);
    for (int sgi = 0; sgi < b->n_segments; ++sgi) {
        const int g = b->seg_adapter[sgi];
        int lo = b->seg_offset[sgi];
        const int hi = b->seg_offset[sgi + 1];
        if (g < 0) continue;
        while (lo < hi) {
            const int mt = lo / L.tile;
            const int e = std::min(hi, (mt + 1) * L.tile);
            auto& v = per[mt];
            if (!v.empty() && v.back().adapter == g && v.back().hi == lo) v.back().hi = e;
            else v.push_back(BasePiece{lo, e, g, 0});
            lo = e;
        }
    }
    std::vector<int32_t> off(L.n_mt + 1, 0);
    for (int m = 0; m < L.n_mt; ++m) off[m + 1] = off[m] + (int32_t)per[m].size();
    L.off_piece_list = align_up((size_t)(L.n_mt + 1) * sizeof(int32_t), 16);
    L.pieces_blob.assign(L.off_piece_list + (size_t)off[L.n_mt] * sizeof(BasePiece), 0);
    std::memcpy(L.pieces_blob.data(), off.data(), off.size() * sizeof(int32_t));
    size_t at = L.off_piece_list;
    for (const auto& v : per)
        for (const BasePiece& pc : v) {
            std::memcpy(L.pieces_blob.data() + at, &pc, sizeof pc);
            at += sizeof pc;
        }
    L.off_pieces = align_up(L.off_v + L.v_bytes);
    L.off_part = align_up(L.off_pieces + std::max<size_t>(L.pieces_blob.size(), 16));
    choose_split(L.n_mt * L.n_nt, t->h_in, t->n_cu, L);
    L.part_bytes = (size_t)(L.n_mt * L.n_nt - L.n_whole) * L.split * ((size_t)L.tile * L.tile * sizeof(float));
    if (L.split < 2) L.part_bytes = 0;
    L.total = L.off_part + L.part_bytes;
    return LORA_OK;
}

}  // namespace

int lora_base_workspace_bytes(lora_table_t t, const lora_batch_t* b, size_t* bytes) {
    if (int rc = check_table(t)) return rc;
    if (!bytes) return fail(LORA_E_ARG, "bytes is NULL");
    BaseLayout L;
    if (int rc = build_base(t, b, L)) return rc;
    *bytes = L.total;
    return LORA_OK;
}

int lora_base_inspect(const lora_batch_t* b, int32_t h_in, int32_t h_out, int32_t n_adapters, const int32_t* ranks,
                      int32_t n_cu, int32_t n_xcd, lora_base_info_t* out) {
    if (!out) return fail(LORA_E_ARG, "out is NULL");
    if (h_in <= 0 || h_out <= 0 || h_in % 8 || h_out % 8)
        return fail(LORA_E_SHAPE, "h_in and h_out must be positive multiples of 8");
    if ((uint64_t)std::max(h_in, h_out) * kMaxRank * 2 > kMaxSpan)
        return fail(LORA_E_SHAPE, "h_in and h_out must be at most 4 Mi elements (factors below 2 GiB)");
    if (n_adapters < 0 || (n_adapters > 0 && !ranks)) return fail(LORA_E_ARG, "bad adapter ranks");
    if (n_cu < 0) return fail(LORA_E_ARG, "negative n_cu");
    lora_table_s t;                           // host-side table: ranks and shapes only
    t.h_in = h_in;
    t.h_out = h_out;
    t.n = n_adapters;
    t.n_cu = n_cu;
    t.n_xcd = std::max(1, std::min(n_xcd, 64));
    t.host.assign(n_adapters, DevAdapter{});
    for (int i = 0; i < n_adapters; ++i) {
        if (ranks[i] < 1 || ranks[i] > kMaxRank)
            return fail(LORA_E_RANK, "adapter " + std::to_string(i) + " has rank " + std::to_string(ranks[i]) +
                                         " outside [1, 256]");
        t.host[i].rank = ranks[i];
        t.host[i].scale = 1.f;
    }
    BaseLayout L;
    if (int rc = build_base(&t, b, L)) return rc;
    const int bk = base_bk(L.tile);
    const int n_tiles = L.n_mt * L.n_nt;
    const int per_xcd = (L.n_whole + t.n_xcd - 1) / t.n_xcd;
    const int n_split = L.split > 1 ? n_tiles - L.n_whole : 0;
    out->tile = L.tile;
    out->n_mt = L.n_mt;
    out->n_nt = L.n_nt;
    out->n_whole = L.n_whole;
    out->split = L.split;
    out->chunk = L.chunk;
    out->n_stages = ((h_in + 2 * bk - 1) / (2 * bk)) * 2;
    out->stage_k = bk;
    out->per_xcd = per_xcd;
    out->grid = t.n_xcd * per_xcd + n_split * L.split;
    out->panel = kBasePanel;
    out->workspace_bytes = L.total;
    return LORA_OK;
}

}  // extern "C"

namespace {

// The operand checks of lora_base_apply and lora_base_plan_apply.
int check_base_operands(const lora_table_s* t, int n_rows, const void* x, int64_t ldx, const void* wt, int64_t ldw,
                        void* y, int64_t ldy, uint64_t* w_span_out) {
    if (int rc = check_x(t, x, ldx, n_rows)) return rc;
    if (int rc = check_y(t, y, ldy, n_rows)) return rc;
    if (!wt) return fail(LORA_E_ARG, "wt is NULL");
    if (!aligned16(wt)) return fail(LORA_E_ALIGN, "wt not 16-byte aligned");
    if (int rc = check_ld("ldw", ldw, t->h_in)) return rc;
    const uint64_t w_span = span_bytes(t->h_out, ldw, t->h_in);
    if (w_span > kMaxSpan) return fail(LORA_E_SHAPE, "wt spans more than 2 GiB");
    if (int rc = check_overlap(x, ldx, t->h_in, y, ldy, t->h_out, n_rows)) return rc;
    const uintptr_t ws0 = (uintptr_t)wt, we = ws0 + w_span;
    const uintptr_t ys = (uintptr_t)y, ye = ys + span_bytes(n_rows, ldy, t->h_out);
    if (ws0 < ye && ys < we) return fail(LORA_E_OVERLAP, "wt and y overlap");
    *w_span_out = w_span;
    return LORA_OK;
}

// Everything after the upload: the shrink of every adapted row into the dense
// float32 v, then the GEMM with the delta in its epilogue.  The work list and
// the tile pieces are at their layout offsets in w.  Kernels only (a graph
// may record it).
int base_run(const lora_table_s* t, const BaseLayout& L, int n_rows, unsigned char* w, const void* x, int64_t ldx,
             const void* wt, int64_t ldw, uint64_t w_span, void* y, int64_t ldy, hipStream_t s) {
    float* v = (float*)(w + L.off_v);
    const HostPlan& p = L.p;
    if (p.n_active > 0) {
        // v = x . A_g for every adapted row, into the dense float32 buffer
        if (int rc = enqueue(t, p, w, x, ldx, nullptr, 0, s, true)) return rc;
        KernelArgs ra = make_args(t, p, w, kSpinLimit);
        ra.items = (const DevItem*)(w + p.off_reduce_all);
        ra.n_items = (int32_t)p.reduce_all.size();
        ra.v = v;
        ra.ldv = L.ldv;
        LORA_HIP_TRY(launch_reduce(ra, (const uint32_t*)w, s));
    }
    BaseArgs a{};
    a.x = x;
    a.wt = wt;
    a.y = y;
    a.v = v;
    a.table = t->dev;
    a.piece_off = (const int32_t*)(w + L.off_pieces);
    a.pieces = (const BasePiece*)(w + L.off_pieces + L.off_piece_list);
    a.ldx = ldx;
    a.ldw = ldw;
    a.ldy = ldy;
    a.ldv = L.ldv;
    a.M = n_rows;
    a.N = t->h_out;
    a.K = t->h_in;
    a.tile = L.tile;
    a.n_mt = L.n_mt;
    a.n_nt = L.n_nt;
    a.n_xcd = std::max(1, t->n_xcd);
    a.n_whole = L.n_whole;
    a.per_xcd = (L.n_whole + a.n_xcd - 1) / a.n_xcd;
    a.split = L.split;
    a.chunk = L.chunk;
    a.part = L.split > 1 ? (float*)(w + L.off_part) : nullptr;
    a.x_bytes = (uint32_t)span_bytes(n_rows, ldx, t->h_in);
    a.w_bytes = (uint32_t)w_span;
    a.y_bytes = (uint32_t)span_bytes(n_rows, ldy, t->h_out);
    a.v_bytes = (uint32_t)L.v_bytes;
    a.b_span_ok = 1;
    LORA_HIP_TRY(launch_base(a, t->dtype, s));
    return LORA_OK;
}

}  // namespace

struct lora_base_plan_s {
    const lora_table_s* table = nullptr;
    int device = 0;
    int n_rows = 0;
    BaseLayout L;
    unsigned char* dmem = nullptr;
};

extern "C" {

int lora_base_apply(lora_table_t t, const lora_batch_t* b, const void* x, int64_t ldx, const void* wt,
                    int64_t ldw, void* y, int64_t ldy, void* ws, size_t ws_bytes, void* stream) {
    if (int rc = check_table(t)) return rc;
    BaseLayout L;
    if (int rc = build_base(t, b, L)) return rc;
    const int n_rows = b->n_rows;
    if (n_rows == 0) return LORA_OK;
    uint64_t w_span = 0;
    if (int rc = check_base_operands(t, n_rows, x, ldx, wt, ldw, y, ldy, &w_span)) return rc;
    if (!ws) return fail(LORA_E_ARG, "workspace is NULL");
    if (!aligned16(ws)) return fail(LORA_E_ALIGN, "workspace not 16-byte aligned");
    if (ws_bytes < L.total)
        return fail(LORA_E_WORKSPACE, "workspace has " + std::to_string(ws_bytes) + " bytes, needs " +
                                          std::to_string(L.total));
    DeviceGuard dg(t->device);
    hipStream_t s = (hipStream_t)stream;
    if (int rc = check_not_capturing(s, "lora_base_apply")) return rc;
    unsigned char* w = (unsigned char*)ws;
    if (int rc = stage_upload(t->device, L.p.blob.data(), L.p.plan_bytes, w, s)) return rc;
    if (int rc = stage_upload(t->device, L.pieces_blob.data(), L.pieces_blob.size(), w + L.off_pieces, s)) return rc;
    return base_run(t, L, n_rows, w, x, ldx, wt, ldw, w_span, y, ldy, s);
}

int lora_base_plan_create(lora_base_plan_t* out, lora_table_t t, const lora_batch_t* b, void* stream) {
    if (!out) return fail(LORA_E_ARG, "out is NULL");
    *out = nullptr;
    if (int rc = check_table(t)) return rc;
    auto* pl = new (std::nothrow) lora_base_plan_s();
    if (!pl) return fail(LORA_E_NOMEM, "plan allocation failed");
    if (int rc = build_base(t, b, pl->L)) {
        delete pl;
        return rc;
    }
    DeviceGuard dg(t->device);
    hipStream_t s = (hipStream_t)stream;
    if (int rc = check_not_capturing(s, "lora_base_plan_create")) {
        delete pl;
        return rc;
    }
    pl->table = t;
    pl->device = t->device;
    pl->n_rows = b->n_rows;
    hipError_t e = hipMalloc((void**)&pl->dmem, std::max<size_t>(pl->L.total, 256));
    if (e != hipSuccess) {
        delete pl;
        return fail(LORA_E_NOMEM, std::string("hipMalloc of the base plan: ") + hipGetErrorString(e));
    }
    const BaseLayout& L = pl->L;
    e = hipMemcpyAsync(pl->dmem, L.p.blob.data(), L.p.plan_bytes, hipMemcpyHostToDevice, s);
    if (e == hipSuccess && !L.pieces_blob.empty())
        e = hipMemcpyAsync(pl->dmem + L.off_pieces, L.pieces_blob.data(), L.pieces_blob.size(), hipMemcpyHostToDevice,
                           s);
    if (e == hipSuccess) e = hipStreamSynchronize(s);
    if (e != hipSuccess) {
        (void)hipFree(pl->dmem);
        delete pl;
        return fail(LORA_E_HIP, std::string("base plan upload: ") + hipGetErrorString(e));
    }
    *out = pl;
    return LORA_OK;
}

int lora_base_plan_apply(lora_base_plan_t pl, lora_table_t t, const void* x, int64_t ldx, const void* wt, int64_t ldw,
                         void* y, int64_t ldy, void* stream) {
    if (!pl || !pl->dmem) return fail(LORA_E_ARG, "plan is NULL");
    const lora_table_s* tt = t ? t : pl->table;
    if (int rc = check_compatible(pl->L.p, tt)) return rc;
    if (tt->device != pl->device) return fail(LORA_E_ARG, "table is on another device than the plan");
    if (pl->n_rows == 0) return LORA_OK;
    uint64_t w_span = 0;
    if (int rc = check_base_operands(tt, pl->n_rows, x, ldx, wt, ldw, y, ldy, &w_span)) return rc;
    DeviceGuard dg(tt->device);
    return base_run(tt, pl->L, pl->n_rows, pl->dmem, x, ldx, wt, ldw, w_span, y, ldy, (hipStream_t)stream);
}

int lora_base_plan_destroy(lora_base_plan_t pl) {
    if (!pl) return fail(LORA_E_ARG, "plan is NULL");
    if (pl->dmem) {
        DeviceGuard dg(pl->device);
        (void)hipFree(pl->dmem);
    }
    delete pl;
    return LORA_OK;
}

int lora_apply_fused_static(lora_table_t t, const lora_batch_t* b, const void* x, int64_t ldx, void* y,
                            int64_t ldy, void* stream) {
    if (int rc = check_table(t)) return rc;
    HostPlan p;
    if (int rc = build_plan(t, b, p)) return rc;
    if (p.n_active == 0) return LORA_OK;
    if (int rc = check_x(t, x, ldx, b->n_rows)) return rc;
    if (int rc = check_y(t, y, ldy, b->n_rows)) return rc;
    if (int rc = check_overlap(x, ldx, t->h_in, y, ldy, t->h_out, b->n_rows)) return rc;
    if (p.total_bytes > kScratchBytes)
        return fail(LORA_E_WORKSPACE, "the batch needs " + std::to_string(p.total_bytes) +
                                          " bytes of workspace; the static scratch holds " +
                                          std::to_string(kScratchBytes) + " (use lora_apply_fused)");
    DeviceGuard dg(t->device);
    if (!dg.ok) return fail(LORA_E_HIP, "hipSetDevice failed");
    hipStream_t s = (hipStream_t)stream;
    if (int rc = check_not_capturing(s, "lora_apply_fused_static")) return rc;
    unsigned char* w = nullptr;
    if (int rc = scratch_address(t->device, &w)) return rc;
    // from pageable host memory: HIP performs this copy synchronously, so the
    // host-side work list may go when the call returns (and the copy is
    // ordered after the stream's earlier work, which may still read scratch)
    LORA_HIP_TRY(hipMemcpyAsync(w, p.blob.data(), p.plan_bytes, hipMemcpyHostToDevice, s));
    return enqueue(t, p, w, x, ldx, y, ldy, s);
}

int lora_plan_bytes(lora_table_t t, const lora_batch_t* b, size_t* bytes) {
    if (int rc = check_table(t)) return rc;
    if (!bytes) return fail(LORA_E_ARG, "bytes is NULL");
    HostPlan p;
    if (int rc = build_plan(t, b, p)) return rc;
    *bytes = p.plan_total_bytes;
    return LORA_OK;
}

}  // extern "C"

namespace {

// A plan of n projections sharing x (n = 1: an ordinary plan).
int plan_create(lora_plan_t* out, int n, const lora_table_t* tables, const lora_batch_t* b, size_t min_bytes,
                void* stream) {
    if (!out) return fail(LORA_E_ARG, "out is NULL");
    *out = nullptr;
    const lora_table_s* t = tables[0];
    if (int rc = check_table(t)) return rc;
    hipStream_t s = (hipStream_t)stream;
    if (int rc = check_not_capturing(s, "lora_plan_create")) return rc;
    auto* pl = new (std::nothrow) lora_plan_s();
    if (!pl) return fail(LORA_E_NOMEM, "plan allocation failed");
    pl->table = t;
    pl->device = t->device;
    for (int i = 1; i < n; ++i)
        if (tables[i]->device != t->device) {
            delete pl;
            return fail(LORA_E_ARG, "the projections' tables are on different devices");
        }
    if (int rc = n > 1 ? build_plan_multi(tables, n, b, pl->plan) : build_plan(t, b, pl->plan)) {
        delete pl;
        return rc;
    }
    for (int i = 1; i < n; ++i)
        if (int rc = check_compatible_proj(pl->plan, tables[i], i)) {
            delete pl;
            return rc;
        }
    pl->n_rows = b->n_rows;
    pl->capacity = align_up(std::max(pl->plan.plan_total_bytes, min_bytes));
    DeviceGuard dg(t->device);
    hipError_t e = hipMalloc((void**)&pl->dmem, pl->capacity);
    for (auto& st : pl->stage) {
        if (e == hipSuccess) e = hipHostMalloc(&st.host, pl->capacity, hipHostMallocDefault);
        if (e == hipSuccess) e = hipEventCreateWithFlags(&st.ev, hipEventDisableTiming);
    }
    if (e != hipSuccess) {
        plan_free(pl);
        return fail(LORA_E_NOMEM, std::string("plan memory: ") + hipGetErrorString(e));
    }
    int rc = plan_upload(pl, s);
    if (rc == LORA_OK && hipStreamSynchronize(s) != hipSuccess) rc = fail(LORA_E_HIP, "plan upload failed");
    if (rc != LORA_OK) {
        plan_free(pl);
        return rc;
    }
    *out = pl;
    return LORA_OK;
}

}  // namespace

extern "C" {

int lora_plan_create_reserved(lora_plan_t* out, lora_table_t t, const lora_batch_t* b, size_t min_bytes,
                              void* stream) {
    return plan_create(out, 1, &t, b, min_bytes, stream);
}

int lora_plan_create(lora_plan_t* out, lora_table_t t, const lora_batch_t* b, void* stream) {
    return lora_plan_create_reserved(out, t, b, 0, stream);
}

int lora_plan_create_multi(lora_plan_t* out, int32_t n, const lora_table_t* tables, const lora_batch_t* b,
                           void* stream) {
    if (!out) return fail(LORA_E_ARG, "out is NULL");
    *out = nullptr;
    if (n < 1 || n > kMaxProj) return fail(LORA_E_ARG, "n must be in [1, " + std::to_string(kMaxProj) + "]");
    if (!tables) return fail(LORA_E_ARG, "tables is NULL");
    for (int i = 0; i < n; ++i)
        if (int rc = check_table(tables[i])) return rc;
    return plan_create(out, n, tables, b, 0, stream);
}

int lora_plan_apply_multi(lora_plan_t pl, const lora_table_t* tables, const void* x, int64_t ldx, void* const* ys,
                          const int64_t* ldys, void* stream) {
    if (!pl || !pl->dmem) return fail(LORA_E_ARG, "plan is NULL");
    const int n = pl->plan.n_proj;
    if (!tables || !ys || !ldys || !x) return fail(LORA_E_ARG, "tables, ys, ldys or x is NULL");
    for (int i = 0; i < n; ++i) {
        const lora_table_s* tt = tables[i] ? tables[i] : (i == 0 ? pl->table : nullptr);
        if (!tt) return fail(LORA_E_ARG, "table " + std::to_string(i) + " is NULL");
        if (int rc = check_compatible_proj(pl->plan, tt, i)) return rc;
        if (tt->device != pl->device) return fail(LORA_E_ARG, "table is on another device than the plan");
        if (!ys[i]) return fail(LORA_E_ARG, "y " + std::to_string(i) + " is NULL");
        if (pl->plan.n_active == 0) continue;
        if (int rc = check_x(tt, x, ldx, pl->n_rows)) return rc;
        if (int rc = check_y(tt, ys[i], ldys[i], pl->n_rows)) return rc;
        if (int rc = check_overlap(x, ldx, tt->h_in, ys[i], ldys[i], tt->h_out, pl->n_rows)) return rc;
        for (int j = 0; j < i; ++j)
            if (int rc = check_overlap(ys[j], ldys[j], pl->plan.proj_h_out.empty() ? tt->h_out : pl->plan.proj_h_out[j],
                                       ys[i], ldys[i], tt->h_out, pl->n_rows))
                return rc;
    }
    if (pl->plan.n_active == 0) return LORA_OK;
    const lora_table_s* t0 = tables[0] ? tables[0] : pl->table;
    DeviceGuard dg(pl->device);
    KernelArgs a{};
    if (int rc = step_args(t0, pl->plan, pl->dmem, x, ldx, ys[0], ldys[0], pl->spin_limit, a)) return rc;
    a.n_proj = n;
    for (int i = 0; i < n; ++i) {
        const lora_table_s* tt = tables[i] ? tables[i] : pl->table;
        a.ptable[i] = tt->dev;
        a.py[i] = ys[i];
        a.pldy[i] = ldys[i];
        a.py_bytes[i] = (uint32_t)span_bytes(pl->n_rows, ldys[i], tt->h_out);
        a.ph_out[i] = tt->h_out;
    }
    LORA_HIP_TRY(launch_step(a, (const uint32_t*)pl->dmem, t0->dtype, (hipStream_t)stream));
    return LORA_OK;
}

int lora_plan_update(lora_plan_t pl, lora_table_t t, const lora_batch_t* b, void* stream) {
    if (!pl || !pl->dmem) return fail(LORA_E_ARG, "plan is NULL");
    const lora_table_s* tt = t ? t : pl->table;
    if (int rc = check_table(tt)) return rc;
    if (tt->device != pl->device) return fail(LORA_E_ARG, "table is on another device than the plan");
    hipStream_t s = (hipStream_t)stream;
    DeviceGuard dg(pl->device);
    if (int rc = check_not_capturing(s, "lora_plan_update")) return rc;
    if (pl->plan.n_proj > 1)
        return fail(LORA_E_ARG, "a plan of several projections is re-planned with lora_plan_create_multi");
    HostPlan np;
    if (int rc = build_plan(tt, b, np)) return rc;
    if (np.plan_total_bytes > pl->capacity)
        return fail(LORA_E_WORKSPACE, "the batch needs " + std::to_string(np.plan_total_bytes) +
                                          " bytes of plan memory; the plan holds " + std::to_string(pl->capacity) +
                                          " (lora_plan_create_reserved sets the capacity)");
    pl->plan = std::move(np);
    pl->table = tt;
    pl->n_rows = b->n_rows;
    return plan_upload(pl, s);
}

static int plan_run(lora_plan_t pl, lora_table_t t, const void* x, int64_t ldx, void* y, int64_t ldy,
                    void* stream) {
    if (!pl || !pl->dmem) return fail(LORA_E_ARG, "plan is NULL");
    if (pl->plan.n_proj > 1) return fail(LORA_E_ARG, "a plan of several projections runs through lora_plan_apply_multi");
    const lora_table_s* tt = t ? t : pl->table;
    if (int rc = check_compatible(pl->plan, tt)) return rc;
    if (tt->device != pl->device) return fail(LORA_E_ARG, "table is on another device than the plan");
    if (pl->plan.n_active == 0) return LORA_OK;
    if (x)
        if (int rc = check_x(tt, x, ldx, pl->n_rows)) return rc;
    if (y)
        if (int rc = check_y(tt, y, ldy, pl->n_rows)) return rc;
    if (x && y)
        if (int rc = check_overlap(x, ldx, tt->h_in, y, ldy, tt->h_out, pl->n_rows)) return rc;
    DeviceGuard dg(tt->device);
    if (x && y)
        return enqueue_step(tt, pl->plan, pl->dmem, x, ldx, y, ldy, pl->spin_limit, (hipStream_t)stream);
    return enqueue(tt, pl->plan, pl->dmem, x, ldx, y, ldy, (hipStream_t)stream);
}

int lora_plan_apply(lora_plan_t pl, lora_table_t t, const void* x, int64_t ldx, void* y, int64_t ldy,
                    void* stream) {
    if (!x || !y) return fail(LORA_E_ARG, "x or y is NULL");
    return plan_run(pl, t, x, ldx, y, ldy, stream);
}

int lora_plan_shrink(lora_plan_t pl, lora_table_t t, const void* x, int64_t ldx, void* stream) {
    if (!x) return fail(LORA_E_ARG, "x is NULL");
    return plan_run(pl, t, x, ldx, nullptr, 0, stream);
}

int lora_plan_expand(lora_plan_t pl, lora_table_t t, void* y, int64_t ldy, void* stream) {
    if (!y) return fail(LORA_E_ARG, "y is NULL");
    return plan_run(pl, t, nullptr, 0, y, ldy, stream);
}

int lora_plan_status(lora_plan_t pl, void* stream) {
    if (!pl || !pl->dmem) return fail(LORA_E_ARG, "plan is NULL");
    DeviceGuard dg(pl->device);
    hipStream_t s = (hipStream_t)stream;
    int32_t flag = 0;
    LORA_HIP_TRY(hipMemcpyAsync(&flag, pl->dmem + sizeof(uint32_t), sizeof(flag), hipMemcpyDeviceToHost, s));
    LORA_HIP_TRY(hipStreamSynchronize(s));
    if (flag == kStatusOk) return LORA_OK;
    LORA_HIP_TRY(arm_step(pl->plan, pl->dmem, s));
    LORA_HIP_TRY(hipStreamSynchronize(s));
    if (flag == kStatusStale)
        return fail(LORA_E_STALE, "a launch recorded for an earlier batch of this plan ran after lora_plan_update "
                                  "and did nothing");
    return fail(LORA_E_SYNC, "a step launch gave up waiting for its shrink items; its results are invalid");
}

int lora_plan_set_spin_limit(lora_plan_t pl, int32_t polls) {
    if (!pl) return fail(LORA_E_ARG, "plan is NULL");
    if (polls < 0) return fail(LORA_E_ARG, "negative spin limit");
    pl->spin_limit = polls;
    return LORA_OK;
}

int lora_plan_destroy(lora_plan_t pl) {
    if (!pl) return fail(LORA_E_ARG, "plan is NULL");
    plan_free(pl);
    return LORA_OK;
}

}  // extern "C"
