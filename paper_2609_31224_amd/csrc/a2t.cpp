// libA2T host side: argument validation, the per-stream host state, the
// eviction planner of Sec. 3.3, and kernel launches.  Public API: include/a2t.h.
//
// The host state mirrors what the device holds, so no call needs to read the
// device back to plan work: per stream it knows the kept-region size, the
// ring head and size, and the queue of not-yet-evicted units with their row
// counts.  Eviction is planned from those counts (positions are what the
// paper's budget counts) and the device then derives the per-row mask,
// compaction indices and row moves itself.
#include "../../include/a2t.h"
#include "a2t_internal.h"

#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdlib>
#include <cstring>
#include <deque>
#include <map>
#include <string>
#include <vector>

using namespace a2t;

namespace {

struct UnitRec {
    int32_t unit;
    int32_t rows;       // rows of this unit still in the ring
    int32_t evictable;  // ACOUSTIC/DELIM rows among them
};

// FIFO of the units with rows in the ring, in a buffer sized at creation: every
// queued unit holds at least one ring row, so unit_rows entries always suffice.
class UnitQueue {
public:
    void init(size_t cap) { buf_.assign(std::max<size_t>(cap, 1), UnitRec{}); }
    size_t size() const { return n_; }
    bool empty() const { return n_ == 0; }
    UnitRec& operator[](size_t i) { return buf_[(h_ + i) % buf_.size()]; }
    const UnitRec& operator[](size_t i) const { return buf_[(h_ + i) % buf_.size()]; }
    UnitRec& back() { return (*this)[n_ - 1]; }
    const UnitRec& back() const { return (*this)[n_ - 1]; }
    bool full() const { return n_ == buf_.size(); }
    void push_back(const UnitRec& u) {
        buf_[(h_ + n_) % buf_.size()] = u;
        ++n_;
    }
    void pop_front(size_t k) {
        h_ = (h_ + k) % buf_.size();
        n_ -= k;
    }

private:
    std::vector<UnitRec> buf_;
    size_t h_ = 0, n_ = 0;
};

struct StreamState {
    int64_t last_pos = -1;
    int32_t cur_unit = -2;          // -2: nothing appended yet
    int32_t last_evicted = -2;
    int32_t kept = 0;               // T
    int32_t head = 0;               // ring head slot
    int32_t ring = 0;               // U
    int32_t peak = 0;
    UnitQueue units;
    std::vector<uint8_t> ring_seg;  // class of every ring slot (host mirror of the device's)
    // open step
    int32_t step_rows = 0;
    int32_t step_slot0 = 0;
    std::vector<uint8_t> appended;  // per layer, for the open step
    std::vector<uint8_t> step_seg;
    std::vector<int32_t> step_pos;
    int32_t step_unit = 0;
    // stats
    int64_t evicted_total = 0;
    int64_t moved_total = 0;
    int32_t budget_unmet = 0;
    int32_t last_evict_pre = -1;

    int32_t resident() const { return kept + ring; }
    bool step_complete() const {
        for (uint8_t a : appended)
            if (!a) return false;
        return true;
    }
};

struct ProfEvent {
    std::string name;
    hipEvent_t start, stop;
};

// One stream's eviction, planned on the host.  The device pass moves over the
// `span` oldest ring rows: it keeps `n_keep` of them (copied to the kept region)
// and drops `evicted`.
struct EvictPlan {
    int n_units = 0;          // whole units popped from the queue
    int32_t part_rows = 0;    // rows consumed from the next unit (rules that stop inside a unit)
    int32_t part_evictable = 0;
    int32_t span = 0, n_keep = 0, evicted = 0, u_last = -2, R_pre = 0;
    int32_t sink = -1;        // A2T_RULE_SINK_RECENT: the sink count (rows kept by index)
    bool unmet = false;
};

}  // namespace

struct a2t_cache {
    a2t_config cfg{};
    bool host_only = false;
    hipStream_t stream = nullptr;
    int poisoned = 0;
    DevState dev{};
    std::vector<StreamState> ss;
    // pinned staging slots for step metadata, reused round-robin behind events
    uint8_t* stage = nullptr;      // host address
    uint8_t* stage_dev = nullptr;  // the same memory as seen by kernels
    size_t slot_bytes = 0;
    int n_slots = 0;
    int next_slot = 0;
    std::vector<hipEvent_t> slot_ev;
    std::vector<uint8_t> slot_live;
    // per-call scratch, sized at creation (no allocation on the hot path)
    std::vector<uint32_t> seen;      // stream id -> call stamp
    uint32_t stamp = 0;
    std::vector<int32_t> tmp_nq, tmp_row0, tmp_in0, tmp_extra;
    std::vector<EvictPlan> evict_plans;
    bool own_pools = true;           // false: the K/V pools belong to the caller
    // the library's fixed split workspace on this cache's device (a2t_append_attn_noalloc)
    float* static_ws = nullptr;
    int64_t static_ws_floats = 0;
    // device-planned steps (a2t_dev_*): the plan the device writes, the call
    // sequence the host checks, a host copy of the device's per-stream state
    DevPlan* dplan = nullptr;
    bool dev_mode = false;
    bool dev_step_open = false;
    int dev_count = 0;
    int dev_max_splits = 1;
    int32_t dev_ids[kMaxDesc] = {};
    std::vector<uint8_t> dev_layers;
    std::vector<DevStream> dss_host;
    std::vector<int32_t> uid_host;
    std::vector<uint8_t> seg_host;
    // attention tuning
    int target_wgs = 1024;
    int force_splits = 0;
    // the last split plan (every layer of a step plans the same resident counts)
    int plan_n = 0;
    int plan_force = -1;
    int64_t plan_limit = -1;
    std::vector<int> plan_tiles, plan_splits, plan_tmp, plan_order;
    std::vector<int64_t> plan_heap;
    bool force_valu = false;
    // profiling
    bool prof_on = false;
    std::string prof_filter;
    std::deque<ProfEvent> prof_pending;
    std::vector<hipEvent_t> prof_free;
    std::map<std::string, std::pair<int64_t, double>> prof_acc;
};

namespace {

int hip_fail(a2t_cache* c) {
    if (c) c->poisoned = 1;
    return A2T_ERR_HIP;
}

struct DeviceGuard {
    int prev = -1;
    bool changed = false;
    explicit DeviceGuard(int dev) {
        if (hipGetDevice(&prev) == hipSuccess && prev != dev) {
            changed = hipSetDevice(dev) == hipSuccess;
        }
    }
    ~DeviceGuard() {
        if (changed) (void)hipSetDevice(prev);
    }
};

bool env_flag(const char* name) {
    const char* v = std::getenv(name);
    return v && *v && std::strcmp(v, "0") != 0;
}
int env_int(const char* name, int dflt) {
    const char* v = std::getenv(name);
    return (v && *v) ? std::atoi(v) : dflt;
}

// ---- profiling ---------------------------------------------------------------
void prof_harvest(a2t_cache* c, bool wait) {
    while (!c->prof_pending.empty()) {
        ProfEvent& e = c->prof_pending.front();
        if (wait) {
            if (hipEventSynchronize(e.stop) != hipSuccess) return;
        } else if (hipEventQuery(e.stop) != hipSuccess) {
            return;
        }
        float ms = 0.f;
        if (hipEventElapsedTime(&ms, e.start, e.stop) == hipSuccess) {
            auto& acc = c->prof_acc[e.name];
            acc.first += 1;
            acc.second += ms;
        }
        c->prof_free.push_back(e.start);
        c->prof_free.push_back(e.stop);
        c->prof_pending.pop_front();
    }
}

// Times the one kernel that a launcher issues inside the scope: the launcher
// takes kt() and records the events at the dispatch's own begin and end.
struct ProfScope {
    a2t_cache* c;
    ProfEvent ev;
    KTimer t;
    ProfScope(a2t_cache* cc, const char* name) : c(cc) {
        if (!c->prof_on) return;
        if (!c->prof_filter.empty() && std::strstr(name, c->prof_filter.c_str()) == nullptr) return;
        // recycle finished pairs only when the pool is empty (a2t_profile_reserve
        // fills it beforehand, so a timed launch costs the host no more than a
        // plain one)
        if (c->prof_free.size() < 2) prof_harvest(c, false);
        if (c->prof_free.size() < 2) {
            hipEvent_t a, b;
            if (hipEventCreate(&a) != hipSuccess || hipEventCreate(&b) != hipSuccess) return;
            c->prof_free.push_back(a);
            c->prof_free.push_back(b);
        }
        ev.name = name;
        ev.stop = c->prof_free.back();
        c->prof_free.pop_back();
        ev.start = c->prof_free.back();
        c->prof_free.pop_back();
        t.start = ev.start;
        t.stop = ev.stop;
    }
    const KTimer& kt() const { return t; }
    ~ProfScope() {
        if (t.start) c->prof_pending.push_back(ev);
    }
};

// ---- staging -------------------------------------------------------------------
uint8_t* stage_acquire(a2t_cache* c, int* slot_out) {
    const int s = c->next_slot;
    c->next_slot = (c->next_slot + 1) % c->n_slots;
    if (c->slot_live[s]) {
        if (hipEventSynchronize(c->slot_ev[s]) != hipSuccess) return nullptr;
        c->slot_live[s] = 0;
    }
    *slot_out = s;
    return c->stage + (size_t)s * c->slot_bytes;
}
bool stage_release(a2t_cache* c, int slot) {
    if (hipEventRecord(c->slot_ev[slot], c->stream) != hipSuccess) return false;
    c->slot_live[slot] = 1;
    return true;
}

int check_streams(a2t_cache* c, int32_t n, const int32_t* ids) {
    if (n < 1 || n > c->cfg.n_streams || !ids) return A2T_ERR_INVALID;
    if (++c->stamp == 0) {  // wrapped: clear the stamps
        std::fill(c->seen.begin(), c->seen.end(), 0u);
        c->stamp = 1;
    }
    for (int i = 0; i < n; ++i) {
        if (ids[i] < 0 || ids[i] >= c->cfg.n_streams || c->seen[ids[i]] == c->stamp)
            return A2T_ERR_INVALID;
        c->seen[ids[i]] = c->stamp;
    }
    return A2T_OK;
}

bool is_evictable(uint8_t seg) { return seg == A2T_SEG_ACOUSTIC || seg == A2T_SEG_DELIM; }

// Key splits per stream for one attention launch.  A workgroup of the MFMA
// kernel occupies a whole CU (its LDS ring) and the dispatcher hands the next
// workgroup to the first CU that frees up, so a launch takes about the makespan
// of its workgroups dispatched in order over `slots` (= CU count) CUs.  For each
// tile budget per workgroup (>= 2 tiles) every stream gets the fewest splits that
// respect it; a workgroup costs its tiles plus a fixed part (setup, first-load
// latency, partial write: ~5 us, measured, ~4 tiles).  Streams are dispatched longest workgroups first
// (attn_launch orders the descriptors that way), and the budget with the
// shortest simulated makespan wins (ties: fewer workgroups, i.e. fewer split
// partials).  The partials must fit the workspace.
constexpr int kWgFixedTiles = 4;

int64_t launch_makespan(int n, const int* tiles, const int* splits, int Hkv, int slots,
                        std::vector<int>& order, std::vector<int64_t>& heap) {
    int64_t wgs = 0, largest = 0;
    order.resize(n);
    for (int i = 0; i < n; ++i) {
        order[i] = i;
        wgs += (int64_t)splits[i] * Hkv;
        largest = std::max<int64_t>(largest, (tiles[i] + splits[i] - 1) / splits[i]);
    }
    if (wgs <= slots) return largest + kWgFixedTiles;
    auto cost = [&](int i) { return (int64_t)(tiles[i] + splits[i] - 1) / splits[i] + kWgFixedTiles; };
    std::stable_sort(order.begin(), order.end(), [&](int a, int b) { return cost(a) > cost(b); });
    // min-heap of CU finish times
    heap.assign(slots, 0);
    auto gt = std::greater<int64_t>();
    for (int i : order) {
        const int64_t ci = cost(i);
        for (int64_t k = 0; k < (int64_t)splits[i] * Hkv; ++k) {
            std::pop_heap(heap.begin(), heap.end(), gt);
            heap.back() += ci;
            std::push_heap(heap.begin(), heap.end(), gt);
        }
    }
    return *std::max_element(heap.begin(), heap.end());
}

void plan_splits(a2t_cache* c, int n, const int* tiles, const int64_t* floats_per_split,
                 int* splits, int64_t ws_limit) {
    // every layer of a step plans the same resident counts: reuse the last plan
    // while its partials fit the workspace (query counts may differ)
    if (c->plan_n == n && std::equal(tiles, tiles + n, c->plan_tiles.begin()) &&
        c->plan_force == c->force_splits && c->plan_limit == ws_limit) {
        int64_t ws = 0;
        for (int i = 0; i < n; ++i)
            ws += stream_partials(c->plan_splits[i], floats_per_split[i]);
        if (ws <= ws_limit) {
            std::copy(c->plan_splits.begin(), c->plan_splits.begin() + n, splits);
            return;
        }
    }
    const int Hkv = c->cfg.n_kv_heads;
    if (c->force_splits <= 0) {
        int max_tiles = 1;
        for (int i = 0; i < n; ++i) max_tiles = std::max(max_tiles, tiles[i]);
        int64_t best_cost = INT64_MAX, best_w = 0;
        int best_budget = max_tiles;
        std::vector<int>& sp = c->plan_tmp;
        sp.resize(n);
        for (int budget = 2; budget <= std::max(2, max_tiles); ++budget) {
            int64_t w = 0, ws = 0;
            for (int i = 0; i < n; ++i) {
                sp[i] = std::max(1, std::min((tiles[i] + budget - 1) / budget, kMaxSplits));
                w += (int64_t)sp[i] * Hkv;
                ws += stream_partials(sp[i], floats_per_split[i]);
            }
            if (ws > ws_limit) continue;
            const int64_t cost = launch_makespan(n, tiles, sp.data(), Hkv, c->target_wgs,
                                                 c->plan_order, c->plan_heap);
            if (cost < best_cost || (cost == best_cost && w < best_w)) {
                best_cost = cost;
                best_w = w;
                best_budget = budget;
            }
        }
        for (int i = 0; i < n; ++i)
            splits[i] = std::max(1, std::min((tiles[i] + best_budget - 1) / best_budget, kMaxSplits));
        if (best_cost == INT64_MAX) {
            // nothing fits the workspace: shrink below
        } else {
            c->plan_n = n;
            c->plan_force = c->force_splits;
            c->plan_limit = ws_limit;
            c->plan_tiles.assign(tiles, tiles + n);
            c->plan_splits.assign(splits, splits + n);
            return;
        }
    } else {
        for (int i = 0; i < n; ++i) splits[i] = std::max(1, std::min({c->force_splits, tiles[i], kMaxSplits}));
    }
    // shrink uniformly until the partials fit the workspace
    for (;;) {
        int64_t ws = 0;
        int mx = 1;
        for (int i = 0; i < n; ++i) {
            ws += stream_partials(splits[i], floats_per_split[i]);
            mx = std::max(mx, splits[i]);
        }
        if (ws <= ws_limit || mx == 1) break;
        for (int i = 0; i < n; ++i) splits[i] = std::max(1, splits[i] / 2);
    }
    c->plan_n = n;
    c->plan_force = c->force_splits;
    c->plan_limit = ws_limit;
    c->plan_tiles.assign(tiles, tiles + n);
    c->plan_splits.assign(splits, splits + n);
}

// Where a launch's split partials go: the cache's workspace (default) or the
// library's fixed device array (the no-allocation entry point, which plans
// without the workspace limit and never times its launches).
struct WsChoice {
    float* ws;
    int64_t floats;
};

// Floats of split partials one launch over these streams writes at the
// planner's choice (ws_limit as in plan_splits); `extra` rows are added to each
// stream's resident count (a step that is about to be appended).
int64_t planned_partials(a2t_cache* c, int n, const int32_t* ids, const int32_t* n_q,
                         const int32_t* extra, int64_t ws_limit) {
    const int G = c->cfg.n_q_heads / c->cfg.n_kv_heads;
    const int64_t rf = partial_row_floats(c->cfg.head_dim, c->cfg.dtype == A2T_F32 || c->force_valu);
    int tiles[kMaxDesc], nsplit[kMaxDesc];
    int64_t floats[kMaxDesc];
    for (int i = 0; i < n; ++i) {
        const int64_t R = c->ss[ids[i]].resident() + (extra ? extra[i] : 0);
        tiles[i] = (int)std::max<int64_t>(1, (R + kTileKeys - 1) / kTileKeys);
        floats[i] = (int64_t)c->cfg.n_kv_heads * G * n_q[i] * rf;
    }
    plan_splits(c, n, tiles, floats, nsplit, ws_limit);
    int64_t total = 0;
    for (int i = 0; i < n; ++i)
        total += stream_partials(nsplit[i], floats[i]);
    return total;
}

// the kernels move K, V, Q and O rows 16 bytes at a time
static bool unaligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) != 0; }

// One attention launch (plus merge) over up to kMaxDesc streams.
// With in_row0 non-null (bf16 MFMA path only) the launch also appends each
// stream's open-step rows of `layer` from k_in / v_in.
int attn_launch(a2t_cache* c, int layer, int n, const int32_t* ids, const int32_t* n_q,
                const int32_t* q_row0, const void* q, void* o, const int32_t* in_row0 = nullptr, const void* k_in = nullptr,
                const void* v_in = nullptr, const WsChoice* wsc = nullptr) {
    AttnBatch b{};
    b.count = n;
    b.layer = layer;
    const int G = c->cfg.n_q_heads / c->cfg.n_kv_heads;
    // bf16 caches use the MFMA kernel for decode too: with one query row per
    // stream it is still bound by streaming the resident K/V, and its staged
    // tile pipeline keeps more bytes in flight than the VALU kernel.
    const bool valu = c->cfg.dtype == A2T_F32 || c->force_valu;
    const int64_t rf = partial_row_floats(c->cfg.head_dim, valu);
    int max_rows = 0, tiles[kMaxDesc], nsplit[kMaxDesc];
    int64_t floats[kMaxDesc];
    for (int i = 0; i < n; ++i) {
        const StreamState& s = c->ss[ids[i]];
        tiles[i] = std::max(1, (s.resident() + kTileKeys - 1) / kTileKeys);
        max_rows = std::max(max_rows, n_q[i]);
        floats[i] = (int64_t)c->cfg.n_kv_heads * G * n_q[i] * rf;
    }
    plan_splits(c, n, tiles, floats, nsplit, wsc ? INT64_MAX : c->dev.ws_floats);
    // descriptors in order of falling tiles per split: the dispatcher starts the
    // longest workgroups first
    int ord[kMaxDesc];
    for (int i = 0; i < n; ++i) ord[i] = i;
    std::stable_sort(ord, ord + n, [&](int a, int b2) {
        return (tiles[a] + nsplit[a] - 1) / nsplit[a] > (tiles[b2] + nsplit[b2] - 1) / nsplit[b2];
    });
    int splits = 1;
    int64_t off = 0;
    for (int k = 0; k < n; ++k) {
        const int i = ord[k];
        const StreamState& s = c->ss[ids[i]];
        AttnDesc& d = b.d[k];
        d.s = ids[i];
        d.kept = s.kept;
        d.head = s.head;
        d.R = s.resident();
        d.n_q = n_q[i];
        d.q_row0 = q_row0[i];
        d.rope_row0 = s.step_rows - n_q[i];
        d.splits = nsplit[i];
        const int n_tiles = (d.R + kTileKeys - 1) / kTileKeys;
        d.tile_q = n_tiles / d.splits;
        d.tile_r = n_tiles % d.splits;
        splits = std::max(splits, nsplit[i]);
        d.n_new = in_row0 ? s.step_rows : 0;
        d.in_row0 = in_row0 ? in_row0[i] : 0;
        d.ws_off = off;
        off += stream_partials(d.splits, (int64_t)c->cfg.n_kv_heads * G * d.n_q * rf);
    }
    // a fused step's own rows: when the launch's workgroups (with one more split
    // per tile holding them) still fit one round over the CUs, those tiles get
    // one-tile splits of their own, so that the workgroup that also rotates and
    // stores the rows is not the last of the launch to finish
    if (in_row0 && !wsc) {
        const int Hkv = c->cfg.n_kv_heads;
        int64_t wgs = 0, ws = 0;
        int32_t tq[kMaxDesc], tr[kMaxDesc], ns[kMaxDesc];
        bool any = false;
        for (int k = 0; k < n; ++k) {
            const AttnDesc& d = b.d[k];
            const int n_tiles = (d.R + kTileKeys - 1) / kTileKeys;
            const int qmax = (n_tiles + d.splits - 1) / d.splits;
            const int t_old = (d.R - d.n_new) / kTileKeys, m = n_tiles - t_old;
            tq[k] = d.tile_q, tr[k] = d.tile_r, ns[k] = d.splits;
            if (d.splits > 1 && qmax >= 2 && d.n_new > 0 && t_old >= 1 && m >= 1) {
                const int s_old = (t_old + qmax - 1) / qmax;
                if (s_old + m <= kMaxSplits) {
                    ns[k] = s_old + m;
                    tq[k] = t_old / s_old;
                    tr[k] = (t_old % s_old) | (m << 16);
                    any = true;
                }
            }
            wgs += (int64_t)ns[k] * Hkv;
            ws += stream_partials(ns[k], (int64_t)Hkv * G * d.n_q * rf);
        }
        if (any && wgs <= c->target_wgs && ws <= c->dev.ws_floats) {
            int64_t o2 = 0;
            for (int k = 0; k < n; ++k) {
                AttnDesc& d = b.d[k];
                d.splits = ns[k], d.tile_q = tq[k], d.tile_r = tr[k];
                d.ws_off = o2;
                o2 += stream_partials(d.splits, (int64_t)Hkv * G * d.n_q * rf);
                splits = std::max(splits, (int)d.splits);
            }
            off = o2;
        }
    }
    b.max_splits = splits;
    b.max_rows = max_rows;
    hipError_t e;
    if (wsc) {
        // the caller checked the partials against the fixed array before any state changed
        if (off > wsc->floats) return A2T_ERR_CAPACITY;
        DevState st = c->dev;
        st.ws = wsc->ws;
        st.ws_floats = wsc->floats;
        const KTimer none{};
        e = valu ? launch_attn_valu(st, b, q, o, c->stream, none)
                 : launch_attn_tile(st, b, q, o, k_in, v_in, c->stream, none);
        if (e == hipSuccess && splits > 1) e = launch_attn_merge(st, b, o, c->stream, none, !valu);
        return e == hipSuccess ? A2T_OK : hip_fail(c);
    }
    {
        ProfScope ps(c, valu ? "attn_valu" : "attn_tile");
        e = valu ? launch_attn_valu(c->dev, b, q, o, c->stream, ps.kt())
                 : launch_attn_tile(c->dev, b, q, o, k_in, v_in, c->stream, ps.kt());
    }
    if (e != hipSuccess) return hip_fail(c);
    if (splits > 1) {
        ProfScope ps(c, "attn_merge");
        if (launch_attn_merge(c->dev, b, o, c->stream, ps.kt(), !valu) != hipSuccess) return hip_fail(c);
    }
    return A2T_OK;
}

int attn_common(a2t_cache* c, int32_t layer, int32_t n_streams, const int32_t* ids,
                const int32_t* n_q, const void* q, void* o, bool decode,
                const WsChoice* wsc = nullptr) {
    if (!c) return A2T_ERR_INVALID;
    if (c->poisoned) return A2T_ERR_HIP;
    if (c->dev_mode) return A2T_ERR_STATE;
    if (layer < 0 || layer >= c->cfg.n_layers) return A2T_ERR_INVALID;
    int rc = check_streams(c, n_streams, ids);
    if (rc) return rc;
    if (!q || !o || unaligned16(q) || unaligned16(o) || (!decode && !n_q)) return A2T_ERR_INVALID;
    std::vector<int32_t>& nq = c->tmp_nq;
    std::vector<int32_t>& row0 = c->tmp_row0;
    int32_t acc = 0;
    for (int i = 0; i < n_streams; ++i) {
        const StreamState& s = c->ss[ids[i]];
        nq[i] = decode ? 1 : n_q[i];
        if (nq[i] < 1) return A2T_ERR_INVALID;
        if (s.step_rows == 0 || !s.appended[layer]) return A2T_ERR_STATE;
        if (nq[i] > s.step_rows) return A2T_ERR_STATE;
        row0[i] = acc;
        acc += nq[i];
    }
    if (c->host_only) return A2T_ERR_NODEV;
    DeviceGuard dg(c->cfg.device);
    for (int i0 = 0; i0 < n_streams; i0 += kMaxDesc) {
        const int n = std::min(kMaxDesc, n_streams - i0);
        rc = attn_launch(c, layer, n, ids + i0, nq.data() + i0, row0.data() + i0, q, o, nullptr,
                         nullptr, nullptr, wsc);
        if (rc) return rc;
    }
    return A2T_OK;
}

void free_device(a2t_cache* c) {
    if (c->own_pools) {
        // a library-allocated pool is one allocation per tensor: ring, then kept regions
        if (c->dev.k_unit) (void)hipFree(c->dev.k_unit);
        if (c->dev.v_unit) (void)hipFree(c->dev.v_unit);
    }
    void* ptrs[] = {c->dev.unit_pos, c->dev.unit_uid, c->dev.unit_seg, c->dev.kept_pos,
                    c->dev.kept_uid, c->dev.kept_seg, c->dev.rope, c->dev.ev_mask,
                    c->dev.ev_slot, c->dev.ws, c->dev.dss, c->dplan};
    for (void* p : ptrs)
        if (p) (void)hipFree(p);
    if (c->stage) (void)hipHostFree(c->stage);
    for (hipEvent_t e : c->slot_ev) (void)hipEventDestroy(e);
    for (auto& e : c->prof_pending) {
        (void)hipEventDestroy(e.start);
        (void)hipEventDestroy(e.stop);
    }
    for (hipEvent_t e : c->prof_free) (void)hipEventDestroy(e);
}

}  // namespace

extern "C" {

int a2t_abi_version(void) { return A2T_ABI_VERSION; }

const char* a2t_status_str(int status) {
    switch (status) {
        case A2T_OK: return "ok";
        case A2T_ERR_INVALID: return "invalid argument";
        case A2T_ERR_POS: return "position/unit order or metadata mismatch";
        case A2T_ERR_CAPACITY: return "cache region capacity exceeded";
        case A2T_ERR_STATE: return "call out of order";
        case A2T_ERR_OOM: return "out of memory";
        case A2T_ERR_HIP: return "HIP error or device fault (cache poisoned)";
        case A2T_ERR_NODEV: return "no usable gfx950 device";
        default: return "unknown status";
    }
}

int a2t_cache_create(const a2t_config* cfg, void* hip_stream, a2t_cache** out) {
    if (!cfg || !out) return A2T_ERR_INVALID;
    *out = nullptr;
    const a2t_config& k = *cfg;
    if (k.n_layers < 1 || k.n_streams < 1 || k.n_kv_heads < 1 || k.n_q_heads < 1) return A2T_ERR_INVALID;
    if (k.n_q_heads % k.n_kv_heads) return A2T_ERR_INVALID;
    const int G = k.n_q_heads / k.n_kv_heads;
    if (G != 1 && G != 2 && G != 4 && G != 8) return A2T_ERR_INVALID;
    if (k.head_dim != 64 && k.head_dim != 128) return A2T_ERR_INVALID;
    if (k.dtype != A2T_F32 && k.dtype != A2T_BF16) return A2T_ERR_INVALID;
    if (k.unit_rows < 1 || k.kept_rows < 0) return A2T_ERR_INVALID;
    if (k.max_step_rows < 1 || k.max_step_rows > 1024) return A2T_ERR_INVALID;
    if (k.rope_theta < 0 || k.attn_scale < 0) return A2T_ERR_INVALID;
    if ((int64_t)k.unit_rows + k.kept_rows > (int64_t)1 << 30) return A2T_ERR_INVALID;
    if ((k.k_pool == nullptr) != (k.v_pool == nullptr)) return A2T_ERR_INVALID;
    if ((reinterpret_cast<uintptr_t>(k.k_pool) | reinterpret_cast<uintptr_t>(k.v_pool)) & 255u)
        return A2T_ERR_INVALID;

    a2t_cache* c = new (std::nothrow) a2t_cache();
    if (!c) return A2T_ERR_OOM;
    c->cfg = k;
    if (c->cfg.rope_theta == 0) c->cfg.rope_theta = 1.0e6;
    if (c->cfg.attn_scale == 0) c->cfg.attn_scale = 1.0 / std::sqrt((double)k.head_dim);
    c->host_only = (k.flags & A2T_FLAG_HOST_ONLY) != 0;
    c->stream = static_cast<hipStream_t>(hip_stream);
    c->ss.resize(k.n_streams);
    for (auto& s : c->ss) {
        s.appended.assign(k.n_layers, 1);
        s.units.init((size_t)k.unit_rows);
        s.ring_seg.assign((size_t)k.unit_rows, 0);
        s.step_seg.reserve((size_t)k.max_step_rows);
        s.step_pos.reserve((size_t)k.max_step_rows);
    }
    c->seen.assign(k.n_streams, 0u);
    c->tmp_nq.assign(k.n_streams, 0);
    c->tmp_row0.assign(k.n_streams, 0);
    c->tmp_in0.assign(k.n_streams, 0);
    c->tmp_extra.assign(k.n_streams, 0);
    c->evict_plans.assign(k.n_streams, EvictPlan{});
    {
        // one workgroup of the attention kernel per CU: a launch runs in rounds of CU count
        int cus = 0;
        if (c->host_only ||
            hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, k.device) != hipSuccess || cus <= 0)
            cus = 256;
        c->target_wgs = std::max(1, env_int("A2T_TARGET_WGS", cus));
    }
    c->force_splits = std::max(0, env_int("A2T_SPLITS", 0));
    c->force_valu = env_flag("A2T_FORCE_VALU");
    // the split planner's scratch, so that no attention call allocates
    for (auto* v : {&c->plan_tiles, &c->plan_splits, &c->plan_tmp, &c->plan_order}) v->reserve(kMaxDesc);
    c->plan_heap.reserve((size_t)c->target_wgs);

    DevState& d = c->dev;
    d.L = k.n_layers;
    d.S = k.n_streams;
    d.Hq = k.n_q_heads;
    d.Hkv = k.n_kv_heads;
    d.G = k.n_q_heads / k.n_kv_heads;
    d.D = k.head_dim;
    d.dtype = k.dtype;
    d.unit_rows = k.unit_rows;
    d.kept_rows = k.kept_rows;
    d.max_step_rows = k.max_step_rows;
    d.theta = c->cfg.rope_theta;
    d.scale_log2e = (float)(c->cfg.attn_scale * 1.4426950408889634);
    if (c->host_only) {
        *out = c;
        return A2T_OK;
    }

    int ndev = 0;
    if (hipGetDeviceCount(&ndev) != hipSuccess || k.device < 0 || k.device >= ndev) {
        delete c;
        return A2T_ERR_NODEV;
    }
    hipDeviceProp_t prop;
    if (hipGetDeviceProperties(&prop, k.device) != hipSuccess ||
        std::strncmp(prop.gcnArchName, "gfx950", 6) != 0) {
        delete c;
        return A2T_ERR_NODEV;
    }
    DeviceGuard dg(k.device);
    const int64_t elt = k.dtype == A2T_F32 ? 4 : 2;
    const int64_t lsh = (int64_t)k.n_layers * k.n_streams * k.n_kv_heads * k.head_dim * elt;
    const int64_t S = k.n_streams;
    const int64_t tot = (int64_t)k.unit_rows + k.kept_rows;
    // workspace for key-split partials (none with A2T_FLAG_NO_WORKSPACE: such a
    // cache splits only through a2t_append_attn_noalloc and the library's fixed array)
    const bool no_ws = (k.flags & A2T_FLAG_NO_WORKSPACE) != 0;
    int64_t ws = no_ws ? 0 : (int64_t)env_int("A2T_WS_MB", 256) << 20;
    bool ok = true;
    auto alloc = [&](void** p, int64_t bytes) {
        if (!ok) return;
        if (hipMalloc(p, std::max<int64_t>(bytes, 256)) != hipSuccess) ok = false;
    };
    // K and V pools: [L][S][Hkv][unit_rows][D] ring, then [L][S][Hkv][kept_rows][D] kept
    c->own_pools = (k.k_pool == nullptr);
    if (c->own_pools) {
        alloc(&d.k_unit, lsh * tot);
        alloc(&d.v_unit, lsh * tot);
    } else {
        d.k_unit = k.k_pool;
        d.v_unit = k.v_pool;
    }
    if (ok) {
        d.k_kept = static_cast<char*>(d.k_unit) + lsh * k.unit_rows;
        d.v_kept = static_cast<char*>(d.v_unit) + lsh * k.unit_rows;
    }
    alloc((void**)&d.unit_pos, S * k.unit_rows * 4);
    alloc((void**)&d.unit_uid, S * k.unit_rows * 4);
    alloc((void**)&d.unit_seg, S * k.unit_rows);
    alloc((void**)&d.kept_pos, S * std::max(1, k.kept_rows) * 4);
    alloc((void**)&d.kept_uid, S * std::max(1, k.kept_rows) * 4);
    alloc((void**)&d.kept_seg, S * std::max(1, k.kept_rows));
    alloc((void**)&d.rope, S * k.max_step_rows * (k.head_dim / 2) * 8);
    alloc((void**)&d.ev_mask, S * tot);
    alloc((void**)&d.ev_slot, S * tot * 4);
    if (!no_ws) alloc((void**)&d.ws, ws);
    d.ws_floats = ws / 4;
    alloc((void**)&d.dss, S * (int64_t)sizeof(DevStream));
    alloc((void**)&c->dplan, (int64_t)sizeof(DevPlan));
    if (ok && static_scratch(k.device, &c->static_ws, &c->static_ws_floats) != hipSuccess) {
        c->static_ws = nullptr;   // the no-allocation entry point reports NODEV
        c->static_ws_floats = 0;
        (void)hipGetLastError();
    }
    // staging: per slot, seg (u8) + pos (i32) for every stream's max step, + unit ids
    c->n_slots = 16;
    c->slot_bytes = (size_t)S * k.max_step_rows * 5 + (size_t)kMaxDesc * 4 * ((S + kMaxDesc - 1) / kMaxDesc) + 256;
    c->slot_bytes = (c->slot_bytes + 255) & ~(size_t)255;
    if (ok && hipHostMalloc((void**)&c->stage, c->slot_bytes * c->n_slots,
                            hipHostMallocMapped | hipHostMallocCoherent) != hipSuccess) {
        c->stage = nullptr;
        ok = false;
    }
    if (ok && hipHostGetDevicePointer((void**)&c->stage_dev, c->stage, 0) != hipSuccess) ok = false;
    c->slot_ev.resize(c->n_slots, nullptr);
    c->slot_live.assign(c->n_slots, 0);
    for (int i = 0; ok && i < c->n_slots; ++i)
        if (hipEventCreateWithFlags(&c->slot_ev[i], hipEventDisableTiming) != hipSuccess) ok = false;
    if (!ok) {
        free_device(c);
        delete c;
        (void)hipGetLastError();
        return A2T_ERR_OOM;
    }
    *out = c;
    return A2T_OK;
}

int a2t_cache_destroy(a2t_cache* c) {
    if (!c) return A2T_OK;
    if (!c->host_only) {
        DeviceGuard dg(c->cfg.device);
        (void)hipStreamSynchronize(c->stream);
        free_device(c);
    }
    delete c;
    return A2T_OK;
}

int a2t_set_stream(a2t_cache* c, void* hip_stream) {
    if (!c) return A2T_ERR_INVALID;
    c->stream = static_cast<hipStream_t>(hip_stream);
    return A2T_OK;
}

// a2t_append; with launch_rows false the rows' K/V are left for a fused
// attention launch to store (metadata and the rotary table are still written).
static int append_impl(a2t_cache* c, int32_t layer, int32_t n_streams, const int32_t* ids,
                       const int32_t* n_rows, const void* kin, const void* vin,
                       const uint8_t* seg, const int32_t* pos, const int32_t* unit_id,
                       bool launch_rows) {
    if (!c) return A2T_ERR_INVALID;
    if (c->poisoned) return A2T_ERR_HIP;
    if (c->dev_mode) return A2T_ERR_STATE;
    const a2t_config& k = c->cfg;
    if (layer < A2T_ALL_LAYERS || layer >= k.n_layers) return A2T_ERR_INVALID;
    int rc = check_streams(c, n_streams, ids);
    if (rc) return rc;
    if (!n_rows) return A2T_ERR_INVALID;
    if (!c->host_only && (!kin || !vin || unaligned16(kin) || unaligned16(vin))) return A2T_ERR_INVALID;
    const bool opens = (layer == 0 || layer == A2T_ALL_LAYERS);
    if (opens && (!seg || !pos || !unit_id)) return A2T_ERR_INVALID;

    int64_t total = 0;
    for (int i = 0; i < n_streams; ++i) {
        if (n_rows[i] < 1 || n_rows[i] > k.max_step_rows) return A2T_ERR_INVALID;
        total += n_rows[i];
    }
    // validate every stream before touching any state
    int64_t off = 0;
    for (int i = 0; i < n_streams; ++i) {
        const StreamState& s = c->ss[ids[i]];
        const int n = n_rows[i];
        if (opens) {
            if (!s.step_complete()) return A2T_ERR_STATE;
            const int u = unit_id[i];
            if (u < -1) return A2T_ERR_INVALID;
            int64_t last = s.last_pos;
            for (int r = 0; r < n; ++r) {
                const uint8_t sg = seg[off + r];
                if (sg > A2T_SEG_RESPONSE) return A2T_ERR_INVALID;
                if (pos[off + r] < 0) return A2T_ERR_INVALID;
                if ((u == -1) != (sg == A2T_SEG_PREFIX)) return A2T_ERR_INVALID;
                if ((int64_t)pos[off + r] <= last) return A2T_ERR_POS;
                last = pos[off + r];
            }
            if (u == -1 && s.cur_unit >= 0) return A2T_ERR_POS;
            if (s.cur_unit != -2 && u < s.cur_unit) return A2T_ERR_POS;
            if ((int64_t)s.ring + n > k.unit_rows) return A2T_ERR_CAPACITY;
            // a new unit needs a queue entry (never short: every entry holds a ring row)
            if (!(s.units.size() && s.units.back().unit == u) && s.units.full()) return A2T_ERR_CAPACITY;
        } else {
            if (s.step_rows == 0 || s.appended[layer]) return A2T_ERR_STATE;
            if (n != s.step_rows) return A2T_ERR_POS;
            if (seg || pos) {
                for (int r = 0; r < n; ++r) {
                    if (seg && seg[off + r] != s.step_seg[r]) return A2T_ERR_POS;
                    if (pos && pos[off + r] != s.step_pos[r]) return A2T_ERR_POS;
                }
            }
            if (unit_id && unit_id[i] != s.step_unit) return A2T_ERR_POS;
        }
        off += n;
    }

    // state update
    off = 0;
    for (int i = 0; i < n_streams; ++i) {
        StreamState& s = c->ss[ids[i]];
        const int n = n_rows[i];
        if (opens) {
            const int u = unit_id[i];
            int ev = 0;
            for (int r = 0; r < n; ++r) ev += is_evictable(seg[off + r]);
            s.step_rows = n;
            s.step_slot0 = (s.head + s.ring) % k.unit_rows;
            for (int r = 0; r < n; ++r) s.ring_seg[(s.step_slot0 + r) % k.unit_rows] = seg[off + r];
            s.step_seg.assign(seg + off, seg + off + n);
            s.step_pos.assign(pos + off, pos + off + n);
            s.step_unit = u;
            std::fill(s.appended.begin(), s.appended.end(), layer == A2T_ALL_LAYERS ? 1 : 0);
            if (layer == 0) s.appended[0] = 1;
            s.ring += n;
            if (s.units.size() && s.units.back().unit == u) {
                s.units.back().rows += n;
                s.units.back().evictable += ev;
            } else {
                s.units.push_back(UnitRec{u, n, ev});
            }
            s.cur_unit = std::max(s.cur_unit, u);
            s.last_pos = pos[off + n - 1];
            s.peak = std::max(s.peak, s.resident());
            s.budget_unmet = 0;
        } else {
            s.appended[layer] = 1;
        }
        off += n;
    }
    if (c->host_only) return A2T_OK;

    DeviceGuard dg(k.device);
    // 1. step registration: metadata + rotary table (once per step)
    if (opens) {
        int64_t row = 0;
        for (int i0 = 0; i0 < n_streams; i0 += kMaxDesc) {
            const int n = std::min(kMaxDesc, n_streams - i0);
            int slot;
            uint8_t* sp = stage_acquire(c, &slot);
            if (!sp) return hip_fail(c);
            StepBatch sb{};
            sb.count = n;
            int64_t rows_here = 0;
            for (int i = 0; i < n; ++i) rows_here += n_rows[i0 + i];
            int32_t* spos = reinterpret_cast<int32_t*>(sp);
            int32_t* suid = spos + rows_here;
            uint8_t* sseg = reinterpret_cast<uint8_t*>(suid + n);
            std::memcpy(spos, pos + row, rows_here * 4);
            std::memcpy(sseg, seg + row, rows_here);
            int64_t r0 = 0;
            sb.max_n = 0;
            for (int i = 0; i < n; ++i) {
                const StreamState& s = c->ss[ids[i0 + i]];
                sb.max_n = std::max(sb.max_n, n_rows[i0 + i]);
                sb.d[i] = StepDesc{ids[i0 + i], n_rows[i0 + i], s.step_slot0, (int32_t)r0};
                suid[i] = unit_id[i0 + i];
                r0 += n_rows[i0 + i];
            }
            const ptrdiff_t shift = c->stage_dev - c->stage;
            hipError_t e;
            {
                ProfScope ps(c, "step_meta");
                e = launch_step_meta(c->dev, sb, reinterpret_cast<const uint8_t*>(sseg) + shift,
                                     reinterpret_cast<const int32_t*>(reinterpret_cast<uint8_t*>(spos) + shift),
                                     reinterpret_cast<const int32_t*>(reinterpret_cast<uint8_t*>(suid) + shift),
                                     c->stream, ps.kt());
            }
            if (e != hipSuccess || !stage_release(c, slot)) return hip_fail(c);
            row += rows_here;
        }
    }
    // 2. rotate and store K, store V
    if (launch_rows) {
        int64_t in_row = 0;
        for (int i0 = 0; i0 < n_streams; i0 += kMaxDesc) {
            const int n = std::min(kMaxDesc, n_streams - i0);
            AppendBatch ab{};
            ab.count = n;
            ab.layer0 = layer == A2T_ALL_LAYERS ? 0 : layer;
            ab.total_rows = (int32_t)total;
            int max_n = 0;
            for (int i = 0; i < n; ++i) {
                const StreamState& s = c->ss[ids[i0 + i]];
                ab.d[i] = AppendDesc{ids[i0 + i], n_rows[i0 + i], s.step_slot0, (int32_t)in_row};
                in_row += n_rows[i0 + i];
                max_n = std::max(max_n, n_rows[i0 + i]);
            }
            ab.max_n = max_n;
            hipError_t e;
            {
                ProfScope ps(c, "append");
                e = launch_append(c->dev, ab, layer == A2T_ALL_LAYERS ? k.n_layers : 1, kin, vin,
                                  c->stream, ps.kt());
            }
            if (e != hipSuccess) return hip_fail(c);
        }
    }
    return A2T_OK;
}

int a2t_append(a2t_cache* c, int32_t layer, int32_t n_streams, const int32_t* ids,
               const int32_t* n_rows, const void* kin, const void* vin, const uint8_t* seg,
               const int32_t* pos, const int32_t* unit_id) {
    return append_impl(c, layer, n_streams, ids, n_rows, kin, vin, seg, pos, unit_id, true);
}

int a2t_chunk_attn(a2t_cache* c, int32_t layer, int32_t n_streams, const int32_t* ids,
                   const int32_t* n_q, const void* q, void* o) {
    return attn_common(c, layer, n_streams, ids, n_q, q, o, false);
}

}  // extern "C"

namespace {

int append_attn_impl(a2t_cache* c, int32_t layer, int32_t n_streams, const int32_t* ids,
                     const int32_t* n_rows, const void* kin, const void* vin, const uint8_t* seg,
                     const int32_t* pos, const int32_t* unit_id, const int32_t* n_q, const void* q,
                     void* o, const WsChoice* wsc) {
    const bool fused = c->cfg.dtype == A2T_BF16 && !c->force_valu;
    int rc = append_impl(c, layer, n_streams, ids, n_rows, kin, vin, seg, pos, unit_id, !fused);
    if (rc) return rc;
    if (!fused) return attn_common(c, layer, n_streams, ids, n_q, q, o, false, wsc);
    DeviceGuard dg(c->cfg.device);
    std::vector<int32_t>& row0 = c->tmp_row0;
    std::vector<int32_t>& in0 = c->tmp_in0;
    int32_t acc = 0, acc_in = 0;
    for (int i = 0; i < n_streams; ++i) {
        row0[i] = acc;
        in0[i] = acc_in;
        acc += n_q[i];
        acc_in += n_rows[i];
    }
    for (int i0 = 0; i0 < n_streams; i0 += kMaxDesc) {
        const int n = std::min(kMaxDesc, n_streams - i0);
        rc = attn_launch(c, layer, n, ids + i0, n_q + i0, row0.data() + i0, q, o, in0.data() + i0,
                         kin, vin, wsc);
        if (rc) return rc;
    }
    return A2T_OK;
}

int append_attn_args(a2t_cache* c, int32_t layer, int32_t n_streams, const int32_t* n_rows,
                     const int32_t* n_q, const void* q, const void* o) {
    if (!c) return A2T_ERR_INVALID;
    if (c->poisoned) return A2T_ERR_HIP;
    if (c->dev_mode) return A2T_ERR_STATE;
    if (layer < 0 || layer >= c->cfg.n_layers) return A2T_ERR_INVALID;
    if (!n_rows || !n_q || !q || !o || unaligned16(q) || unaligned16(o) || n_streams < 1 ||
        n_streams > c->cfg.n_streams)
        return A2T_ERR_INVALID;
    for (int i = 0; i < n_streams; ++i)
        if (n_q[i] < 1 || n_q[i] > n_rows[i]) return A2T_ERR_INVALID;
    if (c->host_only) return A2T_ERR_NODEV;
    return A2T_OK;
}

}  // namespace

extern "C" {

int a2t_append_attn(a2t_cache* c, int32_t layer, int32_t n_streams, const int32_t* ids,
                    const int32_t* n_rows, const void* kin, const void* vin, const uint8_t* seg,
                    const int32_t* pos, const int32_t* unit_id, const int32_t* n_q,
                    const void* q, void* o) {
    int rc = append_attn_args(c, layer, n_streams, n_rows, n_q, q, o);
    if (rc) return rc;
    return append_attn_impl(c, layer, n_streams, ids, n_rows, kin, vin, seg, pos, unit_id, n_q, q,
                            o, nullptr);
}

int a2t_append_attn_noalloc(a2t_cache* c, int32_t layer, int32_t n_streams, const int32_t* ids,
                            const int32_t* n_rows, const void* kin, const void* vin,
                            const uint8_t* seg, const int32_t* pos, const int32_t* unit_id,
                            const int32_t* n_q, const void* q, void* o) {
    int rc = append_attn_args(c, layer, n_streams, n_rows, n_q, q, o);
    if (rc) return rc;
    if (!c->static_ws) return A2T_ERR_NODEV;
    if ((rc = check_streams(c, n_streams, ids))) return rc;
    // every launch's split partials must fit the fixed array: checked before the
    // append changes any state (layer 0 opens the step: its rows join R)
    std::vector<int32_t>& extra = c->tmp_extra;
    for (int i = 0; i < n_streams; ++i) extra[i] = layer == 0 ? n_rows[i] : 0;
    for (int i0 = 0; i0 < n_streams; i0 += kMaxDesc) {
        const int n = std::min(kMaxDesc, n_streams - i0);
        if (planned_partials(c, n, ids + i0, n_q + i0, extra.data() + i0, INT64_MAX) >
            c->static_ws_floats)
            return A2T_ERR_CAPACITY;
    }
    const WsChoice wsc{c->static_ws, c->static_ws_floats};
    return append_attn_impl(c, layer, n_streams, ids, n_rows, kin, vin, seg, pos, unit_id, n_q, q,
                            o, &wsc);
}

int a2t_decode_attn(a2t_cache* c, int32_t layer, int32_t n_streams, const int32_t* ids,
                    const void* q, void* o) {
    return attn_common(c, layer, n_streams, ids, nullptr, q, o, true);
}

}  // extern "C"

namespace {

// Number of ACOUSTIC/DELIM rows among `n` ring rows starting at `slot`.
int32_t evictable_in(const StreamState& s, int32_t slot, int32_t n, int32_t ring_rows) {
    int32_t e = 0;
    for (int32_t r = 0; r < n; ++r) {
        int32_t x = slot + r;
        if (x >= ring_rows) x -= ring_rows;
        e += is_evictable(s.ring_seg[x]);
    }
    return e;
}

// Sec. 3.3 and its variants, planned from the host mirror of one stream.
// A2T_RULE_UNIT: while R > B, the oldest unit outside the W most recent units
// that still holds acoustic/structural rows loses all of them.  A2T_RULE_ROW:
// the same rows one at a time, so the last unit touched may lose only part of
// them.  A2T_RULE_SINK_RECENT: everything but the n_sink oldest and the
// B - n_sink newest rows.
int plan_stream(const a2t_cache* c, const StreamState& s, int rule, int32_t budget,
                int32_t window, int32_t n_sink, EvictPlan& p) {
    p = EvictPlan{};
    const int32_t ring_rows = c->cfg.unit_rows;
    int32_t R = s.resident();
    p.R_pre = R;
    if (rule == A2T_RULE_SINK_RECENT) {
        if (R > budget) {
            if (s.kept > n_sink) return A2T_ERR_STATE;   // the kept region holds non-sink rows
            const int32_t sinks_left = n_sink - s.kept;  // the oldest ring rows are still sinks
            p.sink = n_sink;
            p.evicted = R - budget;
            p.n_keep = sinks_left;
            p.span = sinks_left + p.evicted;             // <= ring, since budget >= n_sink
            int32_t rest = p.span;
            size_t t = 0;
            while (t < s.units.size() && rest >= s.units[t].rows) {
                rest -= s.units[t].rows;
                p.u_last = s.units[t].unit;
                ++t;
            }
            p.n_units = (int)t;
            if (rest > 0) {
                p.part_rows = rest;
                p.part_evictable = evictable_in(s, (s.head + p.span - rest) % ring_rows, rest, ring_rows);
                p.u_last = s.units[t].unit;
            }
            R = budget;
        }
        p.unmet = R > budget;
        return A2T_OK;
    }
    const int64_t limit = (int64_t)s.cur_unit - window;
    if (rule == A2T_RULE_ROW) {
        // walk the ring from its head: every eligible ACOUSTIC/DELIM row goes, oldest
        // first, until R <= B; units whose remaining rows hold none are skipped whole
        const int32_t need = R - budget;
        int32_t x = 0;            // ring offset of the next row
        for (size_t t = 0; p.evicted < need && t < s.units.size(); ++t) {
            const UnitRec& u = s.units[t];
            if ((int64_t)u.unit > limit) break;
            if (u.evictable == 0) {
                x += u.rows;
                continue;
            }
            int32_t ev = 0;
            for (int32_t r = 0; r < u.rows && ev < u.evictable && p.evicted < need; ++r) {
                if (is_evictable(s.ring_seg[(s.head + x + r) % ring_rows])) {
                    ++ev;
                    ++p.evicted;
                    p.span = x + r + 1;     // the pass ends at the newest evicted row
                    p.u_last = u.unit;
                }
            }
            x += u.rows;
        }
        // units wholly inside the pass leave the queue; the next one loses its first rows
        int32_t rest = p.span;
        size_t t = 0;
        while (t < s.units.size() && rest > 0 && rest >= s.units[t].rows) rest -= s.units[t++].rows;
        p.n_units = (int)t;
        if (rest > 0) {
            p.part_rows = rest;
            p.part_evictable = evictable_in(s, (s.head + p.span - rest) % ring_rows, rest, ring_rows);
        }
        p.n_keep = p.span - p.evicted;
        R -= p.evicted;
        p.unmet = R > budget;
        return A2T_OK;
    }
    size_t next = 0;
    while (R > budget) {
        size_t j = next;
        while (j < s.units.size() && s.units[j].evictable == 0) ++j;
        if (j >= s.units.size() || (int64_t)s.units[j].unit > limit) break;
        for (size_t t = next; t <= j; ++t) {
            p.span += s.units[t].rows;
            p.n_keep += s.units[t].rows - s.units[t].evictable;
        }
        p.evicted += s.units[j].evictable;
        R -= s.units[j].evictable;
        p.u_last = s.units[j].unit;
        next = j + 1;
    }
    p.n_units = (int)next;
    p.unmet = R > budget;
    return A2T_OK;
}

int evict_impl(a2t_cache* c, int32_t n_streams, const int32_t* ids, const int32_t* budget,
               int32_t window, int32_t rule, int32_t n_sink, int32_t* n_evicted,
               uint8_t* budget_unmet) {
    if (!c) return A2T_ERR_INVALID;
    if (c->poisoned) return A2T_ERR_HIP;
    if (c->dev_mode) return A2T_ERR_STATE;
    int rc = check_streams(c, n_streams, ids);
    if (rc) return rc;
    if (!budget || window < 0) return A2T_ERR_INVALID;
    if (rule != A2T_RULE_UNIT && rule != A2T_RULE_ROW && rule != A2T_RULE_SINK_RECENT)
        return A2T_ERR_INVALID;
    if (n_sink < 0) return A2T_ERR_INVALID;
    EvictPlan* plans = c->evict_plans.data();   // sized n_streams at creation
    for (int i = 0; i < n_streams; ++i) {
        if (budget[i] < 0) return A2T_ERR_INVALID;
        if (rule == A2T_RULE_SINK_RECENT && budget[i] < n_sink) return A2T_ERR_INVALID;
        const StreamState& s = c->ss[ids[i]];
        if (!s.step_complete()) return A2T_ERR_STATE;
        rc = plan_stream(c, s, rule, budget[i], window, n_sink, plans[i]);
        if (rc) return rc;
        if ((int64_t)s.kept + plans[i].n_keep > c->cfg.kept_rows) return A2T_ERR_CAPACITY;
    }
    // device work for the streams that evict
    if (!c->host_only) {
        DeviceGuard dg(c->cfg.device);
        EvictBatch eb{};
        auto flush = [&]() -> int {
            if (eb.count == 0) return A2T_OK;
            hipError_t e;
            {
                ProfScope ps(c, "evict");
                e = launch_evict(c->dev, eb, c->stream, ps.kt());
            }
            eb.count = 0;
            return e == hipSuccess ? A2T_OK : hip_fail(c);
        };
        for (int i = 0; i < n_streams; ++i) {
            const EvictPlan& p = plans[i];
            if (p.evicted == 0) continue;
            const StreamState& s = c->ss[ids[i]];
            eb.d[eb.count++] = EvictDesc{ids[i], s.kept, s.head, p.R_pre, p.span, p.u_last, p.n_keep, p.sink};
            if (eb.count == kMaxDesc && (rc = flush())) return rc;
        }
        if ((rc = flush())) return rc;
    }
    // host state
    for (int i = 0; i < n_streams; ++i) {
        StreamState& s = c->ss[ids[i]];
        const EvictPlan& p = plans[i];
        if (p.evicted > 0) {
            s.units.pop_front((size_t)p.n_units);
            if (p.part_rows) {
                s.units[0].rows -= p.part_rows;
                s.units[0].evictable -= p.part_evictable;
            }
            s.kept += p.n_keep;
            s.head = (int32_t)(((int64_t)s.head + p.span) % c->cfg.unit_rows);
            s.ring -= p.span;
            s.last_evicted = p.u_last;
            s.evicted_total += p.evicted;
            s.moved_total += p.n_keep;
            s.last_evict_pre = p.R_pre;
        }
        s.budget_unmet = p.unmet ? 1 : 0;
        s.step_rows = 0;
        std::fill(s.appended.begin(), s.appended.end(), 1);
        if (n_evicted) n_evicted[i] = p.evicted;
        if (budget_unmet) budget_unmet[i] = p.unmet ? 1 : 0;
    }
    return A2T_OK;
}

}  // namespace

extern "C" {

int a2t_evict(a2t_cache* c, int32_t n_streams, const int32_t* ids, const int32_t* budget,
              int32_t window, int32_t* n_evicted, uint8_t* budget_unmet) {
    return evict_impl(c, n_streams, ids, budget, window, A2T_RULE_UNIT, 0, n_evicted, budget_unmet);
}

int a2t_evict_rule(a2t_cache* c, int32_t n_streams, const int32_t* ids, const int32_t* budget,
                   int32_t window, int32_t rule, int32_t n_sink, int32_t* n_evicted,
                   uint8_t* budget_unmet) {
    return evict_impl(c, n_streams, ids, budget, window, rule, n_sink, n_evicted, budget_unmet);
}

int a2t_stream_info_get(const a2t_cache* c, int32_t stream, a2t_stream_info* out) {
    if (!c || !out || stream < 0 || stream >= c->cfg.n_streams) return A2T_ERR_INVALID;
    if (c->dev_mode) return A2T_ERR_STATE;   // the device holds the state (a2t_dev_end)
    const StreamState& s = c->ss[stream];
    out->resident = s.resident();
    out->peak = s.peak;
    out->kept = s.kept;
    out->ring = s.ring;
    out->ring_head = s.head;
    out->cur_unit = s.cur_unit;
    out->last_evicted_unit = s.last_evicted;
    out->step_rows = s.step_rows;
    out->last_pos = s.last_pos;
    out->evicted_total = s.evicted_total;
    out->moved_total = s.moved_total;
    out->budget_unmet = s.budget_unmet;
    out->last_evict_pre = s.last_evict_pre;
    return A2T_OK;
}

int a2t_resident(const a2t_cache* c, int32_t stream, int32_t* n, int32_t* peak) {
    if (!c || stream < 0 || stream >= c->cfg.n_streams) return A2T_ERR_INVALID;
    if (c->dev_mode) return A2T_ERR_STATE;   // the device holds the state (a2t_dev_end)
    const StreamState& s = c->ss[stream];
    if (n) *n = s.resident();
    if (peak) *peak = s.peak;
    return A2T_OK;
}

int a2t_sync(a2t_cache* c) {
    if (!c) return A2T_ERR_INVALID;
    if (c->host_only) return A2T_OK;
    if (c->poisoned) return A2T_ERR_HIP;
    DeviceGuard dg(c->cfg.device);
    if (hipStreamSynchronize(c->stream) != hipSuccess) return hip_fail(c);
    if (hipGetLastError() != hipSuccess) return hip_fail(c);
    return A2T_OK;
}

int a2t_read_layout(a2t_cache* c, int32_t stream, int32_t* pos, uint8_t* seg, int32_t* unit) {
    if (!c || stream < 0 || stream >= c->cfg.n_streams) return A2T_ERR_INVALID;
    if (c->host_only) return A2T_ERR_NODEV;
    if (c->dev_mode) return A2T_ERR_STATE;
    int rc = a2t_sync(c);
    if (rc) return rc;
    DeviceGuard dg(c->cfg.device);
    const StreamState& s = c->ss[stream];
    const int64_t kb = (int64_t)stream * c->cfg.kept_rows, ub = (int64_t)stream * c->cfg.unit_rows;
    const int T = s.kept, U = s.ring, head = s.head, cap = c->cfg.unit_rows;
    const int first = std::min(U, cap - head), second = U - first;
    auto get = [&](void* dst, const void* src_kept, const void* src_ring, size_t elt) -> bool {
        if (!dst) return true;
        char* d = static_cast<char*>(dst);
        const char* sk = static_cast<const char*>(src_kept) + kb * elt;
        const char* sr = static_cast<const char*>(src_ring) + ub * elt;
        if (T && hipMemcpy(d, sk, T * elt, hipMemcpyDeviceToHost) != hipSuccess) return false;
        if (first && hipMemcpy(d + T * elt, sr + head * elt, first * elt, hipMemcpyDeviceToHost) != hipSuccess) return false;
        if (second && hipMemcpy(d + (T + first) * elt, sr, second * elt, hipMemcpyDeviceToHost) != hipSuccess) return false;
        return true;
    };
    if (!get(pos, c->dev.kept_pos, c->dev.unit_pos, 4) || !get(seg, c->dev.kept_seg, c->dev.unit_seg, 1) ||
        !get(unit, c->dev.kept_uid, c->dev.unit_uid, 4))
        return hip_fail(c);
    return A2T_OK;
}

int a2t_read_last_evict(a2t_cache* c, int32_t stream, int32_t* n_pre, uint8_t* mask,
                        int32_t* new_slot) {
    if (!c || stream < 0 || stream >= c->cfg.n_streams) return A2T_ERR_INVALID;
    if (c->host_only) return A2T_ERR_NODEV;
    if (c->dev_mode) return A2T_ERR_STATE;
    const StreamState& s = c->ss[stream];
    if (s.last_evict_pre < 0) return A2T_ERR_STATE;
    int rc = a2t_sync(c);
    if (rc) return rc;
    DeviceGuard dg(c->cfg.device);
    const int64_t eb = (int64_t)stream * ((int64_t)c->cfg.unit_rows + c->cfg.kept_rows);
    const int n = s.last_evict_pre;
    if (n_pre) *n_pre = n;
    if (mask && hipMemcpy(mask, c->dev.ev_mask + eb, n, hipMemcpyDeviceToHost) != hipSuccess) return hip_fail(c);
    if (new_slot && hipMemcpy(new_slot, c->dev.ev_slot + eb, (size_t)n * 4, hipMemcpyDeviceToHost) != hipSuccess)
        return hip_fail(c);
    return A2T_OK;
}

int a2t_read_kv(a2t_cache* c, int32_t layer, int32_t stream, void* kout, void* vout) {
    if (!c || stream < 0 || stream >= c->cfg.n_streams || layer < 0 || layer >= c->cfg.n_layers)
        return A2T_ERR_INVALID;
    if (c->host_only) return A2T_ERR_NODEV;
    if (c->dev_mode) return A2T_ERR_STATE;
    int rc = a2t_sync(c);
    if (rc) return rc;
    DeviceGuard dg(c->cfg.device);
    const StreamState& s = c->ss[stream];
    const a2t_config& k = c->cfg;
    const size_t elt = k.dtype == A2T_F32 ? 4 : 2;
    const size_t row = (size_t)k.head_dim * elt;       // one head of one row
    const size_t dpitch = row * k.n_kv_heads;          // host row pitch
    const int T = s.kept, U = s.ring, head = s.head, cap = k.unit_rows;
    const int first = std::min(U, cap - head), second = U - first;
    for (int which = 0; which < 2; ++which) {
        char* dst = static_cast<char*>(which ? vout : kout);
        if (!dst) continue;
        const char* kept = static_cast<const char*>(which ? c->dev.v_kept : c->dev.k_kept);
        const char* ring = static_cast<const char*>(which ? c->dev.v_unit : c->dev.k_unit);
        for (int g = 0; g < k.n_kv_heads; ++g) {
            const char* kb = kept + pool_index(c->dev, layer, stream, g, k.kept_rows, 0) * elt;
            const char* ub = ring + pool_index(c->dev, layer, stream, g, k.unit_rows, 0) * elt;
            if (T && hipMemcpy2D(dst + g * row, dpitch, kb, row, row, T, hipMemcpyDeviceToHost) != hipSuccess)
                return hip_fail(c);
            if (first && hipMemcpy2D(dst + (size_t)T * dpitch + g * row, dpitch, ub + (size_t)head * row, row,
                                     row, first, hipMemcpyDeviceToHost) != hipSuccess)
                return hip_fail(c);
            if (second && hipMemcpy2D(dst + (size_t)(T + first) * dpitch + g * row, dpitch, ub, row, row,
                                      second, hipMemcpyDeviceToHost) != hipSuccess)
                return hip_fail(c);
        }
    }
    return A2T_OK;
}

int a2t_profile_enable(a2t_cache* c, const char* kernel_filter) {
    if (!c) return A2T_ERR_INVALID;
    if (c->host_only) return A2T_ERR_NODEV;
    c->prof_on = kernel_filter != nullptr;
    c->prof_filter = kernel_filter ? kernel_filter : "";
    return A2T_OK;
}

int a2t_profile_reserve(a2t_cache* c, int32_t n_launches) {
    if (!c || n_launches < 0) return A2T_ERR_INVALID;
    if (c->host_only) return A2T_ERR_NODEV;
    DeviceGuard dg(c->cfg.device);
    while ((int64_t)c->prof_free.size() < 2 * (int64_t)n_launches) {
        hipEvent_t e = nullptr;
        if (hipEventCreate(&e) != hipSuccess) {
            (void)hipGetLastError();
            return A2T_ERR_OOM;
        }
        c->prof_free.push_back(e);
    }
    return A2T_OK;
}

int a2t_kernel_time(a2t_cache* c, const char* kernel, int64_t* launches, double* total_ms) {
    if (!c || !kernel) return A2T_ERR_INVALID;
    if (c->host_only) return A2T_ERR_NODEV;
    DeviceGuard dg(c->cfg.device);
    prof_harvest(c, true);
    int64_t n = 0;
    double ms = 0;
    for (auto it = c->prof_acc.begin(); it != c->prof_acc.end();) {
        if (std::strstr(it->first.c_str(), kernel)) {
            n += it->second.first;
            ms += it->second.second;
            it = c->prof_acc.erase(it);
        } else {
            ++it;
        }
    }
    if (launches) *launches = n;
    if (total_ms) *total_ms = ms;
    return A2T_OK;
}

// ---- device-planned steps --------------------------------------------------------
int a2t_dev_begin(a2t_cache* c) {
    if (!c) return A2T_ERR_INVALID;
    if (c->poisoned) return A2T_ERR_HIP;
    if (c->host_only) return A2T_ERR_NODEV;
    if (c->cfg.dtype != A2T_BF16 || c->force_valu) return A2T_ERR_INVALID;
    if (c->dev_mode) return A2T_ERR_STATE;
    for (const StreamState& s : c->ss)
        if (!s.step_complete() || s.step_rows != 0) return A2T_ERR_STATE;
    c->dss_host.resize(c->cfg.n_streams);
    for (int i = 0; i < c->cfg.n_streams; ++i) {
        const StreamState& s = c->ss[i];
        DevStream& d = c->dss_host[i];
        d = DevStream{};
        d.kept = s.kept;
        d.head = s.head;
        d.ring = s.ring;
        d.cur_unit = s.cur_unit;
        d.last_pos = s.last_pos;
        d.peak = s.peak;
        d.last_evicted = s.last_evicted;
        d.evicted_total = s.evicted_total;
        d.moved_total = s.moved_total;
        d.budget_unmet = s.budget_unmet;
        d.last_evict_pre = s.last_evict_pre;
    }
    DeviceGuard dg(c->cfg.device);
    if (hipStreamSynchronize(c->stream) != hipSuccess ||
        hipMemcpy(c->dev.dss, c->dss_host.data(), sizeof(DevStream) * c->dss_host.size(),
                  hipMemcpyHostToDevice) != hipSuccess)
        return hip_fail(c);
    c->dev_mode = true;
    c->dev_step_open = false;
    c->dev_layers.assign(c->cfg.n_layers, 0);
    return A2T_OK;
}

int a2t_dev_end(a2t_cache* c) {
    if (!c) return A2T_ERR_INVALID;
    if (c->poisoned) return A2T_ERR_HIP;
    if (!c->dev_mode || c->dev_step_open) return A2T_ERR_STATE;
    DeviceGuard dg(c->cfg.device);
    const int S = c->cfg.n_streams, cap = c->cfg.unit_rows;
    c->uid_host.resize((size_t)S * cap);
    c->seg_host.resize((size_t)S * cap);
    if (hipStreamSynchronize(c->stream) != hipSuccess ||
        hipMemcpy(c->dss_host.data(), c->dev.dss, sizeof(DevStream) * S, hipMemcpyDeviceToHost) != hipSuccess ||
        hipMemcpy(c->uid_host.data(), c->dev.unit_uid, (size_t)S * cap * 4, hipMemcpyDeviceToHost) != hipSuccess ||
        hipMemcpy(c->seg_host.data(), c->dev.unit_seg, (size_t)S * cap, hipMemcpyDeviceToHost) != hipSuccess)
        return hip_fail(c);
    int err = A2T_OK;
    for (int i = 0; i < S; ++i) {
        const DevStream& d = c->dss_host[i];
        StreamState& s = c->ss[i];
        if (d.error && err == A2T_OK) err = d.error;
        s.kept = d.kept;
        s.head = d.head;
        s.ring = d.ring;
        s.cur_unit = d.cur_unit;
        s.last_pos = d.last_pos;
        s.peak = d.peak;
        s.last_evicted = d.last_evicted;
        s.evicted_total = d.evicted_total;
        s.moved_total = d.moved_total;
        s.budget_unmet = d.budget_unmet;
        s.last_evict_pre = d.last_evict_pre;
        s.step_rows = 0;
        std::fill(s.appended.begin(), s.appended.end(), 1);
        // the unit queue and class ring from the ring slots' metadata
        s.units.pop_front(s.units.size());
        for (int x = 0; x < s.ring; ++x) {
            const int slot = (s.head + x) % cap;
            const int32_t u = c->uid_host[(size_t)i * cap + slot];
            const uint8_t sg = c->seg_host[(size_t)i * cap + slot];
            s.ring_seg[slot] = sg;
            if (s.units.size() && s.units.back().unit == u) {
                s.units.back().rows += 1;
                s.units.back().evictable += is_evictable(sg);
            } else {
                s.units.push_back(UnitRec{u, 1, is_evictable(sg) ? 1 : 0});
            }
        }
    }
    c->dev_mode = false;
    return err;
}

int a2t_dev_open(a2t_cache* c, int32_t n_streams, const int32_t* ids, const int32_t* n_rows,
                 const int32_t* unit_id, const uint8_t* seg, const int32_t* pos) {
    if (!c) return A2T_ERR_INVALID;
    if (c->poisoned) return A2T_ERR_HIP;
    if (!c->dev_mode || c->dev_step_open) return A2T_ERR_STATE;
    if (n_streams > kMaxDesc || !n_rows || !unit_id || !seg || !pos) return A2T_ERR_INVALID;
    int rc = check_streams(c, n_streams, ids);
    if (rc) return rc;
    DevStepArgs a{};
    a.count = n_streams;
    a.target_wgs = c->target_wgs;
    a.max_splits = std::max(1, std::min(kMaxSplits, c->target_wgs / c->cfg.n_kv_heads));
    for (int i = 0; i < n_streams; ++i) a.ids[i] = ids[i];
    DeviceGuard dg(c->cfg.device);
    if (launch_dev_open(c->dev, a, n_rows, unit_id, seg, pos, c->dplan, c->stream) != hipSuccess ||
        launch_step_meta_dev(c->dev, c->dplan, n_streams, seg, pos, unit_id, c->stream) != hipSuccess)
        return hip_fail(c);
    c->dev_step_open = true;
    c->dev_count = n_streams;
    c->dev_max_splits = a.max_splits;
    std::copy(ids, ids + n_streams, c->dev_ids);
    std::fill(c->dev_layers.begin(), c->dev_layers.end(), 0);
    return A2T_OK;
}

int a2t_dev_append_attn(a2t_cache* c, int32_t layer, const void* k, const void* v, const void* q,
                        void* o) {
    if (!c) return A2T_ERR_INVALID;
    if (c->poisoned) return A2T_ERR_HIP;
    if (!c->dev_mode || !c->dev_step_open) return A2T_ERR_STATE;
    if (layer < 0 || layer >= c->cfg.n_layers || !k || !v || !q || !o) return A2T_ERR_INVALID;
    if (unaligned16(k) || unaligned16(v) || unaligned16(q) || unaligned16(o)) return A2T_ERR_INVALID;
    if (c->dev_layers[layer]) return A2T_ERR_STATE;
    DeviceGuard dg(c->cfg.device);
    if (launch_attn_tile_dev(c->dev, c->dplan, c->dev_count, c->dev_max_splits, layer, q, o, k, v,
                             c->stream) != hipSuccess ||
        launch_attn_merge_dev(c->dev, c->dplan, c->dev_count, c->dev_max_splits, o, c->stream) !=
            hipSuccess)
        return hip_fail(c);
    c->dev_layers[layer] = 1;
    return A2T_OK;
}

int a2t_dev_evict(a2t_cache* c, const int32_t* budget, int32_t window, int32_t* n_evicted,
                  uint8_t* budget_unmet) {
    return a2t_dev_evict_rule(c, budget, window, A2T_RULE_UNIT, 0, n_evicted, budget_unmet);
}

int a2t_dev_evict_rule(a2t_cache* c, const int32_t* budget, int32_t window, int32_t rule,
                       int32_t n_sink, int32_t* n_evicted, uint8_t* budget_unmet) {
    if (!c) return A2T_ERR_INVALID;
    if (c->poisoned) return A2T_ERR_HIP;
    if (!c->dev_mode || !c->dev_step_open) return A2T_ERR_STATE;
    if (!budget || window < 0 || n_sink < 0) return A2T_ERR_INVALID;
    if (rule != A2T_RULE_UNIT && rule != A2T_RULE_ROW && rule != A2T_RULE_SINK_RECENT)
        return A2T_ERR_INVALID;
    for (uint8_t l : c->dev_layers)
        if (!l) return A2T_ERR_STATE;
    DevStepArgs a{};
    a.count = c->dev_count;
    a.window = window;
    a.rule = rule;
    a.n_sink = rule == A2T_RULE_SINK_RECENT ? n_sink : 0;
    std::copy(c->dev_ids, c->dev_ids + c->dev_count, a.ids);
    DeviceGuard dg(c->cfg.device);
    if (launch_dev_evict(c->dev, a, budget, n_evicted, budget_unmet, c->dplan, c->stream) != hipSuccess)
        return hip_fail(c);
    c->dev_step_open = false;
    return A2T_OK;
}

}  // extern "C"
