// Internal interface between the libA2T host code and its HIP kernels.
// Not part of the public ABI (include/a2t.h is).
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>
#include <string.h>

#include <cstring>

namespace a2t {

// Largest number of stream descriptors one launch carries in its kernel
// arguments; calls over more streams are split into several launches.
constexpr int kMaxDesc = 64;
// Keys per attention tile (rows staged per LDS tile).
constexpr int kTileKeys = 64;
// Most key splits of one attention launch.
constexpr int kMaxSplits = 128;
// Query rows per workgroup of the split merge.
constexpr int kMergeRows = 4;

// State of one stream kept on the device for device-planned steps (the host's
// per-stream mirror, moved to the device while the caller drives the cache
// with a2t_dev_* calls).
struct DevStream {
    int32_t kept, head, ring, cur_unit;
    int64_t last_pos;
    int32_t step_rows, step_slot0;
    int32_t peak, last_evicted;
    int64_t evicted_total, moved_total;
    int32_t budget_unmet, last_evict_pre;
    int32_t error;      // first a2t_status a device-planned step hit on this stream (0: none)
    int32_t pad_;
};

// Device-side buffers of a cache and its shape.
struct DevState {
    void* k_unit;   // [L][S][Hkv][unit_rows][D]  rotated keys of the rows eviction has not
    void* v_unit;   //                             passed over yet (ring); V likewise
    void* k_kept;   // [L][S][Hkv][kept_rows][D]  rows retained from the part eviction has
    void* v_kept;   //                             passed over, in order (right after the ring)
    int32_t* unit_pos;  // [S][unit_rows] metadata of ring slots
    int32_t* unit_uid;
    uint8_t* unit_seg;
    int32_t* kept_pos;  // [S][kept_rows] metadata of kept slots
    int32_t* kept_uid;
    uint8_t* kept_seg;
    float2* rope;       // [S][max_step_rows][D/2] (cos, sin) of the open step's rows
    uint8_t* ev_mask;   // [S][unit_rows + kept_rows] last eviction, 1 = evicted
    int32_t* ev_slot;   // [S][unit_rows + kept_rows] last eviction, new slot or -1
    float* ws;          // split-K attention partials
    int64_t ws_floats;
    DevStream* dss;     // [S] device-planned steps: per-stream state
    int32_t L, S, Hq, Hkv, D, dtype;
    int32_t G;          // query heads per KV head (Hq / Hkv)
    int32_t unit_rows, kept_rows, max_step_rows;
    float scale_log2e;  // softmax scale * log2(e)
    double theta;
};

__host__ __device__ inline int64_t pool_index(const DevState& st, int layer, int s, int g,
                                              int rows, int slot) {
    return ((((int64_t)layer * st.S + s) * st.Hkv + g) * rows + slot) * st.D;
}

// ---- step registration: staged host metadata -> device metadata + rotary table
struct StepDesc {
    int32_t s;        // stream
    int32_t n;        // rows in the step
    int32_t slot0;    // ring slot of the first row
    int32_t row0;     // offset of the stream's rows in the staged arrays
};
template <int N>
struct StepBatchT {
    int32_t count;
    int32_t max_n;
    StepDesc d[N];
};
using StepBatch = StepBatchT<kMaxDesc>;

// ---- append
struct AppendDesc {
    int32_t s;
    int32_t n;
    int32_t slot0;    // ring slot of the first row
    int32_t in_row0;  // first row in the packed k/v input
};
template <int N>
struct AppendBatchT {
    int32_t count;
    int32_t max_n;
    int32_t layer0;       // first layer written
    int32_t total_rows;   // rows per layer in the packed input (A2T_ALL_LAYERS stride)
    AppendDesc d[N];
};
using AppendBatch = AppendBatchT<kMaxDesc>;

// ---- attention (chunk and decode)
struct AttnDesc {
    int32_t s;
    int32_t kept;      // T: rows in the kept region
    int32_t head;      // ring head slot
    int32_t R;         // resident rows (keys)
    int32_t n_q;       // query rows (the stream's last n_q rows)
    int32_t q_row0;    // first row of this stream in the packed q/o
    int32_t rope_row0; // row of the first query in the step's rotary table
    int32_t splits;    // key splits; 1 = write o directly
    int32_t n_new;     // fused append: the last n_new keys come from the input k/v (else 0)
    int32_t in_row0;   // fused append: first row of this stream in the input k/v
    int32_t tile_q;    // key tiles per split: split sp < splits - m takes tile_q tiles,
    int32_t tile_r;    //   one more if sp < r, from tile sp * tile_q + min(sp, r); the last
                       //   m splits take one tile each (r = tile_r & 0xffff, m = tile_r >> 16)
    int64_t ws_off;    // float offset of this stream's partials in the workspace
};
template <int N>
struct AttnBatchT {
    int32_t count;
    int32_t layer;
    int32_t max_splits;
    int32_t max_rows;  // max n_q over the batch
    AttnDesc d[N];
};
using AttnBatch = AttnBatchT<kMaxDesc>;

// ---- eviction / compaction
struct EvictDesc {
    int32_t s;
    int32_t kept;      // T before eviction
    int32_t head;      // ring head before eviction
    int32_t R_pre;     // resident rows before eviction
    int32_t span;      // oldest ring rows passed over (up to and including the last evicted
                       // row, or every row of the units up to u_last)
    int32_t u_last;    // unit id of the newest evicted row
    int32_t n_keep;    // rows of the span that are retained (moved to the kept region)
    int32_t sink;      // >= 0: the span's rows with cache index < sink are kept, every
                       // other one is evicted (sink + recent rule); -1: retained rows
                       // are those of a class that is never evicted
};
template <int N>
struct EvictBatchT {
    int32_t count;
    EvictDesc d[N];
};
using EvictBatch = EvictBatchT<kMaxDesc>;

// ---- device-planned steps: descriptors written by device kernels
// Descriptors read through a pointer to device memory instead of from the
// kernel arguments; `layer` and `max_rows` still come with the launch.  The
// kernels index `b.d[i]` and read `b.layer` / `b.max_rows` the same way for
// both kinds of batch.
template <class Desc>
struct DescPtr {
    const Desc* p;
    __device__ const Desc& operator[](int i) const { return p[i]; }
};
template <class Desc>
struct DevBatch {
    DescPtr<Desc> d;
    int32_t layer;
    int32_t max_rows;
};

// What a device-planned step's kernels read: written by dev_open_kernel
// (metadata, attention) and dev_evict_plan_kernel (eviction).
struct DevPlan {
    StepDesc step[kMaxDesc];
    AttnDesc attn[kMaxDesc];
    EvictDesc evict[kMaxDesc];
};

// Kernel argument of the device planners: the streams of the step and limits.
struct DevStepArgs {
    int32_t count;
    int32_t max_splits;   // key splits the attention grid was sized for
    int32_t target_wgs;   // workgroups one attention launch spreads over at most
    int32_t window;       // recent units protected (eviction)
    int32_t rule;         // a2t_rule of the eviction
    int32_t n_sink;       // sink rows (A2T_RULE_SINK_RECENT)
    int32_t ids[kMaxDesc];
};

// Kernel arguments are copied per launch: a launch carries a batch sized to
// its stream count (1, 8 or kMaxDesc descriptors), not always the largest.
template <template <int> class BT, int N>
inline BT<N> shrink_batch(const BT<kMaxDesc>& b) {
    BT<N> s;
    static_assert(offsetof(BT<N>, d) == offsetof(BT<kMaxDesc>, d), "batch header layout");
    std::memcpy(&s, &b, offsetof(BT<N>, d) + sizeof(b.d[0]) * (b.count < N ? b.count : N));
    return s;
}

// Optional dispatch timestamps: with start non-null the launcher issues its one
// kernel through hipExtLaunchKernel, which records start/stop at the kernel's
// own begin and end (no extra packets on the stream between them).
struct KTimer {
    hipEvent_t start = nullptr;
    hipEvent_t stop = nullptr;
};

// Launchers (kernels.hip).  Each issues one kernel and returns the hipError_t
// of the launch.
hipError_t launch_step_meta(const DevState& st, const StepBatch& b, const uint8_t* seg,
                            const int32_t* pos, const int32_t* uid, hipStream_t stream,
                            const KTimer& kt);
hipError_t launch_append(const DevState& st, const AppendBatch& b, int n_layers,
                         const void* k, const void* v, hipStream_t stream, const KTimer& kt);
// MFMA chunk attention (bf16 cache, D 64 or 128).  With k_in/v_in non-null it
// also appends each stream's n_new newest rows (rotating K) from that input.
hipError_t launch_attn_tile(const DevState& st, const AttnBatch& b, const void* q, void* o,
                            const void* k_in, const void* v_in, hipStream_t stream,
                            const KTimer& kt);
// VALU attention, one (row, kv head) per workgroup column (fp32 caches, decode).
hipError_t launch_attn_valu(const DevState& st, const AttnBatch& b, const void* q, void* o,
                            hipStream_t stream, const KTimer& kt);
// h16: the partials come from the MFMA kernel (fp16 O rows), else from the VALU kernel (fp32)
hipError_t launch_attn_merge(const DevState& st, const AttnBatch& b, void* o,
                             hipStream_t stream, const KTimer& kt, bool h16);
// Floats of key-split partials per query row and head: O (fp16 from the MFMA kernel,
// fp32 from the VALU kernel) and the fp32 (max, sum) pair.
inline int64_t partial_row_floats(int head_dim, bool valu) { return (valu ? head_dim : head_dim / 2) + 2; }
// Floats one stream's key-split partials take in the workspace (none without a
// split), rounded up to 64 floats (256 bytes) so that every stream's rows start
// 16-byte aligned for the kernels' 16-byte stores and loads.
__host__ __device__ inline int64_t stream_partials(int splits, int64_t floats_per_split) {
    return splits > 1 ? (splits * floats_per_split + 63) / 64 * 64 : 0;
}
hipError_t launch_evict(const DevState& st, const EvictBatch& b, hipStream_t stream,
                        const KTimer& kt);

// Device-planned steps (bf16 caches: the fused MFMA path).  dev_open: validate the step's device-resident
// metadata (n_rows, unit [count]; seg, pos [count][max_step_rows]), open it in
// every listed stream and write the metadata, attention and step descriptors
// to `plan`.  Then the per-layer launches read `plan` (metadata + rotary
// table once, attention + merge per layer).  dev_evict: plan Sec. 3.3's
// eviction on the device (budget [count], n_evicted / budget_unmet [count]
// out, may be null) and run it.
hipError_t launch_dev_open(const DevState& st, const DevStepArgs& a, const int32_t* n_rows,
                           const int32_t* unit, const uint8_t* seg, const int32_t* pos,
                           DevPlan* plan, hipStream_t stream);
hipError_t launch_step_meta_dev(const DevState& st, const DevPlan* plan, int count,
                                const uint8_t* seg, const int32_t* pos, const int32_t* unit,
                                hipStream_t stream);
hipError_t launch_attn_tile_dev(const DevState& st, const DevPlan* plan, int count,
                                int max_splits, int layer, const void* q, void* o,
                                const void* k_in, const void* v_in, hipStream_t stream);
hipError_t launch_attn_merge_dev(const DevState& st, const DevPlan* plan, int count,
                                 int max_splits, void* o, hipStream_t stream);
hipError_t launch_dev_evict(const DevState& st, const DevStepArgs& a, const int32_t* budget,
                            int32_t* n_evicted, uint8_t* budget_unmet, DevPlan* plan,
                            hipStream_t stream);

// The library's fixed split workspace (a file-scope device array of kernels.hip)
// on `device`, which must be the current device: its device address and size
// in floats.  The address is looked up once per device and kept.
hipError_t static_scratch(int device, float** ptr, int64_t* floats);

}  // namespace a2t
