// Internal interface between the libA2T host code and its HIP kernels.
// Not part of the public ABI (include/a2t.h is).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace a2t {

// Largest number of stream descriptors one launch carries in its kernel
// arguments; calls over more streams are split into several launches.
constexpr int kMaxDesc = 64;
// Keys per attention tile (rows staged per LDS tile).
constexpr int kTileKeys = 64;

// Device-side buffers of a cache and its shape.
struct DevState {
    void* k_unit;   // [L][S][Hkv][unit_rows][D]  rotated keys of not-yet-evicted units (ring)
    void* v_unit;   // [L][S][Hkv][unit_rows][D]
    void* k_kept;   // [L][S][Hkv][kept_rows][D]  rows retained from evicted units, in order
    void* v_kept;   // [L][S][Hkv][kept_rows][D]
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
    int32_t L, S, Hq, Hkv, D, dtype;
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
struct StepBatch {
    int32_t count;
    StepDesc d[kMaxDesc];
};

// ---- append
struct AppendDesc {
    int32_t s;
    int32_t n;
    int32_t slot0;    // ring slot of the first row
    int32_t in_row0;  // first row in the packed k/v input
};
struct AppendBatch {
    int32_t count;
    int32_t max_n;
    int32_t layer0;       // first layer written
    int32_t total_rows;   // rows per layer in the packed input (A2T_ALL_LAYERS stride)
    AppendDesc d[kMaxDesc];
};

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
    int64_t ws_off;    // float offset of this stream's partials in the workspace
};
struct AttnBatch {
    int32_t count;
    int32_t layer;
    int32_t max_splits;
    int32_t max_rows;  // max n_q over the batch
    AttnDesc d[kMaxDesc];
};

// ---- eviction / compaction
struct EvictDesc {
    int32_t s;
    int32_t kept;      // T before eviction
    int32_t head;      // ring head before eviction
    int32_t R_pre;     // resident rows before eviction
    int32_t span;      // ring rows passed over (all rows of units up to u_last)
    int32_t u_last;    // newest evicted unit id
    int32_t n_keep;    // rows of the span that are retained (moved to the kept region)
};
struct EvictBatch {
    int32_t count;
    EvictDesc d[kMaxDesc];
};

// Launchers (kernels.hip).  Each returns the hipError_t of the launch.
hipError_t launch_step_meta(const DevState& st, const StepBatch& b, const uint8_t* seg,
                            const int32_t* pos, const int32_t* uid, hipStream_t stream);
hipError_t launch_append(const DevState& st, const AppendBatch& b, int n_layers,
                         const void* k, const void* v, hipStream_t stream);
// MFMA chunk attention (bf16 cache, D 64 or 128).
hipError_t launch_attn_mfma(const DevState& st, const AttnBatch& b, const void* q, void* o,
                            hipStream_t stream);
// VALU attention, one (row, kv head) per workgroup column (fp32 caches, decode).
hipError_t launch_attn_valu(const DevState& st, const AttnBatch& b, const void* q, void* o,
                            hipStream_t stream);
hipError_t launch_attn_merge(const DevState& st, const AttnBatch& b, void* o,
                             hipStream_t stream);
hipError_t launch_evict(const DevState& st, const EvictBatch& b, hipStream_t stream);

}  // namespace a2t
