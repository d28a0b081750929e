/*
 * a2t.h — C ABI of libA2T, the MI355X (gfx950) streaming KV step of
 * acoustic-to-text KV compression for full-duplex speech models.
 *
 * One cache holds, for every layer and every stream, the resident key/value
 * rows of a duplex session.  Per step (one listening unit, or one decode
 * token while speaking) the caller
 *   1. appends the step's rows, layer by layer          (a2t_append),
 *   2. runs attention for the step's new rows            (a2t_chunk_attn /
 *                                                         a2t_decode_attn),
 *   3. after the last layer, evicts under a budget and compacts (a2t_evict).
 *
 * Paper passages (Sec. = section of the paper):
 *   Sec. 3.1  a unit is ~10 audio tokens plus marker and decision; its
 *             transcript segment, delimited by two ASR tokens, follows the
 *             first decision and stays in context.
 *   Sec. 3.3  after each unit, if the resident positions (prefix and text
 *             included) exceed budget B, evict the acoustic and structural
 *             rows (unit marker, audio, decision, ASR delimiters, terminators)
 *             of the oldest unit outside the W most recent units; repeat until
 *             the cache fits or no eligible unit remains.  Transcript tokens,
 *             response text and the system prefix are kept.  Position ids
 *             advance with every fed token whatever is evicted, so kept keys
 *             keep their rotary positions and are never re-encoded.
 *
 * Conventions
 *   - Return value: A2T_OK (0) or a negative a2t_status.  Every argument is
 *     validated before any state changes or any work is enqueued, so a call
 *     that fails changes nothing.
 *   - "device" pointers are HIP device memory (e.g. torch CUDA tensors on
 *     ROCm); "host" pointers are ordinary CPU memory, read before the call
 *     returns.  Device buffers must stay valid until the HIP stream reaches
 *     the enqueued work; outputs are ready after the stream does.  The K, V,
 *     Q and O buffers of the append and attention calls must be 16-byte
 *     aligned (the kernels move them 16 bytes at a time): A2T_ERR_INVALID
 *     otherwise.
 *   - All compute is enqueued on the cache's HIP stream (a2t_set_stream).
 *     Nothing in a2t_append / a2t_append_attn / a2t_chunk_attn /
 *     a2t_decode_attn / a2t_evict / a2t_evict_rule allocates memory (every
 *     buffer is sized at creation); the a2t_read_* calls synchronise.  The
 *     calls that open a step (layer 0 or A2T_ALL_LAYERS) stage its metadata
 *     in one of 16 pinned slots: with 16 earlier steps still queued on the
 *     device, opening one more waits until the oldest has run (back-pressure,
 *     not a synchronisation of the whole device).
 *   - A device fault or launch failure poisons the cache: that call and every
 *     later one return A2T_ERR_HIP.
 *   - One host thread at a time per cache.
 *   - Element types: A2T_F32 (float) or A2T_BF16 (bfloat16, raw 16-bit).
 *     Q, K, V and O all use the cache's dtype; arithmetic is fp32 with
 *     fp64-accurate rotary angles.
 *   - Rotary encoding: rotate-half, x'[i] = x[i] cos a - x[i+D/2] sin a,
 *     x'[i+D/2] = x[i+D/2] cos a + x[i] sin a, a = pos * theta^(-2i/D), i < D/2.
 *     Query head h reads KV head h / (n_q_heads / n_kv_heads).
 *   - Causality: a step's query row i sees every resident row up to and
 *     including itself (the rows of the step are appended before attention).
 *
 * Cache order and layout
 *   The resident rows of a stream are kept in the order they were appended
 *   (position order).  Eviction removes rows and keeps the survivors in that
 *   order: survivor i moves to slot new_slot[i] = number of survivors before
 *   it.  Physically a stream's rows live in two dense regions per layer:
 *   the "kept" region (rows retained from the part of the stream eviction
 *   has already passed over, in order) followed, logically, by a ring of the
 *   newer rows.  Eviction always removes the oldest eligible rows, so it
 *   advances the ring head past the rows it passes over and moves only their
 *   retained rows into the kept region; a2t_read_layout / a2t_read_kv return
 *   the rows in cache order.
 */
#ifndef A2T_H
#define A2T_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define A2T_ABI_VERSION 2
#define A2T_ALL_LAYERS (-1)

typedef struct a2t_cache a2t_cache;

typedef enum a2t_status {
    A2T_OK = 0,
    A2T_ERR_INVALID = -1,   /* bad argument: null pointer, out-of-range id/size/class */
    A2T_ERR_POS = -2,       /* position not strictly increasing, unit id decreasing,
                               or metadata that contradicts the registered step */
    A2T_ERR_CAPACITY = -3,  /* a region of the cache would overflow */
    A2T_ERR_STATE = -4,     /* call out of order (layer not appended, step open, ...) */
    A2T_ERR_OOM = -5,       /* device or pinned-host allocation failed (create only) */
    A2T_ERR_HIP = -6,       /* HIP runtime error or device fault; the cache is poisoned */
    A2T_ERR_NODEV = -7      /* no usable gfx950 device, or a host-only cache was asked
                               for device work */
} a2t_status;

typedef enum a2t_dtype { A2T_F32 = 0, A2T_BF16 = 1 } a2t_dtype;

/* Row classes (Sec. 3.3).  ACOUSTIC covers every structural state the paper
 * evicts besides the ASR delimiters: unit marker, audio tokens, native
 * decision, terminators.  DELIM is the ASR start/end delimiter.  TEXT is a
 * transcript token, RESPONSE a model-generated response token, PREFIX the
 * system prefix (unit id -1).  ACOUSTIC and DELIM rows are evictable. */
typedef enum a2t_seg {
    A2T_SEG_PREFIX = 0,
    A2T_SEG_ACOUSTIC = 1,
    A2T_SEG_DELIM = 2,
    A2T_SEG_TEXT = 3,
    A2T_SEG_RESPONSE = 4
} a2t_seg;

/* Cache creation flags. */
#define A2T_FLAG_HOST_ONLY 1u  /* no device: bookkeeping and eviction planning only
                                  (append/evict update the host state; attention and
                                  device reads return A2T_ERR_NODEV) */
#define A2T_FLAG_NO_WORKSPACE 2u  /* allocate no key-split workspace (256 MiB by default):
                                  the attention calls then run one split per stream,
                                  except a2t_append_attn_noalloc, which splits into the
                                  library's fixed array */

typedef struct a2t_config {
    int32_t n_layers;       /* L >= 1 */
    int32_t n_streams;      /* S >= 1 independent sessions */
    int32_t n_q_heads;      /* Hq, a multiple of n_kv_heads */
    int32_t n_kv_heads;     /* Hkv >= 1 */
    int32_t head_dim;       /* D: 64 or 128 */
    int32_t dtype;          /* a2t_dtype */
    int32_t unit_rows;      /* per (layer, stream): capacity of the ring of rows of
                               units not yet evicted */
    int32_t kept_rows;      /* per (layer, stream): capacity of the region of rows
                               retained from evicted units (and the prefix) */
    int32_t max_step_rows;  /* most rows one stream appends in one step (<= 1024) */
    uint32_t flags;         /* A2T_FLAG_* */
    double rope_theta;      /* rotary base; 0 selects 1e6 */
    double attn_scale;      /* softmax scale; 0 selects 1/sqrt(head_dim) */
    int32_t device;         /* HIP device ordinal */
    int32_t reserved;
    /* Optional caller-owned K and V pools (device memory of `device`, 256-byte
     * aligned), each L*S*Hkv*(unit_rows + kept_rows)*D elements of the cache
     * dtype: the ring of every (layer, stream, KV head) first, then the kept
     * regions ([L][S][Hkv][unit_rows][D] followed by [L][S][Hkv][kept_rows][D]).
     * Both NULL: the library allocates and frees them.  Both set: the caller
     * keeps them alive until a2t_cache_destroy returns; the library never frees
     * them.  Only one set: A2T_ERR_INVALID.  Ignored for host-only caches. */
    void* k_pool;
    void* v_pool;
} a2t_config;

/* Per-stream bookkeeping, for tests and reporting. */
typedef struct a2t_stream_info {
    int32_t resident;       /* R: rows in the cache now */
    int32_t peak;           /* largest R seen right after an append */
    int32_t kept;           /* rows in the kept region */
    int32_t ring;           /* rows in the unit ring */
    int32_t ring_head;      /* ring slot of the oldest not-yet-evicted row */
    int32_t cur_unit;       /* newest unit id appended (-2 if none) */
    int32_t last_evicted_unit;  /* newest unit id evicted (-2 if none) */
    int32_t step_rows;      /* rows of the open step (0 if none) */
    int64_t last_pos;       /* last position id appended (-1 if none) */
    int64_t evicted_total;  /* rows evicted since creation */
    int64_t moved_total;    /* rows copied into the kept region since creation */
    int32_t budget_unmet;   /* 1 if the last a2t_evict left R > budget */
    int32_t last_evict_pre; /* R before the last eviction that removed rows (-1 if none) */
} a2t_stream_info;

/* Create a cache.  Allocates every device buffer it will ever use (the K/V
 * pools unless the caller passes them, metadata, attention workspace), the
 * host bookkeeping of every stream (sized by unit_rows and max_step_rows) and
 * a small pinned-host staging area.
 * hip_stream: the hipStream_t to enqueue on (NULL = the default stream).
 * Pools hold L*S*Hkv*(unit_rows+kept_rows)*D elements for each of K and V.
 * Tuning read from the environment at creation (for tests and measurements;
 * results stay within the attention tolerances whatever they are):
 *   A2T_WS_MB       key-split workspace in MiB (default 256; a launch whose
 *                   planned partials do not fit plans fewer splits)
 *   A2T_TARGET_WGS  attention workgroups one launch spreads over (default:
 *                   the device's CU count, one 8-wave workgroup per CU)
 *   A2T_SPLITS      force this many key splits per stream (0 = planned)
 *   A2T_FORCE_VALU  nonzero: the VALU attention kernel for bf16 caches too */
int a2t_cache_create(const a2t_config* cfg, void* hip_stream, a2t_cache** out);

/* Wait for the stream, then free everything the cache owns.  NULL is a no-op. */
int a2t_cache_destroy(a2t_cache* c);

/* Change the HIP stream later calls enqueue on. */
int a2t_set_stream(a2t_cache* c, void* hip_stream);

/* Append one step's rows (Sec. 3.1, Sec. 3.3).
 *   layer       0..L-1, or A2T_ALL_LAYERS.
 *   stream_ids  host [n_streams], distinct ids in 0..S-1.
 *   n_rows      host [n_streams], 1..max_step_rows rows per stream.
 *   k, v        device, pre-rotation, packed in stream order:
 *               [sum n_rows][Hkv][D] for one layer,
 *               [L][sum n_rows][Hkv][D] for A2T_ALL_LAYERS.
 *   seg         host [sum n_rows] a2t_seg per row.
 *   pos         host [sum n_rows] position ids, strictly increasing within a
 *               stream and across its steps (gaps allowed), < 2^31.
 *   unit_id     host [n_streams] unit id of every row of the stream's step:
 *               -1 for a prefix step (PREFIX rows only), otherwise >= 0 and not
 *               below the stream's newest unit id.  A decode step repeats the
 *               newest unit id.
 * Layer 0 (or A2T_ALL_LAYERS) opens a new step for each listed stream: it
 * requires the previous step to be appended on every layer, and seg/pos/
 * unit_id.  Layers 1..L-1 then append the same n_rows; their seg/pos/unit_id
 * may be NULL (if given they must equal the registered values).
 * K rows are stored rotated by their position; V rows as given.
 * Errors: INVALID, POS, CAPACITY (ring full), STATE (layer already appended
 * this step, or layer 0 before the previous step finished). */
int a2t_append(a2t_cache* c, int32_t layer, int32_t n_streams, const int32_t* stream_ids,
               const int32_t* n_rows, const void* k, const void* v, const uint8_t* seg,
               const int32_t* pos, const int32_t* unit_id);

/* Causal chunk attention for the step's newest rows (Sec. 3.1: the unit's
 * tokens are processed over the resident cache).
 *   n_q   host [n_streams]: queries are the stream's last n_q rows appended
 *         this step (1 <= n_q <= step rows); their stored positions rotate q.
 *   q     device [sum n_q][Hq][D], pre-rotation.
 *   o     device [sum n_q][Hq][D], written with softmax(scale q.K^T) V over the
 *         resident rows of `layer` up to each query's own row.
 * Scores, the softmax and the output sums are fp32.  When a launch splits a
 * stream's keys over several workgroups, each split's output rows of a bf16
 * cache are held in fp16 until they are combined (normalised by the split's
 * own sum, so each value lies within the range of the V entries): bf16 V
 * entries must stay within fp16's range (|v| <= 65504).  fp32 caches keep
 * fp32 split outputs.
 * The layer must have appended the current step.  Errors: INVALID, STATE. */
int a2t_chunk_attn(a2t_cache* c, int32_t layer, int32_t n_streams, const int32_t* stream_ids,
                   const int32_t* n_q, const void* q, void* o);

/* a2t_append on one layer followed by a2t_chunk_attn on that layer, in one
 * launch where the kernels allow it (bf16 caches): the workgroups whose key
 * tiles hold the step's new rows rotate and store them while staging them
 * for attention.  Arguments as in the two calls (layer 0..L-1 only; n_q
 * host [n_streams] with 1 <= n_q <= n_rows; q and o packed [sum n_q][Hq][D]).
 * Results and cache contents are the same as the two calls. */
int a2t_append_attn(a2t_cache* c, int32_t layer, int32_t n_streams, const int32_t* stream_ids,
                    const int32_t* n_rows, const void* k, const void* v, const uint8_t* seg,
                    const int32_t* pos, const int32_t* unit_id, const int32_t* n_q,
                    const void* q, void* o);

/* a2t_append_attn for callers that cannot allocate memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc).  Same
 * arguments, results and cache contents as a2t_append_attn; the key-split
 * partials go to a fixed 16 MiB device array of the library (one per GPU, held
 * until the process ends) instead of the cache's workspace, so it also works
 * on a cache created with A2T_FLAG_NO_WORKSPACE.  Splits are planned as
 * a2t_append_attn plans them without a workspace limit; a call whose launch
 * would write more than 16 MiB of partials (4,194,304 floats; a stream's
 * partials are splits x n_q x n_q_heads x (head_dim / 2 + 2) floats for a bf16
 * cache, fp16 output rows with an fp32 maximum and sum, and x (head_dim + 2)
 * for an fp32 cache: about 4 MiB for 22 query rows x 32 heads x head dim 128
 * at ~4,100 resident rows, 23 splits) is
 * rejected with A2T_ERR_CAPACITY before anything changes.  Every call on a GPU
 * shares that GPU's array: calls that overlap on one GPU (two caches on
 * different streams, or two host threads) race and must be serialised by the
 * caller; calls in order on one stream are safe.  Its launches are never timed
 * (a2t_profile_enable does not apply).  Errors: those of a2t_append_attn,
 * CAPACITY as above, NODEV if the array is not available on the device. */
int a2t_append_attn_noalloc(a2t_cache* c, int32_t layer, int32_t n_streams,
                            const int32_t* stream_ids, const int32_t* n_rows, const void* k,
                            const void* v, const uint8_t* seg, const int32_t* pos,
                            const int32_t* unit_id, const int32_t* n_q, const void* q, void* o);

/* Decode attention while speaking: one query per stream, the stream's newest
 * row (Sec. 3.1: response tokens are decoded one by one over the cache).
 *   q, o  device [n_streams][Hq][D].  Errors as a2t_chunk_attn. */
int a2t_decode_attn(a2t_cache* c, int32_t layer, int32_t n_streams, const int32_t* stream_ids,
                    const void* q, void* o);

/* Online budgeted eviction and compaction after a step (Sec. 3.3).
 * For each listed stream: while R > budget[i] and some unit u <= cur - window
 * still holds ACOUSTIC/DELIM rows, remove every ACOUSTIC/DELIM row of the
 * oldest such unit.  Survivors keep their positions and order.  One pass
 * moves the retained rows of all evicted units, in every layer.
 *   budget       host [n_streams], >= 0.
 *   window       recent units protected (cur-window+1 .. cur), >= 0.
 *   n_evicted    optional host [n_streams] out: rows removed.
 *   budget_unmet optional host [n_streams] out: 1 if R > budget afterwards.
 * Requires every layer to have appended the stream's step.  A budget that
 * cannot be met is not an error.  Errors: INVALID, STATE, CAPACITY (kept
 * region full). */
int a2t_evict(a2t_cache* c, int32_t n_streams, const int32_t* stream_ids, const int32_t* budget,
              int32_t window, int32_t* n_evicted, uint8_t* budget_unmet);

/* Variants of the eviction rule, for ablations and comparisons; a2t_evict
 * applies A2T_RULE_UNIT.
 *   A2T_RULE_UNIT         Sec. 3.3: whole units, oldest first, outside the
 *                         window (see a2t_evict).
 *   A2T_RULE_ROW          the same eligible rows (ACOUSTIC/DELIM rows of units
 *                         u <= cur - window), removed one at a time, oldest
 *                         first, until R <= budget: an ablation of the rule's
 *                         whole-unit granularity; a unit may lose only part of
 *                         its rows.
 *   A2T_RULE_SINK_RECENT  the StreamingLLM comparison (Sec. 2 and Table 1: sink
 *                         positions plus a recent window): when R > budget,
 *                         every row except the n_sink oldest and the
 *                         budget - n_sink newest is removed, whatever its
 *                         class; window is ignored.  Requires budget >= n_sink;
 *                         a stream whose kept region holds rows other than its
 *                         sinks (left there by another rule) cannot switch to
 *                         it (A2T_ERR_STATE). */
typedef enum a2t_rule {
    A2T_RULE_UNIT = 0,
    A2T_RULE_ROW = 1,
    A2T_RULE_SINK_RECENT = 2
} a2t_rule;

/* a2t_evict with a choice of rule (a2t_rule) and, for A2T_RULE_SINK_RECENT,
 * the sink count (>= 0; ignored by the other rules).  Survivors keep their
 * positions and order under every rule, and one pass moves the retained rows
 * of every layer.  Arguments and outputs otherwise as a2t_evict.
 * Errors: INVALID (unknown rule, n_sink < 0, budget < n_sink under
 * A2T_RULE_SINK_RECENT, and those of a2t_evict), STATE, CAPACITY. */
int a2t_evict_rule(a2t_cache* c, int32_t n_streams, const int32_t* stream_ids,
                   const int32_t* budget, int32_t window, int32_t rule, int32_t n_sink,
                   int32_t* n_evicted, uint8_t* budget_unmet);

/* ---------------------------------------------------------------------------
 * Device-planned steps: the same listening or decode step (append + chunk
 * attention on every layer, then Sec. 3.3's eviction check) with every
 * per-step decision taken on the device, from step metadata the caller leaves
 * in device memory.  Each call below enqueues kernels whose arguments do not
 * depend on the step, so a caller can capture a whole step (or one layer's
 * call among its own kernels) in a HIP graph once and replay it for every
 * later step, rewriting only the contents of its device buffers in between.
 *
 * Between a2t_dev_begin and a2t_dev_end the device holds each stream's state
 * (rows, ring head, newest unit and position, the per-unit eviction plan): the
 * host-planned calls (a2t_append*, a2t_*_attn, a2t_evict*, a2t_stream_info_get,
 * a2t_read_*) return A2T_ERR_STATE.  Only bf16 caches (the fused MFMA path);
 * at most 64 streams per step; eviction follows Sec. 3.3's whole-unit rule
 * (a2t_dev_evict) or a variant of it (a2t_dev_evict_rule).
 * ------------------------------------------------------------------------- */

/* Hand the host's per-stream state to the device (synchronises).  Errors:
 * INVALID (fp32 cache), STATE (already begun, or a host step still open),
 * NODEV (host-only cache). */
int a2t_dev_begin(a2t_cache* c);

/* Take the state back (synchronises): the host's bookkeeping then describes
 * the cache as the device-planned steps left it.  Returns A2T_OK, or the first
 * status a device-planned step reported for some stream (see a2t_dev_open);
 * the cache is consistent either way.  Errors: STATE (not begun, or a step is
 * open). */
int a2t_dev_end(a2t_cache* c);

/* Open one step for n_streams listed streams (host ids, distinct).  Device
 * arrays, read when the stream reaches the work:
 *   n_rows   [n_streams]  rows of each stream's step (1..max_step_rows)
 *   unit_id  [n_streams]  as in a2t_append
 *   seg      [n_streams][max_step_rows]  a2t_seg per row (first n_rows used)
 *   pos      [n_streams][max_step_rows]  position ids, strictly increasing
 * The device checks what a2t_append checks; a stream whose step fails a check
 * records the status (returned by a2t_dev_end) and takes no part in this or
 * any later device-planned step.  The device then plans each stream's key
 * splits (the smallest budget of key tiles per split whose workgroups fit one
 * round over the CUs, as the host plans a single stream).
 * Errors (host-side, nothing enqueued): INVALID (ids, null pointers, more than
 * 64 streams), STATE (not begun, or the previous step not evicted). */
int a2t_dev_open(a2t_cache* c, int32_t n_streams, const int32_t* stream_ids, const int32_t* n_rows,
                 const int32_t* unit_id, const uint8_t* seg, const int32_t* pos);

/* a2t_append_attn for one layer of the open step.  k, v: device
 * [n_streams][max_step_rows][Hkv][D]; q, o: device [n_streams][max_step_rows]
 * [Hq][D]: listed stream i's rows start at row i * max_step_rows (only its
 * first n_rows are read or written).  Errors: INVALID, STATE (no open step,
 * or the layer already appended). */
int a2t_dev_append_attn(a2t_cache* c, int32_t layer, const void* k, const void* v, const void* q,
                        void* o);

/* Sec. 3.3's eviction for the open step's streams, planned on the device:
 * while R > budget[i], the oldest unit outside the window that still holds
 * acoustic/structural rows loses all of them.  budget: device [n_streams]
 * (negative counts as 0); n_evicted, budget_unmet: optional device
 * [n_streams] outputs.  Closes the step.  Errors: INVALID, STATE (no open
 * step, or a layer not appended).  A kept region that would overflow is
 * reported by a2t_dev_end (CAPACITY) and that stream evicts nothing. */
int a2t_dev_evict(a2t_cache* c, const int32_t* budget, int32_t window, int32_t* n_evicted,
                  uint8_t* budget_unmet);

/* a2t_dev_evict with a choice of rule (a2t_rule, as in a2t_evict_rule) and,
 * for A2T_RULE_SINK_RECENT, the sink count (>= 0; ignored by the other rules).
 * The rule's conditions on the device values are checked per stream on the
 * device: a budget below n_sink (A2T_ERR_INVALID) or a kept region holding
 * rows other than the sinks (A2T_ERR_STATE) is recorded for that stream like
 * a2t_dev_open's checks (reported by a2t_dev_end; the stream evicts nothing
 * and takes no part in later device-planned steps).  Errors (host-side,
 * nothing enqueued): INVALID (unknown rule, n_sink < 0, and those of
 * a2t_dev_evict), STATE. */
int a2t_dev_evict_rule(a2t_cache* c, const int32_t* budget, int32_t window, int32_t rule,
                       int32_t n_sink, int32_t* n_evicted, uint8_t* budget_unmet);

/* Bookkeeping of one stream (host state, no synchronisation). */
int a2t_stream_info_get(const a2t_cache* c, int32_t stream, a2t_stream_info* out);

/* A stream's resident row count R and its peak (Sec. 3.3: the budget is checked
 * against R after each unit; the peak is the largest R right after an append).
 * n, peak: host, either may be NULL.  Host bookkeeping only, no device access.
 * Errors: INVALID (stream out of range), STATE (device-planned steps hold the
 * state: a2t_dev_end first). */
int a2t_resident(const a2t_cache* c, int32_t stream, int32_t* n, int32_t* peak);

/* Copy one stream's layout to host, in cache order (synchronises).
 * pos, seg, unit: host [resident] (any may be NULL).  The values are read from
 * the device metadata, not from the host state. */
int a2t_read_layout(a2t_cache* c, int32_t stream, int32_t* pos, uint8_t* seg, int32_t* unit);

/* The device-computed result of the stream's last eviction that removed rows
 * (synchronises).  n_pre: rows before it.  mask: host [n_pre], 1 = evicted.
 * new_slot: host [n_pre], survivor index or -1.  Either array may be NULL.
 * Returns A2T_ERR_STATE if the stream never evicted. */
int a2t_read_last_evict(a2t_cache* c, int32_t stream, int32_t* n_pre, uint8_t* mask,
                        int32_t* new_slot);

/* Copy one layer's resident K (rotated) and V of a stream to host in cache
 * order (synchronises).  k, v: host [resident][Hkv][D] in the cache dtype. */
int a2t_read_kv(a2t_cache* c, int32_t layer, int32_t stream, void* k, void* v);

/* Wait for all work enqueued by this cache.  Reports device faults. */
int a2t_sync(a2t_cache* c);

/* Kernel timing with HIP events on the cache's stream (for benchmarks).
 * kernel_filter: NULL disables timing; "" times every kernel; otherwise only
 * kernels whose name contains the string ("step_meta", "append",
 * "attn_tile", "attn_valu", "attn_merge", "evict").  While enabled, each
 * matching launch carries a start/stop event pair recorded at the dispatch's
 * own begin and end.  a2t_kernel_time waits for the
 * stream, then reports for the kernels whose name contains `kernel` the
 * number of launches and their summed duration in milliseconds since the
 * last report, and resets those counters. */
int a2t_profile_enable(a2t_cache* c, const char* kernel_filter);
int a2t_kernel_time(a2t_cache* c, const char* kernel, int64_t* launches, double* total_ms);
/* Creates start/stop event pairs ahead of time so that the next n_launches
 * timed dispatches take them from a pool instead of creating events (or
 * collecting finished ones) while the work is being issued.  The pool is
 * freed with the cache.  Errors: INVALID (n_launches < 0), NODEV, OOM (event
 * creation failed; the pairs created so far stay in the pool). */
int a2t_profile_reserve(a2t_cache* c, int32_t n_launches);

/* Static strings. */
const char* a2t_status_str(int status);
int a2t_abi_version(void);

/* ---------------------------------------------------------------------------
 * Adaptation objective (Sec. 3.2): the training loss that teaches the side
 * channel while keeping native behaviour, on given logits.
 *
 *   L = L_ASR + L_native + L_dec + L_turn (unit weights)
 *
 * Rows are prediction positions.  Student logits cover the extended vocabulary
 * (the teacher's `vocab` tokens followed by `n_added` added tokens); the
 * teacher's distribution over `vocab` is extended with zero probability on the
 * added tokens.  Per row, `kind`:
 *   A2T_ROW_ASR     a transcription token or delimiter: cross-entropy of the
 *                   student (temperature 1) against `target`; L_ASR is the mean
 *                   over these rows;
 *   A2T_ROW_NATIVE  a native prediction position aligned with the teacher:
 *                   T^2 KL(P_T || P_S) at temperature T; L_native is the mean
 *                   over these rows;
 *   A2T_ROW_NONE    no loss, zero gradient.
 * L_dec averages the native rows' divergences within each decision group
 * (`dec_group` 0 listen, 1 speak, 2 other; -1 not a unit's first decision) and
 * then over the groups present; L_turn does the same over `turn_group`
 * (1 turn end, 0 continuation, -1 none).
 * ------------------------------------------------------------------------- */
#define A2T_ROW_NONE 0
#define A2T_ROW_ASR 1
#define A2T_ROW_NATIVE 2

typedef struct a2t_distill a2t_distill;

/* Scratch for up to max_rows rows per call (per-row losses and weights, a
 * pinned staging area); the only allocating calls.  dtype: A2T_F32 or
 * A2T_BF16 for logits and gradient.  hip_stream: as for a2t_cache_create.
 * Errors: INVALID (sizes < 1, n_added < 0, dtype), OOM, HIP, NODEV. */
int a2t_distill_create(int32_t max_rows, int32_t vocab, int32_t n_added, int32_t dtype,
                       int32_t device, void* hip_stream, a2t_distill** out);
int a2t_distill_destroy(a2t_distill* d);

/* One evaluation over n_rows rows, asynchronous on the handle's stream.
 *   student         device [n_rows][student_stride], vocab + n_added logits per row
 *   teacher         device [n_rows][teacher_stride], vocab logits per row
 *                   (strides in elements, multiples of 8; pointers 16-byte aligned)
 *   kind, target, dec_group, turn_group
 *                   host [n_rows]; target in [0, vocab + n_added) on ASR rows
 *   temperature     T > 0 of the divergence (the paper uses 1)
 *   losses          device float[5] out: L_ASR, L_native, L_dec, L_turn, L
 *   grad            device [n_rows][student_stride] out, dL/d student logits in
 *                   the logits dtype, or NULL (loss only)
 * Host arrays are consumed before the call returns; device buffers must stay
 * valid until the stream reaches the work.  Errors: INVALID (n_rows out of
 * [1, max_rows], strides, alignment, kinds, groups, targets, T), HIP. */
int a2t_distill_loss(a2t_distill* d, int32_t n_rows, const void* student, int64_t student_stride,
                     const void* teacher, int64_t teacher_stride, const int8_t* kind,
                     const int32_t* target, const int8_t* dec_group, const int8_t* turn_group,
                     float temperature, float* losses, void* grad);

/* Timing of the per-row kernel (for benchmarks): with enable != 0 every later
 * a2t_distill_loss records start/stop events at that dispatch's own begin and
 * end; a2t_distill_kernel_time waits for them and reports the number of
 * timed launches and their summed duration in milliseconds since the last
 * report.  Errors: INVALID, HIP. */
int a2t_distill_profile_enable(a2t_distill* d, int32_t enable);
/* Creates event pairs for the next n_launches timed calls ahead of time (as
 * a2t_profile_reserve).  Errors: INVALID, OOM. */
int a2t_distill_profile_reserve(a2t_distill* d, int32_t n_launches);
int a2t_distill_kernel_time(a2t_distill* d, int64_t* launches, double* total_ms);

#ifdef __cplusplus
}
#endif

#endif /* A2T_H */
