// HIP kernels of libA2T for gfx950 (CDNA4, wave64).
//
//   step_meta   writes a step's row metadata into the stream's ring slots and
//               the step's rotary table (cos, sin of pos * theta^(-2i/D),
//               evaluated in fp64, stored fp32).
//   append      rotates the step's keys by their positions and stores K and V
//               rows into the ring (Sec. 3.3: keys keep their original rotary
//               positions; they are never re-encoded later).
//   attn_tile   causal chunk attention of a step's new rows over the resident
//               cache: 64-key tiles DMA'd into a 4-stage LDS ring, bf16 MFMA
//               16x16x32 for Q.K^T and P.V, online softmax with wave
//               shuffles, key splits for parallelism; also bf16 decode (one
//               query row per stream).
//   attn_valu   the same attention on the vector ALU, one query row per
//               workgroup column: fp32 caches (chunk and decode).
//   attn_merge  combines key-split partials (fixed order, deterministic): split
//               groups combined in LDS, or one thread per row walking every
//               split when a launch's streams have few splits.
//   evict       eviction and compaction (Sec. 3.3): a ballot/prefix-sum scan
//               over the passed-over ring rows keeps TEXT/RESPONSE/PREFIX rows
//               and drops ACOUSTIC/DELIM rows of evicted units, moves the kept
//               rows into the kept region in every layer, and writes the
//               eviction mask and compaction indices over the whole cache.
#include "a2t_internal.h"
#include "a2t.h"

#include <hip/hip_ext.h>
#include <math.h>

#include <mutex>
#include <type_traits>

namespace a2t {
namespace {

constexpr uint8_t kSegAcoustic = 1;
constexpr uint8_t kSegDelim = 2;

typedef __attribute__((__vector_size__(8 * sizeof(__bf16)))) __bf16 bf16x8;
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef _Float16 f16x8 __attribute__((ext_vector_type(8)));

struct bf16_t {
    uint16_t bits;
};

__device__ __forceinline__ float bf16_to_f32(uint16_t b) {
    return __uint_as_float((uint32_t)b << 16);
}
__device__ __forceinline__ uint16_t f32_to_bf16(float f) {
    uint32_t u = __float_as_uint(f);
    if ((u & 0x7fffffffu) > 0x7f800000u) return 0x7fc0;  // NaN
    u += 0x7fffu + ((u >> 16) & 1u);                       // round to nearest even
    return (uint16_t)(u >> 16);
}

template <typename T> struct Elt;
template <> struct Elt<float> {
    __device__ static float load(const float* p) { return *p; }
    __device__ static void store(float* p, float x) { *p = x; }
};
template <> struct Elt<bf16_t> {
    __device__ static float load(const bf16_t* p) { return bf16_to_f32(p->bits); }
    __device__ static void store(bf16_t* p, float x) { p->bits = f32_to_bf16(x); }
};

// Physical row of logical key j (cache order): kept region first, then the ring.
__device__ __forceinline__ int64_t key_row(const DevState& st, int layer, int s, int g, int kept,
                                           int head, int j, bool* in_kept) {
    if (j < kept) {
        *in_kept = true;
        return pool_index(st, layer, s, g, st.kept_rows, j);
    }
    int slot = head + (j - kept);
    if (slot >= st.unit_rows) slot -= st.unit_rows;
    *in_kept = false;
    return pool_index(st, layer, s, g, st.unit_rows, slot);
}

// 8 consecutive elements <-> fp32, with one or two 16-byte accesses.
__device__ __forceinline__ void load8(const float* p, float x[8]) {
    const float4 a = reinterpret_cast<const float4*>(p)[0];
    const float4 b = reinterpret_cast<const float4*>(p)[1];
    x[0] = a.x; x[1] = a.y; x[2] = a.z; x[3] = a.w;
    x[4] = b.x; x[5] = b.y; x[6] = b.z; x[7] = b.w;
}
__device__ __forceinline__ void load8(const bf16_t* p, float x[8]) {
    const uint4 r = *reinterpret_cast<const uint4*>(p);
    const uint32_t w[4] = {r.x, r.y, r.z, r.w};
#pragma unroll
    for (int e = 0; e < 4; ++e) {
        x[2 * e] = __uint_as_float(w[e] << 16);
        x[2 * e + 1] = __uint_as_float(w[e] & 0xffff0000u);
    }
}
__device__ __forceinline__ void store8(float* p, const float x[8]) {
    reinterpret_cast<float4*>(p)[0] = make_float4(x[0], x[1], x[2], x[3]);
    reinterpret_cast<float4*>(p)[1] = make_float4(x[4], x[5], x[6], x[7]);
}
__device__ __forceinline__ void store8(bf16_t* p, const float x[8]) {
    uint32_t w[4];
#pragma unroll
    for (int e = 0; e < 4; ++e)
        w[e] = (uint32_t)f32_to_bf16(x[2 * e]) | ((uint32_t)f32_to_bf16(x[2 * e + 1]) << 16);
    *reinterpret_cast<uint4*>(p) = make_uint4(w[0], w[1], w[2], w[3]);
}
__device__ __forceinline__ void copy8(float* d, const float* s) {
    reinterpret_cast<float4*>(d)[0] = reinterpret_cast<const float4*>(s)[0];
    reinterpret_cast<float4*>(d)[1] = reinterpret_cast<const float4*>(s)[1];
}
__device__ __forceinline__ void copy8(bf16_t* d, const bf16_t* s) {
    *reinterpret_cast<uint4*>(d) = *reinterpret_cast<const uint4*>(s);
}

// ------------------------------------------------------------------ step_meta
// grid (row, stream): one workgroup per new row, one thread per rotary pair.
template <class BT>
__global__ __launch_bounds__(64) void step_meta_kernel(DevState st, BT b,
                                                       const uint8_t* seg, const int32_t* pos,
                                                       const int32_t* uid) {
    const StepDesc d = b.d[blockIdx.y];
    const int r = blockIdx.x;
    if (r >= d.n) return;
    const int p = pos[d.row0 + r];
    const int half = st.D / 2;
    if (threadIdx.x == 0) {
        int slot = d.slot0 + r;
        if (slot >= st.unit_rows) slot -= st.unit_rows;
        const int64_t mb = (int64_t)d.s * st.unit_rows;
        st.unit_pos[mb + slot] = p;
        st.unit_seg[mb + slot] = seg[d.row0 + r];
        st.unit_uid[mb + slot] = uid[blockIdx.y];
    }
    const int i = threadIdx.x;
    if (i < half) {
        const double inv = pow(st.theta, (-2.0 * i) / st.D);
        double sn, cs;
        sincos((double)p * inv, &sn, &cs);
        st.rope[((int64_t)d.s * st.max_step_rows + r) * half + i] = make_float2((float)cs, (float)sn);
    }
}

// --------------------------------------------------------------------- append
// One thread per 8-element chunk of a new row (all heads, all rows of the
// batch); every thread issues its loads at once, then writes its chunk.
template <typename T, class BT>
__global__ __launch_bounds__(256) void append_kernel(DevState st, BT b, const T* k,
                                                     const T* v) {
    const AppendDesc d = b.d[blockIdx.y];
    const int D = st.D, half = D / 2, Hkv = st.Hkv;
    const int cph = D / 8;              // chunks per head row
    const int cpr = Hkv * cph;          // chunks per row
    const int q = blockIdx.x * blockDim.x + threadIdx.x;
    const int r = q / cpr;
    if (r >= d.n) return;
    const int c = q - r * cpr;
    const int g = c / cph, d0 = (c - g * cph) * 8;
    const int layer = b.layer0 + blockIdx.z;
    int slot = d.slot0 + r;
    if (slot >= st.unit_rows) slot -= st.unit_rows;
    const int64_t in = ((int64_t)blockIdx.z * b.total_rows + d.in_row0 + r) * Hkv * D + g * D;
    const bool lower = d0 < half;
    const int i0 = lower ? d0 : d0 - half;
    const float4* cs4 = reinterpret_cast<const float4*>(
        st.rope + ((int64_t)d.s * st.max_step_rows + r) * half + i0);
    float x[8], y[8];
    load8(k + in + d0, x);
    load8(k + in + (lower ? d0 + half : d0 - half), y);
    float4 cs[4];
#pragma unroll
    for (int e = 0; e < 4; ++e) cs[e] = cs4[e];
    const int64_t o = pool_index(st, layer, d.s, g, st.unit_rows, slot) + d0;
    copy8(reinterpret_cast<T*>(st.v_unit) + o, v + in + d0);
    float out[8];
#pragma unroll
    for (int e = 0; e < 4; ++e) {
        // cs[e] = (cos, sin) of pairs i0+2e and i0+2e+1
        const float c0 = cs[e].x, s0 = cs[e].y, c1 = cs[e].z, s1 = cs[e].w;
        if (lower) {
            out[2 * e] = x[2 * e] * c0 - y[2 * e] * s0;
            out[2 * e + 1] = x[2 * e + 1] * c1 - y[2 * e + 1] * s1;
        } else {
            out[2 * e] = x[2 * e] * c0 + y[2 * e] * s0;
            out[2 * e + 1] = x[2 * e + 1] * c1 + y[2 * e + 1] * s1;
        }
    }
    store8(reinterpret_cast<T*>(st.k_unit) + o, out);
}

// ----------------------------------------------------------------- attn_valu
// One workgroup = (key split, kv head g, query row i, stream).  256 threads
// form 16 key groups of 16 lanes; a lane holds D/16 consecutive elements of a
// row.  Scores are reduced across the 16 lanes with xor shuffles; every key
// group runs its own online softmax, and the 16 states are merged in LDS.
template <typename T, int D, int G, class BT>
__global__ __launch_bounds__(256) void attn_valu_kernel(DevState st, BT b, const T* q,
                                                        T* o) {
    constexpr int DPL = D / 16;
    __shared__ float s_m[16], s_l[16];
    __shared__ float s_acc[16][D];

    const AttnDesc d = b.d[blockIdx.z];
    const int sp = blockIdx.x;
    const int g = blockIdx.y / b.max_rows, i = blockIdx.y - g * b.max_rows;
    if (sp >= d.splits || i >= d.n_q) return;
    const int tid = threadIdx.x, l16 = tid & 15, kg = tid >> 4;
    const int d0 = l16 * DPL;
    const int lim = d.R - d.n_q + i + 1;  // keys 0 .. lim-1 are visible
    const int n_tiles = (d.R + kTileKeys - 1) / kTileKeys;
    const int t0 = sp * n_tiles / d.splits, t1 = (sp + 1) * n_tiles / d.splits;
    const int kb = t0 * kTileKeys;
    const int ke = min(lim, t1 * kTileKeys);

    float qf[G][DPL];
    const float2* cs = st.rope + ((int64_t)d.s * st.max_step_rows + d.rope_row0 + i) * (D / 2);
#pragma unroll
    for (int hh = 0; hh < G; ++hh) {
        const T* qp = q + ((int64_t)(d.q_row0 + i) * st.Hq + g * G + hh) * D;
#pragma unroll
        for (int e = 0; e < DPL; ++e) {
            const int dd = d0 + e;
            float r;
            if (dd < D / 2) {
                const float2 c = cs[dd];
                r = Elt<T>::load(qp + dd) * c.x - Elt<T>::load(qp + dd + D / 2) * c.y;
            } else {
                const float2 c = cs[dd - D / 2];
                r = Elt<T>::load(qp + dd) * c.x + Elt<T>::load(qp + dd - D / 2) * c.y;
            }
            qf[hh][e] = r * st.scale_log2e;
        }
    }

    float m[G], l[G], acc[G][DPL];
#pragma unroll
    for (int hh = 0; hh < G; ++hh) {
        m[hh] = -INFINITY;
        l[hh] = 0.f;
#pragma unroll
        for (int e = 0; e < DPL; ++e) acc[hh][e] = 0.f;
    }
    const T* kbase_k = reinterpret_cast<const T*>(st.k_kept);
    const T* kbase_v = reinterpret_cast<const T*>(st.v_kept);
    const T* ubase_k = reinterpret_cast<const T*>(st.k_unit);
    const T* ubase_v = reinterpret_cast<const T*>(st.v_unit);

    for (int j = kb + kg; j < ke; j += 16) {
        bool in_kept;
        const int64_t row = key_row(st, b.layer, d.s, g, d.kept, d.head, j, &in_kept);
        const T* kp = (in_kept ? kbase_k : ubase_k) + row + d0;
        const T* vp = (in_kept ? kbase_v : ubase_v) + row + d0;
        float kv[DPL], vv[DPL];
#pragma unroll
        for (int e = 0; e < DPL; ++e) {
            kv[e] = Elt<T>::load(kp + e);
            vv[e] = Elt<T>::load(vp + e);
        }
#pragma unroll
        for (int hh = 0; hh < G; ++hh) {
            float s = 0.f;
#pragma unroll
            for (int e = 0; e < DPL; ++e) s += qf[hh][e] * kv[e];
            s += __shfl_xor(s, 8, 16);
            s += __shfl_xor(s, 4, 16);
            s += __shfl_xor(s, 2, 16);
            s += __shfl_xor(s, 1, 16);
            const float mn = fmaxf(m[hh], s);
            const float corr = exp2f(m[hh] - mn);
            const float p = exp2f(s - mn);
            l[hh] = l[hh] * corr + p;
#pragma unroll
            for (int e = 0; e < DPL; ++e) acc[hh][e] = acc[hh][e] * corr + p * vv[e];
            m[hh] = mn;
        }
    }

    // merge the 16 key groups, one query head at a time
    const int Mrows = G * d.n_q;
#pragma unroll
    for (int hh = 0; hh < G; ++hh) {
#pragma unroll
        for (int e = 0; e < DPL; ++e) s_acc[kg][d0 + e] = acc[hh][e];
        if (l16 == 0) {
            s_m[kg] = m[hh];
            s_l[kg] = l[hh];
        }
        __syncthreads();
        for (int dd = tid; dd < D; dd += blockDim.x) {
            float mx = -INFINITY;
#pragma unroll
            for (int k = 0; k < 16; ++k) mx = fmaxf(mx, s_m[k]);
            float L = 0.f, O = 0.f;
            if (mx != -INFINITY) {
#pragma unroll
                for (int k = 0; k < 16; ++k) {
                    const float w = exp2f(s_m[k] - mx);
                    L += w * s_l[k];
                    O += w * s_acc[k][dd];
                }
            }
            const int mrow = i * G + hh;
            if (d.splits == 1) {
                Elt<T>::store(o + ((int64_t)(d.q_row0 + i) * st.Hq + g * G + hh) * D + dd, O / L);
            } else {
                float* po = st.ws + d.ws_off;
                po[(((int64_t)sp * st.Hkv + g) * Mrows + mrow) * D + dd] = O;
                if (dd == 0) {
                    float* pml = po + (int64_t)d.splits * st.Hkv * Mrows * D;
                    pml[(((int64_t)sp * st.Hkv + g) * Mrows + mrow) * 2 + 0] = mx;
                    pml[(((int64_t)sp * st.Hkv + g) * Mrows + mrow) * 2 + 1] = L;
                }
            }
        }
        __syncthreads();
    }
}

// ----------------------------------------------------------------- attn_tile
// One workgroup = (key split, kv head g, stream), 8 waves.  The M = G*n_q
// query rows of the head group are processed 128 at a time; each wave owns 16
// of them.
//
// S^T = K . Q^T with mfma_f32_16x16x32_bf16: A = K rows (16 keys x 32 dims),
// B = Q^T (32 dims x 16 queries); the accumulator gives lane l the scores of
// keys 4*(l/16)+e, e<4, for query l%16.  P^T then feeds P.V directly as the
// B operand of O^T = V^T . P^T: within a 32-key chunk, k-slot 8*(l/16)+j maps
// to key 16*(j/4) + 4*(l/16) + j%4, which is exactly what lane l holds; the A
// operand reads the same keys of V.  No cross-lane transposes of P.
constexpr int kMfmaThreads = 512;

__device__ __forceinline__ uint32_t pack_bf16x2(float a, float b) {
    typedef __attribute__((__vector_size__(2 * sizeof(__bf16)))) __bf16 bf16x2;
    const bf16x2 v = {(__bf16)a, (__bf16)b};   // v_cvt_pk_bf16_f32, round to nearest even
    return __builtin_bit_cast(uint32_t, v);
}

// max / sum over the four lanes l, l^16, l^32, l^48 (the lanes holding one
// query column of a 16x16 accumulator), with the gfx950 row-swap permutes
__device__ __forceinline__ uint32_t pack_f16x2(float a, float b) {
    return (uint32_t)__builtin_bit_cast(uint16_t, (_Float16)a) |
           ((uint32_t)__builtin_bit_cast(uint16_t, (_Float16)b) << 16);
}
__device__ __forceinline__ float quad_max(float x) {
    const auto a = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x), false, false);
    x = fmaxf(__uint_as_float(a[0]), __uint_as_float(a[1]));
    const auto b = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
    return fmaxf(__uint_as_float(b[0]), __uint_as_float(b[1]));
}
__device__ __forceinline__ float quad_sum(float x) {
    const auto a = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x), false, false);
    x = __uint_as_float(a[0]) + __uint_as_float(a[1]);
    const auto b = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
    return __uint_as_float(b[0]) + __uint_as_float(b[1]);
}

// Tiles of 64 keys go from HBM straight into a 4-stage LDS ring
// (global_load_lds, 16 bytes per lane, no staging registers), so three tiles
// are in flight while one is computed.  Lane j of a DMA instruction fills LDS bytes [16j, 16j+16)
// of its 1 KiB block; the lane's source address picks which logical 16-byte
// chunk lands there, which implements the bank-conflict swizzles:
//   K: physical chunk = logical ^ (row & (CPR-1))   (Q.K^T reads 16 rows of one chunk)
//   V: physical chunk = logical ^ 2 (row & (CPR/2-1))  (transposed reads of 16 rows x 32 B)
// V stays row-major; the P.V operand (8 keys of one dim per lane) is read with
// two ds_read_b64_tr_b16: within each 16-lane group, result lane 4a+b element
// r is element b of the 8 bytes addressed by source lane a+4r.  Waits are
// explicit: before the barrier that publishes tile t each wave waits until
// only its DMAs of later tiles are outstanding.
constexpr int kTileStages = 4;

template <int D>
struct TileBuf {
    uint16_t k[kTileKeys * D];
    uint16_t v[kTileKeys * D];
};

typedef short short4_t __attribute__((ext_vector_type(4)));

// s_waitcnt vmcnt(N) with expcnt and lgkmcnt left alone (gfx9 encoding)
template <int N>
__device__ __forceinline__ void wait_vmem() {
    static_assert(N >= 0 && N < 64, "vmcnt range");
    __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | (7 << 4) | (15 << 8));
}
// workgroup barrier that the compiler may not move memory accesses across; no
// memory fence (the waits that make DMA'd data visible are explicit)
__device__ __forceinline__ void barrier_only() {
    asm volatile("" ::: "memory");
    __builtin_amdgcn_s_barrier();
    asm volatile("" ::: "memory");
}
__device__ __forceinline__ void dma16(const void* src, uint16_t* lds) {
    __builtin_amdgcn_global_load_lds(src, (__attribute__((address_space(3))) void*)lds, 16, 0, 0);
}
__device__ __forceinline__ uint32_t lds_addr(const void* p) {
    return (uint32_t)(uintptr_t)(const __attribute__((address_space(3))) void*)(p);
}
// Transposed LDS read issued as inline assembly: the compiler cannot tell which
// LDS the builtin form reads and would wait for every outstanding DMA before
// it.  The result is valid only after lds_wait_all() names it.
template <int OFF>
__device__ __forceinline__ uint2 lds_tr16_issue(uint32_t addr) {
    uint2 r;
    asm volatile("ds_read_b64_tr_b16 %0, %1 offset:%2" : "=v"(r) : "v"(addr), "i"(OFF));
    return r;
}
// s_waitcnt lgkmcnt(0) that the listed values depend on
__device__ __forceinline__ void lds_wait_all(uint2 (&a)[8], uint2 (&b)[8]) {
    asm volatile("s_waitcnt lgkmcnt(0)"
                 : "+v"(a[0]), "+v"(a[1]), "+v"(a[2]), "+v"(a[3]), "+v"(a[4]), "+v"(a[5]), "+v"(a[6]),
                   "+v"(a[7]), "+v"(b[0]), "+v"(b[1]), "+v"(b[2]), "+v"(b[3]), "+v"(b[4]), "+v"(b[5]),
                   "+v"(b[6]), "+v"(b[7]));
}
__device__ __forceinline__ void lds_wait_all(uint2 (&a)[4], uint2 (&b)[4]) {
    asm volatile("s_waitcnt lgkmcnt(0)"
                 : "+v"(a[0]), "+v"(a[1]), "+v"(a[2]), "+v"(a[3]), "+v"(b[0]), "+v"(b[1]), "+v"(b[2]),
                   "+v"(b[3]));
}

// 16-byte LDS read issued as inline assembly (the compiler keeps only a few
// in flight and waits after each pair); valid only after k_wait() names it
template <int OFF>
__device__ __forceinline__ u32x4 lds_b128_issue(uint32_t addr) {
    u32x4 r;
    asm volatile("ds_read_b128 %0, %1 offset:%2" : "=v"(r) : "v"(addr), "i"(OFF));
    return r;
}
// s_waitcnt lgkmcnt(N) that the listed K operands depend on: LDS reads
// complete in order, so with N reads issued after them these are complete
template <int N>
__device__ __forceinline__ void k_wait(u32x4 (&a)[4], u32x4 (&b)[4]);
template <>
__device__ __forceinline__ void k_wait<8>(u32x4 (&a)[4], u32x4 (&b)[4]) {
    asm volatile("s_waitcnt lgkmcnt(8)"
                 : "+v"(a[0]), "+v"(a[1]), "+v"(a[2]), "+v"(a[3]), "+v"(b[0]), "+v"(b[1]), "+v"(b[2]), "+v"(b[3]));
}
template <>
__device__ __forceinline__ void k_wait<0>(u32x4 (&a)[4], u32x4 (&b)[4]) {
    asm volatile("s_waitcnt lgkmcnt(0)"
                 : "+v"(a[0]), "+v"(a[1]), "+v"(a[2]), "+v"(a[3]), "+v"(b[0]), "+v"(b[1]), "+v"(b[2]), "+v"(b[3]));
}
// 16-byte global load issued as inline assembly, so the compiler does not
// place its own wait (it would wait for every DMA issued after it).  The
// result is valid only after q_wait() names it.
template <int OFF>
__device__ __forceinline__ u32x4 gload16_issue(const void* p) {
    u32x4 r;
    asm volatile("global_load_dwordx4 %0, %1, off offset:%2" : "=v"(r) : "v"(p), "i"(OFF) : "memory");
    return r;
}
// s_waitcnt vmcnt(first three tiles' DMAs) that the listed Q and rotary
// values depend on: the asm-issued loads before those DMAs are complete
__device__ __forceinline__ void q_wait(u32x4 (&a)[4], u32x4 (&b)[8]) {
    asm volatile("s_waitcnt vmcnt(12)"
                 : "+v"(a[0]), "+v"(a[1]), "+v"(a[2]), "+v"(a[3]), "+v"(b[0]), "+v"(b[1]), "+v"(b[2]),
                   "+v"(b[3]), "+v"(b[4]), "+v"(b[5]), "+v"(b[6]), "+v"(b[7])
                 :
                 : "memory");
}
__device__ __forceinline__ void q_wait(u32x4 (&a)[2], u32x4 (&b)[4]) {
    asm volatile("s_waitcnt vmcnt(6)"
                 : "+v"(a[0]), "+v"(a[1]), "+v"(b[0]), "+v"(b[1]), "+v"(b[2]), "+v"(b[3])
                 :
                 : "memory");
}
// qraw[s] = the 16 bytes at qb + 64 s; cs[4 s + e] = the 16 bytes at cb + 256 s + 16 e,
// issued in the order qraw[0], cs[0..3], qraw[1], cs[4..7], ...
template <int S, int E>
struct QLoad {
    template <int KS, int NC>
    static __device__ __forceinline__ void run(u32x4 (&qraw)[KS], u32x4 (&cs)[NC], const char* qb,
                                               const char* cb) {
        if constexpr (E == 0 && S < KS) qraw[S] = gload16_issue<64 * S>(qb);
        if constexpr (S < KS / 2) {
            cs[4 * S + E] = gload16_issue<256 * S + 16 * E>(cb);
            if constexpr (E < 3)
                QLoad<S, E + 1>::run(qraw, cs, qb, cb);
            else
                QLoad<S + 1, 0>::run(qraw, cs, qb, cb);
        } else if constexpr (S < KS) {
            QLoad<S + 1, 0>::run(qraw, cs, qb, cb);
        }
    }
};

template <int D, class BT>
__global__ __launch_bounds__(kMfmaThreads) void attn_tile_kernel(DevState st, BT b,
                                                                 const uint16_t* q, uint16_t* o,
                                                                 const uint16_t* k_in,
                                                                 const uint16_t* v_in) {
    constexpr int KS = D / 32;                  // k-steps of Q.K^T
    constexpr int DB = D / 16;                  // 16-dim blocks of O
    constexpr int CPR = D / 8;                  // 16-byte chunks per row
    constexpr int RPB = 512 / D;                // rows per 1 KiB DMA block
    constexpr int OPS = kTileKeys / RPB / 8;    // K (and V) DMA blocks per wave per tile
    constexpr int OPT = 2 * OPS;                // DMA instructions per wave per tile
    constexpr int QPW = 16;
    constexpr int QPP = QPW * (kMfmaThreads / 64);
    static_assert(OPS >= 1 && RPB * CPR == 64, "tile shape");
    __shared__ TileBuf<D> ring[kTileStages];

    const AttnDesc d = b.d[blockIdx.z];
    // workgroup (split sp, KV head g) is linear block sp * Hkv + g: the dispatcher
    // deals consecutive workgroups to the 8 XCDs in turn, so with 8 KV heads all
    // splits of head g run on one XCD and share its L2, where the head's Q and
    // rotary rows are fetched once instead of once per XCD (any other head
    // count gives the same results, only without that sharing)
    const int g = blockIdx.x % st.Hkv, sp = blockIdx.x / st.Hkv;
    // request every descriptor and shape field the prologue uses at once: a
    // branch on one field before the others are requested costs one
    // kernel-argument load latency per level
    asm volatile("" ::"s"(d.s), "s"(d.kept), "s"(d.head), "s"(d.R), "s"(d.n_q), "s"(d.q_row0),
                 "s"(d.rope_row0), "s"(d.splits), "s"(d.n_new), "s"(d.in_row0), "s"(d.tile_q),
                 "s"(d.tile_r));
    asm volatile("" ::"s"(st.G), "s"(st.Hq), "s"(st.Hkv), "s"(st.S), "s"(st.unit_rows),
                 "s"(st.kept_rows), "s"(st.max_step_rows), "s"(b.layer), "s"(st.k_kept),
                 "s"(st.v_kept), "s"(st.k_unit), "s"(st.v_unit), "s"(st.rope));
    asm volatile("" ::"s"(q), "s"(k_in), "s"(v_in), "s"(st.scale_log2e), "s"(st.ws), "s"(d.ws_off));
    if (sp >= d.splits) return;
    const int G = st.G, nq = d.n_q, M = G * nq, R = d.R;
    const int tid = threadIdx.x, w = tid >> 6, lane = tid & 63, l16 = lane & 15, lg = lane >> 4;
    // split sp takes tile_q tiles, one more if sp < r; the last m splits take one
    // tile each (r = tile_r & 0xffff, m = tile_r >> 16)
    const int r1 = d.tile_r & 0xffff, cut = d.splits - (d.tile_r >> 16);
    const int t0 = sp < cut ? sp * d.tile_q + min(sp, r1) : cut * d.tile_q + min(cut, r1) + (sp - cut);
    const int t1 = sp < cut ? t0 + d.tile_q + (sp < r1 ? 1 : 0) : t0 + 1;
    const int vis0 = R - nq;
    const int kept = d.kept, head = d.head, ring_rows = st.unit_rows;
    const int newbase = R - d.n_new;  // fused append: rows newbase .. R-1 come from k_in / v_in

    const uint16_t* kk = reinterpret_cast<const uint16_t*>(st.k_kept) +
                         pool_index(st, b.layer, d.s, g, st.kept_rows, 0);
    const uint16_t* vk = reinterpret_cast<const uint16_t*>(st.v_kept) +
                         pool_index(st, b.layer, d.s, g, st.kept_rows, 0);
    uint16_t* ku = reinterpret_cast<uint16_t*>(st.k_unit) +
                   pool_index(st, b.layer, d.s, g, st.unit_rows, 0);
    uint16_t* vu = reinterpret_cast<uint16_t*>(st.v_unit) +
                   pool_index(st, b.layer, d.s, g, st.unit_rows, 0);
    auto row_off = [&](int j, bool* in_kept) -> int {
        if (j < kept) {
            *in_kept = true;
            return j * D;
        }
        int slot = head + (j - kept);
        if (slot >= ring_rows) slot -= ring_rows;
        *in_kept = false;
        return slot * D;
    };
    // element offset of a tile's row 0 when the whole tile is one contiguous
    // run of resident rows without new rows (else -1)
    auto fast_base = [&](int kb, bool* kept_region) -> int {
        if (kb + kTileKeys > newbase) return -1;
        if (kb + kTileKeys <= kept) {
            *kept_region = true;
            return kb * D;
        }
        if (kb < kept) return -1;
        int slot = head + (kb - kept);
        if (slot >= ring_rows) slot -= ring_rows;
        if (slot + kTileKeys > ring_rows) return -1;
        *kept_region = false;
        return slot * D;
    };
    // this lane's DMA slots: block w*OPS+i holds tile rows (w*OPS+i)*RPB .. +RPB-1;
    // lane j fills physical chunk j % CPR of row j / CPR of its block
    uint32_t kofs[OPS], vofs[OPS];  // byte offsets inside a contiguous tile (fast path)
#pragma unroll
    for (int i = 0; i < OPS; ++i) {
        const int pr = (w * OPS + i) * RPB + lane / CPR, pc = lane % CPR;
        kofs[i] = (uint32_t)(pr * D + (pc ^ (pr & (CPR - 1))) * 8) * 2u;
        vofs[i] = (uint32_t)(pr * D + (pc ^ (2 * (pr & (CPR / 2 - 1)))) * 8) * 2u;
    }
    auto src_of = [&](const uint16_t* reg_kept, const uint16_t* reg_ring, const uint16_t* in,
                      int j, int ch) -> const uint16_t* {
        j = j < R ? j : R - 1;  // rows past R read row R-1: masked keys, zero weight
        if (j >= newbase) return in + ((int64_t)(d.in_row0 + (j - newbase)) * st.Hkv + g) * D + ch * 8;
        bool ik;
        const int off = row_off(j, &ik);
        return (ik ? reg_kept : reg_ring) + off + ch * 8;
    };
    // DMAs write LDS only, so the two paths need not share registers: the fast
    // path is a scalar tile base plus 32-bit lane offsets
    auto issue = [&](int t, TileBuf<D>& buf) {
        // opaque tile index: the prologue's issues sit in the query-pass loop, and
        // hoisted out of it their general-path addresses would be computed
        // unconditionally
        asm volatile("" : "+s"(t));
        const int kb = t * kTileKeys;
        bool in_kept = false;
        const int fb = fast_base(kb, &in_kept);
        if (fb >= 0) {
            const char* kf = reinterpret_cast<const char*>((in_kept ? kk : ku) + fb);
            const char* vf = reinterpret_cast<const char*>((in_kept ? vk : vu) + fb);
#pragma unroll
            for (int i = 0; i < OPS; ++i) {
                dma16(kf + kofs[i], &buf.k[(w * OPS + i) * 512]);
                dma16(vf + vofs[i], &buf.v[(w * OPS + i) * 512]);
            }
        } else {
#pragma unroll
            for (int i = 0; i < OPS; ++i) {
                const int pr = (w * OPS + i) * RPB + lane / CPR, pc = lane % CPR;
                dma16(src_of(kk, ku, k_in, kb + pr, pc ^ (pr & (CPR - 1))), &buf.k[(w * OPS + i) * 512]);
                dma16(src_of(vk, vu, v_in, kb + pr, pc ^ (2 * (pr & (CPR / 2 - 1)))),
                      &buf.v[(w * OPS + i) * 512]);
            }
            // keeps the two paths' DMAs apart: merged into one, they would
            // compute the general path's per-lane addresses for every tile
            asm volatile("" ::: "memory");
        }
    };
    // a tile index past the range issues the same number of DMAs, all lanes
    // reading the first 16 bytes of the kept region into the (unused) stage, so
    // every path has the same count of outstanding loads
    auto issue_or_dummy = [&](int t, TileBuf<D>& buf) {
        if (t < t1) {
            issue(t, buf);
        } else {
#pragma unroll
            for (int i = 0; i < OPS; ++i) {
                dma16(kk, &buf.k[(w * OPS + i) * 512]);
                dma16(kk, &buf.v[(w * OPS + i) * 512]);
            }
        }
    };
    // fused append on a tile holding the step's rows: rotate their keys in LDS
    // (rotate-half partner = logical chunk ^ CPR/2 of the same row) and store
    // K and V rows to their ring slots.  Every wave calls it (barriers inside).
    auto fixup = [&](int t, TileBuf<D>& buf) {
        const int kb = t * kTileKeys;
        constexpr int PER = kTileKeys * CPR / kMfmaThreads;
#pragma unroll 1
        for (int e = 0; e < PER; ++e) {
            const int idx = tid + kMfmaThreads * e, r = idx / CPR, c = idx % CPR, j = kb + r;
            const bool mine = j >= newbase && j < R;
            uint4 rot = make_uint4(0, 0, 0, 0), vv = rot;
            if (mine) {
                const uint4 kv = *reinterpret_cast<const uint4*>(&buf.k[r * D + (c ^ (r & (CPR - 1))) * 8]);
                const int cp = c ^ (CPR / 2);
                const uint4 pv = *reinterpret_cast<const uint4*>(&buf.k[r * D + (cp ^ (r & (CPR - 1))) * 8]);
                vv = *reinterpret_cast<const uint4*>(&buf.v[r * D + (c ^ (2 * (r & (CPR / 2 - 1)))) * 8]);
                const int d0 = c * 8;
                const bool lower = d0 < D / 2;
                const int i0 = lower ? d0 : d0 - D / 2;
                const float4* cs4 = reinterpret_cast<const float4*>(
                    st.rope + ((int64_t)d.s * st.max_step_rows + (j - newbase)) * (D / 2) + i0);
                const uint32_t xw[4] = {kv.x, kv.y, kv.z, kv.w};
                const uint32_t yw[4] = {pv.x, pv.y, pv.z, pv.w};
                uint32_t ow[4];
#pragma unroll
                for (int e2 = 0; e2 < 4; ++e2) {
                    const float4 c4 = cs4[e2];
                    const float x0 = __uint_as_float(xw[e2] << 16), x1 = __uint_as_float(xw[e2] & 0xffff0000u);
                    const float y0 = __uint_as_float(yw[e2] << 16), y1 = __uint_as_float(yw[e2] & 0xffff0000u);
                    const float r0 = lower ? x0 * c4.x - y0 * c4.y : x0 * c4.x + y0 * c4.y;
                    const float r1 = lower ? x1 * c4.z - y1 * c4.w : x1 * c4.z + y1 * c4.w;
                    ow[e2] = pack_bf16x2(r0, r1);
                }
                rot = make_uint4(ow[0], ow[1], ow[2], ow[3]);
            }
            __syncthreads();  // every partner chunk of this pass was read before any is overwritten
            if (mine) {
                *reinterpret_cast<uint4*>(&buf.k[r * D + (c ^ (r & (CPR - 1))) * 8]) = rot;
                bool ik;
                const int off = row_off(j, &ik);
                *reinterpret_cast<uint4*>(ku + off + c * 8) = rot;
                *reinterpret_cast<uint4*>(vu + off + c * 8) = vv;
            }
            __syncthreads();  // rotated keys visible; the stores are done before later waits count
        }
    };

    const float2* rope = st.rope + ((int64_t)d.s * st.max_step_rows + d.rope_row0) * (D / 2);

    for (int qg0 = 0; qg0 < M; qg0 += QPP) {
        const int mw = qg0 + QPW * w;
        const bool active = mw < M;
        const int mq = mw + l16;

        // load order: Q and its rotary rows, then the first three tiles, all
        // before any wait (compiler barriers keep the order).  Q heads the
        // memory queue, so it is rotated while the tiles stream in; every
        // wave's requests go out in tile order, so tile t0 of every workgroup
        // tends to arrive first and its compute overlaps the later tiles'
        // transfer.  Unconditional loads (rows past M read row M-1 and are
        // zeroed below): a branch here would merge loaded registers and force
        // an early wait.
        u32x4 qraw[KS];
        u32x4 csr[KS / 2 * 4];
        {
            const int mqc = mq < M ? mq : M - 1;
            const int i = mqc / G, hh = mqc - i * G;
            const uint16_t* qp = q + ((int64_t)(d.q_row0 + i) * st.Hq + g * G + hh) * D;
            const float2* cp = rope + (int64_t)i * (D / 2);
            QLoad<0, 0>::run(qraw, csr, reinterpret_cast<const char*>(qp + 8 * lg),
                             reinterpret_cast<const char*>(cp + 8 * lg));
        }
        asm volatile("" ::: "memory");
        issue_or_dummy(t0, ring[0]);
        issue_or_dummy(t0 + 1, ring[1]);
        issue_or_dummy(t0 + 2, ring[2]);
        static_assert(OPT == KS, "q_wait counts three tiles of DMAs: 12 at head dim 128, 6 at 64");
        q_wait(qraw, csr);
        float4 cs[KS / 2][4];
#pragma unroll
        for (int s = 0; s < KS / 2; ++s)
#pragma unroll
            for (int e2 = 0; e2 < 4; ++e2) cs[s][e2] = __builtin_bit_cast(float4, csr[4 * s + e2]);

        // Q^T operand: rotated, scaled by scale*log2(e), bf16
        bf16x8 qop[KS];
        {
            float x[KS][8];
            const float qs = mq < M ? st.scale_log2e : 0.f;
#pragma unroll
            for (int s = 0; s < KS; ++s) {
                const uint32_t rw[4] = {qraw[s][0], qraw[s][1], qraw[s][2], qraw[s][3]};
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    x[s][2 * e] = __uint_as_float(rw[e] << 16);
                    x[s][2 * e + 1] = __uint_as_float(rw[e] & 0xffff0000u);
                }
            }
#pragma unroll
            for (int s = 0; s < KS / 2; ++s) {
#pragma unroll
                for (int e = 0; e < 8; ++e) {
                    const float4 c4 = cs[s][e >> 1];
                    const float cc = (e & 1) ? c4.z : c4.x, sn = (e & 1) ? c4.w : c4.y;
                    const float a = x[s][e], bb = x[s + KS / 2][e];
                    x[s][e] = (a * cc - bb * sn) * qs;
                    x[s + KS / 2][e] = (bb * cc + a * sn) * qs;
                }
            }
#pragma unroll
            for (int s = 0; s < KS; ++s)
                qop[s] = __builtin_bit_cast(
                    bf16x8, make_uint4(pack_bf16x2(x[s][0], x[s][1]), pack_bf16x2(x[s][2], x[s][3]),
                                       pack_bf16x2(x[s][4], x[s][5]), pack_bf16x2(x[s][6], x[s][7])));
        }

        uint32_t koff[KS];  // byte offset of this lane's K operand of k-step s, key block 0
#pragma unroll
        for (int s = 0; s < KS; ++s) koff[s] = (uint32_t)(l16 * D + ((4 * s + lg) ^ (l16 & (CPR - 1))) * 8) * 2u;
        uint32_t vtr_off[DB];
        {
            const int r0 = 4 * lg + (l16 >> 2);  // rows 32c + r0 and +16 share r0's swizzle
#pragma unroll
            for (int db = 0; db < DB; ++db) {
                const int dim = db * 16 + 4 * (l16 & 3);
                vtr_off[db] = (uint32_t)(r0 * D + (((dim >> 3) ^ (2 * (r0 & (CPR / 2 - 1)))) << 3) + (dim & 7)) * 2u;
            }
        }
        float mrun = -INFINITY, lrun = 0.f;
        f32x4 acc[DB];
#pragma unroll
        for (int db = 0; db < DB; ++db) acc[db] = f32x4{0.f, 0.f, 0.f, 0.f};
        const int lim = (mq < M) ? vis0 + mq / G : -1;

        auto compute = [&](int t, const TileBuf<D>& buf) {
            const int kbase = t * kTileKeys;
            f32x4 sacc[4];
#pragma unroll
            for (int kb = 0; kb < 4; ++kb) sacc[kb] = f32x4{0.f, 0.f, 0.f, 0.f};
            // every K operand of the tile requested before the first product:
            // rows kb*16 + l16 share the swizzle of row l16, so key block kb is
            // an immediate offset from the k-step's address
            const uint32_t kbuf = lds_addr(&buf.k[0]);
            u32x4 kop[KS][4];
#pragma unroll
            for (int s = 0; s < KS; ++s) {
                kop[s][0] = lds_b128_issue<0>(kbuf + koff[s]);
                kop[s][1] = lds_b128_issue<16 * D * 2>(kbuf + koff[s]);
                kop[s][2] = lds_b128_issue<32 * D * 2>(kbuf + koff[s]);
                kop[s][3] = lds_b128_issue<48 * D * 2>(kbuf + koff[s]);
            }
#pragma unroll
            for (int h = 0; h < KS; h += 2) {
                if (h == 0)
                    k_wait<4 * (KS - 2)>(kop[0], kop[1]);
                else
                    k_wait<0>(kop[KS - 2], kop[KS - 1]);
#pragma unroll
                for (int s = h; s < h + 2; ++s)
#pragma unroll
                    for (int kb = 0; kb < 4; ++kb)
                        sacc[kb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, kop[s][kb]),
                                                                           qop[s], sacc[kb], 0, 0, 0);
            }
            // the V operands of keys 0..31 are requested before the softmax, those
            // of keys 32..63 under the products of the first half: the LDS reads'
            // latency overlaps the exponentials and the MFMAs
            const uint32_t vb = lds_addr(&buf.v[0]);
            uint2 lo0[DB], hi0[DB];
#pragma unroll
            for (int db = 0; db < DB; ++db) {
                lo0[db] = lds_tr16_issue<0>(vb + vtr_off[db]);
                hi0[db] = lds_tr16_issue<16 * D * 2>(vb + vtr_off[db]);
            }
            if (kbase + kTileKeys - 1 > vis0) {
#pragma unroll
                for (int kb = 0; kb < 4; ++kb)
#pragma unroll
                    for (int e = 0; e < 4; ++e)
                        if (kbase + kb * 16 + 4 * lg + e > lim) sacc[kb][e] = -INFINITY;
            }
            float tmax = -INFINITY;
#pragma unroll
            for (int kb = 0; kb < 4; ++kb)
#pragma unroll
                for (int e = 0; e < 4; ++e) tmax = fmaxf(tmax, sacc[kb][e]);
            tmax = quad_max(tmax);
            // lazily raised softmax reference: rescale only on a jump above 2^8
            if (__any(tmax > mrun + 8.f)) {
                const float mn = fmaxf(mrun, tmax);
                const float corr = __builtin_amdgcn_exp2f(mrun - ((mn == -INFINITY) ? 0.f : mn));
                lrun *= corr;
#pragma unroll
                for (int db = 0; db < DB; ++db) acc[db] *= corr;
                mrun = mn;
            }
            const float mu = (mrun == -INFINITY) ? 0.f : mrun;
            uint32_t pk[4][2];
#pragma unroll
            for (int kb = 0; kb < 4; ++kb) {
                float p[4];
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    p[e] = __builtin_amdgcn_exp2f(sacc[kb][e] - mu);
                    lrun += p[e];
                }
                pk[kb][0] = pack_bf16x2(p[0], p[1]);
                pk[kb][1] = pack_bf16x2(p[2], p[3]);
            }
            // k-slots 8*lg+0..3 hold keys 32c + 4lg + 0..3 and 8*lg+4..7 keys
            // 32c+16+4lg+0..3; this lane's transposed reads start at row 32c+4lg+(l16>>2)
            // (+16) and dims 16db + 4(l16&3) (the row offsets are immediates)
            lds_wait_all(lo0, hi0);
            uint2 lo1[DB], hi1[DB];
#pragma unroll
            for (int db = 0; db < DB; ++db) {
                lo1[db] = lds_tr16_issue<32 * D * 2>(vb + vtr_off[db]);
                hi1[db] = lds_tr16_issue<48 * D * 2>(vb + vtr_off[db]);
            }
            {
                const bf16x8 pop = __builtin_bit_cast(bf16x8, make_uint4(pk[0][0], pk[0][1], pk[1][0], pk[1][1]));
#pragma unroll
                for (int db = 0; db < DB; ++db) {
                    const bf16x8 a = __builtin_bit_cast(bf16x8, make_uint4(lo0[db].x, lo0[db].y, hi0[db].x, hi0[db].y));
                    acc[db] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, pop, acc[db], 0, 0, 0);
                }
            }
            lds_wait_all(lo1, hi1);
            {
                const bf16x8 pop = __builtin_bit_cast(bf16x8, make_uint4(pk[2][0], pk[2][1], pk[3][0], pk[3][1]));
#pragma unroll
                for (int db = 0; db < DB; ++db) {
                    const bf16x8 a = __builtin_bit_cast(bf16x8, make_uint4(lo1[db].x, lo1[db].y, hi1[db].x, hi1[db].y));
                    acc[db] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, pop, acc[db], 0, 0, 0);
                }
            }
        };

        // one tile: wait for its DMA (only later tiles' DMA may stay in flight),
        // publish it, refill the stage freed by the previous tile, compute
        auto step = [&](int t, TileBuf<D>& cur, TileBuf<D>& nxt) {
            const int rem = t1 - 1 - t;
            if (rem >= 2)
                wait_vmem<2 * OPT>();
            else if (rem == 1)
                wait_vmem<OPT>();
            else
                wait_vmem<0>();
            barrier_only();
            if (t * kTileKeys + kTileKeys > newbase && newbase < R) fixup(t, cur);
            if (t + kTileStages - 1 < t1) issue(t + kTileStages - 1, nxt);
            if (active) compute(t, cur);
        };
#pragma unroll 1
        for (int t = t0; t < t1; ++t) {
            const int k = (t - t0) & (kTileStages - 1);
            step(t, ring[k], ring[(k + kTileStages - 1) & (kTileStages - 1)]);
        }

        if (active) lrun = quad_sum(lrun);
        if (active && d.splits > 1) {
            // key-split partial: O / sum in fp16 (a row with no visible key in this
            // split stores zeros, which its zero weight in the merge ignores) and fp32
            // (max, sum).  A lane holds dims 16 db + 4 lg .. + 3 of its row; lanes
            // lg and lg ^ 1 swap halves of a block pair so that each lane stores 8
            // adjacent dims (16 bytes): even lg the pair's first block, odd lg its
            // second.  Every lane of the wave takes part in the swaps.  Split
            // partials are read once, by the merge launch: non-temporal stores send
            // them on to memory now instead of leaving dirty L2 lines for the
            // end-of-kernel write-back.
            const float inv = lrun > 0.f ? 1.f / lrun : 0.f;
            u32x4 ho[DB / 2];
#pragma unroll
            for (int j = 0; j < DB / 2; ++j) {
                const f32x4 a0 = acc[2 * j], a1 = acc[2 * j + 1];
                const uint32_t h00 = pack_f16x2(a0[0] * inv, a0[1] * inv), h01 = pack_f16x2(a0[2] * inv, a0[3] * inv);
                const uint32_t h10 = pack_f16x2(a1[0] * inv, a1[1] * inv), h11 = pack_f16x2(a1[2] * inv, a1[3] * inv);
                // odd rows (16 lanes) of the first operand trade with even rows of the second
                const auto s0 = __builtin_amdgcn_permlane16_swap(h00, h10, false, false);
                const auto s1 = __builtin_amdgcn_permlane16_swap(h01, h11, false, false);
                ho[j] = (lg & 1) ? u32x4{s0[0], s1[0], h10, h11} : u32x4{h00, h01, s0[1], s1[1]};
            }
            if (mq < M) {
                float* po = st.ws + d.ws_off;
                _Float16* prow = reinterpret_cast<_Float16*>(po) + (((int64_t)sp * st.Hkv + g) * M + mq) * D;
#pragma unroll
                for (int j = 0; j < DB / 2; ++j)
                    __builtin_nontemporal_store(ho[j], reinterpret_cast<u32x4*>(prow + 32 * j + 16 * (lg & 1) + 4 * (lg & ~1)));
                if (lg == 0) {
                    float* pml = po + (int64_t)d.splits * st.Hkv * M * (D / 2);
                    float* mp = pml + (((int64_t)sp * st.Hkv + g) * M + mq) * 2;
                    __builtin_nontemporal_store(mrun, mp);
                    __builtin_nontemporal_store(lrun, mp + 1);
                }
            }
        }
        if (active && mq < M) {
            const int i = mq / G, hh = mq - i * G;
            if (d.splits == 1) {
                const float inv = 1.f / lrun;
                uint16_t* op = o + ((int64_t)(d.q_row0 + i) * st.Hq + g * G + hh) * D;
#pragma unroll
                for (int db = 0; db < DB; ++db) {
                    const f32x4 a = acc[db];
                    *reinterpret_cast<uint2*>(op + db * 16 + 4 * lg) =
                        make_uint2(pack_bf16x2(a[0] * inv, a[1] * inv), pack_bf16x2(a[2] * inv, a[3] * inv));
                }
            }
        }
        if (qg0 + QPP < M) __syncthreads();  // the stages are reused by the next pass over the keys
    }
}

// ----------------------------------------------------------------- attn_merge
// grid (row groups x kv heads, stream).  A workgroup combines the key-split
// partials of kMergeRows query rows: each thread owns 8 output elements of one
// row (the MFMA kernel's fp16 partials; 4 from the VALU kernel's fp32 ones, one
// 16-byte load per split either way) and the splits s = sg, sg + NSG, ... of
// its split group sg (NSG = 4 at head dim 128 with fp16 partials, 2 with fp32),
// read B at a time with all loads of a batch in flight together (the launch
// picks B = 12 when a thread would otherwise take two rounds of 8, else 8,
// which holds fewer registers).  The split groups' running (max, sum, O) then
// combine in LDS in group order.  Spreading a row's splits over NSG threads
// spreads the partials over more workgroups than one thread per row would: the
// partials come from memory and a CU streams only so many bytes per
// microsecond.  The order of every sum is fixed, so the result is deterministic.
// One row group (kMergeRows query rows of KV head g) of the merge; every thread
// of the workgroup calls it (one barrier inside).
template <typename T, int B, bool H16>
__device__ __forceinline__ void merge_row_group(const DevState& st, const AttnDesc& d, T* o, int g,
                                                int rg, float4* s_o, float2* s_ml) {
    // EPT output elements per thread: 4 from fp32 partials (one 16-byte load per
    // split), 8 from fp16 partials (also one 16-byte load)
    constexpr int MR = kMergeRows, EPT = H16 ? 8 : 4;
    const int G = st.G, M = G * d.n_q, D = st.D;
    const int tpr = D / EPT;        // threads per query row
    const int tsg = MR * tpr;       // threads per split group
    const int nsg = 256 / tsg;      // split groups
    const int sg = threadIdx.x / tsg, r = threadIdx.x - sg * tsg;
    const int rr = r / tpr, de = (r - rr * tpr) * EPT;
    const int mq = rg * MR + rr;
    const bool live = mq < M;
    const int mqc = live ? mq : M - 1;
    // floats per stored O row: D (fp32) or D / 2 (fp16); (max, sum) pairs after the O rows
    const int ow = H16 ? D / 2 : D;
    const float* po = st.ws + d.ws_off;
    const float* pml = po + (int64_t)d.splits * st.Hkv * M * ow;
    const int64_t ostride = (int64_t)st.Hkv * M * ow, mstride = (int64_t)st.Hkv * M * 2;
    const float* orow = po + ((int64_t)g * M + mqc) * ow + (H16 ? de / 2 : de);
    const float* mrow = pml + ((int64_t)g * M + mqc) * 2;
    float mx = -INFINITY, L = 0.f, O[EPT];
#pragma unroll
    for (int e2 = 0; e2 < EPT; ++e2) O[e2] = 0.f;
    for (int s0 = sg; s0 < d.splits; s0 += B * nsg) {
        float2 ml[B];
        u32x4 ov[B];
#pragma unroll
        for (int j = 0; j < B; ++j) {
            const int s = s0 + j * nsg;
            if (s < d.splits) {
                ml[j] = *reinterpret_cast<const float2*>(mrow + s * mstride);
                ov[j] = *reinterpret_cast<const u32x4*>(orow + s * ostride);
            } else {
                ml[j] = make_float2(-INFINITY, 0.f);
                ov[j] = u32x4{0u, 0u, 0u, 0u};
            }
        }
        float bm = mx;
#pragma unroll
        for (int j = 0; j < B; ++j) bm = fmaxf(bm, ml[j].x);
        if (bm == -INFINITY) continue;
        const float c = (mx == -INFINITY) ? 0.f : exp2f(mx - bm);
        L *= c;
#pragma unroll
        for (int e2 = 0; e2 < EPT; ++e2) O[e2] *= c;
#pragma unroll
        for (int j = 0; j < B; ++j) {
            // fp32 partials hold O unnormalised (weight exp2(m - bm)); fp16 partials hold
            // O / sum (weight exp2(m - bm) * sum), which keeps them within fp16 range
            const float w0 = (ml[j].x == -INFINITY) ? 0.f : exp2f(ml[j].x - bm);
            L += w0 * ml[j].y;
            if constexpr (H16) {
                const float w = w0 * ml[j].y;
                const f16x8 h = __builtin_bit_cast(f16x8, ov[j]);
#pragma unroll
                for (int e2 = 0; e2 < 8; ++e2) O[e2] += w * (float)h[e2];
            } else {
#pragma unroll
                for (int e2 = 0; e2 < 4; ++e2) O[e2] += w0 * __uint_as_float(ov[j][e2]);
            }
        }
        mx = bm;
    }
    s_o[threadIdx.x] = make_float4(O[0], O[1], O[2], O[3]);
    if constexpr (H16) s_o[256 + threadIdx.x] = make_float4(O[4], O[5], O[6], O[7]);
    s_ml[threadIdx.x] = make_float2(mx, L);
    __syncthreads();
    if (sg != 0 || !live) return;
    float bm = -INFINITY;
    for (int k = 0; k < nsg; ++k) bm = fmaxf(bm, s_ml[k * tsg + r].x);
    float Lt = 0.f, Ot[EPT];
#pragma unroll
    for (int e2 = 0; e2 < EPT; ++e2) Ot[e2] = 0.f;
    for (int k = 0; k < nsg; ++k) {
        const float2 ml = s_ml[k * tsg + r];
        if (ml.x == -INFINITY) continue;
        const float w = exp2f(ml.x - bm);
        const float4 ov = s_o[k * tsg + r];
        Lt += w * ml.y;
        Ot[0] += w * ov.x;
        Ot[1] += w * ov.y;
        Ot[2] += w * ov.z;
        Ot[3] += w * ov.w;
        if constexpr (H16) {
            const float4 ov2 = s_o[256 + k * tsg + r];
            Ot[4] += w * ov2.x;
            Ot[5] += w * ov2.y;
            Ot[6] += w * ov2.z;
            Ot[7] += w * ov2.w;
        }
    }
    const float inv = 1.f / Lt;
    const int i = mq / G, hh = mq - i * G;
    T* op = o + ((int64_t)(d.q_row0 + i) * st.Hq + g * G + hh) * D + de;
#pragma unroll
    for (int e2 = 0; e2 < EPT; ++e2) Elt<T>::store(op + e2, Ot[e2] * inv);
}

// Merge for launches whose streams have few key splits (fp16 partials of the
// MFMA kernel): one thread per (query row, 8 output elements) walks every split
// of its row itself, 8 at a time with all loads of a batch in flight, so a
// workgroup covers 256 / (D / 8) rows (16 at head dim 128) and needs no LDS.
// Splits combine in split order: deterministic.
template <class BT>
__global__ __launch_bounds__(256) void attn_merge_few_kernel(DevState st, BT b, bf16_t* o) {
    constexpr int B = 8;
    const AttnDesc d = b.d[blockIdx.z];
    if (d.splits <= 1) return;
    const int D = st.D, G = st.G, M = G * d.n_q;
    const int tpr = D / 8, rows = 256 / tpr;
    // row group rg of KV head g is linear block rg * Hkv + g, on the XCD of head g
    const int g = blockIdx.x % st.Hkv, rg = blockIdx.x / st.Hkv;
    const int rr = threadIdx.x / tpr, de = (threadIdx.x - rr * tpr) * 8;
    const int mq = rg * rows + rr;
    if (mq >= M) return;
    const int ow = D / 2;   // floats per stored fp16 O row
    const float* po = st.ws + d.ws_off;
    const float* pml = po + (int64_t)d.splits * st.Hkv * M * ow;
    const int64_t ostride = (int64_t)st.Hkv * M * ow, mstride = (int64_t)st.Hkv * M * 2;
    const float* orow = po + ((int64_t)g * M + mq) * ow + de / 2;
    const float* mrow = pml + ((int64_t)g * M + mq) * 2;
    float mx = -INFINITY, L = 0.f, O[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) O[e] = 0.f;
    for (int s0 = 0; s0 < d.splits; s0 += B) {
        float2 ml[B];
        u32x4 ov[B];
#pragma unroll
        for (int j = 0; j < B; ++j) {
            const int s = s0 + j;
            if (s < d.splits) {
                ml[j] = *reinterpret_cast<const float2*>(mrow + s * mstride);
                ov[j] = *reinterpret_cast<const u32x4*>(orow + s * ostride);
            } else {
                ml[j] = make_float2(-INFINITY, 0.f);
                ov[j] = u32x4{0u, 0u, 0u, 0u};
            }
        }
        float bm = mx;
#pragma unroll
        for (int j = 0; j < B; ++j) bm = fmaxf(bm, ml[j].x);
        if (bm == -INFINITY) continue;
        const float c = (mx == -INFINITY) ? 0.f : exp2f(mx - bm);
        L *= c;
#pragma unroll
        for (int e = 0; e < 8; ++e) O[e] *= c;
#pragma unroll
        for (int j = 0; j < B; ++j) {
            // fp16 partials hold O / sum: weight exp2(m - bm) * sum
            const float w0 = (ml[j].x == -INFINITY) ? 0.f : exp2f(ml[j].x - bm);
            const float w = w0 * ml[j].y;
            L += w;
            const f16x8 h = __builtin_bit_cast(f16x8, ov[j]);
#pragma unroll
            for (int e = 0; e < 8; ++e) O[e] += w * (float)h[e];
        }
        mx = bm;
    }
    const float inv = 1.f / L;
    const int i = mq / G, hh = mq - i * G;
    uint16_t* op = reinterpret_cast<uint16_t*>(o) + ((int64_t)(d.q_row0 + i) * st.Hq + g * G + hh) * D + de;
    *reinterpret_cast<uint2*>(op) = make_uint2(pack_bf16x2(O[0] * inv, O[1] * inv), pack_bf16x2(O[2] * inv, O[3] * inv));
    *reinterpret_cast<uint2*>(op + 4) = make_uint2(pack_bf16x2(O[4] * inv, O[5] * inv), pack_bf16x2(O[6] * inv, O[7] * inv));
}

// launches whose streams have at most this many key splits merge with one thread
// per row and element group (at most two load rounds of 8 per thread)
constexpr int kMergeFewSplits = 16;
// H16: the partials of the MFMA attention kernel (fp16 O rows); else fp32 (VALU kernel)
template <typename T, int B, class BT, bool H16 = false>
__global__ __launch_bounds__(256) void attn_merge_kernel(DevState st, BT b, T* o) {
    __shared__ float4 s_o[H16 ? 512 : 256];
    __shared__ float2 s_ml[256];
    const AttnDesc d = b.d[blockIdx.z];
    if (d.splits <= 1) return;
    // row group rg of KV head g is linear block rg * Hkv + g: the XCD of head g,
    // like the attention workgroups that wrote its partials.  A grid with fewer
    // row groups than the step has (device-planned steps, whose grid is fixed)
    // strides over them.
    const int g = blockIdx.x % st.Hkv, groups = gridDim.x / st.Hkv;
    const int M = st.G * d.n_q;
    for (int rg = blockIdx.x / st.Hkv; rg * kMergeRows < M; rg += groups) {
        merge_row_group<T, B, H16>(st, d, o, g, rg, s_o, s_ml);
        __syncthreads();   // s_o / s_ml are reused by the next row group
    }
}

// ---------------------------------------------------------------------- evict
// grid (L + 1, streams).  Workgroups 0..L-1 move the retained rows of the
// passed-over ring span into the kept region of their layer; workgroup L
// writes the kept-region metadata and the mask / compaction indices over the
// whole pre-eviction cache.  Each workgroup ranks the span's rows itself
// (wave ballot + popcount, then a cross-wave prefix in LDS).
template <int ELT, class BT>
__global__ __launch_bounds__(256) void evict_kernel(DevState st, BT b) {
    __shared__ int s_wave[4];
    __shared__ int s_src[256];
    __shared__ int s_dst[256];
    const EvictDesc d = b.d[blockIdx.y];
    if (d.span == 0) return;   // a device-planned stream that evicts nothing this step
    const int which = blockIdx.x;
    const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
    const int64_t mb = (int64_t)d.s * st.unit_rows;
    const int64_t kb = (int64_t)d.s * st.kept_rows;
    const int64_t eb = (int64_t)d.s * (st.unit_rows + st.kept_rows);
    const bool index_wg = (which == st.L);

    if (index_wg) {
        const int tail0 = d.kept + d.span;
        const int shift = d.span - d.n_keep;
        for (int j = tid; j < d.kept; j += 256) {
            st.ev_mask[eb + j] = 0;
            st.ev_slot[eb + j] = j;
        }
        for (int j = tail0 + tid; j < d.R_pre; j += 256) {
            st.ev_mask[eb + j] = 0;
            st.ev_slot[eb + j] = j - shift;
        }
    }

    constexpr int CH = 16 / ELT;  // elements per 16-byte chunk
    const int cph = st.D / CH;    // chunks per head row
    const int cpr = 2 * st.Hkv * cph;  // chunks per cache row (K and V)

    int running = 0;
    for (int base = 0; base < d.span; base += 256) {
        const int x = base + tid;
        const bool in = x < d.span;
        int slot = 0;
        bool keep = false;
        if (in) {
            slot = d.head + x;
            if (slot >= st.unit_rows) slot -= st.unit_rows;
            if (d.sink >= 0) {
                keep = d.kept + x < d.sink;
            } else {
                const uint8_t sg = st.unit_seg[mb + slot];
                const int uid = st.unit_uid[mb + slot];
                keep = !((sg == kSegAcoustic || sg == kSegDelim) && uid <= d.u_last);
            }
        }
        const uint64_t bal = __ballot(keep);
        const int below = __popcll(bal & ((1ull << lane) - 1ull));
        if (lane == 0) s_wave[w] = __popcll(bal);
        __syncthreads();
        int before = 0, total = 0;
#pragma unroll
        for (int ww = 0; ww < 4; ++ww) {
            before += (ww < w) ? s_wave[ww] : 0;
            total += s_wave[ww];
        }
        const int rank = running + before + below;
        if (index_wg) {
            if (in) {
                const int j = d.kept + x;
                st.ev_mask[eb + j] = keep ? 0 : 1;
                st.ev_slot[eb + j] = keep ? d.kept + rank : -1;
                if (keep) {
                    st.kept_pos[kb + d.kept + rank] = st.unit_pos[mb + slot];
                    st.kept_seg[kb + d.kept + rank] = st.unit_seg[mb + slot];
                    st.kept_uid[kb + d.kept + rank] = st.unit_uid[mb + slot];
                }
            }
        } else {
            if (in && keep) {
                s_src[before + below] = slot;
                s_dst[before + below] = d.kept + rank;
            }
            __syncthreads();
            const int layer = which;
            for (int c = tid; c < total * cpr; c += 256) {
                const int r = c / cpr;
                int rem = c - r * cpr;
                const int kv = rem / (st.Hkv * cph);
                rem -= kv * st.Hkv * cph;
                const int g = rem / cph, ch = rem - g * cph;
                const char* src = reinterpret_cast<const char*>(kv ? st.v_unit : st.k_unit) +
                                  (pool_index(st, layer, d.s, g, st.unit_rows, s_src[r]) * ELT) +
                                  ch * 16;
                char* dst = reinterpret_cast<char*>(kv ? st.v_kept : st.k_kept) +
                            (pool_index(st, layer, d.s, g, st.kept_rows, s_dst[r]) * ELT) + ch * 16;
                *reinterpret_cast<uint4*>(dst) = *reinterpret_cast<const uint4*>(src);
            }
        }
        running += total;
        __syncthreads();
    }
}

// ------------------------------------------------------ device-planned steps
constexpr int kDevMergeGroups = 32;   // merge workgroups per KV head of a device-planned launch

// One workgroup: thread i opens the step of stream a.ids[i] from the metadata
// the caller left in device memory, with the checks a2t_append makes on the
// host; a stream that fails one records the status (sticky) and takes no part
// in the step.  The step's q/k/v/o rows sit at a fixed place per listed stream
// (stream i from row i * max_step_rows).  Thread 0 then plans the key splits:
// the smallest tile budget per split (>= 2) whose workgroups fit one round of
// target_wgs and whose partials fit the workspace, as the host planner picks
// for a single stream.
__global__ __launch_bounds__(64) void dev_open_kernel(DevState st, DevStepArgs a,
                                                      const int32_t* n_rows, const int32_t* unit,
                                                      const uint8_t* seg, const int32_t* pos,
                                                      DevPlan* plan) {
    __shared__ int s_n[kMaxDesc];
    __shared__ int s_R[kMaxDesc];
    const int i = threadIdx.x;
    const int MS = st.max_step_rows;
    if (i < a.count) {
        const int s = a.ids[i];
        DevStream& ds = st.dss[s];
        const int n = n_rows[i], u = unit[i];
        int err = ds.error;
        if (!err && ds.step_rows != 0) err = A2T_ERR_STATE;
        if (!err && (n < 1 || n > MS || u < -1)) err = A2T_ERR_INVALID;
        if (!err && u == -1 && ds.cur_unit >= 0) err = A2T_ERR_POS;
        if (!err && ds.cur_unit != -2 && u < ds.cur_unit) err = A2T_ERR_POS;
        if (!err && (int64_t)ds.ring + n > st.unit_rows) err = A2T_ERR_CAPACITY;
        int64_t last = ds.last_pos;
        for (int r = 0; !err && r < n; ++r) {
            const int sg = seg[(int64_t)i * MS + r];
            const int p = pos[(int64_t)i * MS + r];
            if (sg > A2T_SEG_RESPONSE || p < 0 || (u == -1) != (sg == A2T_SEG_PREFIX))
                err = A2T_ERR_INVALID;
            else if (p <= last)
                err = A2T_ERR_POS;
            last = p;
        }
        int slot0 = 0, n_act = 0;
        if (err) {
            ds.error = err;
        } else {
            slot0 = ds.head + ds.ring;
            if (slot0 >= st.unit_rows) slot0 -= st.unit_rows;
            ds.ring += n;
            ds.step_rows = n;
            ds.step_slot0 = slot0;
            ds.cur_unit = ds.cur_unit > u ? ds.cur_unit : u;
            ds.last_pos = pos[(int64_t)i * MS + n - 1];
            ds.peak = ds.peak > ds.kept + ds.ring ? ds.peak : ds.kept + ds.ring;
            ds.budget_unmet = 0;
            n_act = n;
        }
        plan->step[i] = StepDesc{s, n_act, slot0, i * MS};
        AttnDesc& d = plan->attn[i];
        d.s = s;
        d.kept = ds.kept;
        d.head = ds.head;
        d.R = ds.kept + ds.ring;
        d.n_q = n_act;
        d.rope_row0 = 0;
        d.n_new = n_act;
        s_n[i] = n_act;
        s_R[i] = d.R;
    }
    __syncthreads();
    if (i != 0) return;
    const int64_t row_floats = st.D / 2 + 2;   // split partials of one query row and head (fp16 O)
    int max_tiles = 1;
    for (int k = 0; k < a.count; ++k)
        if (s_n[k]) max_tiles = max(max_tiles, (s_R[k] + kTileKeys - 1) / kTileKeys);
    int budget = max_tiles;
    for (int b = 2; b <= max_tiles; ++b) {
        int64_t wgs = 0, ws = 0;
        for (int k = 0; k < a.count; ++k) {
            if (!s_n[k]) continue;
            const int t = max(1, (s_R[k] + kTileKeys - 1) / kTileKeys);
            const int sp = min((t + b - 1) / b, a.max_splits);
            wgs += (int64_t)sp * st.Hkv;
            ws += stream_partials(sp, (int64_t)st.Hq * s_n[k] * row_floats);
        }
        if (wgs <= a.target_wgs && ws <= st.ws_floats) {
            budget = b;
            break;
        }
    }
    int64_t off = 0;
    for (int k = 0; k < a.count; ++k) {
        AttnDesc& d = plan->attn[k];
        d.q_row0 = k * MS;
        d.in_row0 = k * MS;
        d.ws_off = off;
        if (!s_n[k]) {
            d.splits = 0;   // every workgroup of this stream returns at once
            d.tile_q = d.tile_r = 0;
            continue;
        }
        const int t = max(1, (s_R[k] + kTileKeys - 1) / kTileKeys);
        int sp = min((t + budget - 1) / budget, a.max_splits);
        if (sp > 1 && off + stream_partials(sp, (int64_t)st.Hq * s_n[k] * row_floats) > st.ws_floats) sp = 1;
        d.splits = sp;
        d.tile_q = t / sp;
        d.tile_r = t % sp;
        off += stream_partials(sp, (int64_t)st.Hq * s_n[k] * row_floats);
    }
}

// One workgroup per listed stream: Sec. 3.3's eviction planned on the device.
// R > B evicts, oldest first, whole units u <= cur - W that hold acoustic or
// structural rows, until R <= B or none is left: the shortest prefix of such
// units whose evictable rows reach R - B (all of them if none does).  The pass
// covers every ring row of the units up to the last one evicted; the scan ranks
// the ring's eligible evictable rows with wave ballots and a cross-wave prefix.
__global__ __launch_bounds__(256) void dev_evict_plan_kernel(DevState st, DevStepArgs a,
                                                             const int32_t* budget,
                                                             int32_t* n_evicted,
                                                             uint8_t* budget_unmet, DevPlan* plan) {
    __shared__ int s_wave[4];
    __shared__ int s_cut, s_last, s_span;
    const int i = blockIdx.x, tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
    const int s = a.ids[i];
    DevStream& ds = st.dss[s];
    const int kept = ds.kept, head = ds.head, ring = ds.ring, cur = ds.cur_unit;
    const int R = kept + ring, B = max(budget[i], 0);   // a negative budget counts as 0
    const int64_t mb = (int64_t)s * st.unit_rows;
    auto slot_of = [&](int x) {
        int slot = head + x;
        return slot >= st.unit_rows ? slot - st.unit_rows : slot;
    };
    EvictDesc e{s, kept, head, R, 0, -2, 0, -1};
    const bool open = ds.error == 0 && ds.step_rows != 0;
    int evicted = 0;
    if (open && R > B && a.rule == A2T_RULE_SINK_RECENT) {
        // every row but the n_sink oldest and the B - n_sink newest: the pass covers
        // the ring's remaining sinks and the R - B rows after them
        const int n_sink = a.n_sink;
        if (B < n_sink || kept > n_sink) {
            if (tid == 0) ds.error = B < n_sink ? A2T_ERR_INVALID : A2T_ERR_STATE;
        } else {
            const int sinks_left = n_sink - kept;
            e.span = sinks_left + (R - B);   // <= ring, since B >= n_sink >= kept
            e.u_last = st.unit_uid[mb + slot_of(e.span - 1)];
            e.n_keep = sinks_left;
            e.sink = n_sink;
            evicted = R - B;
            if ((int64_t)kept + e.n_keep > st.kept_rows) {
                e.span = 0;
                evicted = 0;
                if (tid == 0) ds.error = A2T_ERR_CAPACITY;
            }
        }
    } else if (open && R > B) {
        const int need = R - B;
        const int64_t limit = (int64_t)cur - a.window;
        if (tid == 0) {
            s_cut = -1;
            s_last = -1;
        }
        __syncthreads();
        // the first eligible evictable row at which the running count reaches
        // need, else the last eligible evictable row
        int running = 0;
        for (int base = 0; base < ring; base += 256) {
            const int x = base + tid;
            bool el = false;
            if (x < ring) {
                const int slot = slot_of(x);
                const uint8_t sg = st.unit_seg[mb + slot];
                el = (sg == A2T_SEG_ACOUSTIC || sg == A2T_SEG_DELIM) && st.unit_uid[mb + slot] <= limit;
            }
            const uint64_t bal = __ballot(el);
            const int below = __popcll(bal & ((1ull << lane) - 1ull));
            if (lane == 0) s_wave[w] = __popcll(bal);
            __syncthreads();
            int before = 0, total = 0;
            for (int ww = 0; ww < 4; ++ww) {
                before += ww < w ? s_wave[ww] : 0;
                total += s_wave[ww];
            }
            if (el) {
                const int rank = running + before + below + 1;   // eligible rows up to x
                if (rank == need) s_cut = x;
                if (rank == running + total) s_last = x;          // the chunk's last one
            }
            running += total;
            __syncthreads();
            if (s_cut >= 0) break;
        }
        const int xc = s_cut >= 0 ? s_cut : s_last;
        if (xc >= 0) {
            const int ucut = st.unit_uid[mb + slot_of(xc)];
            // whole units: the pass ends at the first ring row of a later unit; per
            // row: at the newest evicted row itself
            if (tid == 0) s_span = a.rule == A2T_RULE_ROW ? xc + 1 : ring;
            __syncthreads();
            for (int base = xc + 1; a.rule != A2T_RULE_ROW && base < ring; base += 256) {
                const int x = base + tid;
                if (x < ring && st.unit_uid[mb + slot_of(x)] > ucut) atomicMin(&s_span, x);
                __syncthreads();
                if (s_span < ring) break;
            }
            const int span = s_span;
            // evictable rows inside the pass (all of them are eligible)
            int cnt = 0;
            for (int x = tid; x < span; x += 256) {
                const uint8_t sg = st.unit_seg[mb + slot_of(x)];
                cnt += (sg == A2T_SEG_ACOUSTIC || sg == A2T_SEG_DELIM);
            }
            for (int o = 32; o >= 1; o >>= 1) cnt += __shfl_xor(cnt, o);
            __syncthreads();
            if (lane == 0) s_wave[w] = cnt;
            __syncthreads();
            evicted = s_wave[0] + s_wave[1] + s_wave[2] + s_wave[3];
            e.span = span;
            e.u_last = ucut;
            e.n_keep = span - evicted;
            if ((int64_t)kept + e.n_keep > st.kept_rows) {
                e.span = 0;   // the kept region would overflow: the stream evicts nothing
                evicted = 0;
                if (tid == 0) ds.error = A2T_ERR_CAPACITY;
            }
        }
    }
    __syncthreads();
    if (tid != 0) return;
    plan->evict[i] = e;
    if (open) {
        if (e.span > 0) {
            ds.kept = kept + e.n_keep;
            int h = head + e.span;
            ds.head = h >= st.unit_rows ? h - st.unit_rows : h;
            ds.ring = ring - e.span;
            ds.last_evicted = e.u_last;
            ds.evicted_total += evicted;
            ds.moved_total += e.n_keep;
            ds.last_evict_pre = R;
        }
        ds.budget_unmet = R - evicted > B ? 1 : 0;
        ds.step_rows = 0;
    }
    if (n_evicted) n_evicted[i] = evicted;
    if (budget_unmet) budget_unmet[i] = open && R - evicted > B ? 1 : 0;
}

// ------------------------------------------------------------- fixed workspace
// Key-split partials of a2t_append_attn_noalloc: one launch's partials (every
// split's O rows, then their (max, sum) pairs) in a fixed device array instead
// of a cache's workspace.  16 MiB holds the fp16 partials of a 22-split launch
// over 22 query rows x 32 heads x head dim 128 four times over.
// Every call on a device shares that device's copy; each attention launch
// writes every partial its merge reads, so nothing needs clearing between calls.
constexpr int64_t kScratchFloats = int64_t(4) << 20;
static __device__ __align__(256) float scratch[kScratchFloats];
constexpr int kScratchDevices = 64;

}  // namespace

hipError_t static_scratch(int device, float** ptr, int64_t* floats) {
    static std::mutex mu;
    static float* addr[kScratchDevices] = {};
    if (device < 0 || device >= kScratchDevices) return hipErrorInvalidDevice;
    std::lock_guard<std::mutex> lock(mu);
    if (!addr[device]) {
        // the array's name is a host-side stand-in: kernels get this device address
        void* p = nullptr;
        const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess) return e;
        addr[device] = static_cast<float*>(p);
    }
    *ptr = addr[device];
    *floats = kScratchFloats;
    return hipSuccess;
}

// ------------------------------------------------------------------ launchers
// One dispatch, through hipExtLaunchKernelGGL when the caller asks for timestamps.
#define A2T_DISPATCH(kernel, grid, block, stream, kt, ...)                                        \
    do {                                                                                          \
        if ((kt).start)                                                                           \
            hipExtLaunchKernelGGL(kernel, grid, block, 0, stream, (kt).start, (kt).stop, 0,       \
                                  __VA_ARGS__);                                                   \
        else                                                                                      \
            hipLaunchKernelGGL(kernel, grid, block, 0, stream, __VA_ARGS__);                      \
    } while (0)

// Calls f with the batch shrunk to the smallest of 1, 8 or kMaxDesc descriptors.
template <template <int> class BT, class F>
static hipError_t by_size(const BT<kMaxDesc>& b, F&& f) {
    if (b.count <= 1) return f(shrink_batch<BT, 1>(b));
    if (b.count <= 8) return f(shrink_batch<BT, 8>(b));
    return f(b);
}

hipError_t launch_step_meta(const DevState& st, const StepBatch& b, const uint8_t* seg,
                            const int32_t* pos, const int32_t* uid, hipStream_t stream,
                            const KTimer& kt) {
    return by_size<StepBatchT>(b, [&](const auto& bb) {
        using B = std::decay_t<decltype(bb)>;
        A2T_DISPATCH((step_meta_kernel<B>), dim3(b.max_n, b.count), dim3(64), stream, kt, st, bb,
                           seg, pos, uid);
        return hipGetLastError();
    });
}

hipError_t launch_append(const DevState& st, const AppendBatch& b, int n_layers, const void* k,
                         const void* v, hipStream_t stream, const KTimer& kt) {
    const int cpr = st.Hkv * st.D / 8;
    const dim3 grid((b.max_n * cpr + 255) / 256, b.count, n_layers);
    return by_size<AppendBatchT>(b, [&](const auto& bb) {
        using B = std::decay_t<decltype(bb)>;
        if (st.dtype == 0)
            A2T_DISPATCH((append_kernel<float, B>), grid, dim3(256), stream, kt, st, bb,
                               static_cast<const float*>(k), static_cast<const float*>(v));
        else
            A2T_DISPATCH((append_kernel<bf16_t, B>), grid, dim3(256), stream, kt, st, bb,
                               static_cast<const bf16_t*>(k), static_cast<const bf16_t*>(v));
        return hipGetLastError();
    });
}

// the attention kernels take the shape, the descriptor batch and four pointers by value
static_assert(sizeof(DevState) + sizeof(AttnBatch) + 4 * sizeof(void*) <= 4096,
              "attention kernel arguments must stay within 4 KiB");

hipError_t launch_attn_tile(const DevState& st, const AttnBatch& b, const void* q, void* o,
                            const void* k_in, const void* v_in, hipStream_t stream,
                            const KTimer& kt) {
    const uint16_t* ki = static_cast<const uint16_t*>(k_in);
    const uint16_t* vi = static_cast<const uint16_t*>(v_in);
    const dim3 grid(b.max_splits * st.Hkv, 1, b.count);
    const uint16_t* qq = static_cast<const uint16_t*>(q);
    uint16_t* oo = static_cast<uint16_t*>(o);
    return by_size<AttnBatchT>(b, [&](const auto& bb) {
        using B = std::decay_t<decltype(bb)>;
        if (st.D == 128) {
            A2T_DISPATCH((attn_tile_kernel<128, B>), grid, dim3(kMfmaThreads), stream, kt, st, bb,
                         qq, oo, ki, vi);
        } else if (st.D == 64) {
            A2T_DISPATCH((attn_tile_kernel<64, B>), grid, dim3(kMfmaThreads), stream, kt, st, bb,
                         qq, oo, ki, vi);
        } else {
            return hipErrorInvalidValue;
        }
        return hipGetLastError();
    });
}

template <typename T, int D, class B>
static hipError_t valu_dispatch_g(const DevState& st, const B& b, const void* q, void* o,
                                  hipStream_t stream, const KTimer& kt) {
    const dim3 grid(b.max_splits, st.Hkv * b.max_rows, b.count);
    const T* qq = static_cast<const T*>(q);
    T* oo = static_cast<T*>(o);
    switch (st.Hq / st.Hkv) {
        case 1: A2T_DISPATCH((attn_valu_kernel<T, D, 1, B>), grid, dim3(256), stream, kt, st, b, qq, oo); break;
        case 2: A2T_DISPATCH((attn_valu_kernel<T, D, 2, B>), grid, dim3(256), stream, kt, st, b, qq, oo); break;
        case 4: A2T_DISPATCH((attn_valu_kernel<T, D, 4, B>), grid, dim3(256), stream, kt, st, b, qq, oo); break;
        case 8: A2T_DISPATCH((attn_valu_kernel<T, D, 8, B>), grid, dim3(256), stream, kt, st, b, qq, oo); break;
        default: return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

hipError_t launch_attn_valu(const DevState& st, const AttnBatch& b, const void* q, void* o,
                            hipStream_t stream, const KTimer& kt) {
    return by_size<AttnBatchT>(b, [&](const auto& bb) {
        using B = std::decay_t<decltype(bb)>;
        if (st.dtype == 0) {
            if (st.D == 128) return valu_dispatch_g<float, 128>(st, bb, q, o, stream, kt);
            if (st.D == 64) return valu_dispatch_g<float, 64>(st, bb, q, o, stream, kt);
        } else {
            if (st.D == 128) return valu_dispatch_g<bf16_t, 128>(st, bb, q, o, stream, kt);
            if (st.D == 64) return valu_dispatch_g<bf16_t, 64>(st, bb, q, o, stream, kt);
        }
        (void)sizeof(B);
        return hipErrorInvalidValue;
    });
}

hipError_t launch_attn_merge(const DevState& st, const AttnBatch& b, void* o, hipStream_t stream,
                             const KTimer& kt, bool h16) {
    const int G = st.Hq / st.Hkv;
    if (st.D / 4 * kMergeRows > 256) return hipErrorInvalidValue;
    if (h16 && st.dtype == 0) return hipErrorInvalidValue;   // fp16 partials come from bf16 caches
    const dim3 grid((G * b.max_rows + kMergeRows - 1) / kMergeRows * st.Hkv, 1, b.count);
    const int nsg = 256 / (kMergeRows * st.D / (h16 ? 8 : 4));    // split groups per workgroup
    const bool wide = (b.max_splits + nsg - 1) / nsg > 8;          // more than one round of 8
    const bool few = h16 && b.max_splits <= kMergeFewSplits;
    const int few_rows = 256 / (st.D / 8);
    const dim3 few_grid((G * b.max_rows + few_rows - 1) / few_rows * st.Hkv, 1, b.count);
    return by_size<AttnBatchT>(b, [&](const auto& bb) {
        using B = std::decay_t<decltype(bb)>;
        if (few)
            A2T_DISPATCH((attn_merge_few_kernel<B>), few_grid, dim3(256), stream, kt, st, bb,
                         static_cast<bf16_t*>(o));
        else if (h16 && wide)
            A2T_DISPATCH((attn_merge_kernel<bf16_t, 12, B, true>), grid, dim3(256), stream, kt, st, bb,
                         static_cast<bf16_t*>(o));
        else if (h16)
            A2T_DISPATCH((attn_merge_kernel<bf16_t, 8, B, true>), grid, dim3(256), stream, kt, st, bb,
                         static_cast<bf16_t*>(o));
        else if (st.dtype == 0 && wide)
            A2T_DISPATCH((attn_merge_kernel<float, 12, B>), grid, dim3(256), stream, kt, st, bb,
                         static_cast<float*>(o));
        else if (st.dtype == 0)
            A2T_DISPATCH((attn_merge_kernel<float, 8, B>), grid, dim3(256), stream, kt, st, bb,
                         static_cast<float*>(o));
        else if (wide)
            A2T_DISPATCH((attn_merge_kernel<bf16_t, 12, B>), grid, dim3(256), stream, kt, st, bb,
                         static_cast<bf16_t*>(o));
        else
            A2T_DISPATCH((attn_merge_kernel<bf16_t, 8, B>), grid, dim3(256), stream, kt, st, bb,
                         static_cast<bf16_t*>(o));
        return hipGetLastError();
    });
}

// ---- device-planned steps
hipError_t launch_dev_open(const DevState& st, const DevStepArgs& a, const int32_t* n_rows,
                           const int32_t* unit, const uint8_t* seg, const int32_t* pos,
                           DevPlan* plan, hipStream_t stream) {
    hipLaunchKernelGGL(dev_open_kernel, dim3(1), dim3(64), 0, stream, st, a, n_rows, unit, seg,
                       pos, plan);
    return hipGetLastError();
}

hipError_t launch_step_meta_dev(const DevState& st, const DevPlan* plan, int count,
                                const uint8_t* seg, const int32_t* pos, const int32_t* unit,
                                hipStream_t stream) {
    const DevBatch<StepDesc> b{{plan->step}, 0, 0};
    hipLaunchKernelGGL((step_meta_kernel<DevBatch<StepDesc>>), dim3(st.max_step_rows, count),
                       dim3(64), 0, stream, st, b, seg, pos, unit);
    return hipGetLastError();
}

hipError_t launch_attn_tile_dev(const DevState& st, const DevPlan* plan, int count,
                                int max_splits, int layer, const void* q, void* o,
                                const void* k_in, const void* v_in, hipStream_t stream) {
    const DevBatch<AttnDesc> b{{plan->attn}, layer, st.max_step_rows};
    const dim3 grid(max_splits * st.Hkv, 1, count);
    const uint16_t* qq = static_cast<const uint16_t*>(q);
    uint16_t* oo = static_cast<uint16_t*>(o);
    const uint16_t* ki = static_cast<const uint16_t*>(k_in);
    const uint16_t* vi = static_cast<const uint16_t*>(v_in);
    if (st.D == 128)
        hipLaunchKernelGGL((attn_tile_kernel<128, DevBatch<AttnDesc>>), grid, dim3(kMfmaThreads), 0,
                           stream, st, b, qq, oo, ki, vi);
    else if (st.D == 64)
        hipLaunchKernelGGL((attn_tile_kernel<64, DevBatch<AttnDesc>>), grid, dim3(kMfmaThreads), 0,
                           stream, st, b, qq, oo, ki, vi);
    else
        return hipErrorInvalidValue;
    return hipGetLastError();
}

hipError_t launch_attn_merge_dev(const DevState& st, const DevPlan* plan, int count,
                                 int max_splits, void* o, hipStream_t stream) {
    const int G = st.Hq / st.Hkv;
    if (st.D / 4 * kMergeRows > 256) return hipErrorInvalidValue;
    const DevBatch<AttnDesc> b{{plan->attn}, 0, st.max_step_rows};
    // at most kDevMergeGroups row groups per head; the kernel strides over the rest
    const int groups = std::min((G * st.max_step_rows + kMergeRows - 1) / kMergeRows, kDevMergeGroups);
    const dim3 grid(groups * st.Hkv, 1, count);
    const int nsg = 256 / (kMergeRows * st.D / 8);   // fp16 partials of the MFMA kernel
    if ((max_splits + nsg - 1) / nsg > 8)
        hipLaunchKernelGGL((attn_merge_kernel<bf16_t, 12, DevBatch<AttnDesc>, true>), grid, dim3(256), 0,
                           stream, st, b, static_cast<bf16_t*>(o));
    else
        hipLaunchKernelGGL((attn_merge_kernel<bf16_t, 8, DevBatch<AttnDesc>, true>), grid, dim3(256), 0,
                           stream, st, b, static_cast<bf16_t*>(o));
    return hipGetLastError();
}

hipError_t launch_dev_evict(const DevState& st, const DevStepArgs& a, const int32_t* budget,
                            int32_t* n_evicted, uint8_t* budget_unmet, DevPlan* plan,
                            hipStream_t stream) {
    hipLaunchKernelGGL(dev_evict_plan_kernel, dim3(a.count), dim3(256), 0, stream, st, a, budget,
                       n_evicted, budget_unmet, plan);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    const DevBatch<EvictDesc> b{{plan->evict}, 0, 0};
    if (st.dtype == 0)
        hipLaunchKernelGGL((evict_kernel<4, DevBatch<EvictDesc>>), dim3(st.L + 1, a.count), dim3(256),
                           0, stream, st, b);
    else
        hipLaunchKernelGGL((evict_kernel<2, DevBatch<EvictDesc>>), dim3(st.L + 1, a.count), dim3(256),
                           0, stream, st, b);
    return hipGetLastError();
}

hipError_t launch_evict(const DevState& st, const EvictBatch& b, hipStream_t stream,
                        const KTimer& kt) {
    const dim3 grid(st.L + 1, b.count);
    return by_size<EvictBatchT>(b, [&](const auto& bb) {
        using B = std::decay_t<decltype(bb)>;
        if (st.dtype == 0)
            A2T_DISPATCH((evict_kernel<4, B>), grid, dim3(256), stream, kt, st, bb);
        else
            A2T_DISPATCH((evict_kernel<2, B>), grid, dim3(256), stream, kt, st, bb);
        return hipGetLastError();
    });
}

}  // namespace a2t
