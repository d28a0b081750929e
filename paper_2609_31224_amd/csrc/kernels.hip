// HIP kernels of libA2T for gfx950 (CDNA4, wave64).
//
//   step_meta   writes a step's row metadata into the stream's ring slots and
//               the step's rotary table (cos, sin of pos * theta^(-2i/D),
//               evaluated in fp64, stored fp32).
//   append      rotates the step's keys by their positions and stores K and V
//               rows into the ring (Sec. 3.3: keys keep their original rotary
//               positions; they are never re-encoded later).
//   attn_mfma   causal chunk attention of a step's new rows over the resident
//               cache, bf16 MFMA 16x16x32 for Q.K^T and P.V, online softmax
//               with wave shuffles, key splits for parallelism.
//   attn_valu   the same attention on the vector ALU, one query row per
//               workgroup column: fp32 caches and single-row decode.
//   attn_merge  combines key-split partials (fixed order, deterministic).
//   evict       eviction and compaction (Sec. 3.3): a ballot/prefix-sum scan
//               over the passed-over ring rows keeps TEXT/RESPONSE/PREFIX rows
//               and drops ACOUSTIC/DELIM rows of evicted units, moves the kept
//               rows into the kept region in every layer, and writes the
//               eviction mask and compaction indices over the whole cache.
#include "a2t_internal.h"

#include <math.h>

namespace a2t {
namespace {

constexpr uint8_t kSegAcoustic = 1;
constexpr uint8_t kSegDelim = 2;

typedef __attribute__((__vector_size__(8 * sizeof(__bf16)))) __bf16 bf16x8;
typedef float f32x4 __attribute__((ext_vector_type(4)));

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

// ------------------------------------------------------------------ step_meta
__global__ __launch_bounds__(256) void step_meta_kernel(DevState st, StepBatch b,
                                                        const uint8_t* seg, const int32_t* pos,
                                                        const int32_t* uid) {
    __shared__ int32_t s_pos[1024];
    const StepDesc d = b.d[blockIdx.x];
    const int64_t mb = (int64_t)d.s * st.unit_rows;
    const int u = uid[blockIdx.x];
    for (int r = threadIdx.x; r < d.n; r += blockDim.x) {
        const int p = pos[d.row0 + r];
        s_pos[r] = p;
        int slot = d.slot0 + r;
        if (slot >= st.unit_rows) slot -= st.unit_rows;
        st.unit_pos[mb + slot] = p;
        st.unit_seg[mb + slot] = seg[d.row0 + r];
        st.unit_uid[mb + slot] = u;
    }
    __syncthreads();
    const int half = st.D / 2;
    float2* tab = st.rope + (int64_t)d.s * st.max_step_rows * half;
    for (int idx = threadIdx.x; idx < d.n * half; idx += blockDim.x) {
        const int r = idx / half, i = idx - r * half;
        const double inv = pow(st.theta, (-2.0 * i) / st.D);
        const double a = (double)s_pos[r] * inv;
        double sn, cs;
        sincos(a, &sn, &cs);
        tab[idx] = make_float2((float)cs, (float)sn);
    }
}

// --------------------------------------------------------------------- append
template <typename T>
__global__ __launch_bounds__(256) void append_kernel(DevState st, AppendBatch b, const T* k,
                                                     const T* v) {
    const int r = blockIdx.x;
    const AppendDesc d = b.d[blockIdx.y];
    if (r >= d.n) return;
    const int layer = b.layer0 + blockIdx.z;
    const int D = st.D, half = D / 2, Hkv = st.Hkv;
    int slot = d.slot0 + r;
    if (slot >= st.unit_rows) slot -= st.unit_rows;
    const int64_t in = ((int64_t)blockIdx.z * b.total_rows + d.in_row0 + r) * Hkv * D;
    const float2* cs = st.rope + ((int64_t)d.s * st.max_step_rows + r) * half;
    T* kd = reinterpret_cast<T*>(st.k_unit);
    T* vd = reinterpret_cast<T*>(st.v_unit);
    for (int idx = threadIdx.x; idx < Hkv * half; idx += blockDim.x) {
        const int g = idx / half, i = idx - g * half;
        const float x1 = Elt<T>::load(k + in + g * D + i);
        const float x2 = Elt<T>::load(k + in + g * D + i + half);
        const float2 c = cs[i];
        const int64_t o = pool_index(st, layer, d.s, g, st.unit_rows, slot);
        Elt<T>::store(kd + o + i, x1 * c.x - x2 * c.y);
        Elt<T>::store(kd + o + i + half, x2 * c.x + x1 * c.y);
    }
    for (int idx = threadIdx.x; idx < Hkv * D; idx += blockDim.x) {
        const int g = idx / D, e = idx - g * D;
        vd[pool_index(st, layer, d.s, g, st.unit_rows, slot) + e] = v[in + idx];
    }
}

// ----------------------------------------------------------------- attn_valu
// One workgroup = (key split, kv head g, query row i, stream).  256 threads
// form 16 key groups of 16 lanes; a lane holds D/16 consecutive elements of a
// row.  Scores are reduced across the 16 lanes with xor shuffles; every key
// group runs its own online softmax, and the 16 states are merged in LDS.
template <typename T, int D, int G>
__global__ __launch_bounds__(256) void attn_valu_kernel(DevState st, AttnBatch b, const T* q,
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

// ----------------------------------------------------------------- attn_mfma
// One workgroup = (key split, kv head g, stream), 4 waves.  The M = G*n_q
// query rows of the head group are processed 128 at a time; each wave owns 32
// of them (two 16-column blocks).  Per 64-key tile, K (row-major) and V^T are
// staged in LDS by all 256 threads, with the next tile's global loads issued
// before the current tile's math.
//
// S^T = K . Q^T with mfma_f32_16x16x32_bf16: A = K rows (16 keys x 32 dims),
// B = Q^T (32 dims x 16 queries); the accumulator gives lane l the scores of
// keys 4*(l/16)+e, e<4, for query l%16.  P^T then feeds P.V directly as the
// B operand of O^T = V^T . P^T: within a 32-key chunk, k-slot 8*(l/16)+j maps
// to key 16*(j/4) + 4*(l/16) + j%4, which is exactly what lane l holds; the A
// operand reads the same keys from V^T in LDS.  No cross-lane transposes.
template <int D>
__global__ __launch_bounds__(256) void attn_mfma_kernel(DevState st, AttnBatch b,
                                                        const uint16_t* q, uint16_t* o) {
    constexpr int KS = D / 32;      // k-steps of Q.K^T
    constexpr int DB = D / 16;      // 16-row blocks of V^T
    constexpr int CPR = D / 8;      // 16-byte chunks per K/V row
    constexpr int KROW = D + 8;     // LDS row stride of K (bf16 elements)
    constexpr int VROW = kTileKeys + 8;  // LDS row stride of V^T
    constexpr int NK = kTileKeys * CPR / 256;         // K chunks per thread
    constexpr int NVQ = (kTileKeys / 4) * CPR;        // V (4-key x 8-dim) blocks per tile
    __shared__ __attribute__((aligned(16))) uint16_t Ks[kTileKeys * KROW];
    __shared__ __attribute__((aligned(16))) uint16_t Vt[D * VROW];

    const AttnDesc d = b.d[blockIdx.z];
    const int g = blockIdx.y, sp = blockIdx.x;
    if (sp >= d.splits) return;
    const int G = st.Hq / st.Hkv, nq = d.n_q, M = G * nq, R = d.R;
    const int tid = threadIdx.x, w = tid >> 6, lane = tid & 63, l16 = lane & 15, lg = lane >> 4;
    const int n_tiles = (R + kTileKeys - 1) / kTileKeys;
    const int t0 = sp * n_tiles / d.splits, t1 = (sp + 1) * n_tiles / d.splits;
    const int vis0 = R - nq;  // query row i sees keys 0 .. vis0 + i

    const uint16_t* kk = reinterpret_cast<const uint16_t*>(st.k_kept);
    const uint16_t* vk = reinterpret_cast<const uint16_t*>(st.v_kept);
    const uint16_t* ku = reinterpret_cast<const uint16_t*>(st.k_unit);
    const uint16_t* vu = reinterpret_cast<const uint16_t*>(st.v_unit);

    uint4 kreg[NK];
    uint4 vreg[4];

    auto gload = [&](int t) {
        const int kb = t * kTileKeys;
#pragma unroll
        for (int it = 0; it < NK; ++it) {
            const int c = tid + 256 * it;
            const int row = c / CPR, col = c - row * CPR;
            const int j = kb + row;
            if (j < R) {
                bool in_kept;
                const int64_t r = key_row(st, b.layer, d.s, g, d.kept, d.head, j, &in_kept);
                kreg[it] = *reinterpret_cast<const uint4*>((in_kept ? kk : ku) + r + col * 8);
            } else {
                kreg[it] = make_uint4(0, 0, 0, 0);
            }
        }
        if (tid < NVQ) {
            const int kq = tid / CPR, dc = tid - kq * CPR;
#pragma unroll
            for (int r4 = 0; r4 < 4; ++r4) {
                const int j = kb + 4 * kq + r4;
                if (j < R) {
                    bool in_kept;
                    const int64_t r = key_row(st, b.layer, d.s, g, d.kept, d.head, j, &in_kept);
                    vreg[r4] = *reinterpret_cast<const uint4*>((in_kept ? vk : vu) + r + dc * 8);
                } else {
                    vreg[r4] = make_uint4(0, 0, 0, 0);
                }
            }
        }
    };
    auto lstore = [&]() {
#pragma unroll
        for (int it = 0; it < NK; ++it) {
            const int c = tid + 256 * it;
            const int row = c / CPR, col = c - row * CPR;
            *reinterpret_cast<uint4*>(&Ks[row * KROW + col * 8]) = kreg[it];
        }
        if (tid < NVQ) {
            const int kq = tid / CPR, dc = tid - kq * CPR;
            const uint32_t* v0 = reinterpret_cast<const uint32_t*>(&vreg[0]);
            const uint32_t* v1 = reinterpret_cast<const uint32_t*>(&vreg[1]);
            const uint32_t* v2 = reinterpret_cast<const uint32_t*>(&vreg[2]);
            const uint32_t* v3 = reinterpret_cast<const uint32_t*>(&vreg[3]);
#pragma unroll
            for (int e = 0; e < 8; ++e) {
                const int wd = e >> 1;
                uint32_t a, c2;
                if ((e & 1) == 0) {
                    a = (v0[wd] & 0xffffu) | (v1[wd] << 16);
                    c2 = (v2[wd] & 0xffffu) | (v3[wd] << 16);
                } else {
                    a = (v0[wd] >> 16) | (v1[wd] & 0xffff0000u);
                    c2 = (v2[wd] >> 16) | (v3[wd] & 0xffff0000u);
                }
                *reinterpret_cast<uint2*>(&Vt[(dc * 8 + e) * VROW + 4 * kq]) = make_uint2(a, c2);
            }
        }
    };

    const float2* rope = st.rope + ((int64_t)d.s * st.max_step_rows + d.rope_row0) * (D / 2);

    for (int qg0 = 0; qg0 < M; qg0 += 128) {
        const int mw = qg0 + 32 * w;
        const bool active = mw < M;

        // Q^T operand: rotated, scaled by scale*log2(e), bf16.
        bf16x8 qop[2][KS];
#pragma unroll
        for (int qb = 0; qb < 2; ++qb) {
            const int mq = mw + 16 * qb + l16;
            float x[KS][8];
            if (mq < M) {
                const int i = mq / G, hh = mq - i * G;
                const uint16_t* qp = q + ((int64_t)(d.q_row0 + i) * st.Hq + g * G + hh) * D;
#pragma unroll
                for (int s = 0; s < KS; ++s) {
                    const uint4 raw = *reinterpret_cast<const uint4*>(qp + 32 * s + 8 * lg);
                    const uint32_t* rw = reinterpret_cast<const uint32_t*>(&raw);
#pragma unroll
                    for (int e = 0; e < 8; ++e)
                        x[s][e] = bf16_to_f32((uint16_t)(rw[e >> 1] >> (16 * (e & 1))));
                }
                const float2* cs = rope + (int64_t)i * (D / 2);
#pragma unroll
                for (int s = 0; s < KS / 2; ++s) {
#pragma unroll
                    for (int e = 0; e < 8; ++e) {
                        const float2 c = cs[32 * s + 8 * lg + e];
                        const float a = x[s][e], bb = x[s + KS / 2][e];
                        x[s][e] = (a * c.x - bb * c.y) * st.scale_log2e;
                        x[s + KS / 2][e] = (bb * c.x + a * c.y) * st.scale_log2e;
                    }
                }
            } else {
#pragma unroll
                for (int s = 0; s < KS; ++s)
#pragma unroll
                    for (int e = 0; e < 8; ++e) x[s][e] = 0.f;
            }
#pragma unroll
            for (int s = 0; s < KS; ++s) {
                uint32_t pk[4];
#pragma unroll
                for (int e2 = 0; e2 < 4; ++e2)
                    pk[e2] = (uint32_t)f32_to_bf16(x[s][2 * e2]) |
                             ((uint32_t)f32_to_bf16(x[s][2 * e2 + 1]) << 16);
                qop[qb][s] = __builtin_bit_cast(bf16x8, make_uint4(pk[0], pk[1], pk[2], pk[3]));
            }
        }

        float mrun[2] = {-INFINITY, -INFINITY}, lrun[2] = {0.f, 0.f};
        f32x4 acc[DB][2];
#pragma unroll
        for (int db = 0; db < DB; ++db)
#pragma unroll
            for (int qb = 0; qb < 2; ++qb) acc[db][qb] = f32x4{0.f, 0.f, 0.f, 0.f};

        if (t0 < t1) gload(t0);
        for (int t = t0; t < t1; ++t) {
            __syncthreads();  // every wave is done reading the previous tile
            lstore();
            __syncthreads();
            if (t + 1 < t1) gload(t + 1);
            if (!active) continue;
            const int kbase = t * kTileKeys;

            f32x4 sacc[4][2];
#pragma unroll
            for (int kb = 0; kb < 4; ++kb)
#pragma unroll
                for (int qb = 0; qb < 2; ++qb) sacc[kb][qb] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int s = 0; s < KS; ++s) {
#pragma unroll
                for (int kb = 0; kb < 4; ++kb) {
                    const bf16x8 a = *reinterpret_cast<const bf16x8*>(
                        &Ks[(kb * 16 + l16) * KROW + 32 * s + 8 * lg]);
#pragma unroll
                    for (int qb = 0; qb < 2; ++qb)
                        sacc[kb][qb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
                            a, qop[qb][s], sacc[kb][qb], 0, 0, 0);
                }
            }
            if (kbase + kTileKeys - 1 > vis0) {
#pragma unroll
                for (int qb = 0; qb < 2; ++qb) {
                    const int mq = mw + 16 * qb + l16;
                    const int lim = (mq < M) ? vis0 + mq / G : -1;
#pragma unroll
                    for (int kb = 0; kb < 4; ++kb)
#pragma unroll
                        for (int e = 0; e < 4; ++e) {
                            const int j = kbase + kb * 16 + 4 * lg + e;
                            if (j > lim) sacc[kb][qb][e] = -INFINITY;
                        }
                }
            }

            bf16x8 pop[2][2];
#pragma unroll
            for (int qb = 0; qb < 2; ++qb) {
                float tmax = -INFINITY;
#pragma unroll
                for (int kb = 0; kb < 4; ++kb)
#pragma unroll
                    for (int e = 0; e < 4; ++e) tmax = fmaxf(tmax, sacc[kb][qb][e]);
                tmax = fmaxf(tmax, __shfl_xor(tmax, 16));
                tmax = fmaxf(tmax, __shfl_xor(tmax, 32));
                const float mn = fmaxf(mrun[qb], tmax);
                const float mu = (mn == -INFINITY) ? 0.f : mn;
                const float corr = exp2f(mrun[qb] - mu);
                float rs = 0.f;
                uint32_t pk[4][2];
#pragma unroll
                for (int kb = 0; kb < 4; ++kb) {
                    uint16_t h[4];
#pragma unroll
                    for (int e = 0; e < 4; ++e) {
                        h[e] = f32_to_bf16(exp2f(sacc[kb][qb][e] - mu));
                        rs += bf16_to_f32(h[e]);
                    }
                    pk[kb][0] = (uint32_t)h[0] | ((uint32_t)h[1] << 16);
                    pk[kb][1] = (uint32_t)h[2] | ((uint32_t)h[3] << 16);
                }
                rs += __shfl_xor(rs, 16);
                rs += __shfl_xor(rs, 32);
                lrun[qb] = lrun[qb] * corr + rs;
                mrun[qb] = mn;
#pragma unroll
                for (int db = 0; db < DB; ++db) acc[db][qb] *= corr;
#pragma unroll
                for (int c = 0; c < 2; ++c)
                    pop[c][qb] = __builtin_bit_cast(
                        bf16x8, make_uint4(pk[2 * c][0], pk[2 * c][1], pk[2 * c + 1][0],
                                           pk[2 * c + 1][1]));
            }

#pragma unroll
            for (int c = 0; c < 2; ++c) {
#pragma unroll
                for (int db = 0; db < DB; ++db) {
                    const uint16_t* vr = &Vt[(db * 16 + l16) * VROW + 32 * c + 4 * lg];
                    const uint2 lo = *reinterpret_cast<const uint2*>(vr);
                    const uint2 hi = *reinterpret_cast<const uint2*>(vr + 16);
                    const bf16x8 a = __builtin_bit_cast(bf16x8, make_uint4(lo.x, lo.y, hi.x, hi.y));
#pragma unroll
                    for (int qb = 0; qb < 2; ++qb)
                        acc[db][qb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, pop[c][qb],
                                                                             acc[db][qb], 0, 0, 0);
                }
            }
        }

        if (active) {
#pragma unroll
            for (int qb = 0; qb < 2; ++qb) {
                const int mq = mw + 16 * qb + l16;
                if (mq >= M) continue;
                const int i = mq / G, hh = mq - i * G;
                if (d.splits == 1) {
                    const float inv = 1.f / lrun[qb];
                    uint16_t* op = o + ((int64_t)(d.q_row0 + i) * st.Hq + g * G + hh) * D;
#pragma unroll
                    for (int db = 0; db < DB; ++db) {
                        const f32x4 a = acc[db][qb];
                        const uint32_t lo = (uint32_t)f32_to_bf16(a[0] * inv) |
                                            ((uint32_t)f32_to_bf16(a[1] * inv) << 16);
                        const uint32_t hi = (uint32_t)f32_to_bf16(a[2] * inv) |
                                            ((uint32_t)f32_to_bf16(a[3] * inv) << 16);
                        *reinterpret_cast<uint2*>(op + db * 16 + 4 * lg) = make_uint2(lo, hi);
                    }
                } else {
                    float* po = st.ws + d.ws_off;
                    float* prow = po + (((int64_t)sp * st.Hkv + g) * M + mq) * D;
#pragma unroll
                    for (int db = 0; db < DB; ++db)
                        *reinterpret_cast<f32x4*>(prow + db * 16 + 4 * lg) = acc[db][qb];
                    if (lg == 0) {
                        float* pml = po + (int64_t)d.splits * st.Hkv * M * D;
                        pml[(((int64_t)sp * st.Hkv + g) * M + mq) * 2 + 0] = mrun[qb];
                        pml[(((int64_t)sp * st.Hkv + g) * M + mq) * 2 + 1] = lrun[qb];
                    }
                }
            }
        }
        __syncthreads();
    }
}

// ----------------------------------------------------------------- attn_merge
template <typename T>
__global__ __launch_bounds__(256) void attn_merge_kernel(DevState st, AttnBatch b, T* o) {
    const AttnDesc d = b.d[blockIdx.z];
    if (d.splits <= 1) return;
    const int G = st.Hq / st.Hkv, M = G * d.n_q, D = st.D, g = blockIdx.y;
    const int idx = blockIdx.x * blockDim.x + threadIdx.x;
    if (idx >= M * D) return;
    const int mq = idx / D, dd = idx - mq * D;
    const float* po = st.ws + d.ws_off;
    const float* pml = po + (int64_t)d.splits * st.Hkv * M * D;
    float mx = -INFINITY;
    for (int sp = 0; sp < d.splits; ++sp)
        mx = fmaxf(mx, pml[(((int64_t)sp * st.Hkv + g) * M + mq) * 2]);
    float L = 0.f, O = 0.f;
    for (int sp = 0; sp < d.splits; ++sp) {
        const int64_t r = ((int64_t)sp * st.Hkv + g) * M + mq;
        const float ms = pml[r * 2];
        const float wgt = (ms == -INFINITY) ? 0.f : exp2f(ms - mx);
        L += wgt * pml[r * 2 + 1];
        O += wgt * po[r * D + dd];
    }
    const int i = mq / G, hh = mq - i * G;
    Elt<T>::store(o + ((int64_t)(d.q_row0 + i) * st.Hq + g * G + hh) * D + dd, O / L);
}

// ---------------------------------------------------------------------- evict
// grid (L + 1, streams).  Workgroups 0..L-1 move the retained rows of the
// passed-over ring span into the kept region of their layer; workgroup L
// writes the kept-region metadata and the mask / compaction indices over the
// whole pre-eviction cache.  Each workgroup ranks the span's rows itself
// (wave ballot + popcount, then a cross-wave prefix in LDS).
template <int ELT>
__global__ __launch_bounds__(256) void evict_kernel(DevState st, EvictBatch b) {
    __shared__ int s_wave[4];
    __shared__ int s_src[256];
    __shared__ int s_dst[256];
    const EvictDesc d = b.d[blockIdx.y];
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
            const uint8_t sg = st.unit_seg[mb + slot];
            const int uid = st.unit_uid[mb + slot];
            keep = !((sg == kSegAcoustic || sg == kSegDelim) && uid <= d.u_last);
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

}  // namespace

// ------------------------------------------------------------------ launchers
hipError_t launch_step_meta(const DevState& st, const StepBatch& b, const uint8_t* seg,
                            const int32_t* pos, const int32_t* uid, hipStream_t stream) {
    hipLaunchKernelGGL(step_meta_kernel, dim3(b.count), dim3(256), 0, stream, st, b, seg, pos, uid);
    return hipGetLastError();
}

hipError_t launch_append(const DevState& st, const AppendBatch& b, int n_layers, const void* k,
                         const void* v, hipStream_t stream) {
    const dim3 grid(b.max_n, b.count, n_layers);
    if (st.dtype == 0)
        hipLaunchKernelGGL(append_kernel<float>, grid, dim3(128), 0, stream, st, b,
                           static_cast<const float*>(k), static_cast<const float*>(v));
    else
        hipLaunchKernelGGL(append_kernel<bf16_t>, grid, dim3(128), 0, stream, st, b,
                           static_cast<const bf16_t*>(k), static_cast<const bf16_t*>(v));
    return hipGetLastError();
}

hipError_t launch_attn_mfma(const DevState& st, const AttnBatch& b, const void* q, void* o,
                            hipStream_t stream) {
    const dim3 grid(b.max_splits, st.Hkv, b.count);
    const uint16_t* qq = static_cast<const uint16_t*>(q);
    uint16_t* oo = static_cast<uint16_t*>(o);
    if (st.D == 128)
        hipLaunchKernelGGL(attn_mfma_kernel<128>, grid, dim3(256), 0, stream, st, b, qq, oo);
    else if (st.D == 64)
        hipLaunchKernelGGL(attn_mfma_kernel<64>, grid, dim3(256), 0, stream, st, b, qq, oo);
    else
        return hipErrorInvalidValue;
    return hipGetLastError();
}

template <typename T, int D>
static hipError_t valu_dispatch_g(const DevState& st, const AttnBatch& b, const void* q, void* o,
                                  hipStream_t stream) {
    const dim3 grid(b.max_splits, st.Hkv * b.max_rows, b.count);
    const T* qq = static_cast<const T*>(q);
    T* oo = static_cast<T*>(o);
    switch (st.Hq / st.Hkv) {
        case 1: hipLaunchKernelGGL((attn_valu_kernel<T, D, 1>), grid, dim3(256), 0, stream, st, b, qq, oo); break;
        case 2: hipLaunchKernelGGL((attn_valu_kernel<T, D, 2>), grid, dim3(256), 0, stream, st, b, qq, oo); break;
        case 4: hipLaunchKernelGGL((attn_valu_kernel<T, D, 4>), grid, dim3(256), 0, stream, st, b, qq, oo); break;
        case 8: hipLaunchKernelGGL((attn_valu_kernel<T, D, 8>), grid, dim3(256), 0, stream, st, b, qq, oo); break;
        default: return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

hipError_t launch_attn_valu(const DevState& st, const AttnBatch& b, const void* q, void* o,
                            hipStream_t stream) {
    if (st.dtype == 0) {
        if (st.D == 128) return valu_dispatch_g<float, 128>(st, b, q, o, stream);
        if (st.D == 64) return valu_dispatch_g<float, 64>(st, b, q, o, stream);
    } else {
        if (st.D == 128) return valu_dispatch_g<bf16_t, 128>(st, b, q, o, stream);
        if (st.D == 64) return valu_dispatch_g<bf16_t, 64>(st, b, q, o, stream);
    }
    return hipErrorInvalidValue;
}

hipError_t launch_attn_merge(const DevState& st, const AttnBatch& b, void* o, hipStream_t stream) {
    const int G = st.Hq / st.Hkv;
    const int max_elems = G * b.max_rows * st.D;
    const dim3 grid((max_elems + 255) / 256, st.Hkv, b.count);
    if (st.dtype == 0)
        hipLaunchKernelGGL(attn_merge_kernel<float>, grid, dim3(256), 0, stream, st, b,
                           static_cast<float*>(o));
    else
        hipLaunchKernelGGL(attn_merge_kernel<bf16_t>, grid, dim3(256), 0, stream, st, b,
                           static_cast<bf16_t*>(o));
    return hipGetLastError();
}

hipError_t launch_evict(const DevState& st, const EvictBatch& b, hipStream_t stream) {
    const dim3 grid(st.L + 1, b.count);
    if (st.dtype == 0)
        hipLaunchKernelGGL(evict_kernel<4>, grid, dim3(256), 0, stream, st, b);
    else
        hipLaunchKernelGGL(evict_kernel<2>, grid, dim3(256), 0, stream, st, b);
    return hipGetLastError();
}

}  // namespace a2t
