// The adaptation objective of Sec. 3.2 on given logits: masked cross-entropy
// over transcription rows, T^2 KL(P_T || P_S) at native rows with the teacher
// extended by zero probability on the added tokens, group-balanced means, and
// the gradient with respect to the student logits.  Public API: include/a2t.h.
//
//   distill_row_kernel     one workgroup per row.  Pass 1 streams the student
//                          and teacher rows once (16-byte loads, four chunks
//                          in flight per thread) keeping online statistics:
//                          (max, sum e^x) of the student at temperature T and
//                          at T = 1, and of the teacher at T, plus
//                          A = sum_v e^(w_v - m_w) (w_v - u_v), which gives
//                              KL = A / Z_w - lse(w) + lse(u)
//                          in the same pass (u = s/T, w = t/T).  Pass 2
//                          (optional) writes dL/ds.
//   distill_reduce_kernel  one workgroup: the four weighted sums over rows in
//                          a fixed order (deterministic).
// The weights of the four means are per-row coefficients computed on the host
// from the row metadata.
#include "../../include/a2t.h"

#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdint>
#include <cstring>
#include <new>
#include <vector>

namespace {

constexpr int kDistThreads = 256;
constexpr int kChunk = 8;     // elements per 16-byte (bf16) load
constexpr int kUnroll = 4;    // chunks in flight per thread

struct DistillRow {
    int32_t target;     // ASR target, -1 elsewhere
    float c_asr;        // weight of this row's CE in L_ASR
    float c_nat;        // weight of this row's KL in L_native
    float c_dec;        // ... in L_dec
    float c_turn;       // ... in L_turn
};

struct bf16_t {
    uint16_t bits;
};

__device__ __forceinline__ void load8(const float* p, float (&x)[kChunk]) {
    const float4 a = *reinterpret_cast<const float4*>(p);
    const float4 b = *reinterpret_cast<const float4*>(p + 4);
    x[0] = a.x; x[1] = a.y; x[2] = a.z; x[3] = a.w;
    x[4] = b.x; x[5] = b.y; x[6] = b.z; x[7] = b.w;
}
__device__ __forceinline__ void load8(const bf16_t* p, float (&x)[kChunk]) {
    const uint4 r = *reinterpret_cast<const uint4*>(p);
    const uint32_t w[4] = {r.x, r.y, r.z, r.w};
#pragma unroll
    for (int e = 0; e < 4; ++e) {
        x[2 * e] = __uint_as_float(w[e] << 16);
        x[2 * e + 1] = __uint_as_float(w[e] & 0xffff0000u);
    }
}
__device__ __forceinline__ float load1(const float* p) { return *p; }
__device__ __forceinline__ float load1(const bf16_t* p) { return __uint_as_float((uint32_t)p->bits << 16); }

__device__ __forceinline__ uint32_t pack2(float a, float b) {
    typedef __attribute__((__vector_size__(2 * sizeof(__bf16)))) __bf16 bf16x2;
    const bf16x2 v = {(__bf16)a, (__bf16)b};   // round to nearest even
    return __builtin_bit_cast(uint32_t, v);
}
__device__ __forceinline__ void store8(float* p, const float (&g)[kChunk]) {
    *reinterpret_cast<float4*>(p) = make_float4(g[0], g[1], g[2], g[3]);
    *reinterpret_cast<float4*>(p + 4) = make_float4(g[4], g[5], g[6], g[7]);
}
__device__ __forceinline__ void store8(bf16_t* p, const float (&g)[kChunk]) {
    *reinterpret_cast<uint4*>(p) = make_uint4(pack2(g[0], g[1]), pack2(g[2], g[3]),
                                              pack2(g[4], g[5]), pack2(g[6], g[7]));
}

// (max, sum e^(x - max)) pairs and the teacher triple, combined across lanes
struct Stats {
    float mu, zu;     // student at temperature T
    float m1, z1;     // student at T = 1
    float mw, zw, aw; // teacher at T, with A
};

__device__ __forceinline__ void merge_pair(float& m, float& z, float m2, float z2) {
    const float mn = fmaxf(m, m2);
    if (mn == -INFINITY) return;
    z = z * __expf(m - mn) + z2 * __expf(m2 - mn);
    m = mn;
}
__device__ __forceinline__ void merge_stats(Stats& a, const Stats& b) {
    merge_pair(a.mu, a.zu, b.mu, b.zu);
    merge_pair(a.m1, a.z1, b.m1, b.z1);
    const float mn = fmaxf(a.mw, b.mw);
    if (mn != -INFINITY) {
        const float sa = __expf(a.mw - mn), sb = __expf(b.mw - mn);
        a.zw = a.zw * sa + b.zw * sb;
        a.aw = a.aw * sa + b.aw * sb;
        a.mw = mn;
    }
}
__device__ __forceinline__ Stats shfl_stats(const Stats& s, int mask) {
    Stats o;
    o.mu = __shfl_xor(s.mu, mask);
    o.zu = __shfl_xor(s.zu, mask);
    o.m1 = __shfl_xor(s.m1, mask);
    o.z1 = __shfl_xor(s.z1, mask);
    o.mw = __shfl_xor(s.mw, mask);
    o.zw = __shfl_xor(s.zw, mask);
    o.aw = __shfl_xor(s.aw, mask);
    return o;
}

// grid: one workgroup per row.  Pass 1: statistics; pass 2 (grad != null): dL/ds.
template <typename T>
__global__ __launch_bounds__(kDistThreads) void distill_row_kernel(
    const T* student, int64_t s_stride, const T* teacher, int64_t t_stride, int vocab, int vs,
    const DistillRow* rows, float inv_t, int same_t, float2* rowval, T* grad) {
    const int i = blockIdx.x, tid = threadIdx.x;
    const DistillRow r = rows[i];
    const T* s = student + (int64_t)i * s_stride;
    const T* t = teacher + (int64_t)i * t_stride;
    const float wk = r.c_nat + r.c_dec + r.c_turn;  // KL weight in the gradient
    const float wc = r.c_asr;                       // CE weight in the gradient
    const int vs_pad = (vs + kChunk - 1) / kChunk * kChunk;

    if (wk == 0.f && wc == 0.f) {  // a row without loss: zero gradient
        if (grad) {
            const float z[kChunk] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
            for (int c = tid * kChunk; c < vs_pad; c += kDistThreads * kChunk)
                store8(grad + (int64_t)i * s_stride + c, z);
        }
        if (tid == 0) rowval[i] = make_float2(0.f, 0.f);
        return;
    }

    Stats st{-INFINITY, 0.f, -INFINITY, 0.f, -INFINITY, 0.f, 0.f};
    constexpr int kStep = kDistThreads * kChunk;
    for (int c0 = tid * kChunk; c0 < vs_pad; c0 += kStep * kUnroll) {
        float sv[kUnroll][kChunk], tv[kUnroll][kChunk];
        // all loads of the group first (clamped addresses, masked below)
#pragma unroll
        for (int k = 0; k < kUnroll; ++k) {
            const int c = c0 + k * kStep;
            const int cs = c < vs_pad ? c : vs_pad - kChunk;
            load8(s + cs, sv[k]);
            const int ct = c < vocab ? c : 0;
            load8(t + ct, tv[k]);
        }
#pragma unroll
        for (int k = 0; k < kUnroll; ++k) {
            const int c = c0 + k * kStep;
            if (c >= vs_pad) break;
            float u[kChunk], w[kChunk];
            float cu = -INFINITY, c1 = -INFINITY, cw = -INFINITY;
#pragma unroll
            for (int e = 0; e < kChunk; ++e) {
                const bool vs_ok = c + e < vs, v_ok = c + e < vocab;
                sv[k][e] = vs_ok ? sv[k][e] : -INFINITY;
                u[e] = vs_ok ? sv[k][e] * inv_t : -INFINITY;
                w[e] = v_ok ? tv[k][e] * inv_t : -INFINITY;
                cu = fmaxf(cu, u[e]);
                c1 = fmaxf(c1, sv[k][e]);
                cw = fmaxf(cw, w[e]);
            }
            {
                const float mn = fmaxf(st.mu, cu);
                float acc = 0.f;
#pragma unroll
                for (int e = 0; e < kChunk; ++e) acc += __expf(u[e] - mn);
                st.zu = st.zu * __expf(st.mu - mn) + acc;
                st.mu = mn;
            }
            if (!same_t) {
                const float mn = fmaxf(st.m1, c1);
                float acc = 0.f;
#pragma unroll
                for (int e = 0; e < kChunk; ++e) acc += __expf(sv[k][e] - mn);
                st.z1 = st.z1 * __expf(st.m1 - mn) + acc;
                st.m1 = mn;
            }
            if (cw != -INFINITY) {
                const float mn = fmaxf(st.mw, cw);
                const float sc = __expf(st.mw - mn);
                float zacc = 0.f, aacc = 0.f;
#pragma unroll
                for (int e = 0; e < kChunk; ++e) {
                    const float p = __expf(w[e] - mn);   // 0 past the teacher vocabulary
                    zacc += p;
                    aacc += (w[e] == -INFINITY) ? 0.f : p * (w[e] - u[e]);
                }
                st.zw = st.zw * sc + zacc;
                st.aw = st.aw * sc + aacc;
                st.mw = mn;
            }
        }
    }
    // reduce over the workgroup: waves by xor shuffles, then across waves in LDS
#pragma unroll
    for (int mask = 32; mask >= 1; mask >>= 1) merge_stats(st, shfl_stats(st, mask));
    __shared__ Stats part[kDistThreads / 64];
    if ((tid & 63) == 0) part[tid >> 6] = st;
    __syncthreads();
    Stats tot = part[0];
#pragma unroll
    for (int wv = 1; wv < kDistThreads / 64; ++wv) merge_stats(tot, part[wv]);
    const float lse_u = tot.mu + __logf(tot.zu);
    const float lse_w = tot.mw + __logf(tot.zw);
    const float lse_1 = same_t ? lse_u : tot.m1 + __logf(tot.z1);
    const float tt = 1.f / inv_t;
    if (tid == 0) {
        const float kl = (wk != 0.f) ? tt * tt * (tot.aw / tot.zw - lse_w + lse_u) : 0.f;
        const float ce = (wc != 0.f) ? lse_1 - load1(s + r.target) : 0.f;
        rowval[i] = make_float2(ce, kl);
    }
    if (!grad) return;
    // pass 2: dL/ds_v = wk T (softmax(u)_v - p_t,v) + wc (softmax(s)_v - [v == target])
    T* g = grad + (int64_t)i * s_stride;
    for (int c0 = tid * kChunk; c0 < vs_pad; c0 += kStep * kUnroll) {
        float sv[kUnroll][kChunk], tv[kUnroll][kChunk];
#pragma unroll
        for (int k = 0; k < kUnroll; ++k) {
            const int c = c0 + k * kStep;
            const int cs = c < vs_pad ? c : vs_pad - kChunk;
            load8(s + cs, sv[k]);
            const int ct = c < vocab ? c : 0;
            load8(t + ct, tv[k]);
        }
#pragma unroll
        for (int k = 0; k < kUnroll; ++k) {
            const int c = c0 + k * kStep;
            if (c >= vs_pad) break;
            float gv[kChunk];
#pragma unroll
            for (int e = 0; e < kChunk; ++e) {
                const int v = c + e;
                float x = 0.f;
                if (v < vs) {
                    const float ps = __expf(sv[k][e] * inv_t - lse_u);
                    const float pt = v < vocab ? __expf(tv[k][e] * inv_t - lse_w) : 0.f;
                    x = wk * tt * (ps - pt);
                    if (wc != 0.f) {
                        const float p1 = same_t ? ps : __expf(sv[k][e] - lse_1);
                        x += wc * (p1 - (v == r.target ? 1.f : 0.f));
                    }
                }
                gv[e] = x;
            }
            store8(g + c, gv);
        }
    }
}

// one workgroup: sum_i c_asr ce_i, c_nat kl_i, c_dec kl_i, c_turn kl_i in a fixed order
__global__ __launch_bounds__(kDistThreads) void distill_reduce_kernel(const DistillRow* rows,
                                                                      const float2* rowval, int n,
                                                                      float* losses) {
    const int tid = threadIdx.x;
    float a = 0.f, b = 0.f, c = 0.f, d = 0.f;
    for (int i = tid; i < n; i += kDistThreads) {
        const DistillRow r = rows[i];
        const float2 v = rowval[i];
        a += r.c_asr * v.x;
        b += r.c_nat * v.y;
        c += r.c_dec * v.y;
        d += r.c_turn * v.y;
    }
    __shared__ float4 sh[kDistThreads];
    sh[tid] = make_float4(a, b, c, d);
    __syncthreads();
    for (int w = kDistThreads / 2; w >= 1; w >>= 1) {
        if (tid < w) {
            const float4 x = sh[tid], y = sh[tid + w];
            sh[tid] = make_float4(x.x + y.x, x.y + y.y, x.z + y.z, x.w + y.w);
        }
        __syncthreads();
    }
    if (tid == 0) {
        const float4 t = sh[0];
        losses[0] = t.x;
        losses[1] = t.y;
        losses[2] = t.z;
        losses[3] = t.w;
        losses[4] = ((t.x + t.y) + t.z) + t.w;
    }
}

}  // namespace

// ------------------------------------------------------------------ host API
struct a2t_distill {
    int32_t max_rows = 0, vocab = 0, n_added = 0, dtype = 0, device = 0;
    hipStream_t stream = nullptr;
    DistillRow* rows_dev = nullptr;
    float2* rowval_dev = nullptr;
    DistillRow* stage[2] = {nullptr, nullptr};   // pinned host
    hipEvent_t stage_ev[2] = {nullptr, nullptr};
    bool stage_live[2] = {false, false};
    int next = 0;
    bool poisoned = false;
    // optional dispatch timestamps of the per-row kernel
    bool prof_on = false;
    std::vector<std::pair<hipEvent_t, hipEvent_t>> prof_pending, prof_free;
    int64_t prof_launches = 0;
    double prof_ms = 0.0;
};

namespace {
struct DevGuard {
    int prev = -1;
    explicit DevGuard(int dev) {
        if (hipGetDevice(&prev) != hipSuccess) prev = -1;
        if (prev != dev) (void)hipSetDevice(dev);
    }
    ~DevGuard() {
        if (prev >= 0) (void)hipSetDevice(prev);
    }
};
void free_distill(a2t_distill* d) {
    if (!d) return;
    for (int k = 0; k < 2; ++k) {
        if (d->stage_ev[k]) (void)hipEventDestroy(d->stage_ev[k]);
        if (d->stage[k]) (void)hipHostFree(d->stage[k]);
    }
    if (d->rows_dev) (void)hipFree(d->rows_dev);
    if (d->rowval_dev) (void)hipFree(d->rowval_dev);
    for (auto* v : {&d->prof_pending, &d->prof_free})
        for (auto& e : *v) {
            (void)hipEventDestroy(e.first);
            (void)hipEventDestroy(e.second);
        }
    delete d;
}
}  // namespace

extern "C" int a2t_distill_create(int32_t max_rows, int32_t vocab, int32_t n_added, int32_t dtype,
                                  int32_t device, void* hip_stream, a2t_distill** out) {
    if (!out) return A2T_ERR_INVALID;
    *out = nullptr;
    if (max_rows < 1 || vocab < 1 || n_added < 0 || (dtype != A2T_F32 && dtype != A2T_BF16) ||
        (int64_t)vocab + n_added > (1 << 30))
        return A2T_ERR_INVALID;
    int n_dev = 0;
    if (hipGetDeviceCount(&n_dev) != hipSuccess || device < 0 || device >= n_dev) return A2T_ERR_NODEV;
    DevGuard g(device);
    a2t_distill* d = new (std::nothrow) a2t_distill();
    if (!d) return A2T_ERR_OOM;
    d->max_rows = max_rows;
    d->vocab = vocab;
    d->n_added = n_added;
    d->dtype = dtype;
    d->device = device;
    d->stream = static_cast<hipStream_t>(hip_stream);
    bool ok = hipMalloc(&d->rows_dev, sizeof(DistillRow) * (size_t)max_rows) == hipSuccess &&
              hipMalloc(&d->rowval_dev, sizeof(float2) * (size_t)max_rows) == hipSuccess;
    for (int k = 0; k < 2 && ok; ++k)
        ok = hipHostMalloc(&d->stage[k], sizeof(DistillRow) * (size_t)max_rows, hipHostMallocDefault) ==
                 hipSuccess &&
             hipEventCreateWithFlags(&d->stage_ev[k], hipEventDisableTiming) == hipSuccess;
    if (!ok) {
        free_distill(d);
        return A2T_ERR_OOM;
    }
    *out = d;
    return A2T_OK;
}

extern "C" int a2t_distill_destroy(a2t_distill* d) {
    if (!d) return A2T_ERR_INVALID;
    {
        DevGuard g(d->device);
        (void)hipStreamSynchronize(d->stream);
    }
    free_distill(d);
    return A2T_OK;
}

extern "C" int a2t_distill_loss(a2t_distill* d, int32_t n_rows, const void* student,
                                int64_t student_stride, const void* teacher, int64_t teacher_stride,
                                const int8_t* kind, const int32_t* target, const int8_t* dec_group,
                                const int8_t* turn_group, float temperature, float* losses,
                                void* grad) {
    if (!d) return A2T_ERR_INVALID;
    if (d->poisoned) return A2T_ERR_HIP;
    const int vs = d->vocab + d->n_added;
    if (n_rows < 1 || n_rows > d->max_rows || !student || !teacher || !kind || !target ||
        !dec_group || !turn_group || !losses)
        return A2T_ERR_INVALID;
    if (student_stride < vs || teacher_stride < d->vocab || student_stride % 8 || teacher_stride % 8)
        return A2T_ERR_INVALID;
    auto misaligned = [](const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) != 0; };
    if (misaligned(student) || misaligned(teacher) || (grad && misaligned(grad)) ||
        (reinterpret_cast<uintptr_t>(losses) & 3u))
        return A2T_ERR_INVALID;
    if (!(temperature > 0.f) || !std::isfinite(temperature)) return A2T_ERR_INVALID;
    // row coefficients of the four means (Sec. 3.2)
    int64_t n_asr = 0, n_nat = 0, n_dec[3] = {0, 0, 0}, n_turn[2] = {0, 0};
    for (int i = 0; i < n_rows; ++i) {
        const int k = kind[i];
        if (k < A2T_ROW_NONE || k > A2T_ROW_NATIVE) return A2T_ERR_INVALID;
        if (dec_group[i] < -1 || dec_group[i] > 2 || turn_group[i] < -1 || turn_group[i] > 1)
            return A2T_ERR_INVALID;
        if (k == A2T_ROW_ASR) {
            if (target[i] < 0 || target[i] >= vs) return A2T_ERR_INVALID;
            ++n_asr;
        } else if (k == A2T_ROW_NATIVE) {
            ++n_nat;
            if (dec_group[i] >= 0) ++n_dec[dec_group[i]];
            if (turn_group[i] >= 0) ++n_turn[turn_group[i]];
        }
    }
    const int g_dec = (n_dec[0] > 0) + (n_dec[1] > 0) + (n_dec[2] > 0);
    const int g_turn = (n_turn[0] > 0) + (n_turn[1] > 0);
    DevGuard gd(d->device);
    const int slot = d->next;
    d->next ^= 1;
    if (d->stage_live[slot]) {
        if (hipEventSynchronize(d->stage_ev[slot]) != hipSuccess) {
            d->poisoned = true;
            return A2T_ERR_HIP;
        }
        d->stage_live[slot] = false;
    }
    DistillRow* h = d->stage[slot];
    for (int i = 0; i < n_rows; ++i) {
        DistillRow r{-1, 0.f, 0.f, 0.f, 0.f};
        if (kind[i] == A2T_ROW_ASR) {
            r.target = target[i];
            r.c_asr = (float)(1.0 / (double)n_asr);
        } else if (kind[i] == A2T_ROW_NATIVE) {
            r.c_nat = (float)(1.0 / (double)n_nat);
            if (dec_group[i] >= 0) r.c_dec = (float)(1.0 / ((double)g_dec * n_dec[dec_group[i]]));
            if (turn_group[i] >= 0) r.c_turn = (float)(1.0 / ((double)g_turn * n_turn[turn_group[i]]));
        }
        h[i] = r;
    }
    hipError_t e = hipMemcpyAsync(d->rows_dev, h, sizeof(DistillRow) * (size_t)n_rows,
                                  hipMemcpyHostToDevice, d->stream);
    if (e == hipSuccess) e = hipEventRecord(d->stage_ev[slot], d->stream);
    if (e == hipSuccess) d->stage_live[slot] = true;
    const float inv_t = 1.f / temperature;
    const int same_t = temperature == 1.f;
    if (e == hipSuccess) {
        std::pair<hipEvent_t, hipEvent_t> ev{nullptr, nullptr};
        if (d->prof_on) {
            if (d->prof_free.empty()) {
                hipEvent_t a = nullptr, b = nullptr;
                if (hipEventCreate(&a) == hipSuccess && hipEventCreate(&b) == hipSuccess)
                    d->prof_free.push_back({a, b});
            }
            if (!d->prof_free.empty()) {
                ev = d->prof_free.back();
                d->prof_free.pop_back();
            }
        }
        if (d->dtype == A2T_F32)
            hipExtLaunchKernelGGL((distill_row_kernel<float>), dim3(n_rows), dim3(kDistThreads), 0,
                                  d->stream, ev.first, ev.second, 0, static_cast<const float*>(student),
                                  student_stride, static_cast<const float*>(teacher), teacher_stride,
                                  d->vocab, vs, (const DistillRow*)d->rows_dev, inv_t, same_t,
                                  d->rowval_dev, static_cast<float*>(grad));
        else
            hipExtLaunchKernelGGL((distill_row_kernel<bf16_t>), dim3(n_rows), dim3(kDistThreads), 0,
                                  d->stream, ev.first, ev.second, 0,
                                  static_cast<const bf16_t*>(student), student_stride,
                                  static_cast<const bf16_t*>(teacher), teacher_stride, d->vocab, vs,
                                  (const DistillRow*)d->rows_dev, inv_t, same_t, d->rowval_dev,
                                  static_cast<bf16_t*>(grad));
        e = hipGetLastError();
        if (ev.first) d->prof_pending.push_back(ev);
    }
    if (e == hipSuccess) {
        hipLaunchKernelGGL(distill_reduce_kernel, dim3(1), dim3(kDistThreads), 0, d->stream,
                           d->rows_dev, d->rowval_dev, n_rows, losses);
        e = hipGetLastError();
    }
    if (e != hipSuccess) {
        d->poisoned = true;
        return A2T_ERR_HIP;
    }
    return A2T_OK;
}

extern "C" int a2t_distill_profile_enable(a2t_distill* d, int32_t enable) {
    if (!d) return A2T_ERR_INVALID;
    d->prof_on = enable != 0;
    return A2T_OK;
}

extern "C" int a2t_distill_profile_reserve(a2t_distill* d, int32_t n_launches) {
    if (!d || n_launches < 0) return A2T_ERR_INVALID;
    DevGuard g(d->device);
    while ((int64_t)d->prof_free.size() < (int64_t)n_launches) {
        hipEvent_t a = nullptr, b = nullptr;
        if (hipEventCreate(&a) != hipSuccess || hipEventCreate(&b) != hipSuccess) {
            if (a) (void)hipEventDestroy(a);
            (void)hipGetLastError();
            return A2T_ERR_OOM;
        }
        d->prof_free.push_back({a, b});
    }
    return A2T_OK;
}

extern "C" int a2t_distill_kernel_time(a2t_distill* d, int64_t* launches, double* total_ms) {
    if (!d || !launches || !total_ms) return A2T_ERR_INVALID;
    DevGuard g(d->device);
    for (auto& e : d->prof_pending) {
        if (hipEventSynchronize(e.second) != hipSuccess) return A2T_ERR_HIP;
        float ms = 0.f;
        if (hipEventElapsedTime(&ms, e.first, e.second) == hipSuccess) {
            d->prof_launches += 1;
            d->prof_ms += ms;
        }
        d->prof_free.push_back(e);
    }
    d->prof_pending.clear();
    *launches = d->prof_launches;
    *total_ms = d->prof_ms;
    d->prof_launches = 0;
    d->prof_ms = 0.0;
    return A2T_OK;
}
