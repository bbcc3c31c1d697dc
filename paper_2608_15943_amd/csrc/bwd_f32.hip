// Backward of the KV-shared layer for fp32 models (the small configurations): plain fp32
// on the vector ALUs, the same data flow as the bf16 path.  With S = Q K^T / sqrt(d)
// (masked), P = softmax(S), O = P V (Sec. 2.2, Eq. 2): dV = P^T dO, dP = dO V^T,
// dS = P * (dP - D), D = rowsum(dO * O), dQ = dS K / sqrt(d), dK = dS^T Q / sqrt(d); dQ and
// dK are rotated back through RoPE (orthogonal per position); a consumer's dK, dV add into
// its producer's fp32 sums (Eq. 3).  One thread per output row; d <= 128.
#include <math.h>

#include "common.h"
#include "kernels.h"

namespace kvp {
namespace {

// C[m][n] = R[m][n] + sum_k A(m, k) B(k, n) (R = 0 when res is null; res may equal c) with
// A(m, k) = a[m * sam + k * sak], B(k, n) = b[k * sbk + n * sbn]; C and R row stride ldc.
// One wave per (row, 64 columns): A is read wave-uniformly, B and C along rows.
__global__ __launch_bounds__(256) void gemm_f32s_kernel(const float* __restrict__ a, size_t sam, size_t sak,
                                                        const float* __restrict__ b, size_t sbk, size_t sbn,
                                                        const float* res, float* c, size_t ldc, int M, int N,
                                                        int K) {
    const int n = blockIdx.x * 64 + (threadIdx.x & 63);
    const int m = blockIdx.y * 4 + (threadIdx.x >> 6);
    if (m >= M || n >= N) return;
    float s = 0.f;
    for (int k = 0; k < K; ++k) s = fmaf(a[m * sam + k * sak], b[k * sbk + n * sbn], s);
    const size_t o = (size_t)m * ldc + n;
    c[o] = res ? res[o] + s : s;
}

// Per (token, head): the log-sum-exp of the scaled causal scores and D = dO . O.
template <int D>
__global__ __launch_bounds__(64) void stats_f32_kernel(const float* __restrict__ q, const float* __restrict__ kc,
                                                       const float* __restrict__ dO, const float* __restrict__ O,
                                                       float* __restrict__ lse, float* __restrict__ dsum, int B,
                                                       int S, int a, int g, int cap) {
    const int idx = blockIdx.x * blockDim.x + threadIdx.x;
    if (idx >= B * S * a) return;
    const int r = idx / a, h = idx - r * a, kvh = h / (a / g);
    const int b = r / S, pos = r - b * S;
    const float scale = 1.0f / sqrtf((float)D);
    const float* qr = q + ((size_t)r * a + h) * D;
    const float* kb = kc + ((size_t)b * g + kvh) * cap * D;
    float m = -INFINITY, l = 0.f;
    for (int t = 0; t <= pos; ++t) {
        float s = 0.f;
        for (int i = 0; i < D; ++i) s = fmaf(qr[i], kb[(size_t)t * D + i], s);
        s *= scale;
        const float m_new = fmaxf(m, s);
        l = l * expf(m - m_new) + expf(s - m_new);
        m = m_new;
    }
    lse[idx] = m + logf(l);
    float dd = 0.f;
    for (int i = 0; i < D; ++i) dd = fmaf(dO[((size_t)r * a + h) * D + i], O[((size_t)r * a + h) * D + i], dd);
    dsum[idx] = dd;
}

// dQ of one (token, head): sum over visible keys of dS K, scaled, rotated back.
template <int D>
__global__ __launch_bounds__(64) void dq_f32_kernel(const float* __restrict__ q, const float* __restrict__ kc,
                                                    const float* __restrict__ vc, const float* __restrict__ dO,
                                                    const float* __restrict__ lse, const float* __restrict__ dsum,
                                                    const float2* __restrict__ rope, float* __restrict__ out,
                                                    int ldo, int B, int S, int a, int g, int cap) {
    const int idx = blockIdx.x * blockDim.x + threadIdx.x;
    if (idx >= B * S * a) return;
    const int r = idx / a, h = idx - r * a, kvh = h / (a / g);
    const int b = r / S, pos = r - b * S;
    const float scale = 1.0f / sqrtf((float)D);
    const float* qr = q + ((size_t)r * a + h) * D;
    const float* dor = dO + ((size_t)r * a + h) * D;
    const float* kb = kc + ((size_t)b * g + kvh) * cap * D;
    const float* vb = vc + ((size_t)b * g + kvh) * D * cap;
    float acc[D];
    for (int i = 0; i < D; ++i) acc[i] = 0.f;
    const float L = lse[idx], Dd = dsum[idx];
    for (int t = 0; t <= pos; ++t) {
        float s = 0.f, dp = 0.f;
        for (int i = 0; i < D; ++i) {
            s = fmaf(qr[i], kb[(size_t)t * D + i], s);
            dp = fmaf(dor[i], vb[(size_t)i * cap + t], dp);
        }
        const float ds = expf(s * scale - L) * (dp - Dd);
        for (int i = 0; i < D; ++i) acc[i] = fmaf(ds, kb[(size_t)t * D + i], acc[i]);
    }
    const int half = D / 2;
    float* o = out + (size_t)r * ldo + h * D;
    for (int i = 0; i < half; ++i) {
        const float2 cs = rope[(size_t)pos * half + i];
        const float x1 = acc[i] * scale, x2 = acc[i + half] * scale;
        o[i] = x1 * cs.x + x2 * cs.y;
        o[i + half] = x2 * cs.x - x1 * cs.y;
    }
}

// dK, dV of one (sequence, KV head, key): sum over the later queries of the r heads.
template <int D>
__global__ __launch_bounds__(64) void dkv_f32_kernel(const float* __restrict__ q, const float* __restrict__ kc,
                                                     const float* __restrict__ vc, const float* __restrict__ dO,
                                                     const float* __restrict__ lse, const float* __restrict__ dsum,
                                                     const float2* __restrict__ rope,
                                                     const float* acc_in_k, const float* acc_in_v,
                                                     float* acc_out_k, float* acc_out_v, float* __restrict__ out,
                                                     int ldo, int col_k, int col_v, int B, int S, int a, int g,
                                                     int cap) {
    const int idx = blockIdx.x * blockDim.x + threadIdx.x;
    if (idx >= B * g * S) return;
    const int key = idx % S, bk = idx / S, b = bk / g, kvh = bk - b * g;
    const int r = a / g;
    const float scale = 1.0f / sqrtf((float)D);
    const float* kr = kc + (((size_t)b * g + kvh) * cap + key) * D;
    const float* vb = vc + ((size_t)b * g + kvh) * D * cap;
    float vk[D], dk[D], dv[D];
    for (int i = 0; i < D; ++i) {
        vk[i] = vb[(size_t)i * cap + key];
        dk[i] = 0.f;
        dv[i] = 0.f;
    }
    for (int j = kvh * r; j < (kvh + 1) * r; ++j)
        for (int t = key; t < S; ++t) {
            const size_t qi = ((size_t)(b * S + t) * a + j);
            const float* qr = q + qi * D;
            const float* dor = dO + qi * D;
            float s = 0.f, dp = 0.f;
            for (int i = 0; i < D; ++i) {
                s = fmaf(qr[i], kr[i], s);
                dp = fmaf(dor[i], vk[i], dp);
            }
            const float p = expf(s * scale - lse[qi]);
            const float ds = p * (dp - dsum[qi]);
            for (int i = 0; i < D; ++i) {
                dv[i] = fmaf(p, dor[i], dv[i]);
                dk[i] = fmaf(ds, qr[i], dk[i]);
            }
        }
    const int half = D / 2;
    const size_t ai = idx * (size_t)D;          // [B][g][S][D]
    for (int i = 0; i < half; ++i) {
        const float2 cs = rope[(size_t)key * half + i];
        const float x1 = dk[i] * scale, x2 = dk[i + half] * scale;
        dk[i] = x1 * cs.x + x2 * cs.y;
        dk[i + half] = x2 * cs.x - x1 * cs.y;
    }
    for (int i = 0; i < D; ++i) {
        float yk = dk[i], yv = dv[i];
        if (acc_in_k) {
            yk += acc_in_k[ai + i];
            yv += acc_in_v[ai + i];
        }
        if (acc_out_k) {
            acc_out_k[ai + i] = yk;
            acc_out_v[ai + i] = yv;
        }
        if (out) {
            float* row = out + (size_t)(b * S + key) * ldo + kvh * D;
            row[col_k + i] = yk;
            row[col_v + i] = yv;
        }
    }
}

}  // namespace

hipError_t gemm_f32_strided(const float* a, size_t sam, size_t sak, const float* b, size_t sbk, size_t sbn,
                            const float* res, float* c, size_t ldc, int M, int N, int K, hipStream_t st) {
    if (M < 1 || N < 1) return hipSuccess;
    hipLaunchKernelGGL(gemm_f32s_kernel, dim3((N + 63) / 64, (M + 3) / 4), dim3(256), 0, st, a, sam, sak, b, sbk,
                       sbn, res, c, ldc, M, N, K);
    return hipGetLastError();
}

hipError_t attn_bwd_f32(const AttnBwdF32& p, hipStream_t st) {
    const int nq_items = p.B * p.S * p.a, nk_items = p.B * p.g * p.S;
    const dim3 gq((nq_items + 63) / 64), gk((nk_items + 63) / 64), blk(64);
#define KVP_BWD_F32(DD)                                                                                            \
    hipLaunchKernelGGL(stats_f32_kernel<DD>, gq, blk, 0, st, p.q, p.kc, p.dO, p.O, p.lse, p.dsum, p.B, p.S, p.a,   \
                       p.g, p.cap);                                                                                \
    hipLaunchKernelGGL(dkv_f32_kernel<DD>, gk, blk, 0, st, p.q, p.kc, p.vc, p.dO, p.lse, p.dsum, p.rope,           \
                       p.acc_in_k, p.acc_in_v, p.acc_out_k, p.acc_out_v, p.out_kv, p.ldo, p.col_k, p.col_v, p.B,   \
                       p.S, p.a, p.g, p.cap);                                                                      \
    hipLaunchKernelGGL(dq_f32_kernel<DD>, gq, blk, 0, st, p.q, p.kc, p.vc, p.dO, p.lse, p.dsum, p.rope, p.out_q,   \
                       p.ldo, p.B, p.S, p.a, p.g, p.cap)
    switch (p.d) {
        case 16: KVP_BWD_F32(16); break;
        case 32: KVP_BWD_F32(32); break;
        case 64: KVP_BWD_F32(64); break;
        case 128: KVP_BWD_F32(128); break;
        default: return hipErrorInvalidValue;
    }
#undef KVP_BWD_F32
    return hipGetLastError();
}

}  // namespace kvp
