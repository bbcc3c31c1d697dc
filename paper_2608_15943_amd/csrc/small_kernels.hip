// Smaller kernels of the path:
//   rope_table    -- cos/sin of pos * theta_i in double, stored as fp32 pairs.
//   rope_scatter  -- RoPE on fp32 projections, then Q to its buffer and K, V
//                    (transposed) into the producer's slot; used by decode
//                    (position len_b of each sequence) and by fp32 models.
//   gemm_f32, attn_f32 -- the full-precision path for fp32 models (vector
//                    ALU, no reduced-precision matrix modes).
#include <math.h>

#include "common.h"
#include "kernels.h"

namespace kvp {
namespace {

__device__ __forceinline__ const void* w_row_any(const WRows& w, int n, int K, int esize) {
    const char* base;
    if (n < w.rows[0]) {
        base = (const char*)w.p[0];
    } else if (n < w.rows[0] + w.rows[1]) {
        n -= w.rows[0];
        base = (const char*)w.p[1];
    } else {
        n -= w.rows[0] + w.rows[1];
        base = (const char*)w.p[2];
    }
    return base + (size_t)n * K * esize;
}

// ---------------------------------------------------------------------------
// RoPE
// ---------------------------------------------------------------------------

__global__ void rope_table_kernel(float2* t, int S, int half, int d, double base) {
    const int idx = blockIdx.x * blockDim.x + threadIdx.x;
    if (idx >= S * half) return;
    const int pos = idx / half, i = idx - pos * half;
    const double theta = pow(base, -2.0 * i / d);
    double s, c;
    sincos((double)pos * theta, &s, &c);
    t[idx] = make_float2((float)c, (float)s);
}

template <typename T>
__device__ __forceinline__ void put(T* p, size_t i, float v);
template <>
__device__ __forceinline__ void put<float>(float* p, size_t i, float v) { p[i] = v; }
template <>
__device__ __forceinline__ void put<uint16_t>(uint16_t* p, size_t i, float v) { p[i] = f2bf(v); }

template <typename T>
__global__ __launch_bounds__(256) void rope_scatter_kernel(const float* __restrict__ proj, int nsplit,
                                                           size_t split_stride, int S,
                                                           const int32_t* __restrict__ lens, int a,
                                                           int g, int d, int cap, double base,
                                                           int producer, T* q, T* kc, T* vc) {
    __shared__ float2 cs[64];                 // (cos, sin) of this row's position, d / 2 <= 64
    const int r = blockIdx.x;
    int b, pos;
    if (lens) {
        b = r;
        pos = max(0, min(lens[r], cap - 1));   // never outside the slot
    } else {
        b = r / S;
        pos = r - b * S;
    }
    const int half = d / 2, nq = a * d, nkv = g * d;
    const int ncols = nq + (producer ? 2 * nkv : 0);
    const float* pr = proj + (size_t)r * ncols;
    // Sum of the K slices of the projection (one slice unless the GEMM split K).
    auto val = [&](int c) {
        float v = pr[c];
        for (int s = 1; s < nsplit; ++s) v += pr[(size_t)s * split_stride + c];
        return v;
    };
    for (int i = threadIdx.x; i < half; i += blockDim.x) {
        const double theta = pow(base, -2.0 * i / d);
        double sd, cd;
        sincos((double)pos * theta, &sd, &cd);
        cs[i] = make_float2((float)cd, (float)sd);
    }
    __syncthreads();
    const int heads = a + (producer ? g : 0);
    for (int j = threadIdx.x; j < heads * half; j += blockDim.x) {
        const int h = j / half, i = j - h * half;
        const float c = cs[i].x, s = cs[i].y;
        const float x1 = val(h * d + i), x2 = val(h * d + i + half);
        const float o1 = x1 * c - x2 * s, o2 = x2 * c + x1 * s;
        if (h < a) {
            put(q, (size_t)r * nq + h * d + i, o1);
            put(q, (size_t)r * nq + h * d + i + half, o2);
        } else {
            const size_t kb = (((size_t)b * g + (h - a)) * cap + pos) * d;
            put(kc, kb + i, o1);
            put(kc, kb + i + half, o2);
        }
    }
    if (producer) {
        for (int j = threadIdx.x; j < nkv; j += blockDim.x) {
            const int h = j / d, c = j - h * d;
            put(vc, (((size_t)b * g + h) * d + c) * cap + pos, val(nq + nkv + j));
        }
    }
}

// ---------------------------------------------------------------------------
// fp32 path
// ---------------------------------------------------------------------------

__global__ __launch_bounds__(256) void gemm_f32_kernel(const float* __restrict__ A, WRows W, int M,
                                                       int N, int K, float* __restrict__ out,
                                                       const float* __restrict__ xres) {
    // 32 x 32 output tile (2 x 2 per thread), 64-wide K steps with all of a step's loads in
    // flight at once: the fp32 models' GEMMs are small, so parallelism and latency matter.
    __shared__ float As[64][36], Ws[64][36];
    const int tid = threadIdx.x, tx = tid & 15, ty = tid >> 4;
    const int m0 = blockIdx.y * 32, n0 = blockIdx.x * 32;
    float acc[2][2] = {};
    for (int k0 = 0; k0 < K; k0 += 64) {
        float av_[8], wv_[8];
#pragma unroll
        for (int i = 0; i < 8; ++i) {
            const int id = tid + 256 * i, row = id >> 6, kk = id & 63;
            const int m = m0 + row, n = n0 + row, k = k0 + kk;
            av_[i] = (m < M && k < K) ? A[(size_t)m * K + k] : 0.f;
            wv_[i] = (n < N && k < K) ? ((const float*)w_row_any(W, n, K, 4))[k] : 0.f;
        }
#pragma unroll
        for (int i = 0; i < 8; ++i) {
            const int id = tid + 256 * i, row = id >> 6, kk = id & 63;
            As[kk][row] = av_[i];
            Ws[kk][row] = wv_[i];
        }
        __syncthreads();
#pragma unroll 16
        for (int kk = 0; kk < 64; ++kk) {
            const float a0 = As[kk][ty * 2], a1 = As[kk][ty * 2 + 1];
            const float b0 = Ws[kk][tx * 2], b1 = Ws[kk][tx * 2 + 1];
            acc[0][0] = fmaf(a0, b0, acc[0][0]);
            acc[0][1] = fmaf(a0, b1, acc[0][1]);
            acc[1][0] = fmaf(a1, b0, acc[1][0]);
            acc[1][1] = fmaf(a1, b1, acc[1][1]);
        }
        __syncthreads();
    }
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j) {
            const int m = m0 + ty * 2 + i, n = n0 + tx * 2 + j;
            if (m < M && n < N) {
                const size_t off = (size_t)m * N + n;
                out[off] = xres ? xres[off] + acc[i][j] : acc[i][j];
            }
        }
}

// One wave per (row, query head): the keys [0, pos] go through in chunks of 64, lane j
// scoring key t0 + j (a D-long dot product from its K row); the chunk's maximum and sum are
// wave reductions (online softmax in fp32), and lane j accumulates output dimensions j and
// j + 64 over the chunk's keys, each key's weight broadcast from its lane.
template <int D>
__global__ __launch_bounds__(256) void attn_f32_kernel(const float* __restrict__ q,
                                                       const float* __restrict__ kc,
                                                       const float* __restrict__ vc,
                                                       const int32_t* __restrict__ lens,
                                                       float* __restrict__ o, int rows, int S, int a,
                                                       int g, int cap) {
    constexpr int DPL = (D + 63) / 64;   // output dimensions per lane
    const int wid = (blockIdx.x * blockDim.x + threadIdx.x) >> 6, lane = threadIdx.x & 63;
    if (wid >= rows * a) return;         // wave-uniform
    const int r = wid / a, h = wid - r * a, kvh = h / (a / g);
    int b, pos;
    if (lens) {
        b = r;
        pos = max(0, min(lens[r], cap - 1));
    } else {
        b = r / S;
        pos = r - b * S;
    }
    const float scale = 1.0f / sqrtf((float)D);
    float qv[D];
#pragma unroll
    for (int i = 0; i < D; ++i) qv[i] = q[((size_t)r * a + h) * D + i];
    const float* kb = kc + ((size_t)b * g + kvh) * cap * D;
    const float* vb = vc + ((size_t)b * g + kvh) * D * cap;
    float acc[DPL];
#pragma unroll
    for (int k = 0; k < DPL; ++k) acc[k] = 0.f;
    float m = -INFINITY, l = 0.f;
    for (int t0 = 0; t0 <= pos; t0 += 64) {
        const int t = t0 + lane;
        float sc = -INFINITY;
        if (t <= pos) {
            float d = 0.f;
#pragma unroll
            for (int i = 0; i < D; ++i) d = fmaf(qv[i], kb[(size_t)t * D + i], d);
            sc = d * scale;
        }
        const float m_new = fmaxf(m, wave_max(sc));      // finite: key t0 is always visible
        const float alpha = expf(m - m_new);
        const float p = t <= pos ? expf(sc - m_new) : 0.f;
        l = l * alpha + wave_sum(p);
#pragma unroll
        for (int k = 0; k < DPL; ++k) acc[k] *= alpha;
        const int nk = min(64, pos + 1 - t0);
        for (int j = 0; j < nk; ++j) {
            const float pj = __shfl(p, j);
#pragma unroll
            for (int k = 0; k < DPL; ++k) {
                const int d = lane + 64 * k;
                if (d < D) acc[k] = fmaf(pj, vb[(size_t)d * cap + t0 + j], acc[k]);
            }
        }
        m = m_new;
    }
    const float inv = 1.0f / l;
#pragma unroll
    for (int k = 0; k < DPL; ++k) {
        const int d = lane + 64 * k;
        if (d < D) o[((size_t)r * a + h) * D + d] = acc[k] * inv;
    }
}

}  // namespace

hipError_t rope_table(float2* table, int S, int d, double base, hipStream_t st) {
    const int n = S * (d / 2);
    hipLaunchKernelGGL(rope_table_kernel, dim3((n + 255) / 256), dim3(256), 0, st, table, S, d / 2, d,
                       base);
    return hipGetLastError();
}

hipError_t rope_scatter(const float* proj, int nsplit, size_t split_stride, int rows, int S,
                        const int32_t* lens, int a, int g, int d, int cap, double base, bool producer,
                        bool bf16, void* q, void* kc, void* vc, hipStream_t st) {
    if (rows <= 0) return hipSuccess;
    if (d > 128 || nsplit < 1) return hipErrorInvalidValue;
    if (bf16)
        hipLaunchKernelGGL(rope_scatter_kernel<uint16_t>, dim3(rows), dim3(256), 0, st, proj, nsplit,
                           split_stride, S, lens, a, g, d, cap, base, producer ? 1 : 0, (uint16_t*)q,
                           (uint16_t*)kc, (uint16_t*)vc);
    else
        hipLaunchKernelGGL(rope_scatter_kernel<float>, dim3(rows), dim3(256), 0, st, proj, nsplit,
                           split_stride, S, lens, a, g, d, cap, base, producer ? 1 : 0, (float*)q,
                           (float*)kc, (float*)vc);
    return hipGetLastError();
}

hipError_t gemm_f32(const float* a, const WRows& w, int M, int N, int K, float* out,
                    const float* x_res, hipStream_t st) {
    dim3 grid((N + 31) / 32, (M + 31) / 32);
    hipLaunchKernelGGL(gemm_f32_kernel, grid, dim3(256), 0, st, a, w, M, N, K, out, x_res);
    return hipGetLastError();
}

hipError_t attn_f32(const float* q, const float* kc, const float* vc, const int32_t* lens, float* o,
                    int rows, int S, int a, int g, int d, int cap, hipStream_t st) {
    const int n = rows * a;                  // one wave each, four waves per block
    dim3 grid((n + 3) / 4), block(256);
    switch (d) {
        case 16: hipLaunchKernelGGL(attn_f32_kernel<16>, grid, block, 0, st, q, kc, vc, lens, o, rows, S, a, g, cap); break;
        case 32: hipLaunchKernelGGL(attn_f32_kernel<32>, grid, block, 0, st, q, kc, vc, lens, o, rows, S, a, g, cap); break;
        case 64: hipLaunchKernelGGL(attn_f32_kernel<64>, grid, block, 0, st, q, kc, vc, lens, o, rows, S, a, g, cap); break;
        case 128: hipLaunchKernelGGL(attn_f32_kernel<128>, grid, block, 0, st, q, kc, vc, lens, o, rows, S, a, g, cap); break;
        default: return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

}  // namespace kvp
