// Projections of single-token decode (Sec. 2.2: Q of every layer, K and V of
// producers only; output projection with the residual), M = batch <= 64 rows.
//
// The weights dominate the bytes (N x K bf16 read once; X is <= 64 rows), so
// the kernel is laid out to stream W from HBM at full rate:
//   * a workgroup owns 128 output columns (8 waves x 16) and one slice of K
//     (512 wide when K allows); its X slice (<= 64 rows, <= 64 KB) goes to LDS
//     once, with a 16-byte-chunk XOR swizzle that makes the MFMA operand reads
//     conflict-free;
//   * every wave issues all of its weight loads (16 B per lane per 32-wide k
//     step, immediate offsets from one base) before the single barrier, so W
//     never waits on X;
//   * v_mfma_f32_16x16x32_bf16 with A = X rows, B = W^T, fp32 partial sums per
//     K slice to a workspace; the slices are summed by the epilogue kernels
//     (RoPE + KV append for the projections, residual add for the output
//     projection), in a fixed order.
#include "common.h"
#include "kernels.h"

namespace kvp {
namespace {

typedef __attribute__((address_space(1))) void gvoid_t;
typedef __attribute__((address_space(3))) void lvoid_t;

// Two workgroups per CU (64 KB of LDS and <= 128 VGPRs each).
constexpr int DG_WAVES = 8, DG_THREADS = 64 * DG_WAVES, DG_COLS = 16 * DG_WAVES;
constexpr int DG_KC = 512, DG_SLOTS = DG_KC / 8;

// Width of one K slice: the largest of 512, 384, 256, 128 that divides K (K % 128 == 0).
inline int decode_kc(int K) {
    for (int kc = DG_KC; kc >= 128; kc -= 128)
        if (K % kc == 0) return kc;
    return 0;
}

// part[split][m][n] = sum over the K slice of X[m][k] W[n][k]; STEPS = slice / 32,
// NMB = ceil(M / 16) blocks of 16 rows.
template <int STEPS, int NMB>
__global__ __launch_bounds__(DG_THREADS, 4) void gemm_decode_kernel(const uint16_t* __restrict__ X, WRows W,
                                                                    int M, int N, int K,
                                                                    float* __restrict__ part) {
    // X slice: [row m][slot], slot = chunk ^ (m & 15) for 16-byte chunk `chunk` of the row.
    __shared__ u32x4 xs[64 * DG_SLOTS];
    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int col = lane & 15, kg = lane >> 4;
    const int split = blockIdx.y, k0 = split * (32 * STEPS);
    const bool loads_x = 8 * wave < 16 * NMB;     // waves 0 .. 2 NMB - 1 stage X

    // Rows 8 wave .. 8 wave + 7 of the X slice, one 1 KB row per load; rows past M repeat
    // row M - 1 and chunks past K repeat the last chunk (neither is read back).
    if (loads_x) {
#pragma unroll
        for (int j = 0; j < 8; ++j) {
            const int r = 8 * wave + j;
            const int chunk = lane ^ (r & 15);
            const int kk = min(k0 + 8 * chunk, K - 8);
            __builtin_amdgcn_global_load_lds((gvoid_t*)(X + (size_t)min(r, M - 1) * K + kk),
                                             (lvoid_t*)&xs[r * DG_SLOTS], 16, 0, 0);
        }
    }
    // The wave's 16 columns lie in one weight block (block sizes are multiples of 128).
    int n0 = blockIdx.x * DG_COLS + 16 * wave;
    const void* wbase;
    if (n0 < W.rows[0]) {
        wbase = W.p[0];
    } else if (n0 < W.rows[0] + W.rows[1]) {
        n0 -= W.rows[0];
        wbase = W.p[1];
    } else {
        n0 -= W.rows[0] + W.rows[1];
        wbase = W.p[2];
    }
    // Lane (col, kg) holds k = 32 s + 8 kg .. + 7 of its column for every step s.
    const uint16_t* wr = (const uint16_t*)wbase + (size_t)(n0 + col) * K + k0 + 8 * kg;
    u32x4 wf[STEPS];
#pragma unroll
    for (int s = 0; s < STEPS; ++s) wf[s] = *(const u32x4*)(wr + 32 * s);
    // This wave's X loads were issued before its STEPS weight loads: once at most STEPS
    // are outstanding its rows are in LDS; the barrier covers the other waves' rows.
    if (loads_x) {
        if (STEPS == 16)
            asm volatile("s_waitcnt vmcnt(16)" ::: "memory");
        else if (STEPS == 12)
            asm volatile("s_waitcnt vmcnt(12)" ::: "memory");
        else if (STEPS == 8)
            asm volatile("s_waitcnt vmcnt(8)" ::: "memory");
        else
            asm volatile("s_waitcnt vmcnt(4)" ::: "memory");
    }
    __syncthreads();

    f32x4 acc[NMB];
#pragma unroll
    for (int mb = 0; mb < NMB; ++mb) acc[mb] = f32x4{};
#pragma unroll
    for (int s = 0; s < STEPS; ++s)
#pragma unroll
        for (int mb = 0; mb < NMB; ++mb) {
            const int m = 16 * mb + col;
            const u32x4 xf = xs[m * DG_SLOTS + ((4 * s + kg) ^ (m & 15))];
            acc[mb] = mfma16x16x32(as_bf16x8(xf), as_bf16x8(wf[s]), acc[mb]);
        }
    // Lane (col, kg) holds rows 16 mb + 4 kg + i of its column.
    const int n = blockIdx.x * DG_COLS + 16 * wave + col;
    float* pp = part + (size_t)split * M * N;
#pragma unroll
    for (int mb = 0; mb < NMB; ++mb)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const int m = 16 * mb + 4 * kg + i;
            if (m < M) pp[(size_t)m * N + n] = acc[mb][i];
        }
}

template <int STEPS>
hipError_t launch_decode(const uint16_t* x, const WRows& w, int M, int N, int K, float* part,
                         hipStream_t st) {
    const dim3 grid(N / DG_COLS, K / (32 * STEPS)), block(DG_THREADS);
    switch ((M + 15) / 16) {
        case 1:
            hipLaunchKernelGGL((gemm_decode_kernel<STEPS, 1>), grid, block, 0, st, x, w, M, N, K, part);
            break;
        case 2:
            hipLaunchKernelGGL((gemm_decode_kernel<STEPS, 2>), grid, block, 0, st, x, w, M, N, K, part);
            break;
        case 3:
            hipLaunchKernelGGL((gemm_decode_kernel<STEPS, 3>), grid, block, 0, st, x, w, M, N, K, part);
            break;
        default:
            hipLaunchKernelGGL((gemm_decode_kernel<STEPS, 4>), grid, block, 0, st, x, w, M, N, K, part);
            break;
    }
    return hipGetLastError();
}

// y = x_res + sum over K slices of part (4 consecutive columns per thread).
__global__ __launch_bounds__(256) void decode_resid_kernel(const float* __restrict__ part, int nsplit,
                                                           int MN, const void* __restrict__ xres,
                                                           int xres_f32, uint16_t* __restrict__ y,
                                                           float* __restrict__ yf) {
    const int idx = 4 * (blockIdx.x * blockDim.x + threadIdx.x);
    if (idx >= MN) return;
    f32x4 v = *(const f32x4*)(part + idx);
#pragma unroll 8
    for (int s = 1; s < nsplit; ++s) v += *(const f32x4*)(part + (size_t)s * MN + idx);
    f32x4 r;
    if (xres_f32) {
        r = *(const f32x4*)((const float*)xres + idx);
    } else {
        const u32x2 w = *(const u32x2*)((const uint16_t*)xres + idx);
        r = f32x4{__uint_as_float(w[0] << 16), __uint_as_float(w[0] & 0xFFFF0000u),
                  __uint_as_float(w[1] << 16), __uint_as_float(w[1] & 0xFFFF0000u)};
    }
    r += v;
    u32x2 o;
    o[0] = pack2bf(r[0], r[1]);
    o[1] = pack2bf(r[2], r[3]);
    *(u32x2*)(y + idx) = o;
    if (yf) *(f32x4*)(yf + idx) = r;
}

// Sum of the K slices of sequence b's projections, RoPE at position len_b, then
// Q -> q [B][a * 128] (bf16), K -> K slot row len_b, V -> V^T slot column len_b (or the
// row / column len_b % 64 of page len_b / 64 of sequence b when pages.pt is set).  Work
// item j of a row: a rotary pair (head h < a + g_p, dim i < 64), then the V elements.
__global__ __launch_bounds__(256) void decode_qkv_epi_kernel(const float* __restrict__ part, int nsplit,
                                                             int B, int N, const int32_t* __restrict__ lens,
                                                             int a, int g, int cap, double base,
                                                             int producer, uint16_t* __restrict__ q,
                                                             uint16_t* __restrict__ kc,
                                                             uint16_t* __restrict__ vc, Pages pages) {
    constexpr int D = 128, HALF = 64;
    __shared__ float2 cs[HALF];
    const int b = blockIdx.y;
    const int pos = max(0, min(lens[b], cap - 1));   // never outside the slot (or page table row)
    // Rows (in units of D elements) of head 0's block holding pos and the stride between
    // heads' blocks: the slot of sequence b, or page pos / 64 of the head-major pools.
    size_t kv0, hstride;
    int vld, row;
    if (pages.pt) {
        kv0 = (size_t)page_at(pages, b, pos / kPage) * kPage;
        hstride = (size_t)pages.n * kPage;
        vld = kPage;
        row = pos % kPage;
    } else {
        kv0 = (size_t)b * g * cap;
        hstride = cap;
        vld = cap;
        row = pos;
    }
    if (threadIdx.x < HALF) {
        const double theta = pow(base, -2.0 * threadIdx.x / D);
        double sd, cd;
        sincos((double)pos * theta, &sd, &cd);
        cs[threadIdx.x] = make_float2((float)cd, (float)sd);
    }
    __syncthreads();
    const int heads = a + (producer ? g : 0);
    const int npairs = heads * HALF, nv = producer ? g * D : 0;
    const int j = blockIdx.x * blockDim.x + threadIdx.x;
    if (j >= npairs + nv) return;
    const size_t plane = (size_t)B * N;
    const float* pr = part + (size_t)b * N;
    auto val = [&](int c) {
        float v = pr[c];
#pragma unroll 8
        for (int s = 1; s < nsplit; ++s) v += pr[s * plane + c];
        return v;
    };
    if (j < npairs) {
        const int h = j / HALF, i = j - h * HALF;
        const float c = cs[i].x, sn = cs[i].y;
        const float x1 = val(h * D + i), x2 = val(h * D + i + HALF);
        const float o1 = x1 * c - x2 * sn, o2 = x2 * c + x1 * sn;
        if (h < a) {
            q[(size_t)b * a * D + h * D + i] = f2bf(o1);
            q[(size_t)b * a * D + h * D + i + HALF] = f2bf(o2);
        } else {
            const size_t kb = (kv0 + (size_t)(h - a) * hstride + row) * D;
            kc[kb + i] = f2bf(o1);
            kc[kb + i + HALF] = f2bf(o2);
        }
    } else {
        const int e = j - npairs, h = e / D, c = e - h * D;
        vc[(kv0 + (size_t)h * hstride) * D + (size_t)c * vld + row] = f2bf(val(a * D + g * D + e));
    }
}

// ---------------------------------------------------------------------------
// Small batches (M <= 16): full K per workgroup, epilogue fused.  Workgroup j owns 16
// output columns; wave w multiplies the K slice [512 w, 512 w + 512) in 16 steps of 32
// (v_mfma_f32_16x16x32_bf16, A = X rows read from global memory, B = W^T), exactly as a
// workgroup of gemm_decode_kernel does for one slice, and the waves' 16 x 16 partial tiles
// are added in LDS in slice order, so the sums equal the split path's bit for bit.  The
// sum goes straight to the epilogue (no partial planes, no second kernel): RoPE at the
// sequence's position and Q / K row / V^T column (projections), or the residual add
// (output projection).  In the rotary region a workgroup takes columns 8 s .. 8 s + 7 of a
// head's first half and the same of its second half, so both members of every rotary pair
// are in one workgroup; elsewhere 16 consecutive columns.
// ---------------------------------------------------------------------------
struct FusedQkv {
    uint16_t* q;
    uint16_t* kc;
    uint16_t* vc;
    const int32_t* lens;
    int a, g, cap, producer;
    double base;
    Pages pages;
};
struct FusedResid {
    const void* xres;
    int xres_f32;
    uint16_t* y;
    float* yf;
};

__device__ __forceinline__ const uint16_t* w_row3(const WRows& w, int n, int K) {
    if (n < w.rows[0]) return (const uint16_t*)w.p[0] + (size_t)n * K;
    n -= w.rows[0];
    if (n < w.rows[1]) return (const uint16_t*)w.p[1] + (size_t)n * K;
    n -= w.rows[1];
    return (const uint16_t*)w.p[2] + (size_t)n * K;
}

template <int MODE>   // 0: projections with RoPE + cache append, 1: output projection + residual
__global__ __launch_bounds__(1024) void gemm_decode_fused_kernel(const uint16_t* __restrict__ X, WRows W, int M,
                                                                 int N, int K, FusedQkv fq, FusedResid fr) {
    constexpr int D = 128, HALF = 64;
    __shared__ float red[16][16 * 16];   // [wave][row * 16 + column]
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6, nw = blockDim.x >> 6;
    const int col = lane & 15, kg = lane >> 4;
    const int j = blockIdx.x;
    const int nrot = MODE == 0 ? (fq.a + (fq.producer ? fq.g : 0)) * D : 0;   // rotary columns
    const bool rot = 16 * j < nrot;
    const int n = rot ? (j >> 3) * D + (col < 8 ? 0 : HALF) + (j & 7) * 8 + (col & 7) : 16 * j + col;
    const int k0 = 512 * wave;
    const uint16_t* wr = w_row3(W, n, K) + k0 + 8 * kg;
    const uint16_t* xr = X + (size_t)min(col, M - 1) * K + k0 + 8 * kg;
    u32x4 wf[16], xf[16];
#pragma unroll
    for (int s = 0; s < 16; ++s) {
        wf[s] = *(const u32x4*)(wr + 32 * s);
        xf[s] = *(const u32x4*)(xr + 32 * s);
    }
    f32x4 acc = f32x4{};
#pragma unroll
    for (int s = 0; s < 16; ++s) acc = mfma16x16x32(as_bf16x8(xf[s]), as_bf16x8(wf[s]), acc);
    // Lane (col, kg) holds rows 4 kg + i of its column.
#pragma unroll
    for (int i = 0; i < 4; ++i) red[wave][(4 * kg + i) * 16 + col] = acc[i];
    __syncthreads();
    auto sum = [&](int row, int c) {
        float v = red[0][row * 16 + c];
        for (int w = 1; w < nw; ++w) v += red[w][row * 16 + c];
        return v;
    };
    // Epilogue items (16 rows x 16 columns, or 16 rows x 8 rotary pairs) go over the
    // workgroup's threads (one wave when K = 512).
    if constexpr (MODE == 1) {
        for (int t = threadIdx.x; t < 16 * M; t += blockDim.x) {
            const int row = t >> 4, c = t & 15;
            const size_t off = (size_t)row * N + 16 * j + c;
            const float xv = fr.xres_f32 ? ((const float*)fr.xres)[off]
                                         : __uint_as_float((uint32_t)((const uint16_t*)fr.xres)[off] << 16);
            const float r = xv + sum(row, c);
            fr.y[off] = f2bf(r);
            if (fr.yf) fr.yf[off] = r;
        }
    } else {
        // Rows (in units of D elements) of head 0's block holding pos and the stride between
        // heads' blocks: the slot of sequence b, or page pos / 64 of the head-major pools.
        auto place = [&](int b, int pos, size_t& kv0, size_t& hstride, int& vld, int& prow) {
            if (fq.pages.pt) {
                kv0 = (size_t)page_at(fq.pages, b, pos / kPage) * kPage;
                hstride = (size_t)fq.pages.n * kPage;
                vld = kPage;
                prow = pos % kPage;
            } else {
                kv0 = (size_t)b * fq.g * fq.cap;
                hstride = fq.cap;
                vld = fq.cap;
                prow = pos;
            }
        };
        if (rot) {
            for (int t = threadIdx.x; t < 8 * M; t += blockDim.x) {
                const int row = t >> 3, c = t & 7;
                const int h = j >> 3, i = (j & 7) * 8 + c;
                const int pos = max(0, min(fq.lens[row], fq.cap - 1));
                const double theta = pow(fq.base, -2.0 * i / D);
                double sd, cd;
                sincos((double)pos * theta, &sd, &cd);
                const float cs = (float)cd, sn = (float)sd;
                const float x1 = sum(row, c), x2 = sum(row, c + 8);
                const float o1 = x1 * cs - x2 * sn, o2 = x2 * cs + x1 * sn;
                if (h < fq.a) {
                    fq.q[(size_t)row * fq.a * D + h * D + i] = f2bf(o1);
                    fq.q[(size_t)row * fq.a * D + h * D + i + HALF] = f2bf(o2);
                } else {
                    size_t kv0, hstride;
                    int vld, prow;
                    place(row, pos, kv0, hstride, vld, prow);
                    const size_t kb = (kv0 + (size_t)(h - fq.a) * hstride + prow) * D;
                    fq.kc[kb + i] = f2bf(o1);
                    fq.kc[kb + i + HALF] = f2bf(o2);
                }
            }
        } else {
            for (int t = threadIdx.x; t < 16 * M; t += blockDim.x) {
                const int row = t >> 4, c = t & 15;
                const int pos = max(0, min(fq.lens[row], fq.cap - 1));
                const int e = 16 * j - nrot + c, h = e / D, d = e - h * D;
                size_t kv0, hstride;
                int vld, prow;
                place(row, pos, kv0, hstride, vld, prow);
                fq.vc[(kv0 + (size_t)h * hstride) * D + (size_t)d * vld + prow] = f2bf(sum(row, c));
            }
        }
    }
}

}  // namespace

bool decode_fused_ok(int M, int N, int K) {
    return M >= 1 && M <= 16 && N % 16 == 0 && K % 512 == 0 && K >= 512 && K <= 16 * 512;
}

hipError_t gemm_decode_qkv_fused_bf16(const uint16_t* x, const WRows& w, int B, int N, int K, const int32_t* lens,
                                      int a, int g, int cap, double base, bool producer, uint16_t* q, uint16_t* kc,
                                      uint16_t* vc, const Pages& pages, hipStream_t st) {
    if (!decode_fused_ok(B, N, K) || N != (a + (producer ? 2 * g : 0)) * 128) return hipErrorInvalidValue;
    if (pages.pt && (pages.n < 1 || pages.stride < 1 || cap != kPage * pages.stride)) return hipErrorInvalidValue;
    FusedQkv fq{q, kc, vc, lens, a, g, cap, producer ? 1 : 0, base, pages};
    hipLaunchKernelGGL(gemm_decode_fused_kernel<0>, dim3(N / 16), dim3(64 * (K / 512)), 0, st, x, w, B, N, K, fq,
                       FusedResid{});
    return hipGetLastError();
}

hipError_t gemm_decode_resid_fused_bf16(const uint16_t* x, const WRows& w, int M, int N, int K, const void* x_res,
                                        bool x_f32, uint16_t* y, float* yf, hipStream_t st) {
    if (!decode_fused_ok(M, N, K)) return hipErrorInvalidValue;
    FusedResid fr{x_res, x_f32 ? 1 : 0, y, yf};
    hipLaunchKernelGGL(gemm_decode_fused_kernel<1>, dim3(N / 16), dim3(64 * (K / 512)), 0, st, x, w, M, N, K,
                       FusedQkv{}, fr);
    return hipGetLastError();
}

int decode_gemm_splits(int K) {
    const int kc = decode_kc(K);
    return kc ? K / kc : 0;
}

hipError_t gemm_decode_bf16(const uint16_t* x, const WRows& w, int M, int N, int K, float* part,
                            hipStream_t st) {
    if (M < 1 || M > 64 || N % DG_COLS || K % 128 || K < 128) return hipErrorInvalidValue;
    switch (decode_kc(K)) {
        case 512: return launch_decode<16>(x, w, M, N, K, part, st);
        case 384: return launch_decode<12>(x, w, M, N, K, part, st);
        case 256: return launch_decode<8>(x, w, M, N, K, part, st);
        default: return launch_decode<4>(x, w, M, N, K, part, st);
    }
}

hipError_t decode_resid_bf16(const float* part, int nsplit, int M, int N, const void* x_res, bool x_f32,
                             uint16_t* y, float* yf, hipStream_t st) {
    const int MN = M * N;
    if (MN % 4 || nsplit < 1) return hipErrorInvalidValue;
    hipLaunchKernelGGL(decode_resid_kernel, dim3((MN / 4 + 255) / 256), dim3(256), 0, st, part, nsplit, MN,
                       x_res, x_f32 ? 1 : 0, y, yf);
    return hipGetLastError();
}

hipError_t decode_qkv_epilogue_bf16(const float* part, int nsplit, int B, int N, const int32_t* lens, int a,
                                    int g, int cap, double base, bool producer, uint16_t* q, uint16_t* kc,
                                    uint16_t* vc, const Pages& pages, hipStream_t st) {
    if (nsplit < 1) return hipErrorInvalidValue;
    if (pages.pt && (pages.n < 1 || pages.stride < 1 || cap != kPage * pages.stride)) return hipErrorInvalidValue;
    const int items = (a + (producer ? g : 0)) * 64 + (producer ? g * 128 : 0);
    hipLaunchKernelGGL(decode_qkv_epi_kernel, dim3((items + 255) / 256, B), dim3(256), 0, st, part, nsplit,
                       B, N, lens, a, g, cap, base, producer ? 1 : 0, q, kc, vc, pages);
    return hipGetLastError();
}

}  // namespace kvp
