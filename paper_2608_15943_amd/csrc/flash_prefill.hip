// Causal flash attention for the prefill / training forward (Sec. 2.2, Eq. 2),
// bf16 matrix cores, d_h = 128, GQA: query head j reads KV head j / r.
//
// A consumer layer runs the same kernel on its producer's slot (Eq. 3); the
// kernel only sees a K slot and a V slot.
//
// Workgroup = 4 waves = 128 queries of one (sequence, head); wave w owns 32
// queries.  Keys and values stream through LDS in tiles of 64 positions
// (K: [64][128], V^T: [128][64]; 32 KB per tile, double buffered).
//
// Per tile and wave:
//   S^T[64 x 32] = K_tile Q^T   v_mfma_f32_32x32x16_bf16, A = K from LDS,
//                               B = Q^T held in registers for the whole kernel.
//   The lane that owns query q holds 32 of its 64 scores; the other 32 are in
//   lane q ^ 32, so the row maximum needs one exchange and the row sum none
//   (each lane keeps a partial sum, added at the end).
//   P is rounded to bf16 and used as the B operand of
//   O^T[128 x 32] += V^T_tile P^T  straight from the score registers: the
//   positions a lane holds for a 16-wide k step are the ones it reads from the
//   V^T tile (two 8-byte reads), so P never leaves registers.
// Online softmax in the exp2 domain with a lazily moved maximum: the
// accumulators are rescaled only when some row's maximum grows by more than
// 8 (a factor 256), which keeps every exp2 argument <= 8.
//
// Query tiles are issued heaviest-first (most key tiles under the causal
// mask) and grouped per XCD so that the r heads that share a KV head and
// their key tiles meet in one L2.
#include <math.h>

#include "common.h"
#include "kernels.h"

namespace kvp {
namespace {

constexpr int BQ = 128, BKV = 64, D = 128, NT = 256;
constexpr float kLazy = 8.0f;

struct Tile {
    u32x4 k[4];   // K: 64 rows x 16 chunks = 1024 chunks, 4 per thread
    u32x4 v[4];   // V^T: 128 rows x 8 chunks = 1024 chunks, 4 per thread
};

__global__ __launch_bounds__(NT, 2) void flash_prefill_kernel(
    const uint16_t* __restrict__ Q, const uint16_t* __restrict__ Kc, const uint16_t* __restrict__ Vc,
    uint16_t* __restrict__ O, int B, int S, int a, int g, int cap, float scale_log2) {
    __shared__ u32x4 lk[2][BKV * 16];   // [stage][row * 16 + (chunk ^ (row & 15))]
    __shared__ u32x2 lv[2][D * 16];     // [stage][d * 16 + (unit ^ (d & 15))], unit = 4 positions

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int l32 = lane & 31, hi = lane >> 5;

    // Work item: heaviest query tiles first, then (sequence, head).
    const int nqt = (S + BQ - 1) / BQ;
    const int lid = xcd_remap(blockIdx.x, gridDim.x);
    const int per_qt = a * B;
    const int qt = nqt - 1 - lid / per_qt;
    const int rest = lid - (lid / per_qt) * per_qt;
    const int b = rest / a, head = rest - (rest / a) * a;
    const int kvh = head / (a / g);

    const int ldq = a * D;
    const int q0w = qt * BQ + wave * 32;         // first query of this wave
    const int q_lane = q0w + l32;                // the query whose column this lane holds

    // Q^T fragments: 8 k-steps of 16 dims, lane holds dims 16 ks + 8 hi + 0..7.
    bf16x8 qf[8];
    {
        const uint16_t* qrow = Q + ((size_t)b * S + min(q_lane, S - 1)) * ldq + head * D + 8 * hi;
#pragma unroll
        for (int ks = 0; ks < 8; ++ks) qf[ks] = as_bf16x8(*(const u32x4*)(qrow + 16 * ks));
    }

    const uint16_t* kbase = Kc + ((size_t)b * g + kvh) * cap * D;
    const uint16_t* vbase = Vc + ((size_t)b * g + kvh) * D * cap;

    // Key tiles needed by this workgroup (causal, and never past S).
    const int last_q = min(qt * BQ + BQ - 1, S - 1);
    const int ntiles = last_q / BKV + 1;

    auto load_tile = [&](int t, Tile& tl) {
        const int t0 = t * BKV;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const int id = tid + NT * i;
            const int row = id >> 4, c = id & 15;     // K row = position, chunk of 8 dims
            const int pos = t0 + row;
            if (pos < S)
                tl.k[i] = *(const u32x4*)(kbase + (size_t)pos * D + c * 8);
            else
                tl.k[i] = u32x4{0, 0, 0, 0};
            const int d = id >> 3, vc = id & 7;       // V^T row = dim, chunk of 8 positions
            const int p0 = t0 + vc * 8;
            u32x4 v = *(const u32x4*)(vbase + (size_t)d * cap + p0);
            if (p0 + 8 > S) {                         // zero positions >= S (never valid data)
                const int keep = S - p0;              // 0..7 valid elements
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    const int lo_ok = (2 * e) < keep, hi_ok = (2 * e + 1) < keep;
                    v[e] &= (lo_ok ? 0x0000FFFFu : 0u) | (hi_ok ? 0xFFFF0000u : 0u);
                }
            }
            tl.v[i] = v;
        }
    };
    auto store_tile = [&](int stg, const Tile& tl) {
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const int id = tid + NT * i;
            const int row = id >> 4, c = id & 15;
            lk[stg][row * 16 + (c ^ (row & 15))] = tl.k[i];
            const int d = id >> 3, vc = id & 7;
            const int u0 = 2 * vc, sw = d & 15;
            lv[stg][d * 16 + (u0 ^ sw)] = u32x2{tl.v[i][0], tl.v[i][1]};
            lv[stg][d * 16 + ((u0 + 1) ^ sw)] = u32x2{tl.v[i][2], tl.v[i][3]};
        }
    };

    f32x16 o[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) o[i] = f32x16{};
    float m_run = -INFINITY, l_run = 0.f;

    Tile nxt;
    load_tile(0, nxt);
    store_tile(0, nxt);
    __syncthreads();

    for (int t = 0; t < ntiles; ++t) {
        const int stg = t & 1;
        if (t + 1 < ntiles) load_tile(t + 1, nxt);

        const int t0 = t * BKV;
        if (t0 <= q0w + 31 && q0w < S) {          // some key of the tile is visible to this wave
            // ---- S^T = K Q^T -------------------------------------------------------
            f32x16 s[2] = {f32x16{}, f32x16{}};
#pragma unroll
            for (int ks = 0; ks < 8; ++ks) {
                const int c = 2 * ks + hi;
#pragma unroll
                for (int mb = 0; mb < 2; ++mb) {
                    const int row = 32 * mb + l32;
                    s[mb] = mfma32x32x16(as_bf16x8(lk[stg][row * 16 + (c ^ (row & 15))]), qf[ks], s[mb]);
                }
            }
            // ---- mask: position > query (causal) or >= S ----------------------------
            const bool diag = (t0 + BKV - 1 > q0w) || (t0 + BKV > S);
            if (diag) {
#pragma unroll
                for (int mb = 0; mb < 2; ++mb)
#pragma unroll
                    for (int i = 0; i < 16; ++i) {
                        const int pos = t0 + 32 * mb + 8 * (i >> 2) + 4 * hi + (i & 3);
                        if (pos > q_lane || pos >= S) s[mb][i] = -INFINITY;
                    }
            }
            // ---- online softmax -------------------------------------------------------
            float mx = -INFINITY;
#pragma unroll
            for (int mb = 0; mb < 2; ++mb)
#pragma unroll
                for (int i = 0; i < 16; ++i) mx = fmaxf(mx, s[mb][i]);
            mx = fmaxf(mx, __shfl_xor(mx, 32));
            const float mt = mx * scale_log2;                  // tile max, log2 domain
            const bool grow = mt > m_run + kLazy;
            if (__any(grow)) {
                const float m_new = fmaxf(m_run, mt);
                const float alpha = exp2f(m_run - m_new);      // 0 on the first visible tile
                m_run = m_new;
                l_run *= alpha;
#pragma unroll
                for (int db = 0; db < 4; ++db)
#pragma unroll
                    for (int i = 0; i < 16; ++i) o[db][i] *= alpha;
            }
            bf16x8 pb[2][2];
#pragma unroll
            for (int mb = 0; mb < 2; ++mb)
#pragma unroll
                for (int jp = 0; jp < 2; ++jp) {
                    float p[8];
#pragma unroll
                    for (int e = 0; e < 8; ++e) {
                        p[e] = exp2f(fmaf(s[mb][8 * jp + e], scale_log2, -m_run));
                        l_run += p[e];
                    }
                    u32x4 w;
                    w[0] = pack2bf(p[0], p[1]);
                    w[1] = pack2bf(p[2], p[3]);
                    w[2] = pack2bf(p[4], p[5]);
                    w[3] = pack2bf(p[6], p[7]);
                    pb[mb][jp] = as_bf16x8(w);
                }
            // ---- O^T += V^T P^T -------------------------------------------------------
#pragma unroll
            for (int db = 0; db < 4; ++db) {
                const int d = 32 * db + l32, sw = d & 15;
#pragma unroll
                for (int mb = 0; mb < 2; ++mb)
#pragma unroll
                    for (int jp = 0; jp < 2; ++jp) {
                        const int u1 = 8 * mb + 4 * jp + hi;     // positions 32mb + 16jp + 4hi + 0..3
                        const u32x2 lo = lv[stg][d * 16 + (u1 ^ sw)];
                        const u32x2 up = lv[stg][d * 16 + ((u1 + 2) ^ sw)];
                        const u32x4 w = {lo[0], lo[1], up[0], up[1]};
                        o[db] = mfma32x32x16(as_bf16x8(w), pb[mb][jp], o[db]);
                    }
            }
        }
        if (t + 1 < ntiles) store_tile(stg ^ 1, nxt);
        __syncthreads();
    }

    // ---- normalise and store O[b, q, head, :] -------------------------------------
    if (q_lane < S) {
        const float l_tot = l_run + __shfl_xor(l_run, 32);
        const float inv = 1.0f / l_tot;
        uint16_t* orow = O + ((size_t)b * S + q_lane) * ldq + head * D;
#pragma unroll
        for (int db = 0; db < 4; ++db)
#pragma unroll
            for (int r4 = 0; r4 < 4; ++r4) {
                const int d0 = 32 * db + 8 * r4 + 4 * hi;
                u32x2 w;
                w[0] = pack2bf(o[db][4 * r4 + 0] * inv, o[db][4 * r4 + 1] * inv);
                w[1] = pack2bf(o[db][4 * r4 + 2] * inv, o[db][4 * r4 + 3] * inv);
                *(u32x2*)(orow + d0) = w;
            }
    } else {
        (void)__shfl_xor(l_run, 32);
    }
}

}  // namespace

hipError_t flash_prefill_bf16(const uint16_t* q, const uint16_t* kc, const uint16_t* vc,
                              uint16_t* o, int B, int S, int a, int g, int cap, hipStream_t st) {
    const int nqt = (S + BQ - 1) / BQ;
    const float scale_log2 = (float)(1.4426950408889634 / sqrt((double)D));
    hipLaunchKernelGGL(flash_prefill_kernel, dim3(nqt * a * B), dim3(NT), 0, st, q, kc, vc, o, B, S,
                       a, g, cap, scale_log2);
    return hipGetLastError();
}

}  // namespace kvp
