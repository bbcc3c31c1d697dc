// Causal flash attention for the prefill / training forward (Sec. 2.2, Eq. 2),
// bf16 matrix cores, d_h = 128, GQA: query head j reads KV head j / r.  For training
// it also stores each query's log-sum-exp of the scaled scores (log2 domain), from
// which the backward rebuilds the softmax weights.
//
// A consumer layer runs the same kernel on its producer's slot (Eq. 3); the
// kernel only sees a K slot and a V slot (or, paged, the pools and the sequence's
// page table row: a 128-position tile spans two 64-position pages, looked up once
// per tile).
//
// Workgroup = 8 waves = 256 queries of one (sequence, head); wave w owns 32
// queries; two waves per SIMD.  Keys and values stream through LDS in tiles of
// 128 positions (K: [128][128], V^T: [128][128]; 64 KB per tile, double
// buffered), loaded straight from HBM/L2 into LDS (global_load_lds_dwordx4): no
// staging registers, and the XOR swizzle of the LDS rows is produced by choosing
// which 16-byte chunk each lane fetches.  Eight waves sharing 128-position tiles
// halve both the global->LDS bytes and the barriers per FLOP compared with four
// waves on 64-position tiles (measured: 10 % faster on the 8-layer stage share).
//
// Per tile and wave:
//   S^T[128 x 32] = K_tile Q^T  v_mfma_f32_32x32x16_bf16, A = K rows from LDS,
//                               B = Q^T held in registers for the whole kernel.
//   MFMA row rho of a 32-row block reads the K row whose index has bits 2 and
//   3 of rho swapped; then the 8 scores a lane holds for each 16-position k
//   step of the PV product are 8 consecutive positions, i.e. one 16-byte
//   chunk of a V^T row, and P is used as the B operand of
//   O^T[128 x 32] += V^T_tile P^T straight from the score registers.
//   The lane that owns query q holds 64 of its 128 scores (the other 64 are in
//   lane q ^ 32): the row max needs one exchange, the row sum none.
// Online softmax in the exp2 domain (raw v_exp_f32: arguments never exceed 8,
// tiny results may flush to 0) with a lazily moved maximum: accumulators
// are rescaled only when some row's maximum grows by more than 8 (a factor
// 256), which keeps every exp2 argument <= 8.  On the tile that holds a wave's diagonal
// (or the end of the sequence) the 32-key blocks with no visible key skip their
// QK^T and PV products.
//
// Work mapping: hardware workgroup p runs on XCD p % 8 and is the (p / 8)-th
// dispatched there.  When the B * g (sequence, KV head) groups split evenly
// over the 8 XCDs, XCD x takes whole groups x, x + 8, ... (the r heads sharing
// a KV head, and its key tiles, meet in one L2) and runs their query tiles
// heaviest first (most key tiles under the causal mask); otherwise query tiles
// are dealt heaviest first round-robin over the XCDs.  Either way every XCD
// gets the same mix of tile sizes.  (Giving each XCD a contiguous range of a
// heaviest-first list instead put all the long tiles on the first XCDs: 1.4x
// slower on the 8-layer stage share.)
#include <math.h>
#include <stdint.h>
#include <type_traits>

#include "common.h"
#include "kernels.h"
#include "tokmajor.h"

namespace kvp {
namespace {

constexpr int BQ = 256, BKV = 128, D = 128, NT = 512;
constexpr float kLazy = 8.0f;

typedef __attribute__((address_space(1))) void gvoid_t;
typedef __attribute__((address_space(3))) void lvoid_t;

// 64 lanes x 16 bytes from per-lane global addresses to 1 KB of LDS at lds_base
// (wave-uniform): lane i lands at lds_base + 16 i.
__device__ __forceinline__ void load_lds_1k(const void* gsrc, void* lds_base) {
    __builtin_amdgcn_global_load_lds((gvoid_t*)gsrc, (lvoid_t*)lds_base, 16, 0, 0);
}

// Word 3 of a raw buffer resource: a valid (32-bit) data format, so that dword loads are
// range-checked against the record count and return zeros past it.
constexpr int kRsrcWord3 = 0x00020000;

__device__ __forceinline__ int swap_b23(int r) { return (r & ~12) | ((r & 4) << 1) | ((r & 8) >> 1); }

// LDS fragment reads with their waits placed by hand.  The compiler, at this kernel's register
// pressure, issues the next fragment read right before the MFMA that needs it and waits for it
// there, so every fragment's LDS latency stalls the wave.  These reads go ahead by two k steps
// (three rotating sets of four fragments) and each step waits only for its own set: the
// reads return in order and nothing else uses the LDS counter inside those loops.  A wait
// names the set it completes as an in/out operand, so the MFMAs that read the set cannot be
// scheduled before it.
template <int OFF>
__device__ __forceinline__ u32x4 ds_read16(uint32_t addr) {
    u32x4 v;
    asm volatile("ds_read_b128 %0, %1 offset:%2" : "=v"(v) : "v"(addr), "i"(OFF));
    return v;
}
template <int N>
__device__ __forceinline__ void lgkm_wait(u32x4 (&f)[4]) {
    asm volatile("s_waitcnt lgkmcnt(%4)" : "+v"(f[0]), "+v"(f[1]), "+v"(f[2]), "+v"(f[3]) : "i"(N));
}

// 8 waves of 32 queries; two waves per SIMD (<= 256 registers each), 128 KB of LDS.
template <bool PAGED>
__global__ __launch_bounds__(NT, 2) void flash_prefill_kernel(
    const uint16_t* __restrict__ Q, const uint16_t* __restrict__ Kc, const uint16_t* __restrict__ Vc,
    uint16_t* __restrict__ O, float* __restrict__ lse, uint16_t* __restrict__ Ot, int Sp, int B, int S, int a,
    int g, int cap, float scale_log2, Pages pages) {
    // K: [stage][row * 16 + (chunk ^ (row & 15))]; V^T: [stage][d * 16 + (chunk ^ (d & 15))]
    // (rows of 256 bytes: 128 dims of a position, or 128 positions of a dim).
    __shared__ u32x4 lk[2][BKV * 16];
    __shared__ u32x4 lv[2][D * 16];

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int l32 = lane & 31, hi = lane >> 5;

    // Work item (query tile, sequence, head): see the work mapping above.
    const int nqt = (S + BQ - 1) / BQ;
    int qt, b, head;
    {
        const int G = B * g, r = a / g, p = blockIdx.x;
        if (G % kNumXcd == 0) {
            const int x = p % kNumXcd, k = p / kNumXcd;
            const int per = (G / kNumXcd) * r;            // workgroups per query tile on one XCD
            qt = nqt - 1 - k / per;
            const int rest = k - (k / per) * per;
            const int grp = (rest / r) * kNumXcd + x;     // (sequence, KV head) group
            b = grp / g;
            head = (grp - b * g) * r + rest % r;
        } else {
            const int per_qt = a * B;
            qt = nqt - 1 - p / per_qt;
            const int rest = p - (p / per_qt) * per_qt;
            b = rest / a;
            head = rest - b * a;
        }
    }
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
    // Slots: one buffer resource per slot, sized to it, so a load past its end returns
    // zeros without touching memory; per lane the offsets of its 4 + 4 loads are computed
    // once and a tile adds t0 (one 32-bit add per load).
    const int slot_bytes = PAGED ? 0 : cap * D * 2;   // < 2^31: slots hold fewer than 2^23 positions
    const __amdgpu_buffer_rsrc_t krs = __builtin_amdgcn_make_buffer_rsrc((void*)kbase, 0, slot_bytes, kRsrcWord3);
    const __amdgpu_buffer_rsrc_t vrs = __builtin_amdgcn_make_buffer_rsrc((void*)vbase, 0, slot_bytes, kRsrcWord3);
    uint32_t koff[4], voff[4];
    if constexpr (!PAGED) {
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const int r = 16 * wave + 4 * j + (lane >> 4);
            const int c = (lane & 15) ^ (r & 15);
            koff[j] = (uint32_t)(r * D + 8 * c) * 2u;
            voff[j] = (uint32_t)(r * cap + 8 * c) * 2u;
        }
    }

    // Key tiles needed by this workgroup (causal, and never past S).
    const int last_q = min(qt * BQ + BQ - 1, S - 1);
    const int ntiles = last_q / BKV + 1;

    // Issue the 32 + 32 one-kilobyte loads of tile t (4 + 4 per wave): K rows and V^T rows
    // 16 wave + 4 j + lane / 16, four 256-byte rows per instruction.  Positions past the
    // slot (only in the last tile when cap % 128 == 64) are clamped to the slot's last
    // row / chunk: they lie beyond S, so their scores are masked and their V is zeroed.
    // Paged: the tile's two pages are looked up once per tile (pages past the last one
    // holding a position < S are replaced by that page, so every read stays in a mapped
    // page; rows of positions >= S are masked and their V zeroed as above).  Each wave keeps
    // 64 consecutive entries of the table row in a register (lane i: entry 64 c + i) and
    // reads the two entries with readlane: one table load per 32 tiles.  Wave w's K rows
    // 16 w .. 16 w + 15 all lie in page w / 4 of the tile, so its K base is wave-uniform.
    int pchunk = -1, pgv = 0;
    auto issue_tile = [&](int t, int stg) {
        const int t0 = t * BKV;
        if constexpr (PAGED) {
            const int p0 = t0 / kPage;          // even: both pages of the tile in one chunk of 64
            if ((p0 >> 6) != pchunk) {
                pchunk = p0 >> 6;
                const int e = 64 * pchunk + lane;
                pgv = e < pages.stride ? pages.pt[(size_t)b * pages.stride + e] : 0;
            }
            const int p1 = min(p0 + 1, (S - 1) / kPage);
            const int pg0 = min(max(__builtin_amdgcn_readlane(pgv, p0 & 63), 0), pages.n - 1);
            const int pg1 = min(max(__builtin_amdgcn_readlane(pgv, p1 & 63), 0), pages.n - 1);
            const size_t hb = (size_t)kvh * pages.n;
            const uint16_t* kw = Kc + (hb + (wave >= 4 ? pg1 : pg0)) * kPage * D;
            const uint16_t* v0 = Vc + (hb + pg0) * D * kPage;
            const uint16_t* v1 = Vc + (hb + pg1) * D * kPage;
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                const int r = 16 * wave + 4 * j + (lane >> 4);
                const int c = (lane & 15) ^ (r & 15);
                load_lds_1k(kw + (size_t)(r & (kPage - 1)) * D + 8 * c, &lk[stg][(16 * wave + 4 * j) * 16]);
                load_lds_1k((c >= 8 ? v1 : v0) + r * kPage + 8 * (c & 7), &lv[stg][(16 * wave + 4 * j) * 16]);
            }
            return;
        }
        // K rows t0 + r and V^T row r (dimension r), positions t0 + 8 c .. + 7.  Past the
        // slot (only in the last tile when cap % 128 == 64) K rows read as zeros and V^T
        // chunks read the next row's start: both lie beyond S, so their scores are masked
        // and their V is zeroed.
        const int wu = __builtin_amdgcn_readfirstlane(wave);   // LDS destinations are scalar
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            __builtin_amdgcn_raw_ptr_buffer_load_lds(krs, (lvoid_t*)&lk[stg][(16 * wu + 4 * j) * 16], 16,
                                                     koff[j] + (uint32_t)t0 * (D * 2), 0, 0, 0);
            __builtin_amdgcn_raw_ptr_buffer_load_lds(vrs, (lvoid_t*)&lv[stg][(16 * wu + 4 * j) * 16], 16,
                                                     voff[j] + (uint32_t)t0 * 2, 0, 0, 0);
        }
    };
    auto fix_tail = [&](int t, int stg) {
        const int t0 = t * BKV;
        for (int i = tid; i < D * 16; i += NT) {
            const int d = i >> 4, pc = i & 15, c = pc ^ (d & 15);
            const int keep = S - (t0 + 8 * c);
            u32x4 v = lv[stg][i];
#pragma unroll
            for (int e = 0; e < 4; ++e)
                v[e] &= ((2 * e) < keep ? 0x0000FFFFu : 0u) | ((2 * e + 1) < keep ? 0xFFFF0000u : 0u);
            lv[stg][i] = v;
        }
    };
    f32x16 o[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) o[i] = f32x16{};
    float m_run = -INFINITY, l_run = 0.f;

    const int ksw = swap_b23(l32);          // K row read by this lane inside a 32-row block
    // LDS byte addresses of this lane's fragments in stage 0: K step ks of block 0 (block mb is
    // 8 KB further, since rows 32 mb + ksw share ksw's swizzle) and V^T chunk c of d block 0
    // (d blocks are 8 KB apart likewise); stage 1 is 32 KB further.
    uint32_t kaddr[8], vaddr[8];
#pragma unroll
    for (int ks = 0; ks < 8; ++ks) {
        kaddr[ks] = (uint32_t)(uintptr_t)&lk[0][ksw * 16 + ((2 * ks + hi) ^ (ksw & 15))];
        vaddr[ks] = (uint32_t)(uintptr_t)&lv[0][l32 * 16 + ((2 * ks + hi) ^ (l32 & 15))];
    }
    issue_tile(0, 0);
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    __syncthreads();
    if (BKV > S) {
        fix_tail(0, 0);
        __syncthreads();
    }

    // One tile, with its LDS stage as a compile-time constant: the two stages are 32 KB
    // apart, so every fragment address of stage 1 is stage 0's plus an immediate offset and
    // the per-lane addresses are computed once for the whole loop.
    auto tile = [&](int t, auto stg_t) {
        constexpr int stg = decltype(stg_t)::value;
        const bool more = t + 1 < ntiles;
        bool issued = false;

        const int t0 = t * BKV;
        // The tile body; on a tile that holds this wave's diagonal (or the end of the
        // sequence) the 32-key blocks with no visible key skip their MFMAs.
        auto body = [&](auto diag_t) {
            constexpr bool kDiag = decltype(diag_t)::value;
            int nmb = 4;
            if constexpr (kDiag) nmb = min(min(4, (q0w + 31 - t0) / 32 + 1), (S - t0 + 31) / 32);
            // ---- S^T = K Q^T: 32 MFMAs, each K fragment read once ------------------------
            f32x16 s[4] = {f32x16{}, f32x16{}, f32x16{}, f32x16{}};
            auto kfrag = [&](int mb, int ks) {
                const int row = 32 * mb + ksw;
                return as_bf16x8(lk[stg][row * 16 + ((2 * ks + hi) ^ (row & 15))]);
            };
            if constexpr (kDiag) {
#pragma unroll
                for (int mb = 0; mb < 4; ++mb)
                    if (mb < nmb) {
#pragma unroll
                        for (int ks = 0; ks < 8; ++ks) s[mb] = mfma32x32x16(kfrag(mb, ks), qf[ks], s[mb]);
                    }
            } else if constexpr (PAGED) {
#pragma unroll
            for (int ks = 0; ks < 8; ++ks) {
                const bf16x8 k0 = kfrag(0, ks), k1 = kfrag(1, ks), k2 = kfrag(2, ks), k3 = kfrag(3, ks);
                s[0] = mfma32x32x16(k0, qf[ks], s[0]);
                s[1] = mfma32x32x16(k1, qf[ks], s[1]);
                s[2] = mfma32x32x16(k2, qf[ks], s[2]);
                s[3] = mfma32x32x16(k3, qf[ks], s[3]);
            }
            } else {
                u32x4 kf[3][4];
                auto rd = [&](int ks, u32x4 (&f)[4]) __attribute__((always_inline)) {
                    f[0] = ds_read16<stg * 32768 + 0>(kaddr[ks]);
                    f[1] = ds_read16<stg * 32768 + 8192>(kaddr[ks]);
                    f[2] = ds_read16<stg * 32768 + 16384>(kaddr[ks]);
                    f[3] = ds_read16<stg * 32768 + 24576>(kaddr[ks]);
                };
                rd(0, kf[0]);
                rd(1, kf[1]);
#pragma unroll
                for (int ks = 0; ks < 8; ++ks) {
                    if (ks < 7) lgkm_wait<4>(kf[ks % 3]);
                    else lgkm_wait<0>(kf[ks % 3]);
                    if (ks + 2 < 8) rd(ks + 2, kf[(ks + 2) % 3]);
#pragma unroll
                    for (int mb = 0; mb < 4; ++mb) s[mb] = mfma32x32x16(as_bf16x8(kf[ks % 3][mb]), qf[ks], s[mb]);
                }
            }
            // The next tile goes into the other buffer (read last before the previous barrier)
            // after the K fragment reads of this one, not in the same burst (1-2 % faster).
            if (more) issue_tile(t + 1, stg ^ 1);
            issued = true;
            // Register i of block mb holds position t0 + 32 mb + 16 (i / 8) + 8 hi + i % 8.
            if constexpr (kDiag) {
                // Visible: pos <= q_lane and pos < S, i.e. the register's offset within the
                // lane's positions is at most lim (one compare against a constant each).
                const int lim = min(q_lane, S - 1) - t0 - 8 * hi;
#pragma unroll
                for (int mb = 0; mb < 4; ++mb)
#pragma unroll
                    for (int i = 0; i < 16; ++i)
                        if (32 * mb + 16 * (i >> 3) + (i & 7) > lim) s[mb][i] = -INFINITY;
            }
            // ---- online softmax -------------------------------------------------------
            float mx = -INFINITY;
#pragma unroll
            for (int mb = 0; mb < 4; ++mb)
#pragma unroll
                for (int i = 0; i < 16; ++i) mx = fmaxf(mx, s[mb][i]);
            mx = pair32_max(mx);
            const float mt = mx * scale_log2;                  // tile max, log2 domain
            if (__any(mt > m_run + kLazy)) {
                const float m_new = fmaxf(m_run, mt);
                const float alpha = __builtin_amdgcn_exp2f(m_run - m_new);   // 0 on the first visible tile
                m_run = m_new;
                l_run *= alpha;
#pragma unroll
                for (int db = 0; db < 4; ++db) o[db] *= alpha;
            }
            bf16x8 pb[4][2];
#pragma unroll
            for (int mb = 0; mb < 4; ++mb)
#pragma unroll
                for (int p = 0; p < 2; ++p) {
                    float e[8];
#pragma unroll
                    for (int k = 0; k < 8; ++k) {
                        e[k] = __builtin_amdgcn_exp2f(fmaf(s[mb][8 * p + k], scale_log2, -m_run));
                        l_run += e[k];
                    }
                    u32x4 w;
                    w[0] = pack2bf(e[0], e[1]);
                    w[1] = pack2bf(e[2], e[3]);
                    w[2] = pack2bf(e[4], e[5]);
                    w[3] = pack2bf(e[6], e[7]);
                    pb[mb][p] = as_bf16x8(w);
                }
            // ---- O^T += V^T P^T: 32 MFMAs over 8 chunks of 16 positions -------------------
            if constexpr (kDiag || PAGED) {
#pragma unroll
            for (int c = 0; c < 8; ++c) {
                const int mb = c >> 1, p = c & 1;
                if (kDiag && mb >= nmb) continue;
#pragma unroll
                for (int db = 0; db < 4; ++db) {
                    const int d = 32 * db + l32;
                    const bf16x8 vf = as_bf16x8(lv[stg][d * 16 + ((2 * c + hi) ^ (d & 15))]);
                    o[db] = mfma32x32x16(vf, pb[mb][p], o[db]);
                }
            }
            } else {
                u32x4 vf[3][4];
                auto rd = [&](int c, u32x4 (&f)[4]) __attribute__((always_inline)) {
                    f[0] = ds_read16<stg * 32768 + 0>(vaddr[c]);
                    f[1] = ds_read16<stg * 32768 + 8192>(vaddr[c]);
                    f[2] = ds_read16<stg * 32768 + 16384>(vaddr[c]);
                    f[3] = ds_read16<stg * 32768 + 24576>(vaddr[c]);
                };
                rd(0, vf[0]);
                rd(1, vf[1]);
#pragma unroll
                for (int c = 0; c < 8; ++c) {
                    if (c < 7) lgkm_wait<4>(vf[c % 3]);
                    else lgkm_wait<0>(vf[c % 3]);
                    if (c + 2 < 8) rd(c + 2, vf[(c + 2) % 3]);
#pragma unroll
                    for (int db = 0; db < 4; ++db) o[db] = mfma32x32x16(as_bf16x8(vf[c % 3][db]), pb[c >> 1][c & 1], o[db]);
                }
            }
        };
        if (t0 <= q0w + 31 && q0w < S) {          // some key of the tile is visible to this wave
            if ((t0 + BKV - 1 > q0w) || (t0 + BKV > S)) body(std::true_type{});
            else body(std::false_type{});
        }
        if (more && !issued) issue_tile(t + 1, stg ^ 1);   // this wave saw no key of tile t
        // One barrier: tile t + 1 has landed in LDS (every wave waited for its own loads)
        // and every wave is done reading tile t, whose buffer is refilled next.
        if (t + 1 < ntiles) {
            asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
            __syncthreads();
            if ((t + 2) * BKV > S) {
                fix_tail(t + 1, stg ^ 1);
                __syncthreads();
            }
        }
    };
    for (int t = 0; t < ntiles; t += 2) {
        tile(t, std::integral_constant<int, 0>{});
        if (t + 1 < ntiles) tile(t + 1, std::integral_constant<int, 1>{});
    }

    // ---- normalise and store O[b, q, head, :] -------------------------------------
    // Lanes q and q ^ 32 hold the same query, so both take this branch or neither.  The
    // token-major copy (training) is staged in the K buffers, free once every wave is past
    // its last tile.
    uint16_t* ts = (uint16_t*)&lk[0][0] + wave * (D * 32);
    if (Ot) __syncthreads();
    if (q_lane < S) {
        const float l_tot = pair32_sum(l_run);
        const float inv = 1.0f / l_tot;
        if (lse && hi == 0) lse[((size_t)b * a + head) * Sp + q_lane] = m_run + log2f(l_tot);
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
                if (Ot) tm_put_token(ts, d0, l32, w);
            }
    }
    if (Ot) tm_flush(ts, Ot, (size_t)B * S, head * D, (size_t)b * S + q0w, S - q0w, lane);
}

}  // namespace

hipError_t flash_prefill_bf16(const uint16_t* q, const uint16_t* kc, const uint16_t* vc,
                              uint16_t* o, float* lse, uint16_t* ot, int Sp, int B, int S, int a, int g,
                              int cap, const Pages& pages, hipStream_t st) {
    if (ot && (pages.pt || S % 8 != 0)) return hipErrorInvalidValue;
    const int nqt = (S + BQ - 1) / BQ;
    const float scale_log2 = (float)(1.4426950408889634 / sqrt((double)D));
    if (pages.pt) {
        if (pages.n < 1 || pages.stride < 1 || S > kPage * pages.stride) return hipErrorInvalidValue;
        hipLaunchKernelGGL(flash_prefill_kernel<true>, dim3(nqt * a * B), dim3(NT), 0, st, q, kc, vc, o, lse,
                           nullptr, Sp, B, S, a, g, cap, scale_log2, pages);
    } else {
        hipLaunchKernelGGL(flash_prefill_kernel<false>, dim3(nqt * a * B), dim3(NT), 0, st, q, kc, vc, o, lse,
                           ot, Sp, B, S, a, g, cap, scale_log2, pages);
    }
    return hipGetLastError();
}

}  // namespace kvp
