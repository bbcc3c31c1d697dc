// Internal launch interface of the HIP kernels (not part of the C ABI).
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace kvp {

// B operand of the projection GEMMs: up to three row blocks [rows_i][K]
// stacked along N (W_Q; W_K; W_V), each a separate caller buffer.
struct WRows {
    const void* p[3];
    int rows[3];
};

// KV storage.  Contiguous slots (pt == nullptr): K [B][g][cap][d], V [B][g][d][cap].
// Paged: position p of sequence b lives in page pt[b * stride + p / kPage], row p % kPage,
// of the head-major pools K [g][n][kPage][d] and V [g][n][d][kPage]; entries are clamped
// to [0, n).
constexpr int kPage = 64;
struct Pages {
    const int32_t* pt;
    int stride, n;
};
__device__ __forceinline__ int page_at(const Pages& pg, int b, int j) {
    return min(max(pg.pt[(size_t)b * pg.stride + j], 0), pg.n - 1);
}

// ---- bf16 prefill ---------------------------------------------------------

// Q (all layers) and K, V (producers) projections with RoPE fused into the
// epilogue.  x [M = B*S][K]; writes q [M][n_q] (post-RoPE), K slot rows
// (post-RoPE) and transposed V slot rows at positions s = m % S.
struct QkvOut {
    uint16_t* q;          // [M][n_q]
    uint16_t* kc;         // K slot [Bmax][g][cap][128] or nullptr
    uint16_t* vc;         // V slot [Bmax][g][128][cap] or nullptr
    const float2* rope;   // [S][64] (cos, sin)
    int n_q, n_kv, g, cap, S;
    Pages pages;          // pages.pt != nullptr: kc, vc are page pools
};
hipError_t gemm_qkv_bf16(const uint16_t* x, const WRows& w, int M, int N, int K, const QkvOut& o,
                         hipStream_t st);

// y = x_res + a @ w^T, a [M][K], w [N][K]; x_res [M][N] in bf16 or (x_f32) fp32;
// y [M][N] bf16 and, if yf != nullptr, yf [M][N] fp32 (may alias an fp32 x_res).
hipError_t gemm_resid_bf16(const uint16_t* a, const uint16_t* w, const void* x_res, bool x_f32,
                           uint16_t* y, float* yf, int M, int N, int K, hipStream_t st);

// Causal flash attention: q [B*S][a*128], K/V slots (or pools, pages.pt set) of the
// producer, o [B*S][a*128]; lse (optional) [B][a][Sp]: the row log-sum-exp of the scaled
// scores, log2 domain.
// ot (nullable): a token-major copy O^T [a*128][B*S] of the same bf16 values (the backward's
// dW_O operand); slots only, and S % 8 == 0.
hipError_t flash_prefill_bf16(const uint16_t* q, const uint16_t* kc, const uint16_t* vc,
                              uint16_t* o, float* lse, uint16_t* ot, int Sp, int B, int S, int a, int g,
                              int cap, const Pages& pages, hipStream_t st);

// The slice count gemm_kmajor_out_bf16 should use for an M x N x K product.
int gemm_out_splits(int M, int N, int K);

// C[M][N] = sum_k a[k][m] b[k][n] with a [K][lda], b [K][ldb] K-major (the backward's weight
// gradients; any K; M, N, lda, ldb % 8 == 0), split over `splits` ranges of whole 64-wide K
// tiles, fp32 partials to part + s * M * N.
hipError_t gemm_kmajor_out_bf16(const uint16_t* a, int lda, const uint16_t* b, int ldb, int M, int N, int K,
                                int splits, float* part, hipStream_t st);
// C = a @ w^T in bf16 (a [M][K], w [N][K], K % 64 == 0), no fused work.
// part[s][M][N] (fp32, s < splits) = the K slice s of a @ w^T (a [M][K], w [N][K], both
// K-contiguous); K a multiple of 64 * splits.
hipError_t gemm_nt_out_splits(const uint16_t* a, const uint16_t* w, int M, int N, int K, int splits, float* part,
                              hipStream_t st);
hipError_t gemm_out_bf16(const uint16_t* a, const uint16_t* w, int M, int N, int K, uint16_t* c,
                         hipStream_t st);

// ---- bf16 backward ----------------------------------------------------------

// out[c][r] = in[r][c] for r < R, c < C (row strides in_ld, out_ld).
hipError_t transpose_bf16(const uint16_t* in, uint16_t* out, int R, int C, size_t in_ld, size_t out_ld,
                          hipStream_t st);
hipError_t f32_to_bf16(const float* x, uint16_t* y, size_t n, hipStream_t st);
// Sum of `planes` [M][N] fp32 planes; rows [0, rows0) -> dst0, then rows1 -> dst1, rest -> dst2.
hipError_t reduce_planes(const float* part, int planes, int M, int N, float* dst0, int rows0, float* dst1,
                         int rows1, float* dst2, hipStream_t st);
// D = rowsum(dO * O) [B][a][Sp].
hipError_t attn_bwd_prep_bf16(const uint16_t* dO, const uint16_t* O, float* dsum, int B, int S, int Sp, int a,
                              hipStream_t st);

struct AttnBwdKv {
    const uint16_t* q;      // post-RoPE Q of the layer [B*S][a*128]
    const uint16_t* dO;     // [B*S][a*128]
    const float* lse;       // [B][a][Sp]
    const float* dsum;      // [B][a][Sp]
    const uint16_t* kc;     // producer K slot
    const uint16_t* vc;     // producer V slot (transposed)
    const float2* rope;
    const float* acc_in_k;
    const float* acc_in_v;
    float* acc_out_k;
    float* acc_out_v;
    uint16_t* out;
    uint16_t* out_t;        // nullable: the same rows token-major, [ldo][B*S] (S % 8 == 0)
    int ldo, col_k, col_v;
    int B, S, Sp, a, g, cap;
};
hipError_t flash_bwd_kv_bf16(const AttnBwdKv& p, hipStream_t st);

struct AttnBwdQ {
    const uint16_t* q;
    const uint16_t* dO;
    const float* lse;
    const float* dsum;
    const uint16_t* kc;
    const uint16_t* vc;
    const float2* rope;
    uint16_t* out;
    uint16_t* out_t;        // nullable: dQ token-major, [ldo][B*S] rows head*128 + d (S % 8 == 0)
    int ldo;
    int B, S, Sp, a, g, cap;
};
hipError_t flash_bwd_q_bf16(const AttnBwdQ& p, hipStream_t st);

// ---- bf16 decode ------------------------------------------------------------
// Largest decode grid (waves); the combine keeps one weight per wave of a pair in LDS.
constexpr int kMaxDecodeSplits = 4096;

// Allocation-free decode: the device array behind kvp_decode_step_noalloc (one per GPU,
// held until the process ends).  static_scratch returns its address on the current
// device (looked up on the first call on that device) and its size.
constexpr size_t kStaticScratchBytes = (size_t)64 << 20;
hipError_t static_scratch(void** addr, size_t* bytes);

// Partial-result slots the decode attention writes: one per (wave, pair) piece, at most
// waves + B * g of them, r = a / g rows of decode_partial_floats() floats each.
inline size_t decode_partial_floats() { return 132; }

// Decode projections (M <= 64 rows, N % 128 == 0, K % 128 == 0): fp32 partial sums
// part [decode_gemm_splits(K)][M][N] of x @ w^T, one plane per slice of K (512 wide
// when 512 divides K, else 384, 256 or 128).
int decode_gemm_splits(int K);
hipError_t gemm_decode_bf16(const uint16_t* x, const WRows& w, int M, int N, int K, float* part,
                            hipStream_t st);
// y = x_res + sum of the nsplit planes of part ([M][N] each); x_res bf16 or (x_f32) fp32,
// y bf16 and yf (optional) fp32.  In place (y or yf == x_res) is allowed.
hipError_t decode_resid_bf16(const float* part, int nsplit, int M, int N, const void* x_res, bool x_f32,
                             uint16_t* y, float* yf, hipStream_t st);
// Sum of the nsplit planes of part ([B][N], N = n_q (+ 2 n_kv for a producer)), RoPE at
// position lens[b] (d_h = 128), then q [B][n_q] and, for a producer, the K row and V^T
// column at position lens[b] of the slot.
hipError_t decode_qkv_epilogue_bf16(const float* part, int nsplit, int B, int N, const int32_t* lens, int a,
                                    int g, int cap, double base, bool producer, uint16_t* q, uint16_t* kc,
                                    uint16_t* vc, const Pages& pages, hipStream_t st);
// Small batches (M <= 16, K % 512 == 0, K <= 8192): the same products with the whole K in
// one workgroup per 16 columns and the epilogue fused (RoPE + Q / K / V^T writes as
// decode_qkv_epilogue_bf16, or the residual as decode_resid_bf16); results equal the split
// path's bit for bit.
bool decode_fused_ok(int M, int N, int K);
hipError_t gemm_decode_qkv_fused_bf16(const uint16_t* x, const WRows& w, int B, int N, int K, const int32_t* lens,
                                      int a, int g, int cap, double base, bool producer, uint16_t* q, uint16_t* kc,
                                      uint16_t* vc, const Pages& pages, hipStream_t st);
hipError_t gemm_decode_resid_fused_bf16(const uint16_t* x, const WRows& w, int M, int N, int K, const void* x_res,
                                        bool x_f32, uint16_t* y, float* yf, hipStream_t st);

// Attention of one new query per sequence over positions [0, len_b], on a grid of
// `waves` single-wave workgroups that split the (sequence, KV head, tile) list evenly.
// Paged (pages.pt != nullptr): kc, vc are pools and cap = kPage * pages.stride.
hipError_t decode_attn_bf16(const uint16_t* q, const uint16_t* kc, const uint16_t* vc,
                            const int32_t* lens, float* part, int B, int a, int g, int cap, int waves,
                            const Pages& pages, hipStream_t st);
hipError_t decode_combine_bf16(const float* part, const int32_t* lens, uint16_t* o, int B, int a, int g,
                               int cap, int waves, hipStream_t st);

// ---- shared by both dtypes -------------------------------------------------

// table[pos][i] = (cos, sin)(pos * base^(-2i/d)), evaluated in double.
hipError_t rope_table(float2* table, int S, int d, double base, hipStream_t st);

// RoPE + scatter of fp32 projections proj [rows][n_q + 2*n_kv] (the sum of nsplit
// planes split_stride floats apart): Q -> q [rows][n_q], K -> K slot, V -> V slot
// (transposed).  Row r is sequence r / S at position r % S (lens == nullptr), or
// sequence r at position lens[r].  d <= 128.
hipError_t rope_scatter(const float* proj, int nsplit, size_t split_stride, int rows, int S,
                        const int32_t* lens, int a, int g, int d, int cap, double base, bool producer,
                        bool bf16, void* q, void* kc, void* vc, hipStream_t st);

// ---- fp32 model path (vector ALU, full fp32) -------------------------------

// out [M][N] = a @ w^T (fp32), or y = x_res + a @ w^T when x_res != nullptr.
hipError_t gemm_f32(const float* a, const WRows& w, int M, int N, int K, float* out,
                    const float* x_res, hipStream_t st);

// Attention for fp32 models: row r of q [rows][a*d] is sequence r / S at
// position r % S (lens == nullptr) or sequence r at lens[r]; attends [0, pos].
hipError_t attn_f32(const float* q, const float* kc, const float* vc, const int32_t* lens,
                    float* o, int rows, int S, int a, int g, int d, int cap, hipStream_t st);

// ---- fp32 backward (vector ALU) ---------------------------------------------

// C[m][n] = R[m][n] + sum_k A(m, k) B(k, n) with A(m, k) = a[m * sam + k * sak] and
// B(k, n) = b[k * sbk + n * sbn]; R = res (row stride ldc, may equal c) or 0 when null.
hipError_t gemm_f32_strided(const float* a, size_t sam, size_t sak, const float* b, size_t sbk, size_t sbn,
                            const float* res, float* c, size_t ldc, int M, int N, int K, hipStream_t st);

// Attention backward of one fp32 layer: q, dO, O [B*S][a*d] (q after RoPE), the producer's
// K slot [B][g][cap][d] and V slot [B][g][d][cap]; lse and dsum [B*S*a] are scratch.
// dQ (rotated back, scaled) goes to out_q columns h*d of rows ldo floats apart.  dK, dV
// (dK rotated back and scaled) plus acc_in_* (optional, [B][g][S][d]) go to acc_out_* (same
// layout, may equal acc_in_*) and / or to out_kv row b*S + key at columns col_k / col_v +
// kvh*d.  d in {16, 32, 64, 128}.
struct AttnBwdF32 {
    const float* q;
    const float* dO;
    const float* O;
    const float* kc;
    const float* vc;
    const float2* rope;     // [S][d/2] (cos, sin)
    float* lse;
    float* dsum;
    const float* acc_in_k;
    const float* acc_in_v;
    float* acc_out_k;
    float* acc_out_v;
    float* out_kv;
    float* out_q;
    int ldo, col_k, col_v;
    int B, S, a, g, d, cap;
};
hipError_t attn_bwd_f32(const AttnBwdF32& p, hipStream_t st);

}  // namespace kvp
