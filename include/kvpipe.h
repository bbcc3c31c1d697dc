/*
 * kvpipe.h -- C ABI of the KV-shared attention library for MI355X (gfx950).
 *
 * The library computes the attention block of a transformer stack in which
 * every layer l reads keys and values from a producer layer tau(l) <= l
 * (KV-Pipe, Sec. 2.2, Eq. (3)): a producer (tau(l) = l) projects Q, K and V,
 * applies RoPE and writes its KV cache; a consumer projects Q only and attends
 * against its producer's cache.  It runs as a causal prefill / training
 * forward over S tokens and as a single-token decode step over a long cache.
 * A CPU planner implements the paper's offline FIR-balancing rule
 * (Sec. 2.3-2.7, Algorithm 1; App. A.3 guardrail; App. A.7 FLOPs model), the
 * two position-based placement archetypes it is compared with (Sec. 2.5),
 * and can produce the sharing map.
 *
 * Conventions
 * -----------
 * - Every call returns an int status: KVP_OK (0) or a negative KVP_E_* code.
 *   No C++ exception crosses this boundary.  kvp_last_error() returns a
 *   thread-local message describing the last failure on the calling thread.
 * - The library allocates no device memory at run time.  The caller owns
 *   weights, activations, KV caches and the workspace (its size comes from
 *   kvp_workspace_size; every compute call takes it as ws / ws_bytes, so that
 *   the calls never allocate).  The one piece of device memory the library
 *   holds is the file-scope array that kvp_decode_step_noalloc uses in place
 *   of a workspace (64 MiB per GPU, loaded with the library).  Host-side plan
 *   state lives in an opaque kvp_ctx.
 * - Device pointers are plain `void*` into device memory of the current HIP
 *   device.  Device work is enqueued asynchronously on the caller's stream
 *   (`stream` is a hipStream_t passed as void*, NULL = the null stream); the
 *   call returns once the launches are enqueued.  Buffers must stay valid
 *   until that work completes.  Calls on one ctx must not overlap in time on
 *   different streams: they share the ctx's producer KV slots.
 * - Shapes: h = model width, a = query heads, g = KV heads (a % g == 0,
 *   r = a / g), d_h = head dimension, a * d_h == h.  Query head j reads KV
 *   head floor(j / r).
 * - Layouts (row-major, element type = the model dtype unless stated):
 *     activations x, y   [B, S, h]            (decode: [B, h])
 *     W_Q                [a * d_h, h]          ([out, in])
 *     W_K, W_V           [g * d_h, h]
 *     W_O                [h, a * d_h]
 *     K slot             [B_max][g][kv_capacity][d_h]   post-RoPE keys
 *     V slot             [B_max][g][d_h][kv_capacity]   values, transposed so
 *                        that both attention contractions read contiguous
 *                        runs of the cache (see kvp_set_kv_slot): a deliberate
 *                        departure from a row-major [B][g][kv_capacity][d_h]
 *                        V cache.
 *     attention output   [B, S, a * d_h]      (concatenated heads)
 * - RoPE: rotate-half pairing (x_i, x_{i + d_h/2}), theta_i =
 *   rope_base^(-2i/d_h), absolute positions 0..S-1 in prefill and len_b in
 *   decode; cos/sin are evaluated in double precision.
 * - bf16 models compute every product in bf16 on matrix cores with fp32
 *   accumulation; Q, K, V, the softmax weights P and the attention output
 *   are rounded to bf16.  Between layers the residual stream is carried in
 *   fp32 (workspace), with a bf16 copy as the next projection's operand; the
 *   caller's x and y are bf16.  fp32 models run every step in fp32 on the
 *   vector units (no reduced-precision modes).
 */
#ifndef KVPIPE_H
#define KVPIPE_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* ---- status codes ------------------------------------------------------ */
#define KVP_OK              0
#define KVP_E_INVALID_ARG  -1  /* NULL where a pointer is required, bad enum, bad number */
#define KVP_E_BAD_MAP      -2  /* tau(l) > l, tau(l) < 0, or tau(0) != 0; z_0 = 1           */
#define KVP_E_SHAPE        -3  /* shape outside what the kernels support (see kvp_create)    */
#define KVP_E_WORKSPACE    -4  /* workspace NULL or smaller than kvp_workspace_size()        */
#define KVP_E_CAPACITY     -5  /* B > max_batch, S > max_seq, or a position >= kv_capacity   */
#define KVP_E_HIP          -6  /* a HIP runtime call or a kernel launch failed               */
#define KVP_E_STATE        -7  /* weights or KV slots of some layer were never set           */

/* ---- enums ------------------------------------------------------------- */
#define KVP_DTYPE_BF16      0
#define KVP_DTYPE_FP32      1

#define KVP_PHASE_PREFILL   0
#define KVP_PHASE_DECODE    1
#define KVP_PHASE_BACKWARD  2  /* workspace of kvp_backward (kvp_workspace_size only) */

#define KVP_STOP_FIR_MET        0  /* FIR <= 1 + eps                                    */
#define KVP_STOP_BUDGET         1  /* m conversions made                                */
#define KVP_STOP_NO_CONVERTIBLE 2  /* the chosen stage has no admissible full layer left */

#define KVP_PLACE_UNIFORM           0  /* Sec. 2.5, Uniform split             */
#define KVP_PLACE_SYMMETRIC_BIPOLAR 1  /* Sec. 2.5, Symmetric Bipolar split   */

/* ======================================================================== */
/* Planner (host only; touches no GPU)                                       */
/* ======================================================================== */

/* Shape of one layer for the FLOPs model of App. A.7. */
typedef struct kvp_shape {
    int64_t b;       /* micro-batch size                                          */
    int64_t s;       /* prefill: sequence length; decode: cached context length   */
    int64_t h;       /* hidden size                                               */
    int64_t a;       /* query heads (d = h / a)                                   */
    int64_t g;       /* KV heads (r = a / g)                                      */
    int64_t ffn;     /* SwiGLU MLP width, 0 = attention only                      */
    int32_t causal;  /* prefill only: 1 = score/context FLOPs over s^2/2 pairs,   */
                     /* 0 = over s^2 (Eqs. (qk), (av) as printed)                  */
    int32_t _pad;
} kvp_shape;

/*
 * kvp_layer_flops -- App. A.7, Eqs. (mm_flops)-(gqa_skv_flop_saving).
 * phase = KVP_PHASE_PREFILL: F(0) = 2bsh^2 (1 + 2/r) + score/context + 2bsh^2
 *   [+ 6 b s h ffn], score/context = 4 b s^2 h (causal: 2 b s^2 h).
 * phase = KVP_PHASE_DECODE: one new token per sequence over s cached keys:
 *   F(0) = b (4h^2 + 4h^2/r + 4 s h) [+ 6 b h ffn].
 * F(1) = F(0) - 4 b s h^2 / r (prefill) or - 4 b h^2 / r (decode): a shared
 * layer drops its K and V projections.  Values are exact integers < 2^53.
 * Errors: KVP_E_INVALID_ARG if a pointer is NULL, any size < 1 (ffn < 0), or
 * a does not divide h, or g does not divide a.
 */
int kvp_layer_flops(const kvp_shape* shape, int phase, double* f_full, double* f_share);

/*
 * kvp_fir -- Eqs. (flop_imbalance_main), (favg): FIR = max_i F_i / mean_i F_i.
 * stage_flops[P] already includes the LM head on the last stage.
 * Errors: KVP_E_INVALID_ARG if P < 1, a pointer is NULL, or the mean is <= 0.
 */
int kvp_fir(int P, const double* stage_flops, double* fir);

/* Inputs of Algorithm 1 (caller-owned arrays). */
typedef struct kvp_plan_in {
    int32_t L;                      /* layers                                          */
    int32_t P;                      /* pipeline stages, 1 <= P <= L                     */
    const int32_t* stage_of_layer;  /* [L], non-decreasing, 0..P-1, every stage used    */
    const double* f_full;           /* [L] F_l(0)                                       */
    const double* f_share;          /* [L] F_l(1), with F_l(0) - F_l(1) > 0              */
    double f_lmhead;                /* F_LM-Head, added to stage P-1 (>= 0)              */
    double eps;                     /* tolerance epsilon > 0                            */
    int32_t m;                      /* conversion budget; <= 0 means m = L               */
    int32_t _pad;
    const uint8_t* admissible;      /* [L] or NULL (= all); layer 0 is never converted  */
    double alpha;                   /* App. A.3 guardrail: < 0 = off, else also require */
                                    /* (1-indexed) l >= ceil(alpha L)                   */
} kvp_plan_in;

/* Outputs of Algorithm 1 (caller-owned arrays). */
typedef struct kvp_plan_out {
    uint8_t* z;            /* [L] conversion mask                               */
    double* stage_flops;   /* [P] stage FLOPs after the conversions             */
    double fir;            /* FIR of the returned state                         */
    int32_t n_converted;   /* number of conversions made                        */
    int32_t stop_reason;   /* KVP_STOP_*                                        */
} kvp_plan_out;

/*
 * kvp_plan_fir -- Algorithm 1 (Architecture-Balanced, tail-first).
 * Each pass starts from the last stage; once that stage is within (1 + eps)
 * of the mean it takes the stage with the most FLOPs instead (exact ties go
 * to the highest stage index); it converts the last unconverted admissible
 * layer of that stage, subtracts F(0) - F(1) from the stage and recomputes
 * the mean and FIR.  It stops when FIR <= 1 + eps, after m conversions, or
 * when the chosen stage has no admissible full layer left, and returns that
 * final state.  The arithmetic is IEEE double in a fixed order (stage sums
 * left to right, LM head last, mean = sum / P, FIR = max / mean), so two
 * faithful implementations return the same mask bit for bit.
 * Errors: KVP_E_INVALID_ARG on NULL arrays, L < 1, P < 1, P > L, eps <= 0,
 * a stage index out of range or decreasing, an empty stage, or
 * F(0) - F(1) <= 0 for an admissible layer.
 */
int kvp_plan_fir(const kvp_plan_in* in, kvp_plan_out* out);

/*
 * kvp_stage_flops -- Eq. (stage_flops_z): stage_flops[i] = the sum of F_l(z_l)
 * over the layers l of stage i (left to right), plus f_lmhead on stage P-1,
 * in the order kvp_plan_fir uses.  Arrays are caller-owned: stage_of_layer,
 * f_full, f_share, z of length L; stage_flops of length P (written).
 * Errors: KVP_E_INVALID_ARG on NULL arrays, L < 1, P < 1, P > L or a stage
 * index outside 0..P-1.
 */
int kvp_stage_flops(int L, int P, const int32_t* stage_of_layer, const double* f_full,
                    const double* f_share, const uint8_t* z, double f_lmhead,
                    double* stage_flops);

/*
 * kvp_place -- the two position-based placement archetypes of Sec. 2.5.
 * They place k conversions without looking at FLOPs (the FLOPs-driven
 * Architecture-Balanced archetype is kvp_plan_fir); the caller evaluates the
 * result with kvp_stage_flops and kvp_fir (Table 2).
 *
 * KVP_PLACE_UNIFORM: the k conversions are spaced evenly over the layers of
 *   the last min(k, P) stages, the first on the last layer, moving left:
 *   target_j = hi - round(j (hi - lo) / (k - 1)), halves rounded up, with
 *   hi = L - 1 and lo the first layer of stage P - min(k, P).  With equal
 *   stages and k <= P this is one conversion in each of the last k stages
 *   (App. A.1 Table A1; for LLaMA2-7B on 8 stages and k = 4 the 1-indexed
 *   layers 17, 22, 27, 32 of App. A.4).
 * KVP_PLACE_SYMMETRIC_BIPOLAR: two anchors, the last layer of stage P-1 and
 *   the last layer of the middle stage (P-1)/2; conversions alternate between
 *   them, the last stage first, each anchor moving left from its previous
 *   choice (App. A.1 Table A2: two each in stages 3 and 7 for k = 4, P = 8).
 *   An anchor with no free layer left hands its turns to the other; with
 *   P = 1 the anchors coincide.
 * Under both, a layer is free when it is admissible (the caller mask, the
 * App. A.3 guardrail alpha as in kvp_plan_fir, never layer 0) and not yet
 * converted; a Uniform target that is not free moves to the nearest free
 * layer on its left, else on its right.
 * In: stage_of_layer[L] as in kvp_plan_in; admissible[L] or NULL; k >= 0.
 * Out: z[L] (1 = KV-sharing layer), *n_placed, *stop_reason =
 * KVP_STOP_BUDGET when all k were placed, else KVP_STOP_NO_CONVERTIBLE
 * (no free layer was left).  Integer arithmetic only.
 * Errors: KVP_E_INVALID_ARG on NULL pointers, L < 1, P < 1, P > L, k < 0,
 * an unknown strategy, or a partition that is not 0..P-1, non-decreasing
 * and without empty stages.
 */
int kvp_place(int strategy, int L, int P, const int32_t* stage_of_layer, int k,
              const uint8_t* admissible, double alpha, uint8_t* z, int32_t* n_placed,
              int32_t* stop_reason);

/*
 * kvp_map_from_mask -- Eq. (3) with tau(l) = nearest earlier full-attention
 * layer: tau(l) = l where z_l = 0, else the largest j < l with z_j = 0.
 * Errors: KVP_E_INVALID_ARG on NULL / L < 1; KVP_E_BAD_MAP if z_0 = 1.
 */
int kvp_map_from_mask(int L, const uint8_t* z, int32_t* tau);

/*
 * kvp_canonicalize_map -- checks 0 <= tau(l) <= l and tau(0) = 0 and resolves
 * chains (tau(tau(l)) != tau(l)) to the root producer; in may equal out.
 * Errors: KVP_E_INVALID_ARG on NULL / L < 1; KVP_E_BAD_MAP otherwise.
 */
int kvp_canonicalize_map(int L, const int32_t* in, int32_t* out);

/* ======================================================================== */
/* Attention stack                                                            */
/* ======================================================================== */

typedef struct kvp_model_desc {
    int32_t L;            /* layers                                                  */
    int32_t h;            /* hidden size, == a * d_h                                 */
    int32_t a;            /* query heads                                             */
    int32_t g;            /* KV heads, divides a                                     */
    int32_t d_h;          /* head dim: 128 for bf16; even and <= 256 for fp32        */
    int32_t dtype;        /* KVP_DTYPE_BF16 or KVP_DTYPE_FP32                        */
    double rope_base;     /* RoPE base (> 0), e.g. 10000                             */
    int32_t max_batch;    /* largest B of any call, and the B extent of the KV slots */
    int32_t max_seq;      /* largest prefill S                                       */
    int32_t kv_capacity;  /* positions per sequence in a KV slot; bf16: multiple of 64, < 2^23 */
    int32_t _pad;
} kvp_model_desc;

typedef struct kvp_ctx kvp_ctx;

/*
 * kvp_create -- validates desc, canonicalises tau[L] (see
 * kvp_canonicalize_map) and returns a context with no weights or slots set.
 * bf16 needs d_h == 128, h % 128 == 0 and kv_capacity % 64 == 0.
 * Errors: KVP_E_INVALID_ARG (NULL, non-positive sizes, unknown dtype,
 * max_seq > kv_capacity), KVP_E_BAD_MAP, KVP_E_SHAPE.  *out is NULL on error.
 */
int kvp_create(const kvp_model_desc* desc, const int32_t* tau, kvp_ctx** out);

/* kvp_destroy -- frees the host-side context (NULL is accepted). */
int kvp_destroy(kvp_ctx* ctx);

/*
 * kvp_set_layer -- device pointers of layer l's weights (layouts above).
 * Wk and Wv are required for a producer and must be NULL for a consumer: a
 * consumer has no K/V projection (Eq. 3).  The pointers are kept, not copied.
 * Errors: KVP_E_INVALID_ARG.
 */
int kvp_set_layer(kvp_ctx* ctx, int l, const void* Wq, const void* Wk, const void* Wv,
                  const void* Wo);

/*
 * kvp_set_kv_slot -- device buffers that hold producer l's cache:
 * K [max_batch][g][kv_capacity][d_h] and V [max_batch][g][d_h][kv_capacity].
 * Consumers have no slot; they read tau(l)'s.  Prefill writes positions
 * [0, S) of sequences [0, B); decode writes position len_b of sequence b.
 * Errors: KVP_E_INVALID_ARG (NULL pointer, l not a producer).
 */
int kvp_set_kv_slot(kvp_ctx* ctx, int l, void* K, void* V);

/*
 * kvp_workspace_size -- bytes of device scratch that a call with this phase,
 * batch B and length S (prefill, backward; ignored for decode) needs.  The
 * workspace holds Q, the attention output, the fp32 residual stream and its
 * bf16 copy, the RoPE table (prefill) and split-K partial results (decode);
 * for KVP_PHASE_BACKWARD the gradients in flight, (bf16 models) their
 * transposed copies and transposed weights, (fp32 models) the per-(token,
 * head) softmax statistics, and the producers' fp32 dK/dV sums.
 * Errors: KVP_E_INVALID_ARG, KVP_E_CAPACITY (B > max_batch, S > max_seq).
 */
int kvp_workspace_size(const kvp_ctx* ctx, int phase, int B, int S, size_t* bytes);

/*
 * kvp_prefill -- causal forward of all L layers over x [B, S, h] into
 * y [B, S, h]: for l in order, X_{l+1} = X_l + Attn_l(X_l) W_O^T with the
 * producer / consumer semantics of Sec. 2.2.  Producers write positions
 * [0, S) of their slot.  x and y may not alias; x is not modified.
 * Errors: KVP_E_INVALID_ARG, KVP_E_CAPACITY, KVP_E_WORKSPACE, KVP_E_STATE,
 * KVP_E_HIP.
 */
int kvp_prefill(kvp_ctx* ctx, const void* x, void* y, int B, int S, void* ws, size_t ws_bytes,
                void* stream);

/*
 * kvp_layer_forward -- one layer of kvp_prefill on caller-supplied input x:
 * y = x + O W_O^T, and, if attn_out is not NULL, the attention output O
 * [B, S, a * d_h].  A producer writes its slot; a consumer reads tau(l)'s
 * slot, which must already hold positions [0, S).
 * Errors: as kvp_prefill, plus KVP_E_INVALID_ARG for l out of range.
 */
int kvp_layer_forward(kvp_ctx* ctx, int l, const void* x, void* attn_out, void* y, int B, int S,
                      void* ws, size_t ws_bytes, void* stream);

/*
 * kvp_decode_step -- one new token per sequence through all L layers.
 * x, y [B, h]; len_dev: device int32 [B], len_b = the number of tokens
 * already cached for sequence b; the new token sits at position len_b.
 * Each producer appends its post-RoPE K and V at len_b before attending;
 * every layer attends over positions [0, len_b].  The caller advances the
 * lengths.  max_len (host) must be >= every len_b; it sizes the split-K
 * grid.  Sequences shorter than max_len do proportionally less work.  bf16
 * models run a batch above 64 as consecutive chunks of 64 sequences through
 * the whole stack (each chunk reads the weights once); results do not depend
 * on the chunking.
 * Errors: KVP_E_CAPACITY if max_len >= kv_capacity or B > max_batch (len_b
 * itself is not read on the host; len_b > max_len is undefined behaviour),
 * KVP_E_INVALID_ARG, KVP_E_WORKSPACE, KVP_E_STATE, KVP_E_HIP.
 */
int kvp_decode_step(kvp_ctx* ctx, const void* x, const int32_t* len_dev, int max_len, void* y,
                    int B, void* ws, size_t ws_bytes, void* stream);

/*
 * kvp_decode_step_noalloc -- kvp_decode_step for callers that cannot allocate device
 * memory (code under HIP graph capture, tight serving loops, harnesses that forbid
 * allocation): the same kernels and arithmetic (y and the appended K/V are bit-identical
 * to kvp_decode_step's), with the workspace taken from a device array of the library
 * instead of a caller buffer.  The caller still passes x, y, len_dev and the slots.
 * The array holds 64 MiB (enough for kvp_workspace_size(KVP_PHASE_DECODE, B) at B <= 64
 * and h <= 8192 with the decode kernels' split counts), one copy per GPU, held until the
 * process ends; its address on a device is looked up on the first call there (that
 * call is the only one that may touch the HIP runtime beyond kernel launches).  The call
 * itself allocates nothing and issues kernel launches only.  All calls on one GPU share
 * the array: calls that overlap in time on one GPU (other streams, other contexts, other
 * threads) race on it and give undefined results; calls in sequence on one stream are
 * safe, and nothing in the array needs to start at zero.
 * Errors: as kvp_decode_step; KVP_E_WORKSPACE when the call's workspace exceeds the
 * array; KVP_E_HIP when the array's address cannot be found on the current device.
 */
int kvp_decode_step_noalloc(kvp_ctx* ctx, const void* x, const int32_t* len_dev, int max_len,
                            void* y, int B, void* stream);

/* ======================================================================== */
/* Paged KV storage (capacity-driven serving)                                 */
/* ======================================================================== */
/*
 * Sec. 1 and Sec. 4 credit KV sharing, at inference, with a smaller KV cache and
 * hence larger batches.  Contiguous slots reserve kv_capacity positions for every
 * sequence; paged storage holds each sequence's positions in 64-position pages
 * drawn from one pool per producer, so a fixed amount of HBM holds as many tokens
 * as the pools have pages, whatever the mix of lengths, and a consumer layer adds
 * no pages.
 *
 * Page layout (bf16 models): producer l's head-major pools K [g][n_pages][64][d_h]
 * and V [g][n_pages][d_h][64] (V transposed within the page, as in the slots), so
 * a run of consecutive pages is one contiguous stream per KV head, as a slot is.  A
 * device page table pages [B][stride] (int32, row b for sequence b of the call)
 * maps position p of sequence b to page pages[b][p / 64], row p % 64, in every
 * producer's pool.  Entries are clamped to [0, n_pages) on the device, so a bad
 * entry reads or writes a wrong page of the pool but never leaves it; entries
 * covering positions a call touches must be mapped (kvp_pager_*).
 */

/* kvp_set_kv_pool -- producer l's page pools (device, caller-owned, 16-byte
 * aligned), n_pages pages each.  Consumers have none; they read tau(l)'s.
 * Errors: KVP_E_INVALID_ARG (NULL pool, n_pages < 1, l not a producer),
 * KVP_E_SHAPE (fp32 model). */
int kvp_set_kv_pool(kvp_ctx* ctx, int l, void* K, void* V, int n_pages);

/* kvp_page_bytes -- bytes of one page (K and V) in one producer's pool:
 * 2 * 64 * g * d_h * sizeof(dtype).  A budget of H bytes holds
 * H / (bytes * number of producers) pages.  Errors: KVP_E_INVALID_ARG. */
int kvp_page_bytes(const kvp_ctx* ctx, size_t* bytes);

/*
 * kvp_prefill_paged -- kvp_prefill with the producers' K/V written to and read
 * from the pools: positions [0, S) of sequence b go to the pages of row b of
 * `pages` (device int32 [B][pages_stride]).  Same kernels and arithmetic as
 * kvp_prefill: y is bit-identical and the pages hold the values the slots would.
 * Errors: as kvp_prefill, plus KVP_E_CAPACITY (S > 64 * pages_stride),
 * KVP_E_STATE (a pool never set), KVP_E_SHAPE (fp32 model).
 */
int kvp_prefill_paged(kvp_ctx* ctx, const void* x, void* y, int B, int S, const int32_t* pages,
                      int pages_stride, void* ws, size_t ws_bytes, void* stream);

/*
 * kvp_decode_step_paged -- kvp_decode_step over the pools: every producer
 * appends at position len_b of row b of `pages`, and every layer attends over
 * positions [0, len_b] through it.  Same kernels and arithmetic as
 * kvp_decode_step (bit-identical y).  Errors: as kvp_decode_step, with
 * KVP_E_CAPACITY when max_len >= 64 * pages_stride; KVP_E_STATE, KVP_E_SHAPE.
 */
int kvp_decode_step_paged(kvp_ctx* ctx, const void* x, const int32_t* len_dev, int max_len,
                          const int32_t* pages, int pages_stride, void* y, int B, void* ws,
                          size_t ws_bytes, void* stream);

/*
 * Host page allocator.  One table of max_seqs rows x max_pages_per_seq entries
 * (-1 = unmapped) over n_pages pages; free pages are handed out lowest first
 * from a fresh pager, and a released sequence's pages are reused first.
 *   kvp_pager_reserve  -- grow sequence seq to hold positions [0, n_tokens);
 *                         all or nothing: KVP_E_CAPACITY when the pool or the
 *                         row is too small (nothing changes); never shrinks.
 *   kvp_pager_release  -- return all of seq's pages.
 *   kvp_pager_rows     -- copy the rows of seqs[0..B) to out [B][max_pages_per_seq]
 *                         (host memory; the caller copies it to the device).
 * Host memory only; not thread-safe (one pager per thread).
 */
typedef struct kvp_pager kvp_pager;
int kvp_pager_create(int n_pages, int max_seqs, int max_pages_per_seq, kvp_pager** out);
void kvp_pager_destroy(kvp_pager* p);
int kvp_pager_reserve(kvp_pager* p, int seq, int n_tokens);
int kvp_pager_release(kvp_pager* p, int seq);
int kvp_pager_free_pages(const kvp_pager* p, int* n);
int kvp_pager_rows(const kvp_pager* p, const int32_t* seqs, int B, int32_t* out);

/* ======================================================================== */
/* Training: forward that keeps activations, and the backward pass           */
/* ======================================================================== */
/*
 * Training a KV-shared model (the setting of Sec. 3) needs the gradients of the
 * stack above.  The forward keeps, per layer l, in the caller's `saved` buffer,
 * in the model dtype: the post-RoPE Q_l and the attention output O_l
 * ([B*S, a*d_h]), the layer input X_l for l >= 1 ([B*S, h]; X_0 is the
 * caller's x), and for bf16 models the row log-sum-exp of the scaled scores
 * ([B, a, Sp] fp32, log2 domain, Sp = S rounded up to 64; fp32 models
 * recompute it).  The producers' K/V slots hold what the forward wrote; the
 * backward reads them.  Layout: layer l's record starts at l * stride and holds,
 * in this order and each starting on a 256-byte boundary, Q_l, O_l, X_l (its
 * bytes are reserved, unwritten, for l = 0), (bf16) the log-sum-exp, and (bf16,
 * when B*S is a multiple of 512 and S a multiple of 8) O_l^T ([a*d_h, B*S], the
 * values of O_l token-major, the operand of dW_O); stride = the record's size
 * rounded up to 256 bytes, and the buffer is L * stride bytes.  Callers may read these tensors after the forward (e.g. to
 * check a layer against a reference fed the same X_l).
 *
 * The backward runs the layers last to first.  For layer l with producer
 * p = tau(l): dW_O = G^T O_l and dO = G W_O with G = dLoss/dX_{l+1}; the
 * attention gradients dQ, dK, dV (softmax Jacobian; dQ and dK rotated back
 * through RoPE); a consumer adds its dK, dV to an fp32 buffer of its producer,
 * and the producer adds that sum to its own (Eq. 3: K_p, V_p feed every layer
 * that maps to p); then dW_Q = dQ^T X_l, for a producer dW_K = dK^T X_l and
 * dW_V = dV^T X_l, and G += dQ W_Q (+ dK W_K + dV W_V).  bf16 models: products
 * on bf16 matrix cores with fp32 accumulation, G carried in fp32.  fp32 models:
 * every step in fp32 on the vector ALUs.
 */

/* kvp_train_saved_size -- bytes of the `saved` buffer for a call with B, S.
 * Errors: KVP_E_INVALID_ARG, KVP_E_CAPACITY. */
int kvp_train_saved_size(const kvp_ctx* ctx, int B, int S, size_t* bytes);

/*
 * kvp_train_forward -- kvp_prefill that also fills `saved` (16-byte aligned,
 * at least kvp_train_saved_size bytes).  Workspace: KVP_PHASE_PREFILL.
 * Errors: as kvp_prefill, plus KVP_E_WORKSPACE for a short `saved` buffer.
 */
int kvp_train_forward(kvp_ctx* ctx, const void* x, void* y, int B, int S, void* saved,
                      size_t saved_bytes, void* ws, size_t ws_bytes, void* stream);

/*
 * kvp_set_layer_grads -- device buffers (fp32, caller-owned, 16-byte aligned)
 * that kvp_backward overwrites with layer l's weight gradients, laid out like
 * the weights: dWq [a*d_h, h], dWo [h, a*d_h]; dWk, dWv [g*d_h, h] for a
 * producer, NULL for a consumer (it has no W_K, W_V).
 * Errors: KVP_E_INVALID_ARG (l out of range, NULL / non-NULL mismatch).
 */
int kvp_set_layer_grads(kvp_ctx* ctx, int l, void* dWq, void* dWk, void* dWv, void* dWo);

/*
 * kvp_backward -- gradients of the last kvp_train_forward with the same x,
 * B, S and saved buffer: dy = dLoss/dY [B*S, h] fp32 in, dx = dLoss/dX_0
 * [B*S, h] fp32 out (dx must not alias dy or x), weight gradients into the
 * buffers of kvp_set_layer_grads.  Workspace: KVP_PHASE_BACKWARD.  For fp32
 * models x is the fp32 input and the whole attention backward of a layer is
 * timed as KVP_K_BWD_ATTN_KV.
 * Errors: KVP_E_INVALID_ARG, KVP_E_CAPACITY, KVP_E_WORKSPACE, KVP_E_SHAPE,
 * KVP_E_STATE (weights, slots or gradient buffers of some layer not set),
 * KVP_E_HIP.
 */
int kvp_backward(kvp_ctx* ctx, const void* x, const void* dy, void* dx, int B, int S,
                 const void* saved, size_t saved_bytes, void* ws, size_t ws_bytes, void* stream);

/* ======================================================================== */
/* Kernel timing (tracing)                                                    */
/* ======================================================================== */

/* Kernel kinds reported by kvp_profile_read. */
#define KVP_K_ROPE_TABLE      0  /* prefill: cos/sin table                        */
#define KVP_K_QKV_GEMM        1  /* prefill: Q|K|V (producer) or Q (consumer) GEMM  */
#define KVP_K_FLASH_ATTN      2  /* prefill: causal flash attention                */
#define KVP_K_OPROJ_GEMM      3  /* prefill: output projection + residual          */
#define KVP_K_DEC_GEMM        4  /* decode: Q|K|V / Q projection                   */
#define KVP_K_DEC_ROPE        5  /* decode: RoPE + cache append                    */
#define KVP_K_DEC_ATTN        6  /* decode: split-K attention                      */
#define KVP_K_DEC_COMBINE     7  /* decode: merge of the split results             */
#define KVP_K_DEC_OPROJ       8  /* decode: output projection + residual           */
#define KVP_K_F32_ROPE        9  /* fp32 models: RoPE + scatter (prefill)          */
#define KVP_K_F32_ATTN       10  /* fp32 models: attention                         */
#define KVP_K_BWD_GEMM       11  /* backward: dO, weight-gradient and dX GEMMs      */
#define KVP_K_BWD_ATTN_KV    12  /* backward: attention dK, dV                      */
#define KVP_K_BWD_ATTN_Q     13  /* backward: attention dQ                          */
#define KVP_K_BWD_AUX        14  /* backward: D, transposes, split-K sums, casts    */
#define KVP_NUM_KERNEL_KINDS 15

/*
 * kvp_profile_enable -- enable (1) or disable (0) kernel timing on ctx and
 * reset the counters.  While enabled, every launch of the calls above is
 * bracketed by two HIP events recorded on the call's stream (the stream the
 * kernel runs on).  Events are created by the library on first use and reused.
 * Errors: KVP_E_INVALID_ARG, KVP_E_HIP.
 */
int kvp_profile_enable(kvp_ctx* ctx, int enable);

/*
 * kvp_profile_read -- waits for the recorded events, adds each launch's
 * elapsed time to ms[kind] and 1 to launches[kind] (both arrays of
 * KVP_NUM_KERNEL_KINDS, zeroed by this call first), then resets the counters.
 * Errors: KVP_E_INVALID_ARG, KVP_E_HIP.
 */
int kvp_profile_read(kvp_ctx* ctx, double* ms, int64_t* launches);

/* kvp_get_map -- copies the canonical map tau[L] into the caller's array. */
int kvp_get_map(const kvp_ctx* ctx, int32_t* tau);

/* kvp_status_string -- static name of a status code ("KVP_OK", ...). */
const char* kvp_status_string(int status);

/* kvp_last_error -- thread-local message of the last failing call ("" if none). */
const char* kvp_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* KVPIPE_H */
