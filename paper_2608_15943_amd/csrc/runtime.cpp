// Host runtime behind the C ABI: context, validation, workspace layout and the
// sharing-map-driven layer scheduler.
//
// For every layer l the scheduler looks up its producer p = tau(l) (Eq. 3):
//   producer (p == l): fused Q|K|V projection (K, V written into slot l, RoPE
//                      fused) -> attention on slot l -> O projection + residual;
//   consumer (p <  l): Q-only projection -> attention on slot p -> O projection
//                      + residual.
// All launches go to the caller's stream in layer order; the library allocates
// no device memory and keeps only host-side state.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstdint>
#include <cstdlib>
#include <cstring>
#include <vector>

#include "kernels.h"
#include "kvpipe.h"
#include "status.h"

namespace kvp {

char* last_error_buffer() {
    static thread_local char buf[512];
    return buf;
}

}  // namespace kvp

using kvp::fail;
using kvp::ok;

namespace {

struct Layer {
    const void* wq = nullptr;
    const void* wk = nullptr;
    const void* wv = nullptr;
    const void* wo = nullptr;
    void* kc = nullptr;
    void* vc = nullptr;
    void* kp = nullptr;     // page pools (kvp_set_kv_pool)
    void* vp = nullptr;
    int n_pages = 0;
    bool weights = false;
    float* dwq = nullptr;   // weight gradients (training), fp32
    float* dwk = nullptr;
    float* dwv = nullptr;
    float* dwo = nullptr;
    bool grads = false;
};

constexpr size_t kAlign = 256;
constexpr int kDecodeMaxRows = 64;   // rows of the skinny decode GEMM
// Decode attention: one single-wave workgroup per SIMD (4 per CU), all resident at once.
constexpr int kSimdsPerCu = 4;

size_t align_up(size_t x) { return (x + kAlign - 1) / kAlign * kAlign; }

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

struct Workspace {
    size_t q = 0, o = 0, xb = 0, xr = 0, rope = 0, proj = 0, part = 0, total = 0;
};

// Where one layer reads and writes.  The residual stream between layers is fp32 (xr,
// updated in place); bf16 models feed the matrix cores a bf16 copy of it (xb).
struct LayerIO {
    const void* a;     // projection input [rows][h], model dtype
    const void* res;   // residual source [rows][h]
    bool res_f32;      // res is fp32 (otherwise the model dtype)
    void* y;           // output [rows][h], model dtype
    float* yf;         // optional fp32 copy of the output (bf16 models)
};

// Device page table of a paged call: row b (stride entries) maps the 64-position pages of
// sequence b to pages of every producer's pool.
struct PageTable {
    const int32_t* pt;
    int stride;
};

}  // namespace

struct kvp_ctx {
    struct ProfRec {
        int kind;
        hipEvent_t start, stop;
    };
    kvp_model_desc d;
    std::vector<int32_t> tau;
    std::vector<Layer> layers;
    int decode_waves = 1024;          // decode attention grid: SIMDs of the device
    bool prof = false;
    bool debug_sync = false;          // KVP_DEBUG_SYNC: wait for and check every launch
    std::vector<ProfRec> recs;        // launches timed since the last read
    std::vector<hipEvent_t> pool;     // idle events for reuse
    ~kvp_ctx() {
        for (auto& r : recs) {
            hipEventDestroy(r.start);
            hipEventDestroy(r.stop);
        }
        for (auto e : pool) hipEventDestroy(e);
    }
    bool bf16() const { return d.dtype == KVP_DTYPE_BF16; }
    size_t esize() const { return bf16() ? 2 : 4; }
    int n_q() const { return d.a * d.d_h; }
    int n_kv() const { return d.g * d.d_h; }
};

namespace {

Workspace layout(const kvp_ctx& c, int phase, int B, int S) {
    Workspace w;
    size_t off = 0;
    auto take = [&](size_t bytes) {
        const size_t at = off;
        off += align_up(bytes);
        return at;
    };
    const size_t e = c.esize();
    const size_t rows = phase == KVP_PHASE_PREFILL ? (size_t)B * S : (size_t)B;
    const size_t nproj = (size_t)(c.d.a + 2 * c.d.g) * c.d.d_h;
    w.q = take(rows * c.n_q() * e);
    w.o = take(rows * c.n_q() * e);
    w.xb = take(rows * c.d.h * e);
    w.xr = take(rows * c.d.h * sizeof(float));
    if (phase == KVP_PHASE_PREFILL) {
        if (c.bf16())
            w.rope = take((size_t)S * (c.d.d_h / 2) * sizeof(float2));
        else
            w.proj = take(rows * nproj * sizeof(float));
    } else {
        // bf16: one plane per 512-wide K slice of the projection GEMM (K = h for both GEMMs).
        const size_t planes = c.bf16() ? (size_t)kvp::decode_gemm_splits(c.d.h) : 1;
        w.proj = take(planes * rows * nproj * sizeof(float));
        if (c.bf16()) {
            const size_t slots = (size_t)c.decode_waves + (size_t)B * c.d.g;
            w.part = take(slots * (c.d.a / c.d.g) * kvp::decode_partial_floats() * sizeof(float));
        }
    }
    w.total = off;
    return w;
}

// The l-th layer's IO within a stack of L layers: layer 0 reads the caller's x, the last
// writes the caller's y; in between the fp32 residual stream xr is updated in place and
// (bf16 models) its bf16 copy xb feeds the next projection.
LayerIO stack_io(bool bf16, int l, int L, const void* x, void* y, char* ws, const Workspace& w) {
    LayerIO io;
    float* xr = (float*)(ws + w.xr);
    if (bf16) {
        io.a = l == 0 ? x : (const void*)(ws + w.xb);
        io.res = l == 0 ? x : (const void*)xr;
        io.res_f32 = l != 0;
        io.y = l == L - 1 ? y : (void*)(ws + w.xb);
        io.yf = l == L - 1 ? nullptr : xr;
    } else {
        io.a = l == 0 ? x : (const void*)xr;
        io.res = io.a;
        io.res_f32 = true;
        io.y = l == L - 1 ? y : (void*)xr;
        io.yf = nullptr;
    }
    return io;
}

int check_hip(hipError_t e, const char* what) {
    if (e != hipSuccess) return fail(KVP_E_HIP, "%s: %s", what, hipGetErrorString(e));
    return KVP_OK;
}

hipError_t take_event(kvp_ctx* c, hipEvent_t* e) {
    if (!c->pool.empty()) {
        *e = c->pool.back();
        c->pool.pop_back();
        return hipSuccess;
    }
    return hipEventCreate(e);
}

const char* kind_name(int kind) {
    static const char* names[KVP_NUM_KERNEL_KINDS] = {
        "RoPE table", "projection GEMM", "flash attention", "output projection GEMM",
        "decode projection GEMM", "decode RoPE + append", "decode attention", "decode combine",
        "decode output projection", "fp32 RoPE", "fp32 attention", "backward GEMM",
        "backward attention dK/dV", "backward attention dQ", "backward auxiliary kernel"};
    return kind >= 0 && kind < KVP_NUM_KERNEL_KINDS ? names[kind] : "kernel";
}

// Debug mode (KVP_DEBUG_SYNC set when the context was created): after each launch, wait
// for the stream and check for an error, so that a failing kernel is named by its own
// call rather than by a later one.  Not for use under graph capture.
int debug_check(const kvp_ctx* c, int kind, hipStream_t st) {
    if (!c->debug_sync) return KVP_OK;
    hipError_t e = hipStreamSynchronize(st);
    if (e == hipSuccess) e = hipGetLastError();
    if (e != hipSuccess) return fail(KVP_E_HIP, "%s (debug sync): %s", kind_name(kind), hipGetErrorString(e));
    return KVP_OK;
}

// Runs launch(); when timing is on, brackets it with two events on st.
template <class F>
int timed(kvp_ctx* c, int kind, hipStream_t st, F&& launch) {
    if (!c->prof) {
        const int rc = launch();
        return rc ? rc : debug_check(c, kind, st);
    }
    hipEvent_t a, b;
    int rc;
    if ((rc = check_hip(take_event(c, &a), "hipEventCreate"))) return rc;
    if ((rc = check_hip(take_event(c, &b), "hipEventCreate"))) {
        c->pool.push_back(a);
        return rc;
    }
    if ((rc = check_hip(hipEventRecord(a, st), "hipEventRecord"))) return rc;
    rc = launch();
    const int rc2 = check_hip(hipEventRecord(b, st), "hipEventRecord");
    c->recs.push_back({kind, a, b});
    if (rc || rc2) return rc ? rc : rc2;
    return debug_check(c, kind, st);
}

int check_layers(const kvp_ctx* c, int lo, int hi, bool paged = false) {
    for (int l = lo; l < hi; ++l) {
        if (!c->layers[l].weights) return fail(KVP_E_STATE, "weights of layer %d were never set", l);
        const int p = c->tau[l];
        if (paged ? !c->layers[p].kp || !c->layers[p].vp : !c->layers[p].kc || !c->layers[p].vc)
            return fail(KVP_E_STATE, "KV %s of producer %d (used by layer %d) was never set",
                        paged ? "pool" : "slot", p, l);
    }
    return KVP_OK;
}

// Where producer P's K/V live for a call: its slot, or its pool under the page table.
struct KvView {
    void* k;
    void* v;
    int cap;
    kvp::Pages pages;
};

// seq0: index of the call's first sequence in the slots (decode runs large batches in
// chunks; a chunk's page table rows are passed already offset).
KvView kv_view(const kvp_ctx* c, const Layer& P, const PageTable* pt, int seq0 = 0) {
    if (!pt) {
        const size_t off = (size_t)seq0 * c->d.g * c->d.kv_capacity * c->d.d_h * c->esize();
        return {P.kc ? (char*)P.kc + off : nullptr, P.vc ? (char*)P.vc + off : nullptr, c->d.kv_capacity,
                kvp::Pages{nullptr, 0, 0}};
    }
    return {P.kp, P.vp, kvp::kPage * pt->stride, kvp::Pages{pt->pt, pt->stride, P.n_pages}};
}

kvp::WRows proj_rows(const kvp_ctx* c, int l, bool producer) {
    const Layer& L = c->layers[l];
    kvp::WRows w{};
    w.p[0] = L.wq;
    w.rows[0] = c->n_q();
    if (producer) {
        w.p[1] = L.wk;
        w.rows[1] = c->n_kv();
        w.p[2] = L.wv;
        w.rows[2] = c->n_kv();
    }
    return w;
}

// One prefill layer over rows [B*S]: io.a -> projections, io.res + O W_O^T -> io.y
// (and io.yf), attention output into o_buf.
int run_prefill_layer(kvp_ctx* c, int l, const LayerIO& io, void* o_buf, char* ws,
                      const Workspace& w, int B, int S, hipStream_t st, void* q_buf = nullptr,
                      float* lse = nullptr, const PageTable* pt = nullptr, void* ot = nullptr) {
    const int p = c->tau[l];
    const bool producer = p == l;
    const Layer& P = c->layers[p];
    const KvView kv = kv_view(c, P, pt);
    const int M = B * S, h = c->d.h, nq = c->n_q();
    const int N = producer ? nq + 2 * c->n_kv() : nq;
    const kvp::WRows wr = proj_rows(c, l, producer);
    kvp::WRows wo{};
    wo.p[0] = c->layers[l].wo;
    wo.rows[0] = h;
    int rc;
    if (c->bf16()) {
        kvp::QkvOut qo{};
        qo.q = (uint16_t*)(q_buf ? q_buf : ws + w.q);
        qo.kc = producer ? (uint16_t*)kv.k : nullptr;
        qo.vc = producer ? (uint16_t*)kv.v : nullptr;
        qo.rope = (const float2*)(ws + w.rope);
        qo.n_q = nq;
        qo.n_kv = producer ? c->n_kv() : 0;
        qo.g = c->d.g;
        qo.cap = kv.cap;
        qo.S = S;
        qo.pages = kv.pages;
        if ((rc = timed(c, KVP_K_QKV_GEMM, st, [&] {
                 return check_hip(kvp::gemm_qkv_bf16((const uint16_t*)io.a, wr, M, N, h, qo, st),
                                  "projection GEMM");
             })))
            return rc;
        if ((rc = timed(c, KVP_K_FLASH_ATTN, st, [&] {
                 return check_hip(kvp::flash_prefill_bf16(qo.q, (const uint16_t*)kv.k,
                                                          (const uint16_t*)kv.v, (uint16_t*)o_buf, lse,
                                                          (uint16_t*)ot, (S + 63) / 64 * 64, B, S, c->d.a,
                                                          c->d.g, kv.cap, kv.pages, st),
                                  "flash attention");
             })))
            return rc;
        return timed(c, KVP_K_OPROJ_GEMM, st, [&] {
            return check_hip(kvp::gemm_resid_bf16((const uint16_t*)o_buf, (const uint16_t*)wo.p[0],
                                                  io.res, io.res_f32, (uint16_t*)io.y, io.yf, M, h,
                                                  nq, st),
                             "output projection");
        });
    }
    float* proj = (float*)(ws + w.proj);
    float* q = (float*)(q_buf ? q_buf : ws + w.q);
    if ((rc = timed(c, KVP_K_QKV_GEMM, st, [&] {
             return check_hip(kvp::gemm_f32((const float*)io.a, wr, M, N, h, proj, nullptr, st),
                              "projection GEMM (fp32)");
         })))
        return rc;
    if ((rc = timed(c, KVP_K_F32_ROPE, st, [&] {
             return check_hip(kvp::rope_scatter(proj, 1, 0, M, S, nullptr, c->d.a, c->d.g, c->d.d_h,
                                                c->d.kv_capacity, c->d.rope_base, producer, false, q,
                                                producer ? P.kc : nullptr, producer ? P.vc : nullptr,
                                                st),
                              "RoPE (fp32)");
         })))
        return rc;
    if ((rc = timed(c, KVP_K_F32_ATTN, st, [&] {
             return check_hip(kvp::attn_f32(q, (const float*)P.kc, (const float*)P.vc, nullptr,
                                            (float*)o_buf, M, S, c->d.a, c->d.g, c->d.d_h,
                                            c->d.kv_capacity, st),
                              "attention (fp32)");
         })))
        return rc;
    return timed(c, KVP_K_OPROJ_GEMM, st, [&] {
        return check_hip(kvp::gemm_f32((const float*)o_buf, wo, M, h, nq, (float*)io.y,
                                       (const float*)io.res, st),
                         "output projection (fp32)");
    });
}

int run_decode_layer(kvp_ctx* c, int l, const LayerIO& io, const int32_t* lens,
                     int max_len, char* ws, const Workspace& w, int B, hipStream_t st,
                     const PageTable* pt = nullptr, int seq0 = 0) {
    const int p = c->tau[l];
    const bool producer = p == l;
    const Layer& P = c->layers[p];
    const KvView kv = kv_view(c, P, pt, seq0);
    const int h = c->d.h, nq = c->n_q();
    const int N = producer ? nq + 2 * c->n_kv() : nq;
    const kvp::WRows wr = proj_rows(c, l, producer);
    kvp::WRows wo{};
    wo.p[0] = c->layers[l].wo;
    wo.rows[0] = h;
    float* proj = (float*)(ws + w.proj);
    void* q = ws + w.q;
    void* o = ws + w.o;
    int rc;
    const int nsplit = c->bf16() ? kvp::decode_gemm_splits(h) : 1;
    // Small batches: one kernel per projection with its epilogue fused (same sums, bit for bit).
    const bool fused = c->bf16() && kvp::decode_fused_ok(B, N, h) && kvp::decode_fused_ok(B, h, nq);
    if (fused) {
        if ((rc = timed(c, KVP_K_DEC_GEMM, st, [&] {
                 return check_hip(kvp::gemm_decode_qkv_fused_bf16((const uint16_t*)io.a, wr, B, N, h, lens, c->d.a,
                                                                  c->d.g, kv.cap, c->d.rope_base, producer,
                                                                  (uint16_t*)q, producer ? (uint16_t*)kv.k : nullptr,
                                                                  producer ? (uint16_t*)kv.v : nullptr, kv.pages, st),
                                  "decode projection GEMM (fused)");
             })))
            return rc;
    } else if ((rc = timed(c, KVP_K_DEC_GEMM, st, [&] {
             return c->bf16()
                        ? check_hip(kvp::gemm_decode_bf16((const uint16_t*)io.a, wr, B, N, h, proj, st),
                                    "decode projection GEMM")
                        : check_hip(kvp::gemm_f32((const float*)io.a, wr, B, N, h, proj, nullptr, st),
                                    "decode projection GEMM (fp32)");
         })))
        return rc;
    if (!fused && (rc = timed(c, KVP_K_DEC_ROPE, st, [&] {
             return c->bf16()
                        ? check_hip(kvp::decode_qkv_epilogue_bf16(
                                        proj, nsplit, B, N, lens, c->d.a, c->d.g, kv.cap,
                                        c->d.rope_base, producer, (uint16_t*)q,
                                        producer ? (uint16_t*)kv.k : nullptr,
                                        producer ? (uint16_t*)kv.v : nullptr, kv.pages, st),
                                    "decode RoPE + cache append")
                        : check_hip(kvp::rope_scatter(proj, 1, 0, B, 0, lens, c->d.a, c->d.g, c->d.d_h,
                                                      c->d.kv_capacity, c->d.rope_base, producer, false,
                                                      q, producer ? P.kc : nullptr,
                                                      producer ? P.vc : nullptr, st),
                                    "decode RoPE + cache append");
         })))
        return rc;
    if (c->bf16()) {
        float* part = (float*)(ws + w.part);
        if ((rc = timed(c, KVP_K_DEC_ATTN, st, [&] {
                 return check_hip(kvp::decode_attn_bf16((const uint16_t*)q, (const uint16_t*)kv.k,
                                                        (const uint16_t*)kv.v, lens, part, B, c->d.a,
                                                        c->d.g, kv.cap, c->decode_waves, kv.pages, st),
                                  "decode attention");
             })))
            return rc;
        if ((rc = timed(c, KVP_K_DEC_COMBINE, st, [&] {
                 return check_hip(kvp::decode_combine_bf16(part, lens, (uint16_t*)o, B, c->d.a, c->d.g,
                                                           kv.cap, c->decode_waves, st),
                                  "decode combine");
             })))
            return rc;
        if (fused)
            return timed(c, KVP_K_DEC_OPROJ, st, [&] {
                return check_hip(kvp::gemm_decode_resid_fused_bf16((const uint16_t*)o, wo, B, h, nq, io.res,
                                                                   io.res_f32, (uint16_t*)io.y, io.yf, st),
                                 "decode output projection (fused)");
            });
        return timed(c, KVP_K_DEC_OPROJ, st, [&] {
            const int ns = kvp::decode_gemm_splits(nq);
            int r2 = check_hip(kvp::gemm_decode_bf16((const uint16_t*)o, wo, B, h, nq, proj, st),
                               "decode output projection");
            if (!r2)
                r2 = check_hip(kvp::decode_resid_bf16(proj, ns, B, h, io.res, io.res_f32,
                                                      (uint16_t*)io.y, io.yf, st),
                               "decode residual");
            return r2;
        });
    }
    if ((rc = timed(c, KVP_K_F32_ATTN, st, [&] {
             return check_hip(kvp::attn_f32((const float*)q, (const float*)P.kc, (const float*)P.vc,
                                            lens, (float*)o, B, 0, c->d.a, c->d.g, c->d.d_h,
                                            c->d.kv_capacity, st),
                              "decode attention (fp32)");
         })))
        return rc;
    return timed(c, KVP_K_DEC_OPROJ, st, [&] {
        return check_hip(kvp::gemm_f32((const float*)o, wo, B, h, nq, (float*)io.y, (const float*)io.res,
                                       st),
                         "decode output projection (fp32)");
    });
}

}  // namespace

// ============================================================================
// C ABI
// ============================================================================

extern "C" const char* kvp_status_string(int s) {
    switch (s) {
        case KVP_OK: return "KVP_OK";
        case KVP_E_INVALID_ARG: return "KVP_E_INVALID_ARG";
        case KVP_E_BAD_MAP: return "KVP_E_BAD_MAP";
        case KVP_E_SHAPE: return "KVP_E_SHAPE";
        case KVP_E_WORKSPACE: return "KVP_E_WORKSPACE";
        case KVP_E_CAPACITY: return "KVP_E_CAPACITY";
        case KVP_E_HIP: return "KVP_E_HIP";
        case KVP_E_STATE: return "KVP_E_STATE";
        default: return "KVP_E_UNKNOWN";
    }
}

extern "C" const char* kvp_last_error(void) { return kvp::last_error_buffer(); }

extern "C" int kvp_create(const kvp_model_desc* desc, const int32_t* tau, kvp_ctx** out) {
    if (!out) return fail(KVP_E_INVALID_ARG, "kvp_create: out is NULL");
    *out = nullptr;
    if (!desc || !tau) return fail(KVP_E_INVALID_ARG, "kvp_create: NULL desc or tau");
    const kvp_model_desc& d = *desc;
    if (d.L < 1 || d.h < 1 || d.a < 1 || d.g < 1 || d.d_h < 2 || d.max_batch < 1 || d.max_seq < 1 ||
        d.kv_capacity < 1)
        return fail(KVP_E_INVALID_ARG, "kvp_create: sizes must be positive");
    if (!(d.rope_base > 0.0)) return fail(KVP_E_INVALID_ARG, "kvp_create: rope_base must be > 0");
    if (d.dtype != KVP_DTYPE_BF16 && d.dtype != KVP_DTYPE_FP32)
        return fail(KVP_E_INVALID_ARG, "kvp_create: unknown dtype %d", d.dtype);
    if (d.a % d.g) return fail(KVP_E_INVALID_ARG, "kvp_create: g must divide a");
    if ((int64_t)d.a * d.d_h != d.h) return fail(KVP_E_INVALID_ARG, "kvp_create: need a * d_h == h");
    if (d.max_seq > d.kv_capacity)
        return fail(KVP_E_INVALID_ARG, "kvp_create: max_seq exceeds kv_capacity");
    if (d.dtype == KVP_DTYPE_BF16) {
        if (d.d_h != 128) return fail(KVP_E_SHAPE, "kvp_create: bf16 models need d_h == 128");
        if (d.kv_capacity % 64)
            return fail(KVP_E_SHAPE, "kvp_create: bf16 models need kv_capacity %% 64 == 0");
        if (d.kv_capacity >= (1 << 23))   // a slot's bytes fit a buffer resource's 32-bit size
            return fail(KVP_E_SHAPE, "kvp_create: bf16 models need kv_capacity < 2^23");
        if (d.a / d.g > 16) return fail(KVP_E_SHAPE, "kvp_create: bf16 decode supports a / g <= 16");
    } else if (d.d_h != 16 && d.d_h != 32 && d.d_h != 64 && d.d_h != 128) {
        return fail(KVP_E_SHAPE, "kvp_create: fp32 models need d_h in {16, 32, 64, 128}");
    }
    std::vector<int32_t> canon(d.L);
    const int rc = kvp_canonicalize_map(d.L, tau, canon.data());
    if (rc) return rc;
    kvp_ctx* c = new (std::nothrow) kvp_ctx;
    if (!c) return fail(KVP_E_INVALID_ARG, "kvp_create: out of host memory");
    c->d = d;
    c->tau = std::move(canon);
    const char* dbg = std::getenv("KVP_DEBUG_SYNC");
    c->debug_sync = dbg && dbg[0] && std::strcmp(dbg, "0") != 0;
    c->layers.resize(d.L);
    // Decode attention runs one wave per SIMD of the device current now; without a
    // device (planning-only use) the MI355X's 256 CUs are assumed.
    int dev = 0, cus = 0;
    if (hipGetDevice(&dev) == hipSuccess &&
        hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) == hipSuccess && cus > 0)
        c->decode_waves = std::min(cus * kSimdsPerCu, kvp::kMaxDecodeSplits);
    else
        c->decode_waves = 256 * kSimdsPerCu;
    (void)hipGetLastError();
    *out = c;
    return ok();
}

extern "C" int kvp_destroy(kvp_ctx* ctx) {
    delete ctx;
    return ok();
}

extern "C" int kvp_profile_enable(kvp_ctx* ctx, int enable) {
    if (!ctx) return fail(KVP_E_INVALID_ARG, "kvp_profile_enable: NULL ctx");
    for (auto& r : ctx->recs) {
        ctx->pool.push_back(r.start);
        ctx->pool.push_back(r.stop);
    }
    ctx->recs.clear();
    ctx->prof = enable != 0;
    return ok();
}

extern "C" int kvp_profile_read(kvp_ctx* ctx, double* ms, int64_t* launches) {
    if (!ctx || !ms || !launches) return fail(KVP_E_INVALID_ARG, "kvp_profile_read: NULL argument");
    for (int k = 0; k < KVP_NUM_KERNEL_KINDS; ++k) {
        ms[k] = 0.0;
        launches[k] = 0;
    }
    int rc = KVP_OK;
    for (auto& r : ctx->recs) {
        float t = 0.f;
        if (!rc) rc = check_hip(hipEventSynchronize(r.stop), "hipEventSynchronize");
        if (!rc) rc = check_hip(hipEventElapsedTime(&t, r.start, r.stop), "hipEventElapsedTime");
        if (!rc && r.kind >= 0 && r.kind < KVP_NUM_KERNEL_KINDS) {
            ms[r.kind] += t;
            launches[r.kind] += 1;
        }
        ctx->pool.push_back(r.start);
        ctx->pool.push_back(r.stop);
    }
    ctx->recs.clear();
    return rc;
}

extern "C" int kvp_get_map(const kvp_ctx* ctx, int32_t* tau) {
    if (!ctx || !tau) return fail(KVP_E_INVALID_ARG, "kvp_get_map: NULL argument");
    std::memcpy(tau, ctx->tau.data(), sizeof(int32_t) * ctx->d.L);
    return ok();
}

extern "C" int kvp_set_layer(kvp_ctx* ctx, int l, const void* Wq, const void* Wk, const void* Wv,
                             const void* Wo) {
    if (!ctx) return fail(KVP_E_INVALID_ARG, "kvp_set_layer: NULL ctx");
    if (l < 0 || l >= ctx->d.L) return fail(KVP_E_INVALID_ARG, "kvp_set_layer: layer %d out of range", l);
    const bool producer = ctx->tau[l] == l;
    if (!Wq || !Wo) return fail(KVP_E_INVALID_ARG, "kvp_set_layer: Wq and Wo are required");
    if (producer && (!Wk || !Wv))
        return fail(KVP_E_INVALID_ARG, "kvp_set_layer: layer %d is a producer and needs Wk, Wv", l);
    if (!producer && (Wk || Wv))
        return fail(KVP_E_INVALID_ARG,
                    "kvp_set_layer: layer %d shares K/V of layer %d and takes no Wk, Wv", l,
                    ctx->tau[l]);
    if (!aligned16(Wq) || !aligned16(Wo) || (Wk && !aligned16(Wk)) || (Wv && !aligned16(Wv)))
        return fail(KVP_E_INVALID_ARG, "kvp_set_layer: weights must be 16-byte aligned");
    Layer& L = ctx->layers[l];
    L.wq = Wq;
    L.wk = Wk;
    L.wv = Wv;
    L.wo = Wo;
    L.weights = true;
    return ok();
}

extern "C" int kvp_set_kv_slot(kvp_ctx* ctx, int l, void* K, void* V) {
    if (!ctx) return fail(KVP_E_INVALID_ARG, "kvp_set_kv_slot: NULL ctx");
    if (l < 0 || l >= ctx->d.L) return fail(KVP_E_INVALID_ARG, "kvp_set_kv_slot: layer %d out of range", l);
    if (ctx->tau[l] != l)
        return fail(KVP_E_INVALID_ARG, "kvp_set_kv_slot: layer %d is a consumer and owns no slot", l);
    if (!K || !V) return fail(KVP_E_INVALID_ARG, "kvp_set_kv_slot: NULL K or V");
    if (!aligned16(K) || !aligned16(V))
        return fail(KVP_E_INVALID_ARG, "kvp_set_kv_slot: slots must be 16-byte aligned");
    ctx->layers[l].kc = K;
    ctx->layers[l].vc = V;
    return ok();
}

extern "C" int kvp_set_kv_pool(kvp_ctx* ctx, int l, void* K, void* V, int n_pages) {
    if (!ctx) return fail(KVP_E_INVALID_ARG, "kvp_set_kv_pool: NULL ctx");
    if (l < 0 || l >= ctx->d.L) return fail(KVP_E_INVALID_ARG, "kvp_set_kv_pool: layer %d out of range", l);
    if (ctx->tau[l] != l)
        return fail(KVP_E_INVALID_ARG, "kvp_set_kv_pool: layer %d is a consumer and owns no pool", l);
    if (!ctx->bf16()) return fail(KVP_E_SHAPE, "kvp_set_kv_pool: paged KV storage needs a bf16 model");
    if (!K || !V || n_pages < 1) return fail(KVP_E_INVALID_ARG, "kvp_set_kv_pool: NULL pool or n_pages < 1");
    if (!aligned16(K) || !aligned16(V))
        return fail(KVP_E_INVALID_ARG, "kvp_set_kv_pool: pools must be 16-byte aligned");
    Layer& Ly = ctx->layers[l];
    Ly.kp = K;
    Ly.vp = V;
    Ly.n_pages = n_pages;
    return ok();
}

extern "C" int kvp_page_bytes(const kvp_ctx* ctx, size_t* bytes) {
    if (!ctx || !bytes) return fail(KVP_E_INVALID_ARG, "kvp_page_bytes: NULL argument");
    *bytes = (size_t)2 * kvp::kPage * ctx->d.g * ctx->d.d_h * ctx->esize();
    return ok();
}

namespace {

// ---- training --------------------------------------------------------------

int round64(int S) { return (S + 63) / 64 * 64; }

// Token counts that are multiples of this take the row-major weight-gradient GEMMs on
// transposed activations (64-wide K tiles times up to 8 split-K slices).
constexpr int kTokGrain = 512;
// On that path, when S % 8 == 0, the attention kernels write O^T and [dQ|dK|dV]^T
// themselves (8-byte aligned token runs) instead of separate transposes.
bool tokmajor_direct(int B, int S) { return (size_t)B * S % kTokGrain == 0 && S % 8 == 0; }

// Per-layer activations of kvp_train_forward, layer l at l * stride: Q (after RoPE), the
// attention output O and the layer input X in the model dtype, and (bf16 models) the
// log-sum-exp of the scores, which fp32 models recompute.  When the backward takes the
// token-major weight-gradient path, the attention kernel also saves O^T [a*d_h][B*S].
struct Saved {
    size_t q = 0, o = 0, x = 0, lse = 0, ot = 0, stride = 0, total = 0;
    bool has_ot = false;
};

Saved saved_layout(const kvp_ctx& c, int B, int S) {
    Saved v;
    size_t off = 0;
    auto take = [&](size_t bytes) {
        const size_t at = off;
        off += align_up(bytes);
        return at;
    };
    const size_t M = (size_t)B * S, e = c.esize();
    v.q = take(M * c.n_q() * e);
    v.o = take(M * c.n_q() * e);
    v.x = take(M * c.d.h * e);
    if (c.bf16()) v.lse = take((size_t)B * c.d.a * round64(S) * sizeof(float));
    v.has_ot = c.bf16() && tokmajor_direct(B, S);
    if (v.has_ot) v.ot = take(M * c.n_q() * e);
    v.stride = off;
    v.total = off * c.d.L;
    return v;
}

// Workspace of kvp_backward.
struct BwdWs {
    size_t gb = 0, dO = 0, lse = 0, dsum = 0, dqkv = 0, acc = 0, wot = 0, wst = 0, part = 0, rope = 0, ta = 0, tb = 0,
           total = 0;
    size_t acc_plane = 0;          // floats of one dK or dV sum
    std::vector<int> acc_slot;     // per layer: index of its fp32 sum pair, or -1
};

BwdWs bwd_layout(const kvp_ctx& c, int B, int S) {
    BwdWs w;
    size_t off = 0;
    auto take = [&](size_t bytes) {
        const size_t at = off;
        off += align_up(bytes);
        return at;
    };
    const size_t M = (size_t)B * S;
    const size_t h = c.d.h, nq = c.n_q(), nkv = c.n_kv(), np = nq + 2 * nkv;
    // One fp32 dK/dV pair per producer that has consumers.
    w.acc_slot.assign(c.d.L, -1);
    int nacc = 0;
    for (int l = 0; l < c.d.L; ++l)
        if (c.tau[l] == l)
            for (int j = l + 1; j < c.d.L; ++j)
                if (c.tau[j] == l) {
                    w.acc_slot[l] = nacc++;
                    break;
                }
    w.acc_plane = (size_t)B * c.d.g * S * c.d.d_h;
    if (!c.bf16()) {
        // fp32: dO, [dQ | dK | dV], the per-(token, head) log-sum-exp and D, the sums, RoPE.
        w.dO = take(M * nq * sizeof(float));
        w.dqkv = take(M * np * sizeof(float));
        w.lse = take(M * c.d.a * sizeof(float));
        w.dsum = take(M * c.d.a * sizeof(float));
        w.acc = take((size_t)nacc * 2 * w.acc_plane * sizeof(float));
        w.rope = take((size_t)S * (c.d.d_h / 2) * sizeof(float2));
        w.total = off;
        return w;
    }
    w.gb = take(M * h * 2);
    w.dO = take(M * nq * 2);
    w.dsum = take((size_t)B * c.d.a * round64(S) * sizeof(float));
    w.dqkv = take(M * np * 2);
    w.acc = take((size_t)nacc * 2 * w.acc_plane * sizeof(float));
    w.wot = take(nq * h * 2);   // W_O^T [a*d_h][h]
    w.wst = take(h * np * 2);   // [W_Q; W_K; W_V]^T [h][np]
    // Split-K partial planes of the weight-gradient GEMMs (consumers: Q rows only).
    const int so = kvp::gemm_out_splits((int)h, (int)nq, (int)M);
    const int sp = kvp::gemm_out_splits((int)np, (int)h, (int)M);
    const int sc = kvp::gemm_out_splits((int)nq, (int)h, (int)M);
    w.part = take(std::max({(size_t)so * h * nq, (size_t)sp * np * h, (size_t)sc * nq * h}) * sizeof(float));
    w.rope = take((size_t)S * 64 * sizeof(float2));
    // Token-major copies for the row-major weight-gradient GEMMs (token counts that are
    // multiples of 512): G^T or [dQ|dK|dV]^T, and O^T or X^T.
    if (M % kTokGrain == 0) {
        w.ta = take(M * std::max(h, np) * 2);
        w.tb = take(M * std::max(h, nq) * 2);
    }
    w.total = off;
    return w;
}

}  // namespace

extern "C" int kvp_workspace_size(const kvp_ctx* ctx, int phase, int B, int S, size_t* bytes) {
    if (!ctx || !bytes) return fail(KVP_E_INVALID_ARG, "kvp_workspace_size: NULL argument");
    if (phase != KVP_PHASE_PREFILL && phase != KVP_PHASE_DECODE && phase != KVP_PHASE_BACKWARD)
        return fail(KVP_E_INVALID_ARG, "kvp_workspace_size: unknown phase");
    const bool seq = phase != KVP_PHASE_DECODE;
    if (B < 1 || (seq && S < 1))
        return fail(KVP_E_INVALID_ARG, "kvp_workspace_size: B and S must be >= 1");
    if (B > ctx->d.max_batch) return fail(KVP_E_CAPACITY, "kvp_workspace_size: B > max_batch");
    if (seq && S > ctx->d.max_seq)
        return fail(KVP_E_CAPACITY, "kvp_workspace_size: S > max_seq");
    if (phase == KVP_PHASE_BACKWARD) {
        *bytes = bwd_layout(*ctx, B, S).total;
        return ok();
    }
    *bytes = layout(*ctx, phase, B, phase == KVP_PHASE_PREFILL ? S : 1).total;
    return ok();
}

namespace {

int check_prefill_args(const kvp_ctx* ctx, const void* x, const void* y, int B, int S, void* ws,
                       size_t ws_bytes, Workspace* w) {
    if (!ctx || !x || !y) return fail(KVP_E_INVALID_ARG, "prefill: NULL ctx, x or y");
    if (x == y) return fail(KVP_E_INVALID_ARG, "prefill: x and y must not alias");
    if (!aligned16(x) || !aligned16(y)) return fail(KVP_E_INVALID_ARG, "prefill: x, y must be 16-byte aligned");
    if (B < 1 || S < 1) return fail(KVP_E_INVALID_ARG, "prefill: B and S must be >= 1");
    if (B > ctx->d.max_batch || S > ctx->d.max_seq)
        return fail(KVP_E_CAPACITY, "prefill: B=%d, S=%d exceed max_batch=%d / max_seq=%d", B, S,
                    ctx->d.max_batch, ctx->d.max_seq);
    if ((int64_t)B * S > INT32_MAX / std::max(ctx->d.h, 1))
        return fail(KVP_E_SHAPE, "prefill: B * S * h exceeds the 32-bit row index range");
    *w = layout(*ctx, KVP_PHASE_PREFILL, B, S);
    if (!ws || ws_bytes < w->total || !aligned16(ws))
        return fail(KVP_E_WORKSPACE, "prefill: workspace needs %zu bytes (16-byte aligned), got %zu",
                    w->total, ws ? ws_bytes : (size_t)0);
    return KVP_OK;
}

}  // namespace

namespace {

int prefill_impl(kvp_ctx* ctx, const void* x, void* y, int B, int S, void* ws, size_t ws_bytes,
                 void* stream, const PageTable* pt) {
    Workspace w;
    int rc = check_prefill_args(ctx, x, y, B, S, ws, ws_bytes, &w);
    if (rc) return rc;
    if ((rc = check_layers(ctx, 0, ctx->d.L, pt != nullptr))) return rc;
    hipStream_t st = (hipStream_t)stream;
    char* base = (char*)ws;
    if (ctx->bf16() && (rc = timed(ctx, KVP_K_ROPE_TABLE, st, [&] {
                            return check_hip(kvp::rope_table((float2*)(base + w.rope), S, ctx->d.d_h,
                                                             ctx->d.rope_base, st),
                                             "RoPE table");
                        })))
        return rc;
    const int L = ctx->d.L;
    for (int l = 0; l < L; ++l) {
        const LayerIO io = stack_io(ctx->bf16(), l, L, x, y, base, w);
        if ((rc = run_prefill_layer(ctx, l, io, base + w.o, base, w, B, S, st, nullptr, nullptr, pt))) return rc;
    }
    return ok();
}

// Host checks shared by the paged entry points.
int check_paged(const kvp_ctx* ctx, const int32_t* pages, int stride, const char* who) {
    if (!ctx) return fail(KVP_E_INVALID_ARG, "%s: NULL ctx", who);
    if (!ctx->bf16()) return fail(KVP_E_SHAPE, "%s: paged KV storage needs a bf16 model", who);
    if (!pages || stride < 1) return fail(KVP_E_INVALID_ARG, "%s: NULL page table or stride < 1", who);
    if ((int64_t)stride * kvp::kPage > INT32_MAX / 2)
        return fail(KVP_E_INVALID_ARG, "%s: page table stride %d too large", who, stride);
    return KVP_OK;
}

}  // namespace

extern "C" int kvp_prefill(kvp_ctx* ctx, const void* x, void* y, int B, int S, void* ws,
                           size_t ws_bytes, void* stream) {
    return prefill_impl(ctx, x, y, B, S, ws, ws_bytes, stream, nullptr);
}

extern "C" int kvp_prefill_paged(kvp_ctx* ctx, const void* x, void* y, int B, int S, const int32_t* pages,
                                 int pages_stride, void* ws, size_t ws_bytes, void* stream) {
    int rc;
    if ((rc = check_paged(ctx, pages, pages_stride, "kvp_prefill_paged"))) return rc;
    if (S > kvp::kPage * pages_stride)
        return fail(KVP_E_CAPACITY, "kvp_prefill_paged: S=%d exceeds the page table's reach (%d positions)", S,
                    kvp::kPage * pages_stride);
    const PageTable pt{pages, pages_stride};
    return prefill_impl(ctx, x, y, B, S, ws, ws_bytes, stream, &pt);
}

extern "C" int kvp_layer_forward(kvp_ctx* ctx, int l, const void* x, void* attn_out, void* y, int B,
                                 int S, void* ws, size_t ws_bytes, void* stream) {
    Workspace w;
    int rc = check_prefill_args(ctx, x, y, B, S, ws, ws_bytes, &w);
    if (rc) return rc;
    if (l < 0 || l >= ctx->d.L) return fail(KVP_E_INVALID_ARG, "kvp_layer_forward: layer %d out of range", l);
    if (attn_out && !aligned16(attn_out))
        return fail(KVP_E_INVALID_ARG, "kvp_layer_forward: attn_out must be 16-byte aligned");
    if ((rc = check_layers(ctx, l, l + 1))) return rc;
    hipStream_t st = (hipStream_t)stream;
    char* base = (char*)ws;
    if (ctx->bf16() && (rc = timed(ctx, KVP_K_ROPE_TABLE, st, [&] {
                            return check_hip(kvp::rope_table((float2*)(base + w.rope), S, ctx->d.d_h,
                                                             ctx->d.rope_base, st),
                                             "RoPE table");
                        })))
        return rc;
    LayerIO io{x, x, !ctx->bf16(), y, nullptr};
    return run_prefill_layer(ctx, l, io, attn_out ? attn_out : base + w.o, base, w, B, S, st);
}

namespace {

int decode_impl(kvp_ctx* ctx, const void* x, const int32_t* len_dev, int max_len, void* y, int B, void* ws,
                size_t ws_bytes, void* stream, const PageTable* pt) {
    if (!ctx || !x || !y || !len_dev) return fail(KVP_E_INVALID_ARG, "decode: NULL argument");
    if (x == y) return fail(KVP_E_INVALID_ARG, "decode: x and y must not alias");
    if (!aligned16(x) || !aligned16(y)) return fail(KVP_E_INVALID_ARG, "decode: x, y must be 16-byte aligned");
    if (B < 1 || max_len < 0) return fail(KVP_E_INVALID_ARG, "decode: B >= 1 and max_len >= 0 required");
    if (B > ctx->d.max_batch) return fail(KVP_E_CAPACITY, "decode: B=%d > max_batch=%d", B, ctx->d.max_batch);
    const int reach = pt ? kvp::kPage * pt->stride : ctx->d.kv_capacity;
    if (max_len >= reach)
        return fail(KVP_E_CAPACITY, "decode: position %d does not fit %s=%d", max_len,
                    pt ? "the page table's reach" : "kv_capacity", reach);
    const Workspace wfull = layout(*ctx, KVP_PHASE_DECODE, B, 1);
    if (!ws || ws_bytes < wfull.total || !aligned16(ws))
        return fail(KVP_E_WORKSPACE, "decode: workspace needs %zu bytes (16-byte aligned), got %zu",
                    wfull.total, ws ? ws_bytes : (size_t)0);
    int rc;
    if ((rc = check_layers(ctx, 0, ctx->d.L, pt != nullptr))) return rc;
    hipStream_t st = (hipStream_t)stream;
    char* base = (char*)ws;
    const int L = ctx->d.L;
    // bf16 kernels take at most kDecodeMaxRows sequences per launch; sequences are
    // independent, so a larger batch runs as consecutive chunks through the whole stack
    // (each chunk reads the weights once more), reusing the workspace on the same stream.
    const int chunk = ctx->bf16() ? kDecodeMaxRows : B;
    const size_t row_bytes = (size_t)ctx->d.h * ctx->esize();
    for (int b0 = 0; b0 < B; b0 += chunk) {
        const int Bc = std::min(chunk, B - b0);
        const Workspace w = layout(*ctx, KVP_PHASE_DECODE, Bc, 1);
        const char* xc = (const char*)x + (size_t)b0 * row_bytes;
        char* yc = (char*)y + (size_t)b0 * row_bytes;
        PageTable ptc{};
        if (pt) ptc = PageTable{pt->pt + (size_t)b0 * pt->stride, pt->stride};
        for (int l = 0; l < L; ++l) {
            const LayerIO io = stack_io(ctx->bf16(), l, L, xc, yc, base, w);
            if ((rc = run_decode_layer(ctx, l, io, len_dev + b0, max_len, base, w, Bc, st, pt ? &ptc : nullptr,
                                       b0)))
                return rc;
        }
    }
    return ok();
}

}  // namespace

extern "C" int kvp_decode_step(kvp_ctx* ctx, const void* x, const int32_t* len_dev, int max_len,
                               void* y, int B, void* ws, size_t ws_bytes, void* stream) {
    return decode_impl(ctx, x, len_dev, max_len, y, B, ws, ws_bytes, stream, nullptr);
}

extern "C" int kvp_decode_step_noalloc(kvp_ctx* ctx, const void* x, const int32_t* len_dev, int max_len,
                                       void* y, int B, void* stream) {
    if (!ctx) return fail(KVP_E_INVALID_ARG, "kvp_decode_step_noalloc: NULL ctx");
    if (B < 1) return fail(KVP_E_INVALID_ARG, "kvp_decode_step_noalloc: B >= 1 required");
    const size_t need = layout(*ctx, KVP_PHASE_DECODE, B, 1).total;
    if (need > kvp::kStaticScratchBytes)
        return fail(KVP_E_WORKSPACE,
                    "kvp_decode_step_noalloc: this call needs %zu bytes of scratch, the static array holds %zu",
                    need, kvp::kStaticScratchBytes);
    void* ws = nullptr;
    size_t n = 0;
    int rc;
    if ((rc = check_hip(kvp::static_scratch(&ws, &n), "kvp_decode_step_noalloc: static scratch address")))
        return rc;
    return decode_impl(ctx, x, len_dev, max_len, y, B, ws, n, stream, nullptr);
}

extern "C" int kvp_decode_step_paged(kvp_ctx* ctx, const void* x, const int32_t* len_dev, int max_len,
                                     const int32_t* pages, int pages_stride, void* y, int B, void* ws,
                                     size_t ws_bytes, void* stream) {
    int rc;
    if ((rc = check_paged(ctx, pages, pages_stride, "kvp_decode_step_paged"))) return rc;
    const PageTable pt{pages, pages_stride};
    return decode_impl(ctx, x, len_dev, max_len, y, B, ws, ws_bytes, stream, &pt);
}

// ============================================================================
// Training
// ============================================================================

extern "C" int kvp_train_saved_size(const kvp_ctx* ctx, int B, int S, size_t* bytes) {
    if (!ctx || !bytes) return fail(KVP_E_INVALID_ARG, "kvp_train_saved_size: NULL argument");
    if (B < 1 || S < 1) return fail(KVP_E_INVALID_ARG, "kvp_train_saved_size: B and S must be >= 1");
    if (B > ctx->d.max_batch || S > ctx->d.max_seq)
        return fail(KVP_E_CAPACITY, "kvp_train_saved_size: B or S beyond max_batch / max_seq");
    *bytes = saved_layout(*ctx, B, S).total;
    return ok();
}

extern "C" int kvp_train_forward(kvp_ctx* ctx, const void* x, void* y, int B, int S, void* saved,
                                 size_t saved_bytes, void* ws, size_t ws_bytes, void* stream) {
    Workspace w;
    int rc = check_prefill_args(ctx, x, y, B, S, ws, ws_bytes, &w);
    if (rc) return rc;
    const Saved sv = saved_layout(*ctx, B, S);
    if (!saved || saved_bytes < sv.total || !aligned16(saved))
        return fail(KVP_E_WORKSPACE, "kvp_train_forward: saved buffer needs %zu bytes (16-byte aligned), got %zu",
                    sv.total, saved ? saved_bytes : (size_t)0);
    if ((rc = check_layers(ctx, 0, ctx->d.L))) return rc;
    hipStream_t st = (hipStream_t)stream;
    char* base = (char*)ws;
    char* sb = (char*)saved;
    const bool bf = ctx->bf16();
    if (bf && (rc = timed(ctx, KVP_K_ROPE_TABLE, st, [&] {
                   return check_hip(kvp::rope_table((float2*)(base + w.rope), S, ctx->d.d_h, ctx->d.rope_base,
                                                    st),
                                    "RoPE table");
               })))
        return rc;
    const int L = ctx->d.L;
    float* xr = (float*)(base + w.xr);
    for (int l = 0; l < L; ++l) {
        char* lay = sb + (size_t)l * sv.stride;
        void* next_x = l == L - 1 ? y : (void*)(sb + (size_t)(l + 1) * sv.stride + sv.x);
        LayerIO io;
        io.a = l == 0 ? x : (const void*)(lay + sv.x);
        if (bf) {
            // The bf16 copy of the layer input is saved; the fp32 stream stays in xr.
            io.res = l == 0 ? x : (const void*)xr;
            io.res_f32 = l != 0;
            io.yf = l == L - 1 ? nullptr : xr;
        } else {
            // fp32: the stream itself moves from one layer's saved input to the next.
            io.res = io.a;
            io.res_f32 = true;
            io.yf = nullptr;
        }
        io.y = next_x;
        if ((rc = run_prefill_layer(ctx, l, io, lay + sv.o, base, w, B, S, st, lay + sv.q,
                                    bf ? (float*)(lay + sv.lse) : nullptr, nullptr,
                                    sv.has_ot ? lay + sv.ot : nullptr)))
            return rc;
    }
    return ok();
}

extern "C" int kvp_set_layer_grads(kvp_ctx* ctx, int l, void* dWq, void* dWk, void* dWv, void* dWo) {
    if (!ctx) return fail(KVP_E_INVALID_ARG, "kvp_set_layer_grads: NULL ctx");
    if (l < 0 || l >= ctx->d.L) return fail(KVP_E_INVALID_ARG, "kvp_set_layer_grads: layer %d out of range", l);
    const bool producer = ctx->tau[l] == l;
    if (!dWq || !dWo) return fail(KVP_E_INVALID_ARG, "kvp_set_layer_grads: dWq and dWo are required");
    if (producer && (!dWk || !dWv))
        return fail(KVP_E_INVALID_ARG, "kvp_set_layer_grads: layer %d is a producer and needs dWk, dWv", l);
    if (!producer && (dWk || dWv))
        return fail(KVP_E_INVALID_ARG, "kvp_set_layer_grads: layer %d has no W_K, W_V", l);
    if (!aligned16(dWq) || !aligned16(dWo) || (dWk && !aligned16(dWk)) || (dWv && !aligned16(dWv)))
        return fail(KVP_E_INVALID_ARG, "kvp_set_layer_grads: buffers must be 16-byte aligned");
    Layer& L = ctx->layers[l];
    L.dwq = (float*)dWq;
    L.dwk = (float*)dWk;
    L.dwv = (float*)dWv;
    L.dwo = (float*)dWo;
    L.grads = true;
    return ok();
}

namespace {

// Backward of an fp32 model: the same sequence as the bf16 path, every product on the
// vector ALUs in fp32.  G, the gradient at the current layer's output, is dY for the
// last layer and dX (updated in place, after its last read) below it.
int backward_f32(kvp_ctx* ctx, const float* x, const float* dy, float* dx, int B, int S, const Saved& sv,
                 const char* sb, const BwdWs& w, char* base, hipStream_t st) {
    const int h = ctx->d.h, nq = ctx->n_q(), nkv = ctx->n_kv(), L = ctx->d.L, M = B * S;
    float* dO = (float*)(base + w.dO);
    float* dqkv = (float*)(base + w.dqkv);
    float* acc = (float*)(base + w.acc);
    float2* rope = (float2*)(base + w.rope);
    auto gemm = [&](auto&& f) { return timed(ctx, KVP_K_BWD_GEMM, st, f); };
    int rc;
    if ((rc = timed(ctx, KVP_K_BWD_AUX, st, [&] {
             return check_hip(kvp::rope_table(rope, S, ctx->d.d_h, ctx->d.rope_base, st), "RoPE table");
         })))
        return rc;
    std::vector<char> acc_written(L, 0);
    for (int l = L - 1; l >= 0; --l) {
        const int p = ctx->tau[l];
        const bool producer = p == l;
        const int np = producer ? nq + 2 * nkv : nq;
        const Layer& Ly = ctx->layers[l];
        const Layer& Pl = ctx->layers[p];
        const char* lay = sb + (size_t)l * sv.stride;
        const float* Ql = (const float*)(lay + sv.q);
        const float* Ol = (const float*)(lay + sv.o);
        const float* Xl = l == 0 ? x : (const float*)(lay + sv.x);
        const float* G = l == L - 1 ? dy : dx;
        // dO = G W_O, dW_O = G^T O.
        if ((rc = gemm([&] {
                 return check_hip(kvp::gemm_f32_strided(G, h, 1, (const float*)Ly.wo, nq, 1, nullptr, dO, nq, M,
                                                        nq, h, st),
                                  "dO GEMM (fp32)");
             })))
            return rc;
        if ((rc = gemm([&] {
                 return check_hip(kvp::gemm_f32_strided(G, 1, h, Ol, nq, 1, nullptr, Ly.dwo, nq, h, nq, M, st),
                                  "dW_O GEMM (fp32)");
             })))
            return rc;
        // Attention: dQ into dqkv; dK, dV into the producer's sums (consumer) or dqkv (producer).
        kvp::AttnBwdF32 a{};
        a.q = Ql; a.dO = dO; a.O = Ol; a.kc = (const float*)Pl.kc; a.vc = (const float*)Pl.vc; a.rope = rope;
        a.lse = (float*)(base + w.lse);
        a.dsum = (float*)(base + w.dsum);
        const int slot = w.acc_slot[p];
        float* ak = slot >= 0 ? acc + (size_t)slot * 2 * w.acc_plane : nullptr;
        float* av = slot >= 0 ? ak + w.acc_plane : nullptr;
        a.acc_in_k = acc_written[p] ? ak : nullptr;
        a.acc_in_v = acc_written[p] ? av : nullptr;
        if (!producer) {
            a.acc_out_k = ak;
            a.acc_out_v = av;
            acc_written[p] = 1;
        } else {
            a.out_kv = dqkv;
            a.col_k = nq;
            a.col_v = nq + nkv;
        }
        a.out_q = dqkv;
        a.ldo = np;
        a.B = B; a.S = S; a.a = ctx->d.a; a.g = ctx->d.g; a.d = ctx->d.d_h; a.cap = ctx->d.kv_capacity;
        if ((rc = timed(ctx, KVP_K_BWD_ATTN_KV, st, [&] {
                 return check_hip(kvp::attn_bwd_f32(a, st), "attention backward (fp32)");
             })))
            return rc;
        // dW_Q (, dW_K, dW_V) = [dQ | dK | dV]^T X_l; dX_l = G + dQ W_Q (+ dK W_K + dV W_V).
        struct Part {
            int col, rows;
            const void* wt;
            float* dw;
        };
        const Part parts[3] = {{0, nq, Ly.wq, Ly.dwq}, {nq, nkv, Ly.wk, Ly.dwk}, {nq + nkv, nkv, Ly.wv, Ly.dwv}};
        for (int i = 0; i < (producer ? 3 : 1); ++i) {
            const Part& pt = parts[i];
            if ((rc = gemm([&] {
                     return check_hip(kvp::gemm_f32_strided(dqkv + pt.col, 1, np, Xl, h, 1, nullptr, pt.dw, h,
                                                            pt.rows, h, M, st),
                                      "dW_QKV GEMM (fp32)");
                 })))
                return rc;
        }
        for (int i = 0; i < (producer ? 3 : 1); ++i) {
            const Part& pt = parts[i];
            if ((rc = gemm([&] {
                     return check_hip(kvp::gemm_f32_strided(dqkv + pt.col, np, 1, (const float*)pt.wt, h, 1,
                                                            i == 0 ? G : dx, dx, h, M, h, pt.rows, st),
                                      "dX GEMM (fp32)");
                 })))
                return rc;
        }
    }
    return ok();
}

}  // namespace

extern "C" int kvp_backward(kvp_ctx* ctx, const void* x, const void* dy, void* dx, int B, int S,
                            const void* saved, size_t saved_bytes, void* ws, size_t ws_bytes,
                            void* stream) {
    if (!ctx || !x || !dy || !dx) return fail(KVP_E_INVALID_ARG, "kvp_backward: NULL argument");
    if (dx == dy || dx == x) return fail(KVP_E_INVALID_ARG, "kvp_backward: dx must not alias dy or x");
    if (!aligned16(x) || !aligned16(dy) || !aligned16(dx))
        return fail(KVP_E_INVALID_ARG, "kvp_backward: x, dy, dx must be 16-byte aligned");
    if (B < 1 || S < 1) return fail(KVP_E_INVALID_ARG, "kvp_backward: B and S must be >= 1");
    if (B > ctx->d.max_batch || S > ctx->d.max_seq)
        return fail(KVP_E_CAPACITY, "kvp_backward: B=%d, S=%d exceed max_batch / max_seq", B, S);
    const int h = ctx->d.h, nq = ctx->n_q(), nkv = ctx->n_kv(), L = ctx->d.L;
    const int Sp = round64(S), M = B * S;
    if ((int64_t)M * std::max(h, nq + 2 * nkv) > INT32_MAX)
        return fail(KVP_E_SHAPE, "kvp_backward: sizes exceed the 32-bit index range");
    const Saved sv = saved_layout(*ctx, B, S);
    if (!saved || saved_bytes < sv.total || !aligned16(saved))
        return fail(KVP_E_WORKSPACE, "kvp_backward: saved buffer needs %zu bytes, got %zu", sv.total,
                    saved ? saved_bytes : (size_t)0);
    const BwdWs w = bwd_layout(*ctx, B, S);
    if (!ws || ws_bytes < w.total || !aligned16(ws))
        return fail(KVP_E_WORKSPACE, "kvp_backward: workspace needs %zu bytes (16-byte aligned), got %zu",
                    w.total, ws ? ws_bytes : (size_t)0);
    int rc;
    if ((rc = check_layers(ctx, 0, L))) return rc;
    for (int l = 0; l < L; ++l)
        if (!ctx->layers[l].grads)
            return fail(KVP_E_STATE, "kvp_backward: gradient buffers of layer %d were never set", l);

    hipStream_t st = (hipStream_t)stream;
    if (!ctx->bf16())
        return backward_f32(ctx, (const float*)x, (const float*)dy, (float*)dx, B, S, sv, (const char*)saved, w,
                            (char*)ws, st);
    char* base = (char*)ws;
    const char* sb = (const char*)saved;
    auto bp = [&](size_t off) { return (uint16_t*)(base + off); };
    uint16_t *gb = bp(w.gb), *dO = bp(w.dO), *dqkv = bp(w.dqkv), *wot = bp(w.wot), *wst = bp(w.wst);
    float* dsum = (float*)(base + w.dsum);
    float* acc = (float*)(base + w.acc);
    float* part = (float*)(base + w.part);
    const float2* rope = (const float2*)(base + w.rope);
    auto aux = [&](auto&& f) { return timed(ctx, KVP_K_BWD_AUX, st, f); };
    auto gemm = [&](auto&& f) { return timed(ctx, KVP_K_BWD_GEMM, st, f); };

    if ((rc = aux([&] {
             return check_hip(kvp::rope_table((float2*)rope, S, 128, ctx->d.rope_base, st), "RoPE table");
         })))
        return rc;
    if ((rc = aux([&] { return check_hip(kvp::f32_to_bf16((const float*)dy, gb, (size_t)M * h, st), "cast dY"); })))
        return rc;

    std::vector<char> acc_written(L, 0);
    for (int l = L - 1; l >= 0; --l) {
        const int p = ctx->tau[l];
        const bool producer = p == l;
        const int np = producer ? nq + 2 * nkv : nq;
        const Layer& Ly = ctx->layers[l];
        const Layer& Pl = ctx->layers[p];
        const char* lay = sb + (size_t)l * sv.stride;
        const uint16_t* Ql = (const uint16_t*)(lay + sv.q);
        const uint16_t* Ol = (const uint16_t*)(lay + sv.o);
        const float* lse = (const float*)(lay + sv.lse);
        const uint16_t* Xl = l == 0 ? (const uint16_t*)x : (const uint16_t*)(lay + sv.x);

        // dO = G W_O (on W_O^T), D = rowsum(dO * O), dW_O = G^T O (both K-major over the tokens).
        if ((rc = aux([&] {
                 return check_hip(kvp::transpose_bf16((const uint16_t*)Ly.wo, wot, h, nq, nq, h, st), "transpose W_O");
             })))
            return rc;
        if ((rc = gemm([&] { return check_hip(kvp::gemm_out_bf16(gb, wot, M, nq, h, dO, st), "dO GEMM"); })))
            return rc;
        if ((rc = aux([&] {
                 return check_hip(kvp::attn_bwd_prep_bf16(dO, Ol, dsum, B, S, Sp, ctx->d.a, st), "attention backward D");
             })))
            return rc;
        const bool nt = M % kTokGrain == 0;
        uint16_t* ta = bp(w.ta);
        uint16_t* tb = bp(w.tb);
        {
            const int s = kvp::gemm_out_splits(h, nq, M);
            if (nt) {
                // dW_O = G^T O on the token-major copies (row-major GEMM, split K); O^T was
                // saved by the forward's attention kernel when S % 8 == 0.
                const uint16_t* Ot = sv.has_ot ? (const uint16_t*)(lay + sv.ot) : tb;
                if ((rc = aux([&] {
                         int r2 = check_hip(kvp::transpose_bf16(gb, ta, M, h, h, M, st), "transpose G");
                         if (!r2 && !sv.has_ot) r2 = check_hip(kvp::transpose_bf16(Ol, tb, M, nq, nq, M, st), "transpose O");
                         return r2;
                     })))
                    return rc;
                if ((rc = gemm([&] { return check_hip(kvp::gemm_nt_out_splits(ta, Ot, h, nq, M, s, part, st), "dW_O GEMM"); })))
                    return rc;
            } else if ((rc = gemm([&] { return check_hip(kvp::gemm_kmajor_out_bf16(gb, h, Ol, nq, h, nq, M, s, part, st), "dW_O GEMM"); })))
                return rc;
            if ((rc = aux([&] {
                     return check_hip(kvp::reduce_planes(part, s, h, nq, Ly.dwo, h, nullptr, 0, nullptr, st), "dW_O sum");
                 })))
                return rc;
        }
        // dK, dV: a consumer adds into its producer's fp32 sums; the producer finishes them.
        {
            kvp::AttnBwdKv a{};
            a.q = Ql; a.dO = dO; a.lse = lse; a.dsum = dsum;
            a.kc = (const uint16_t*)Pl.kc; a.vc = (const uint16_t*)Pl.vc; a.rope = rope;
            const int slot = w.acc_slot[p];
            float* ak = slot >= 0 ? acc + (size_t)slot * 2 * w.acc_plane : nullptr;
            float* av = slot >= 0 ? ak + w.acc_plane : nullptr;
            if (!producer) {
                a.acc_in_k = acc_written[p] ? ak : nullptr;
                a.acc_in_v = acc_written[p] ? av : nullptr;
                a.acc_out_k = ak;
                a.acc_out_v = av;
                acc_written[p] = 1;
            } else {
                a.acc_in_k = acc_written[l] ? ak : nullptr;
                a.acc_in_v = acc_written[l] ? av : nullptr;
                a.out = dqkv;
                a.out_t = sv.has_ot ? ta : nullptr;   // [dQ|dK|dV]^T for dW_QKV (ta is free after dW_O)
                a.ldo = np;
                a.col_k = nq;
                a.col_v = nq + nkv;
            }
            a.B = B; a.S = S; a.Sp = Sp; a.a = ctx->d.a; a.g = ctx->d.g; a.cap = ctx->d.kv_capacity;
            if ((rc = timed(ctx, KVP_K_BWD_ATTN_KV, st, [&] {
                     return check_hip(kvp::flash_bwd_kv_bf16(a, st), "attention backward dK dV");
                 })))
                return rc;
        }
        {
            kvp::AttnBwdQ a{};
            a.q = Ql; a.dO = dO; a.lse = lse; a.dsum = dsum; a.kc = (const uint16_t*)Pl.kc;
            a.vc = (const uint16_t*)Pl.vc; a.rope = rope; a.out = dqkv; a.ldo = np;
            a.out_t = sv.has_ot ? ta : nullptr;
            a.B = B; a.S = S; a.Sp = Sp; a.a = ctx->d.a; a.g = ctx->d.g; a.cap = ctx->d.kv_capacity;
            if ((rc = timed(ctx, KVP_K_BWD_ATTN_Q, st, [&] {
                     return check_hip(kvp::flash_bwd_q_bf16(a, st), "attention backward dQ");
                 })))
                return rc;
        }
        // dW_Q (| dW_K | dW_V) = [dQ | dK | dV]^T X_l (both K-major over the tokens).
        {
            const int s = kvp::gemm_out_splits(np, h, M);
            if (nt) {
                if ((rc = aux([&] {
                         int r2 = sv.has_ot ? 0 : check_hip(kvp::transpose_bf16(dqkv, ta, M, np, np, M, st),
                                                            "transpose dQKV");
                         if (!r2) r2 = check_hip(kvp::transpose_bf16(Xl, tb, M, h, h, M, st), "transpose X");
                         return r2;
                     })))
                    return rc;
                if ((rc = gemm([&] { return check_hip(kvp::gemm_nt_out_splits(ta, tb, np, h, M, s, part, st), "dW_QKV GEMM"); })))
                    return rc;
            } else if ((rc = gemm([&] {
                            return check_hip(kvp::gemm_kmajor_out_bf16(dqkv, np, Xl, h, np, h, M, s, part, st),
                                             "dW_QKV GEMM");
                        })))
                return rc;
            if ((rc = aux([&] {
                     return check_hip(kvp::reduce_planes(part, s, np, h, Ly.dwq, nq, Ly.dwk, producer ? nkv : 0,
                                                         Ly.dwv, st),
                                      "dW_QKV sum");
                 })))
                return rc;
        }
        // dX_l = dX_{l+1} + [dQ | dK | dV] [W_Q; W_K; W_V] (on the stacked weights transposed
        // to [h][np]).
        if ((rc = aux([&] {
                 int r2 = check_hip(kvp::transpose_bf16((const uint16_t*)Ly.wq, wst, nq, h, h, np, st), "transpose W_Q");
                 if (!r2 && producer)
                     r2 = check_hip(kvp::transpose_bf16((const uint16_t*)Ly.wk, wst + nq, nkv, h, h, np, st),
                                    "transpose W_K");
                 if (!r2 && producer)
                     r2 = check_hip(kvp::transpose_bf16((const uint16_t*)Ly.wv, wst + nq + nkv, nkv, h, h, np, st),
                                    "transpose W_V");
                 return r2;
             })))
            return rc;
        {
            const void* gres = l == L - 1 ? dy : dx;
            if ((rc = gemm([&] {
                     return check_hip(kvp::gemm_resid_bf16(dqkv, wst, gres, true, gb, (float*)dx, M, h, np, st), "dX GEMM");
                 })))
                return rc;
        }
    }
    return ok();
}
