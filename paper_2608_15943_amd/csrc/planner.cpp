// Offline KV-Pipe planner: App. A.7 FLOPs model, the FIR metric
// (Eqs. flop_imbalance_main, favg), stage FLOPs under a mask (Eq. stage_flops_z),
// Algorithm 1 with the App. A.3 guardrail, and the mask -> producer map.
//
// Host code only.  Built with -ffp-contract=off and without fast-math so that
// every double operation rounds exactly as written: the mask must not depend
// on the compiler.
#include <cmath>
#include <cstdint>
#include <cstring>
#include <vector>

#include "kvpipe.h"
#include "status.h"

namespace {

// Eq. (stage_flops_z): stage sums left to right, the LM head added last.
void stage_sums(const kvp_plan_in& in, const std::vector<uint8_t>& z, std::vector<double>& F) {
    F.assign(in.P, 0.0);
    for (int l = 0; l < in.L; ++l) {
        const int i = in.stage_of_layer[l];
        F[i] = F[i] + (z[l] ? in.f_share[l] : in.f_full[l]);
    }
    F[in.P - 1] = F[in.P - 1] + in.f_lmhead;
}

double mean_of(const std::vector<double>& F) {
    double tot = 0.0;
    for (double v : F) tot = tot + v;
    return tot / static_cast<double>(F.size());
}

double max_of(const std::vector<double>& F) {
    double m = F[0];
    for (double v : F)
        if (v > m) m = v;
    return m;
}

}  // namespace

extern "C" int kvp_layer_flops(const kvp_shape* s, int phase, double* f_full, double* f_share) {
    using namespace kvp;
    if (!s || !f_full || !f_share) return fail(KVP_E_INVALID_ARG, "kvp_layer_flops: NULL pointer");
    if (s->b < 1 || s->s < 1 || s->h < 1 || s->a < 1 || s->g < 1 || s->ffn < 0)
        return fail(KVP_E_INVALID_ARG, "kvp_layer_flops: sizes must be >= 1 (ffn >= 0)");
    if (s->h % s->a || s->a % s->g)
        return fail(KVP_E_INVALID_ARG, "kvp_layer_flops: need a | h and g | a");
    const int64_t d = s->h / s->a, kv_w = s->g * d;
    int64_t tok, attn;
    if (phase == KVP_PHASE_PREFILL) {
        tok = s->b * s->s;
        // Eqs. (qk), (av): 2 b a s^2 d each; causal keeps half of the pairs.
        const int64_t sc = 2 * s->b * s->a * s->s * s->s * d;
        attn = s->causal ? sc : 2 * sc;
    } else if (phase == KVP_PHASE_DECODE) {
        tok = s->b;
        attn = 2 * (2 * s->b * s->a * s->s * d);
    } else {
        return fail(KVP_E_INVALID_ARG, "kvp_layer_flops: unknown phase");
    }
    const int64_t q = 2 * tok * s->h * s->h;          // Eq. (mm_flops) for X W_Q
    const int64_t kv = 2 * (2 * tok * s->h * kv_w);   // X W_K and X W_V, width h / r
    const int64_t out = 2 * tok * s->h * s->h;        // Eq. (wo)
    const int64_t mlp = s->ffn ? 3 * (2 * tok * s->h * s->ffn) : 0;
    const int64_t full = q + kv + attn + out + mlp;
    *f_full = static_cast<double>(full);
    *f_share = static_cast<double>(full - kv);
    return ok();
}

extern "C" int kvp_fir(int P, const double* stage_flops, double* fir) {
    using namespace kvp;
    if (P < 1 || !stage_flops || !fir) return fail(KVP_E_INVALID_ARG, "kvp_fir: bad arguments");
    std::vector<double> F(stage_flops, stage_flops + P);
    const double avg = mean_of(F);
    if (!(avg > 0.0)) return fail(KVP_E_INVALID_ARG, "kvp_fir: mean stage FLOPs must be > 0");
    *fir = max_of(F) / avg;
    return ok();
}

extern "C" int kvp_plan_fir(const kvp_plan_in* in, kvp_plan_out* out) {
    using namespace kvp;
    if (!in || !out || !in->stage_of_layer || !in->f_full || !in->f_share || !out->z ||
        !out->stage_flops)
        return fail(KVP_E_INVALID_ARG, "kvp_plan_fir: NULL pointer");
    const int L = in->L, P = in->P;
    if (L < 1 || P < 1 || P > L) return fail(KVP_E_INVALID_ARG, "kvp_plan_fir: need 1 <= P <= L");
    if (!(in->eps > 0.0)) return fail(KVP_E_INVALID_ARG, "kvp_plan_fir: eps must be > 0");
    if (!(in->f_lmhead >= 0.0)) return fail(KVP_E_INVALID_ARG, "kvp_plan_fir: f_lmhead must be >= 0");
    // The partition: non-decreasing, starts at stage 0, ends at P-1, no stage skipped.
    if (in->stage_of_layer[0] != 0 || in->stage_of_layer[L - 1] != P - 1)
        return fail(KVP_E_INVALID_ARG, "kvp_plan_fir: stages must run from 0 to P-1");
    for (int l = 1; l < L; ++l) {
        const int dlt = in->stage_of_layer[l] - in->stage_of_layer[l - 1];
        if (dlt < 0 || dlt > 1)
            return fail(KVP_E_INVALID_ARG, "kvp_plan_fir: stage_of_layer must be non-decreasing "
                                           "with no empty stage");
    }
    // Admissible layers: caller mask, then the guardrail, never layer 0.
    std::vector<uint8_t> adm(L, 1);
    if (in->admissible)
        for (int l = 0; l < L; ++l) adm[l] = in->admissible[l] ? 1 : 0;
    if (in->alpha >= 0.0) {
        const double lo = std::ceil(in->alpha * static_cast<double>(L));
        for (int l = 0; l < L; ++l)
            if (!(static_cast<double>(l + 1) >= lo)) adm[l] = 0;
    }
    adm[0] = 0;
    for (int l = 0; l < L; ++l)
        if (adm[l] && !(in->f_full[l] - in->f_share[l] > 0.0))
            return fail(KVP_E_INVALID_ARG, "kvp_plan_fir: F(0) - F(1) must be > 0 for every "
                                           "admissible layer");

    const int m = in->m <= 0 ? L : in->m;
    std::vector<uint8_t> z(L, 0);
    std::vector<double> F;
    stage_sums(*in, z, F);
    double avg = mean_of(F);
    if (!(avg > 0.0)) return fail(KVP_E_INVALID_ARG, "kvp_plan_fir: mean stage FLOPs must be > 0");
    double cur = max_of(F) / avg;
    int t = 0, stop;
    const int tail = P - 1;
    for (;;) {
        if (!(cur > 1.0 + in->eps)) { stop = KVP_STOP_FIR_MET; break; }
        if (!(t < m)) { stop = KVP_STOP_BUDGET; break; }
        int target = tail;                               // every pass starts at the tail
        if (F[target] <= (1.0 + in->eps) * avg) {        // tail balanced: take the bottleneck
            double best = F[0];
            target = 0;
            for (int j = 1; j < P; ++j)
                if (F[j] >= best) { best = F[j]; target = j; }   // ties -> later stage
        }
        int chosen = -1;
        for (int l = L - 1; l >= 0; --l)
            if (in->stage_of_layer[l] == target && !z[l] && adm[l]) { chosen = l; break; }
        if (chosen < 0) { stop = KVP_STOP_NO_CONVERTIBLE; break; }
        z[chosen] = 1;
        F[target] = F[target] - (in->f_full[chosen] - in->f_share[chosen]);
        ++t;
        avg = mean_of(F);
        cur = max_of(F) / avg;
    }
    std::memcpy(out->z, z.data(), L);
    std::memcpy(out->stage_flops, F.data(), sizeof(double) * P);
    out->fir = cur;
    out->n_converted = t;
    out->stop_reason = stop;
    return ok();
}

extern "C" int kvp_map_from_mask(int L, const uint8_t* z, int32_t* tau) {
    using namespace kvp;
    if (L < 1 || !z || !tau) return fail(KVP_E_INVALID_ARG, "kvp_map_from_mask: bad arguments");
    if (z[0]) return fail(KVP_E_BAD_MAP, "kvp_map_from_mask: layer 0 has no prior layer to share");
    int32_t last = 0;
    for (int l = 0; l < L; ++l) {
        if (z[l]) {
            tau[l] = last;
        } else {
            tau[l] = l;
            last = l;
        }
    }
    return ok();
}

extern "C" int kvp_canonicalize_map(int L, const int32_t* in, int32_t* out) {
    using namespace kvp;
    if (L < 1 || !in || !out) return fail(KVP_E_INVALID_ARG, "kvp_canonicalize_map: bad arguments");
    std::vector<int32_t> res(L);
    for (int l = 0; l < L; ++l) {
        const int32_t t = in[l];
        if (t < 0 || t > l)
            return fail(KVP_E_BAD_MAP, "kvp_canonicalize_map: tau(%d) = %d is not a prior layer", l, t);
        res[l] = (t == l) ? t : res[t];
    }
    std::memcpy(out, res.data(), sizeof(int32_t) * L);
    return ok();
}
