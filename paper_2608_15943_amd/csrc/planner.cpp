// Offline KV-Pipe planner: App. A.7 FLOPs model, the FIR metric
// (Eqs. flop_imbalance_main, favg), stage FLOPs under a mask (Eq. stage_flops_z),
// the Uniform and Symmetric Bipolar placements (Sec. 2.5), Algorithm 1 with the
// App. A.3 guardrail, and the mask -> producer map.
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

// The partition: non-decreasing, starts at stage 0, ends at P-1, no stage skipped.
bool valid_partition(int L, int P, const int32_t* stage_of_layer) {
    if (stage_of_layer[0] != 0 || stage_of_layer[L - 1] != P - 1) return false;
    for (int l = 1; l < L; ++l) {
        const int dlt = stage_of_layer[l] - stage_of_layer[l - 1];
        if (dlt < 0 || dlt > 1) return false;
    }
    return true;
}

// Admissible layers: caller mask, then the App. A.3 guardrail, never layer 0.
std::vector<uint8_t> admissible_layers(int L, const uint8_t* mask, double alpha) {
    std::vector<uint8_t> adm(L, 1);
    if (mask)
        for (int l = 0; l < L; ++l) adm[l] = mask[l] ? 1 : 0;
    if (alpha >= 0.0) {
        const double lo = std::ceil(alpha * static_cast<double>(L));
        for (int l = 0; l < L; ++l)
            if (!(static_cast<double>(l + 1) >= lo)) adm[l] = 0;
    }
    adm[0] = 0;
    return adm;
}

// Uniform: k targets spaced evenly from the last layer leftward over the layers of the
// last min(k, P) stages (rounded half up); a target that is not free moves to the nearest
// free admissible layer on its left, else on its right.
int place_uniform(int L, int P, const int32_t* stage_of_layer, int k,
                  const std::vector<uint8_t>& adm, std::vector<uint8_t>& z) {
    const int c = k < P ? k : P;
    const int hi = L - 1;
    int lo = hi;
    if (c > 0)
        for (int l = 0; l < L; ++l)
            if (stage_of_layer[l] >= P - c) { lo = l; break; }
    int n = 0;
    for (int j = 0; j < k; ++j) {
        const int64_t span = hi - lo;
        const int t = k == 1 ? hi
                             : hi - static_cast<int>((2 * j * span + (k - 1)) / (2 * static_cast<int64_t>(k - 1)));
        int pick = -1;
        for (int l = t; l >= 0; --l)
            if (adm[l] && !z[l]) { pick = l; break; }
        if (pick < 0)
            for (int l = t + 1; l < L; ++l)
                if (adm[l] && !z[l]) { pick = l; break; }
        if (pick < 0) break;
        z[pick] = 1;
        ++n;
    }
    return n;
}

// Symmetric Bipolar: anchors at the last layer of the last stage and of the middle stage
// (P - 1) / 2; conversions alternate between them, last stage first, each anchor taking the
// nearest free admissible layer at or left of its previous choice.  An exhausted anchor
// hands its turns to the other; with P = 1 there is one anchor.
int place_symmetric(int L, int P, const int32_t* stage_of_layer, int k,
                    const std::vector<uint8_t>& adm, std::vector<uint8_t>& z) {
    const int mid = (P - 1) / 2;
    int last_of_mid = 0;
    for (int l = 0; l < L; ++l)
        if (stage_of_layer[l] == mid) last_of_mid = l;
    int cur[2] = {L - 1, last_of_mid};
    const int na = mid == P - 1 ? 1 : 2;
    int n = 0, turn = 0;
    while (n < k) {
        bool placed = false;
        for (int att = 0; att < na && !placed; ++att) {
            const int a = (turn + att) % na;
            int l = cur[a];
            while (l >= 0 && !(adm[l] && !z[l])) --l;
            cur[a] = l;
            if (l >= 0) {
                z[l] = 1;
                cur[a] = l - 1;
                placed = true;
            }
        }
        if (!placed) break;
        ++n;
        turn = (turn + 1) % na;
    }
    return n;
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
    if (!valid_partition(L, P, in->stage_of_layer))
        return fail(KVP_E_INVALID_ARG, "kvp_plan_fir: stage_of_layer must run from 0 to P-1, "
                                       "non-decreasing, with no empty stage");
    const std::vector<uint8_t> adm = admissible_layers(L, in->admissible, in->alpha);
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

extern "C" int kvp_stage_flops(int L, int P, const int32_t* stage_of_layer, const double* f_full,
                               const double* f_share, const uint8_t* z, double f_lmhead,
                               double* stage_flops) {
    using namespace kvp;
    if (!stage_of_layer || !f_full || !f_share || !z || !stage_flops)
        return fail(KVP_E_INVALID_ARG, "kvp_stage_flops: NULL pointer");
    if (L < 1 || P < 1 || P > L) return fail(KVP_E_INVALID_ARG, "kvp_stage_flops: need 1 <= P <= L");
    for (int l = 0; l < L; ++l)
        if (stage_of_layer[l] < 0 || stage_of_layer[l] >= P)
            return fail(KVP_E_INVALID_ARG, "kvp_stage_flops: stage index out of range");
    kvp_plan_in in{};
    in.L = L;
    in.P = P;
    in.stage_of_layer = stage_of_layer;
    in.f_full = f_full;
    in.f_share = f_share;
    in.f_lmhead = f_lmhead;
    std::vector<uint8_t> zz(z, z + L);
    std::vector<double> F;
    stage_sums(in, zz, F);
    std::memcpy(stage_flops, F.data(), sizeof(double) * P);
    return ok();
}

extern "C" int kvp_place(int strategy, int L, int P, const int32_t* stage_of_layer, int k,
                         const uint8_t* admissible, double alpha, uint8_t* z, int32_t* n_placed,
                         int32_t* stop_reason) {
    using namespace kvp;
    if (!stage_of_layer || !z || !n_placed || !stop_reason)
        return fail(KVP_E_INVALID_ARG, "kvp_place: NULL pointer");
    if (L < 1 || P < 1 || P > L) return fail(KVP_E_INVALID_ARG, "kvp_place: need 1 <= P <= L");
    if (k < 0) return fail(KVP_E_INVALID_ARG, "kvp_place: k must be >= 0");
    if (!valid_partition(L, P, stage_of_layer))
        return fail(KVP_E_INVALID_ARG, "kvp_place: stage_of_layer must run from 0 to P-1, "
                                       "non-decreasing, with no empty stage");
    const std::vector<uint8_t> adm = admissible_layers(L, admissible, alpha);
    std::vector<uint8_t> zz(L, 0);
    int n;
    if (strategy == KVP_PLACE_UNIFORM)
        n = place_uniform(L, P, stage_of_layer, k, adm, zz);
    else if (strategy == KVP_PLACE_SYMMETRIC_BIPOLAR)
        n = place_symmetric(L, P, stage_of_layer, k, adm, zz);
    else
        return fail(KVP_E_INVALID_ARG, "kvp_place: unknown strategy %d", strategy);
    std::memcpy(z, zz.data(), L);
    *n_placed = n;
    *stop_reason = n == k ? KVP_STOP_BUDGET : KVP_STOP_NO_CONVERTIBLE;
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
