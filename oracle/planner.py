"""Oracle for the offline KV-Pipe planner (test infrastructure only).

Follows Sec. 2.3-2.7 (FIR, stage FLOPs under z, the Uniform and Symmetric
Bipolar placements, Algorithm 1), App. A.3 (the safe-layer guardrail) and
App. A.7 (attention FLOPs under MHA/GQA).

Floating-point order is fixed so that a compiled planner doing the same IEEE
double operations in the same order reaches the same mask bit for bit:
stage sums run left to right over the layers of a stage, then the LM head is
added to the last stage; avg = (sum of stages, left to right) / P;
FIR = max / avg; a conversion subtracts (F(0) - F(1)) from the stage.
"""
from __future__ import annotations

import math
from dataclasses import dataclass
from typing import List, Optional, Sequence

STOP_FIR_MET = 0
STOP_BUDGET = 1
STOP_NO_CONVERTIBLE = 2


# ---------------------------------------------------------------------------
# App. A.7: FLOPs of one attention layer.
# ---------------------------------------------------------------------------

def mm_flops(m: int, k: int, n: int) -> int:
    """Eq. (mm_flops): a product of (m x k) by (k x n) costs 2mkn FLOPs."""
    return 2 * m * k * n


def layer_flops_prefill(b: int, s: int, h: int, a: int, g: int, ffn: int = 0,
                        causal: bool = True):
    """(F(0), F(1)) of one layer over a b x s prefill, in integer FLOPs.

    Projections follow Eq. (qkv_gqa) with the K/V width h/r = g*d, d = h/a;
    scores and context follow Eqs. (qk), (av) with s^2 replaced by s^2/2 when
    ``causal`` (the reading under which Table 1's stage FLOPs come out);
    the output projection follows Eq. (wo); an optional SwiGLU MLP adds
    three h x ffn products.  A shared layer drops the K and V projections
    (Eq. gqa_skv_flop_saving).
    """
    if h % a or a % g:
        raise ValueError("need a | h and g | a")
    tokens = b * s
    d = h // a
    kv_width = g * d
    q = mm_flops(tokens, h, h)
    kv = 2 * mm_flops(tokens, h, kv_width)
    score = 2 * b * a * s * s * d          # 2*b*s^2*h, Eq. (qk)
    ctx = 2 * b * a * s * s * d            # Eq. (av)
    attn = (score + ctx) // 2 if causal else score + ctx
    out = mm_flops(tokens, h, h)
    mlp = 3 * mm_flops(tokens, h, ffn) if ffn else 0
    full = q + kv + attn + out + mlp
    return full, full - kv


def layer_flops_decode(b: int, ctx: int, h: int, a: int, g: int, ffn: int = 0):
    """(F(0), F(1)) of one layer for one new token per sequence over ``ctx`` cached keys.

    Per token this is Eq. (attn_gqa_token) with the score/context terms for
    one query against ctx keys: 4h^2 + 4h^2/r + 4*ctx*h.
    """
    if h % a or a % g:
        raise ValueError("need a | h and g | a")
    d = h // a
    kv_width = g * d
    q = mm_flops(b, h, h)
    kv = 2 * mm_flops(b, h, kv_width)
    attn = 2 * (2 * b * a * ctx * d)
    out = mm_flops(b, h, h)
    mlp = 3 * mm_flops(b, h, ffn) if ffn else 0
    full = q + kv + attn + out + mlp
    return full, full - kv


def per_token_attn_flops(h: int, s: int, r: int = 1) -> float:
    """Eqs. (attn_mha_token) / (attn_gqa_token): 4h^2 + 4h^2/r + 4sh (r=1 gives 8h^2 + 4sh)."""
    return 4 * h * h + 4 * h * h / r + 4 * s * h


def gqa_sharing_savings(h: int, r: int, b_elem: int):
    """Eqs. (gqa_skv_flop_saving), (gqa_skv_cache_saving): (4h^2/r, 2(h/r) b_elem) per token."""
    return 4 * h * h / r, 2 * (h / r) * b_elem


# ---------------------------------------------------------------------------
# Sec. 2.3, Eqs. (4)-(6).
# ---------------------------------------------------------------------------

def stage_flops(stage_of_layer: Sequence[int], P: int, f_full: Sequence[float],
                f_share: Sequence[float], z: Sequence[int], f_lmhead: float) -> List[float]:
    """Eq. (stage_flops_z): per-stage sum of F_l(z_l), plus the LM head on the last stage."""
    F = [0.0] * P
    for l, i in enumerate(stage_of_layer):
        F[i] = F[i] + (float(f_share[l]) if z[l] else float(f_full[l]))
    F[P - 1] = F[P - 1] + float(f_lmhead)
    return F


def f_avg(F: Sequence[float]) -> float:
    """Eq. (favg): the mean stage FLOPs (LM head already inside the last stage)."""
    tot = 0.0
    for v in F:
        tot = tot + v
    return tot / len(F)


def fir(F: Sequence[float]) -> float:
    """Eq. (flop_imbalance_main): max stage FLOPs over the average."""
    return max(F) / f_avg(F)


# ---------------------------------------------------------------------------
# Algorithm 1 with the App. A.3 guardrail.
# ---------------------------------------------------------------------------

@dataclass
class PlanResult:
    z: List[int]
    stage_flops: List[float]
    fir: float
    n_converted: int
    stop_reason: int
    fir_trace: List[float]


def guardrail_admissible(L: int, alpha: float) -> List[bool]:
    """App. A.3: C_alpha = {l in 1..L : l >= ceil(alpha L)} (1-indexed), as a 0-indexed mask."""
    lo = math.ceil(alpha * L)
    return [(l + 1) >= lo for l in range(L)]


def plan_fir(stage_of_layer: Sequence[int], P: int, f_full: Sequence[float],
             f_share: Sequence[float], f_lmhead: float, eps: float, m: int = 0,
             admissible: Optional[Sequence[bool]] = None, alpha: float = -1.0) -> PlanResult:
    """Algorithm 1 (Architecture-Balanced), in the paper's order.

    Readings where the paper is silent: layer 0 has no prior layer and is
    never converted; among stages tied at the maximum the highest index is
    taken; ``m <= 0`` means m = L; ``admissible`` (optional) and the
    guardrail C_alpha (alpha >= 0) restrict the layer choice.  The state
    after the last iteration is returned as is.
    """
    L = len(stage_of_layer)
    if m <= 0:
        m = L
    ok = [True] * L if admissible is None else [bool(x) for x in admissible]
    if alpha >= 0.0:
        ca = guardrail_admissible(L, alpha)
        ok = [x and y for x, y in zip(ok, ca)]
    ok[0] = False

    z = [0] * L
    # Stage FLOPs with no layer converted yet, and their FIR (Eqs. 4-5).
    F = stage_flops(stage_of_layer, P, f_full, f_share, z, f_lmhead)
    avg = f_avg(F)
    cur = max(F) / avg
    trace = [cur]
    t = 0
    tail = P - 1
    stop = STOP_FIR_MET
    while True:
        if not cur > 1.0 + eps:
            stop = STOP_FIR_MET
            break
        if not t < m:
            stop = STOP_BUDGET
            break
        target = tail                                   # every pass starts at the tail
        if F[target] <= (1.0 + eps) * avg:              # tail is close enough: take the argmax
            best = F[0]
            target = 0
            for j in range(1, P):
                if F[j] >= best:                        # ties go to the later stage
                    best = F[j]
                    target = j
        chosen = -1
        for l in range(L - 1, -1, -1):                  # last unconverted layer of the stage
            if stage_of_layer[l] == target and z[l] == 0 and ok[l]:
                chosen = l
                break
        if chosen < 0:
            stop = STOP_NO_CONVERTIBLE
            break
        z[chosen] = 1
        F[target] = F[target] - (float(f_full[chosen]) - float(f_share[chosen]))
        t += 1
        avg = f_avg(F)
        cur = max(F) / avg
        trace.append(cur)
    return PlanResult(z=z, stage_flops=F, fir=cur, n_converted=t, stop_reason=stop,
                      fir_trace=trace)


# ---------------------------------------------------------------------------
# Sec. 2.5: the Uniform and Symmetric Bipolar placement archetypes.  Neither
# looks at FLOPs: each places a fixed number k of conversions by position.
# ---------------------------------------------------------------------------

def _placement_admissible(stage_of_layer: Sequence[int], P: int,
                          admissible: Optional[Sequence[bool]], alpha: float) -> List[bool]:
    """Caller mask, then the App. A.3 guardrail; layer 0 (no prior layer) never."""
    L = len(stage_of_layer)
    if L < 1 or P < 1 or P > L:
        raise ValueError("need 1 <= P <= L")
    if stage_of_layer[0] != 0 or stage_of_layer[-1] != P - 1 or any(
            not 0 <= b - a <= 1 for a, b in zip(stage_of_layer, stage_of_layer[1:])):
        raise ValueError("stages must be contiguous, 0..P-1, none empty")
    ok = [True] * L if admissible is None else [bool(x) for x in admissible]
    if alpha >= 0.0:
        ok = [x and y for x, y in zip(ok, guardrail_admissible(L, alpha))]
    ok[0] = False
    return ok


def place_uniform(stage_of_layer: Sequence[int], P: int, k: int,
                  admissible: Optional[Sequence[bool]] = None, alpha: float = -1.0):
    """Uniform split: k conversions spread evenly, anchored at the last layer.

    Reading (the paper gives the rule in words and one example): the k
    conversions are spaced evenly over the layers of the last min(k, P)
    stages, the first at the last layer, moving left:
    target_j = hi - round(j (hi - lo) / (k - 1)), j = 0 .. k-1, with hi the
    last layer, lo the first layer of stage P - min(k, P) and halves rounded
    up.  With equal stages and k <= P this is one conversion in each of the
    last k stages.  A target that is not admissible or already taken moves
    to the nearest free admissible layer on its left, else on its right.
    Returns (z, n placed, stop reason).
    """
    ok = _placement_admissible(stage_of_layer, P, admissible, alpha)
    if k < 0:
        raise ValueError("k must be >= 0")
    L = len(stage_of_layer)
    z = [0] * L
    c = min(k, P)
    hi = L - 1
    lo = next(l for l in range(L) if stage_of_layer[l] >= P - c) if c else hi
    n = 0
    for j in range(k):
        t = hi if k == 1 else hi - (2 * j * (hi - lo) + (k - 1)) // (2 * (k - 1))
        free = [l for l in range(L) if ok[l] and not z[l]]
        left = [l for l in free if l <= t]
        right = [l for l in free if l > t]
        if left:
            z[max(left)] = 1
        elif right:
            z[min(right)] = 1
        else:
            return z, n, STOP_NO_CONVERTIBLE
        n += 1
    return z, n, STOP_BUDGET


def place_symmetric_bipolar(stage_of_layer: Sequence[int], P: int, k: int,
                            admissible: Optional[Sequence[bool]] = None, alpha: float = -1.0):
    """Symmetric Bipolar split: two anchors, each moving left.

    Reading: the anchors are the last layer of the last stage and the last
    layer of the middle stage floor((P - 1) / 2) (stage 3 of 8, as in
    App. A.1, Table A2).  Conversions alternate between the anchors,
    the last stage first; each anchor converts the nearest free admissible
    layer at or left of its previous choice.  An anchor with nothing left
    hands its turns to the other; with P = 1 the two anchors coincide.
    Returns (z, n placed, stop reason).
    """
    ok = _placement_admissible(stage_of_layer, P, admissible, alpha)
    if k < 0:
        raise ValueError("k must be >= 0")
    L = len(stage_of_layer)
    mid = (P - 1) // 2
    last_of_mid = max(l for l in range(L) if stage_of_layer[l] == mid)
    cursors = [L - 1] if mid == P - 1 else [L - 1, last_of_mid]
    z = [0] * L
    n = 0
    turn = 0
    while n < k:
        placed = False
        for attempt in range(len(cursors)):
            a = (turn + attempt) % len(cursors)
            l = cursors[a]
            while l >= 0 and not (ok[l] and not z[l]):
                l -= 1
            cursors[a] = l
            if l >= 0:
                z[l] = 1
                cursors[a] = l - 1
                placed = True
                break
        if not placed:
            return z, n, STOP_NO_CONVERTIBLE
        n += 1
        turn = (turn + 1) % len(cursors)
    return z, n, STOP_BUDGET


def strategy_table(stage_of_layer: Sequence[int], P: int, f_full: Sequence[float],
                   f_share: Sequence[float], f_lmhead: float, k: int, eps: float):
    """The comparison of Sec. 2.7 (Table 2): Baseline, Uniform, Symmetric
    Bipolar and Architecture-Balanced (Algorithm 1 with budget m = k), each
    as (name, z, stage FLOPs, FIR)."""
    rows = []
    z0 = [0] * len(stage_of_layer)
    for name, z in (("baseline", z0),
                    ("uniform", place_uniform(stage_of_layer, P, k)[0]),
                    ("symmetric_bipolar", place_symmetric_bipolar(stage_of_layer, P, k)[0])):
        F = stage_flops(stage_of_layer, P, f_full, f_share, z, f_lmhead)
        rows.append((name, z, F, fir(F)))
    res = plan_fir(stage_of_layer, P, f_full, f_share, f_lmhead, eps, m=k)
    rows.append(("arch_balanced", res.z, res.stage_flops, res.fir))
    return rows


# ---------------------------------------------------------------------------
# Mask -> producer map (Eq. kv_share with the nearest-prior-producer reading).
# ---------------------------------------------------------------------------

def map_from_mask(z: Sequence[int]) -> List[int]:
    """tau(l) = l for a full-attention layer, else the nearest earlier layer with z = 0."""
    if len(z) == 0:
        return []
    if z[0]:
        raise ValueError("layer 0 cannot share: it has no prior layer")
    tau = []
    last = 0
    for l, zl in enumerate(z):
        if zl:
            tau.append(last)
        else:
            tau.append(l)
            last = l
    return tau


def canonicalize_map(tau: Sequence[int]) -> List[int]:
    """Check tau(l) <= l, tau(0) = 0, and resolve chains to their root producer.

    Eq. (kv_share) substitutes K_tau(l) for K_l; if tau(l) itself shares, its
    K is K_tau(tau(l)), so following the chain reaches the layer that
    actually projects K and V.
    """
    L = len(tau)
    out = []
    for l in range(L):
        t = int(tau[l])
        if t < 0 or t > l:
            raise ValueError(f"tau({l}) = {t} is not a prior layer")
        out.append(t if t == l else out[t])
    return out
