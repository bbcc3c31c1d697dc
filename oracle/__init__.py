"""Oracle: a plain, slow, fp64 CPU statement of what the KV-shared attention
path and the FIR planner compute.

TEST INFRASTRUCTURE ONLY.  Only the tests, the smoke check and the
benchmark's CPU-baseline leg may import this package.  It shares no code with
the HIP library or its Python binding, and the library never calls it: a
missing HIP extension is an error on the product path, never a fallback here.

Contents
--------
planner   -- App. A.7 FLOPs model, the FIR metric (Eqs. 4-5), stage FLOPs
             under a conversion mask (Eq. 6), Algorithm 1 (tail-first
             architecture-balanced conversion) with the App. A.3 guardrail,
             and the mask -> producer-map reading.
attention -- Eq. (1)-(2) full attention, Eq. (3) cross-layer KV sharing, RoPE,
             the attention-only residual stack, and single-token decode.
backward  -- the gradients of that stack (attention, RoPE, projections and
             the residual), with a consumer's K/V gradient added to its
             producer's.

Every function is pinned by a test under ``tests/`` against values the paper
prints, closed forms, invariants, library routines or brute force; the few
results with no such pin are marked "parity unpinned" where they are defined.
"""
