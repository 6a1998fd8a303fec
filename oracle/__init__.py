"""Plain float64 CPU oracle for the CAST block-step hot path.

TEST INFRASTRUCTURE ONLY.  Nothing in the product path imports, calls or links
this package: only ``tests/``, ``__graft_entry__.smoke()`` and the
``cpu_baseline`` leg of ``bench.py`` may use it.  It shares no code, tables or
helpers with the HIP library; the two meet only through the seeded input
generators in ``gen/``.

Modules
-------
route  pooled chunk scores and TopK chunk selection   (Sec. 4.4, eq:pooled, eq:topk)
attn   dense softmax attention over routed chunks     (Sec. 4.4, App. B.4 complexity)
par    Phase-Aware Reconstruction                     (Sec. 4.3 eq:cross .. eq:fcpasm,
                                                       App. A.2, Sec. 4.1 eq:block)
coupled  reconstruction-coupled historical routing    (Sec. 4.4 eq:omission .. eq:topk,
                                                       App. B, Algorithm 1)
frame_select  control-aware frame selection         (Sec. 3.1 eq:sensitivity, Sec. 4.2
                                                       eq:debt, eq:score, App. A.1)
diagnostics   spectral diagnostics of reconstructions (App. C eq:oracles .. eq:phaseerror)

Every function computes in float64 on the values it is given (bf16-rounded or
fp32 inputs are widened first), written as the definition in the paper, with
no blocking or fusion beyond what the definition states.
"""
from . import route, attn, par, coupled, frame_select, diagnostics  # noqa: F401
