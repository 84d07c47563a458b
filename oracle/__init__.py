"""CPU oracle for LoPA's per-iteration branch-verification step (arXiv 2512.16229).

TEST INFRASTRUCTURE, NOT PRODUCT CODE. Only tests/, __graft_entry__.smoke() and
bench.py's cpu_baseline leg may import it. It shares no code with the HIP path
(paper_2512_16229_amd/) and imports nothing from it.

Plain, slow, obviously correct numpy, float64 throughout:
  * model.py  - the dLLM forward of one active block for a batch of branches
                against a shared-prefix KV cache (Sec. 3.3 attention pattern,
                Sec. 3.4 static cache), logits -> Conf / candidate tokens (Sec. 3.1).
  * lopa.py   - Eq. 1 threshold fill, anchor + lookahead branches (Alg. 1 steps
                1-2), Eq. 2 branch confidence and selection (Alg. 1 step 3),
                logit reuse (Sec. 3.2) and the decode loop.
  * fp8.py    - E4M3 rounding and per-row / per-channel scaling for the FP8 MLP
                mode of the forward.

Precision modes of the forward (see model.py): "pure" (float64 from the
given weights), "faithful" (float64 arithmetic with bf16 round-to-nearest-even
at the points where a bf16 implementation stores values), "fp8_mlp" (faithful
with the MLP projections in W8A8 E4M3) and "fp8" (also QKV and the LM head). Integer decisions are
compared against "faithful", confidences against "pure".

Parity status per function: every function here is pinned by tests under
tests/ (closed forms, library special cases, invariants, brute force). None is
"parity unpinned" except the published TPF / accuracy / throughput figures,
which need trained weights and datasets that are not available.
"""
from .model import OracleModel, KVCache, bf16_round  # noqa: F401
from . import lopa  # noqa: F401
from . import fp8  # noqa: F401
