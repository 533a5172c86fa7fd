"""CPU reference (oracle) for the speculative-decoding verify step.

TEST INFRASTRUCTURE ONLY. Only the test suite, the smoke check and the
benchmark's CPU-baseline leg may import or run anything in this package; the
product path never does.

Plain, slow, fp64 numpy code written from the paper (arXiv 2505.07680):
  * attention.verify_attention -- the verifier's forward attention over the
    cached context plus the drafted rows, under the logical validity mask
    (Section 2.2 step 2; Section 4.4, Eq. 8);
  * accept.accept_and_diverge -- probabilistic acceptance with residual
    resampling and the bonus token (Section 2.2 steps 3-4), per-position total
    variation distance (Eq. 5) and KL divergence;
  * rollback.rollback -- logical rollback of each sequence's cache to its
    accepted prefix and the common physical length (Section 4.4, Eq. 9);
  * chain -- glue of the three-level chain (which tokens and lengths the next
    level sees, and each level's rollback target);
  * kvcache -- appending a step's K/V rows at a per-sequence or shared
    cursor, compaction of the valid rows, Eq. 9's physical truncation
    (Section 4.4).

It shares no code with the HIP path: inputs arrive as plain numpy arrays
(bf16 as raw uint16 bit patterns, decoded here) and outputs are returned as
numpy arrays.
"""

from .accept import accept_and_diverge, decode_logits
from .attention import decode_bf16, verify_attention
from .rollback import rollback
from . import chain, kvcache

ST_GAMMA = 1
ST_KVLEN = 2
ST_TOKEN = 4
ST_UNIFORM = 8
ST_ROLLBACK_GROW = 16

__all__ = [
    "accept_and_diverge",
    "decode_logits",
    "decode_bf16",
    "verify_attention",
    "rollback",
    "chain",
    "kvcache",
    "ST_GAMMA",
    "ST_KVLEN",
    "ST_TOKEN",
    "ST_UNIFORM",
    "ST_ROLLBACK_GROW",
]
