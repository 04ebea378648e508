"""CPU oracle for the greedy speculative verification step.

TEST INFRASTRUCTURE ONLY.  Nothing in the product path may import, call or
link this package: it is used by the tests, by ``__graft_entry__.smoke()`` to
check one small GPU run, and by ``bench.py``'s CPU-baseline timing.  It shares
no code with the HIP implementation; the only thing both sides consume is the
seeded input generators in ``workloads``.

What it computes (all arithmetic in float64):

* ``model.forward_block`` - the target model's forward over a block of rows
  appended to a committed KV cache: Eq. 3 (the draft appended to the prefix
  and scored in one forward) over the decoder-only architecture the synthetic
  targets use (RMSNorm, rotary positions, grouped-query attention, SwiGLU).
  For bf16 models the values a bf16 pipeline stores are rounded to bf16
  (round-to-nearest-even) at the points listed in ``model``; every other
  quantity stays float64.
* ``accept`` - greedy decoding of each row (Sec. "Reuse", the decode function
  of Eq. 7 is greedy) and the longest accepted prefix of Eq. 7, plus the bonus
  token of the all-accepted case (Sec. "Speculative Decoding"); and the
  greedy walk of a draft tree.
* ``entropy`` - entropy-aware dynamic verification (Eq. 9-10) and fixed
  top-k verification of draft-model tokens (Sec. "Edit").
* ``match`` - the prefix/suffix matcher that resumes Reuse (Sec. "Reuse").
* ``session`` - prefill / verify / rollback / plain greedy decoding (Eq. 1)
  over an oracle-owned KV cache.
* ``sampling`` - stochastic speculative sampling (Eq. 4) with the draws
  given as inputs.
* ``driver`` - the Reuse / Generate phase machine of an edit session with an
  optional draft model.
"""

from .numerics import round_bf16
from .model import forward_block, chain_structure, tree_structure
from .accept import greedy_rows, accept_linear, accept_tree, top2_margin
from .entropy import accept_topk, entropy_threshold, topk_tokens
from .match import match_reuse
from .session import OracleSession
from .driver import OracleEditSession
from .sampling import accept_sample, sample_index, target_probs

__all__ = [
    "round_bf16", "forward_block", "chain_structure", "tree_structure",
    "greedy_rows", "accept_linear", "accept_tree", "top2_margin", "match_reuse",
    "accept_topk", "entropy_threshold", "topk_tokens",
    "OracleSession", "OracleEditSession", "accept_sample", "sample_index", "target_probs",
]
