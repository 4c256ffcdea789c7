"""CPU oracle for the mixed step and its scheduler (test infrastructure only).

This package is a plain, slow, float64 NumPy restatement of what one step of the
paper's heterogeneous batch computes.  It exists to check the GPU library and is
used only by the test suite, by the entry point's smoke check and by the CPU
baseline leg of the benchmark; the product path never imports it.

* ``oracle.model`` -- the single-request definition: an unchunked, uncached
  causal forward pass (Section 3.1: attention and feed-forward layers identical
  for every request type), single-pass pooling heads (Section 3.3) and the
  next-token logits of a generation request recomputed from its whole prefix.
* ``oracle.step`` -- the same arithmetic under the step's contract: a
  type-sorted batch of embedding chunks, generation prefill chunks and decode
  tokens (Section 3.2) that reads and appends a paged KV cache, updates the
  per-request pooling state by Eq. (1)-(2) and the positional heads, finishes
  embeddings after a request's final chunk, and emits next-token logits for
  the last row of a prompt's final chunk and for every decode token.
* ``oracle.sched`` -- intra-batch scheduling (Algorithm 2 with ScheduleRunning
  and ScheduleOne): which items of which requests one iteration's batch holds,
  under the token budget, the chunk cap and the cache capacity.

Where the paper leaves a detail open (the model family's normalisation, RoPE
variant, grouping of query heads, the L2 normalisation of finished embeddings,
the accumulator contract) the reading taken here is stated in each function.
Everything is float64; inputs are upcast on entry.  The oracle imports nothing
from the GPU package and shares no helper with it; only the seeded input
generators in ``workload`` feed both.
"""
from .model import (rmsnorm, rope_rotate, causal_gqa_attention, silu, forward_full,
                    pool_single_pass, l2_normalize, embed_single_pass, decode_full_recompute,
                    lm_logits, greedy_token)
from .step import OracleKV, StepError, step_oracle
from .sched import IBSOracle, SchedConfig, SchedError, Schedule

__all__ = ["rmsnorm", "rope_rotate", "causal_gqa_attention", "silu", "forward_full",
           "pool_single_pass", "l2_normalize", "embed_single_pass", "decode_full_recompute",
           "lm_logits", "greedy_token", "OracleKV", "StepError", "step_oracle", "IBSOracle",
           "SchedConfig", "SchedError", "Schedule"]
