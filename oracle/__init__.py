"""CPU oracle for the true-tail hybrid-state update.

TEST INFRASTRUCTURE ONLY. This package is the plain, slow, float64 statement of
what the maintained update computes. Only the test-suite, the smoke check and
the CPU-baseline leg of the benchmark may import it; the product path (the HIP
library and its Python binding) never does, and shares no code with it.

What it computes (paper: Section 4.1, Eq. 2 and Eq. 3; Section 4.2):
  * range verification against the live spans, and list-based compaction of the
    attention KV rows (Eq. 2), with the position cursor left untouched;
  * rotary position embedding of the replacement tokens at their true tail
    positions, rounded to bf16 as the cache stores them;
  * causal grouped-query softmax attention of the tail over surviving + new KV;
  * the gated delta-rule recurrence continuing from the carried state, token by
    token, plus a chunked form used only to check the invariant that both agree;
  * the short causal convolution of the recurrent layers continuing from its
    carried state (Section 4.1, Fig. 2: convolution state continues);
  * dense refill and fresh gapped prefill of the final context (Section 5.2);
  * the slot-preserving and tail-and-relocate placements of the replacement and the
    relocation of stored keys to other positions (Section 5.2, Section 6.3);
  * the attention diagnostics of Section 5.3: float32 reference-softmax probe
    distributions, memory-group masses, effective group count, boundary-window share
    and total variation distance.

Functions with no independent pin are marked "parity unpinned" in their
docstring; at present there are none.
"""
from .bf16 import bf16_to_f64, f64_to_bf16  # noqa: F401
from .compaction import RangeError, validate_ranges, live_positions, compact  # noqa: F401
from .rope import rope_frequencies, rope_rotate  # noqa: F401
from .attention import causal_gqa_attention  # noqa: F401
from .delta import gated_delta_tokens, gated_delta_chunked  # noqa: F401
from .short_conv import silu, short_conv_continue  # noqa: F401
from .placement import check_new_positions, relocate_keys  # noqa: F401
from .diagnostics import probe_distribution, group_masses, group_summary, tv_distance  # noqa: F401
from .update import (  # noqa: F401
    attention_layer_update,
    delta_layer_update,
    prefill_attention,
    refill_attention,
    gapped_refill_attention,
)
