"""CPU oracle for the per-chunk stream step (score -> select -> compact -> attend).

TEST INFRASTRUCTURE ONLY.  Only the tests, ``__graft_entry__.smoke()`` and the ``cpu_baseline``
leg of ``bench.py`` may import this package.  The product path (the HIP library and its Python
binding) never imports, calls or links it, and this package imports nothing from the product.
The two share only the seeded input generator (``streamgen``), which holds none of the method's
arithmetic.

Plain and slow on purpose: exact int64 integers for scoring, selection and compaction, float64
for attention, loops written in the order of the paper's description.  Every function cites the
passage of the paper (OmniTide: co-designing algorithms and systems for on-device omni-LLM
streaming) it follows; where the paper is silent the reading taken is stated in the docstring.

Pins (tests marked ``not gpu``) tie each function to something other than itself: closed forms,
brute force on tiny inputs, the unit-FIFO special case of selection, the paper's printed
physical-span figures, dense causal attention at full budget, and torch's scaled-dot-product
attention in float64.  No function here is "parity unpinned".
"""
from .errors import OracleError, TagError, BudgetError, CapacityError  # noqa: F401
from .omnipick import (quantize_magnitude, weights_q88, score_units,  # noqa: F401
                       select_units, check_unit_structure)
from .omnipage import compact_kv, page_span, n_pages  # noqa: F401
from .attention import chunk_attention, to_f64  # noqa: F401
from .pipeline import stream_step  # noqa: F401
from .rope import rope_thetas, pair_dims, shift_keys  # noqa: F401
from .spans import plan_spans  # noqa: F401
from .native import (evict_logical, place_chunk, span_of, active_pages,  # noqa: F401
                     packed_span, plan_suffix, pack_suffix, span_attention)
