"""CPU oracle for the STaR-KV compression stage (arxiv 2606.01790).

TEST INFRASTRUCTURE ONLY.  This package is the plain, slow, fp64 reference
that the GPU path is checked against.  Only the test suite, the smoke check
of ``__graft_entry__`` and the ``cpu_baseline`` leg of ``bench.py`` may
import it.  The GPU library never calls it, and it shares no code with the
GPU library: no kernels, headers, helpers or constants.

Every function cites the passage of the paper it follows (section, equation
or algorithm).  Where the paper is silent or ambiguous, the reading taken is
stated in the function's docstring.

Every function is tied by at least one CPU test to a fact outside the
oracle (a closed form, an invariant, a special case that reduces to a
library routine, brute force on tiny inputs, or a hand-written table), and
the planted-mistake tests show that each such pin catches a plausible error.
"""

from .starkv_oracle import (  # noqa: F401
    Params,
    LayerState,
    window_attention_mass,
    avg_pool1d,
    group_scores,
    base_score,
    rank_bins,
    spatial_cells,
    plugin_mi,
    mi_prior,
    lambda_schedule,
    stability,
    temporal_discount,
    entropy_temperature,
    final_score,
    topb_select,
    gather_compact,
    visual_metadata,
    current_frame_span,
    compress_layer,
)
