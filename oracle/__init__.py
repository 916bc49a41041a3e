"""Float64 CPU oracle for RFF linear attention (Flexformer, arXiv 2606.27748).

TEST INFRASTRUCTURE ONLY: imported by tests/, the smoke check and the
benchmark's CPU-baseline leg, never by the product path.
"""
from .flex_oracle import *  # noqa: F401,F403
from .flex_oracle import (feature_map, feature_map_parts, linattn_fwd, linattn_fwd_rows,
                          linattn_bwd, attend_features, conditioning, nonstationary_pairs, decode_step,
                          norm_factor, softmax_weights, awd_loss, awd_grads, STATIONARY,
                          NONSTATIONARY)
