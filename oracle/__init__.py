"""CPU oracle (test infrastructure only): plain fp64 statement of the FF step and scoring.

Only ``tests/``, ``__graft_entry__.smoke()`` and the benchmark's CPU-baseline
leg may import this package.
"""
from .ff_oracle import *  # noqa: F401,F403
from .ff_oracle import (HParams, Layer, StepResult, adam, bf16_round, chunk_bounds,  # noqa: F401
                        chunk_input, embed_labels, ff_loss, goodness, l2_normalise,
                        layer_forward, layer_grads, layer_step, score_labels, sigmoid,
                        softplus, train_pipelined, train_sequential)
