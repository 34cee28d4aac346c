"""CPU ORACLE -- test infrastructure only.

Only ``tests/``, ``__graft_entry__.smoke()`` and ``bench.py``'s CPU-baseline
leg may import this package.  It shares no code with the GPU path (the seeded
input generators in ``lede_inputs`` are the one common dependency) and it is
never used as a fallback for it.

``lede_oracle.c`` holds the decoder arithmetic in fp64; ``model.py`` holds the
decoding loop: greedy autoregressive decoding (the plain definition the
self-speculative loop must reproduce), the draft / verify / accept / commit
step, the page allocator, the Q-network, the reward and the run metrics;
``dqn.py`` holds the offline optimisation of the exit policy's Q-network.
"""
from .build import build, library_path  # noqa: F401
from .model import (OracleDecoder, Pager, StepRecord, accept_length, greedy_ar,  # noqa: F401
                    metrics, reward, ssd_generate, Tolerance)
