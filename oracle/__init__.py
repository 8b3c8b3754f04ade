"""CPU oracle for sampling-based mini-batch GNN training.

TEST INFRASTRUCTURE ONLY.  This package is a plain, slow, float64 statement of
what one training step computes, written from the paper's definitions
(section 2.1, eqs. (1)-(2); section 2.2, eq. (3) and the Neighbor / ShaDow
sampling definitions).  Only the tests, the smoke check and the benchmark's
CPU-baseline leg may import it; the GPU library never calls it, and the two
share no code.  Where the paper leaves a choice open, the reading taken is
stated in the function that makes it.

Modules:
  philox    -- Philox4x64-10 counter-based generator (Salmon et al., SC'11).
  sampling  -- uniform neighbour sampling without replacement (Floyd) and the
               first-occurrence relabelling of every block.
  shadow    -- ShaDow k-hop localised subgraphs (per root, induced edges).
  model     -- feature gather, SAGE-mean / GCN aggregation, dense update,
               softmax cross-entropy, backward, SGD.
  dlb       -- per-batch workload estimate (aggregations of the sampled
               computation graph) and the dynamic load balancer's
               assignment and ratio update (section 3).
  feature_cache -- set-associative LRU cache in GPU memory of a host-resident
               feature table (section 3, GPU Feature Caching).
  optim     -- Adam (Kingma and Ba), the optimiser of the paper's listings.
"""
from . import philox, sampling, shadow, model, dlb, feature_cache, optim  # noqa: F401
