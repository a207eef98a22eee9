"""CPU oracle of the diversity-aware, layer-wise KV-cache eviction path.

TEST INFRASTRUCTURE ONLY.  This package is a plain, slow, obviously-correct restatement of what the
method computes ("Beyond Mean Attention: Diversity-Aware, Layer-Wise Scoring for KV Cache Eviction",
section 3).  Only the test-suite, the smoke check and the benchmark's CPU-baseline leg may import it;
the product path never does, and this package imports nothing from the product package.

Modules
  evict     -- window attention, mean/dispersion statistics, base score, normalisation, top-4B
               candidate restriction, greedy MMR admission and cache compaction (sections 3.1, 3.2)
  profiles  -- per-layer coefficients from the Global / Segments / Curve depth profiles (section 3.3)
  budgets   -- per-layer budgets that fall with depth at the total of a uniform budget (section 3.1)
  decode    -- attention of a generated token over the compacted cache (section 4.3)
"""
from . import budgets, decode, evict, profiles  # noqa: F401
