"""Float64 CPU oracle for the per-device attention of ByteScale's HDP (arXiv 2502.21231).

TEST INFRASTRUCTURE ONLY.  Only the tests, the smoke check and the benchmark's
CPU-baseline leg may import anything here; the HIP library and its Python
binding never do, and share no code, header, table or helper with it.

  attention.py  softmax attention forward / backward / LSE merge (plain definitions)
  plan.py       reference tile classifier and work-list order
  xent.py       softmax cross-entropy: loss, LSE and gradient (plain definition)
  hdp.py        HDP planners: Eq. 3 offload ratio, Alg. 1, Alg. 2 (DP- and PP-Balance)
"""
from . import attention, plan  # noqa: F401
