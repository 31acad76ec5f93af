"""Oracle: plain, slow, obviously correct CPU implementations (float64).

TEST INFRASTRUCTURE ONLY. Only ``tests/``, ``__graft_entry__.smoke()`` and the
``cpu_baseline`` leg of ``bench.py`` may import anything from this package. The
product path (the HIP library and its Python binding) never imports it, and it
imports nothing from the product path.

Modules:
  decode_attention -- softmax decode attention over contiguous/ragged and paged
                      KV caches, split-K partial attention and the log-sum-exp
                      merge (paper Sec. 2.2).
  cost_model       -- the paper's memory-bound decode latency model and the
                      summary-length bound it implies (paper Sec. 3.3).
"""
