"""CPU oracle for the dual-pool paged-decode library.

THIS PACKAGE IS TEST INFRASTRUCTURE.  Only the test-suite, the smoke check in
``__graft_entry__`` and the ``cpu_baseline`` leg of ``bench.py`` may import it.
The product path (``paper_2604_08075_amd``) never imports, links or executes
anything here, and nothing here imports the product path: the two share no
code.  The only module both sides use is ``workloads``, which draws seeded
synthetic inputs and holds none of the method's arithmetic.

Every function is a plain, slow, obviously-correct restatement of what the
paper ("Dual-Pool Token-Budget Routing for Cost-Efficient and Reliable LLM
Serving") defines, computed in IEEE float64 unless the paper fixes another
precision:

* ``numerics``  - exact decode of bfloat16 and OCP FP8 E4M3 bit patterns.
* ``attention`` - paged decode attention (the per-step KV lookup the paper's
  cost model calls memory-bandwidth bound, Sec. 3 effect 4; 16-token
  PagedAttention blocks, Sec. 3 effect 3).
* ``prefill``   - causal chunked-prefill attention over the same paged cache
  (Sec. 1.2: each pool runs chunked prefill internally).
* ``append``    - the KV-cache append of each decode step, with OCP E4M3
  encoding for an FP8 cache (Sec. 4.4, Sec. 4.7).
* ``pool``      - per-sequence KV bytes and concurrent-sequence count
  (Sec. 1.1, Eq. 1 and Eq. 2).
* ``route``     - token-budget estimation, EMA calibration and pool dispatch
  (Sec. 2.1 Eq. 3-5, Sec. 2.2 Algorithm 1); the adaptive threshold that
  Sec. 7 proposes as future work (a reading of this library's own).
* ``cost``      - fleet sizing and the savings model (Sec. 3, boxed equation).

Parity status of each function is recorded in its module header.
"""
