"""CPU oracle for the multipath host<->GPU copy path -- TEST INFRASTRUCTURE ONLY.

This package is a plain, slow, obviously-correct statement of what the GPU path
must produce. Only ``tests/``, ``__graft_entry__.smoke()`` and ``bench.py``'s
``cpu_baseline`` leg may import it; the product path never does. It shares no
code with the HIP library and never loads it.

Every operation here is pure data movement, so the oracle is the plain definition
of each result (byte copy, block-table gather/scatter). See each module's header for
the passage of the paper it follows:

* ``copy``   -- single copy and tensor list (a logical copy must be indistinguishable
  from the native one).
* ``kv``     -- paged-KV fetch (host -> GPU) and offload (GPU -> host) via block
  tables, plus the validity rules for the tables.
* ``naive``  -- an independent byte-at-a-time restatement of ``kv`` from the flat
  index formula, for tiny shapes (used to pin ``kv``).
* ``plan``   -- the micro-task split (fixed-size chunks from offset 0) and the
  exact-once coverage check of a plan.
* ``digest`` -- the order-independent 64-bit checksum used by the dependent check
  kernel of the mixed-contention workload.
"""
from . import copy, digest, kv, naive, plan  # noqa: F401
