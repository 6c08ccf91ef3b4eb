"""fp64 CPU oracle for the ODA decode-step hot path.

TEST INFRASTRUCTURE.  Only ``tests/``, ``__graft_entry__.smoke()`` and the
``cpu_baseline`` leg of ``bench.py`` may import or run anything here; the
product path (the HIP library and its binding) never does, and it shares no
code with this package.

Every function computes the plain definition from the paper in float64,
starting from the exact input values (bf16 and fp32 widen to fp64 exactly):

* ``attention``  -- access sets (§2.1, access-set equation) and masked softmax
                    decode attention over a paged KV cache;
* ``gate``       -- the recall head of App. A.2, the two-layer MLP stand-in,
                    the decision rule of §2.1 / Alg. 1 and its compaction;
* ``step``       -- one decode step (Alg. 1, attention part): Local, score,
                    conditional Full, selected output (App. A.5);
* ``ledger``     -- the bytes each step reads (App. A.6 and B.7 accounting).

Parity status: every function is pinned by ``tests/test_oracle_*.py`` except
the absolute scores of the paper's *trained* heads (no weights exist), which
are "parity unpinned"; synthetic-weight scores are pinned by the structural
tests listed there.
"""
