"""CPU oracle for eviction-masked attention (test infrastructure only).

This package is the plain, slow, obviously correct definition of what the
HIP library computes.  Only the test suite, the smoke check and the CPU
baseline leg of the benchmark may import it; the library never calls it.

* ``attention``   fp64 forward/backward with an explicit boolean mask
                  (Section 2, "KV-streams": one pass over the continuous trace
                  where a mask blocks the deleted span).
* ``stream_sim``  brute-force replay of the streamed, compacted KV cache,
                  token by token (Section 2, "Compaction" and "KV-streams";
                  Section 3, "Summary").
* ``tiles``       per-element counting classifier for Q x K tiles.
* ``paged``       decode attention of one query over the live entries of a
                  streamed KV cache (Section 2, "KV-streams": the inference
                  engine evicts entries in place).

Numbers are fp64 (the paper fixes no precision for this computation).
Shares no code with the HIP path.
"""
