"""Float64 CPU oracle of the gated-delta-rule forward and backward.

TEST INFRASTRUCTURE ONLY.  Only ``tests/``, the smoke check in
``__graft_entry__`` and the CPU-baseline leg of ``bench.py`` may import,
call or run anything in this package.  The product path (the HIP library and
its Python binding) never does, and the two share no code: only the seeded
input generators in ``workloads.py`` (which hold none of the method's
arithmetic) feed both.

Modules:
  gdn_oracle   token-serial recurrence and its hand-derived adjoint (bottom rung)
  chunked_ref  chunkwise reference, checked against the token-serial oracle
  dense_ref    closed forms used only to pin the oracle (brute-force unroll,
               dense masked decayed attention)
  cw_oracle    the channel-wise recurrence (per-channel g, b, w) and its adjoint
"""
