"""CPU oracle for the LASER decode + confidence-probe hot path.

TEST INFRASTRUCTURE ONLY.  Only `tests/`, `__graft_entry__.smoke()` and the
`cpu_baseline` leg of `bench.py` may import or call anything in this package.
The GPU product path never routes through it, and it shares no code with the
GPU path (no kernels, headers, helpers, tables or generators).  Inputs come
from the seeded generators in `paper_2606_31580_amd.synth`, passed in as plain
arrays.

Everything here is written for a reader to check against the paper by eye:
plain numpy in float64, no blocking, fusion or reordering beyond what the
definitions state.

Modules
-------
numerics     bf16 round-to-nearest-even from its definition; bf16 bit decoding.
transformer  decoder step, full causal recompute, LM-head statistics and the
             trial-answer confidence probe (Section 3.1).
controller   load-aware threshold (Eq. 5) with EMA load (Section 4.2), budget
             pre-allocation (Eq. 6-8) and the per-ATP decision of Algorithm 1.
pages        lowest-free-id paged KV bookkeeping (a reading: the paper assumes a
             vLLM-style paged cache, Section 4.2, but specifies no policy).

Parity status (see each module's header):
  * controller, numerics, pages, and attention / RoPE / RMSNorm / SwiGLU /
    softmax statistics are pinned by closed forms, special cases and brute
    force in tests/test_oracle_*.py.
  * Full-model logits of a random-initialised decoder: "parity unpinned" with
    respect to the paper (no worked example exists); pinned only by internal
    invariants (cached decode == full recompute, fp64 vs fp32 agreement).
"""
