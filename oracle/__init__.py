"""CPU oracle for Windowed-MTP draft decode attention.

TEST INFRASTRUCTURE ONLY.  This package is the plain, slow, float64 statement
of what the draft-attention hot path computes.  Only the test suite, the smoke
check and the CPU-baseline leg of the benchmark may import it; the product
path (the HIP library and its Python binding) never does, and shares no code
with it.

Modules
  attention  -- key selection (sink + recent window), exact masked-softmax
                GQA decode attention (Windowed-MTP paper, Section 4
                "Mechanism" and the Appendix A pseudocode of the windowing
                change).
  ring       -- the compact ring-buffer draft KV store: the slot map and an
                operational replay of appends (Section 4 "Memory", Section 6
                "Memory", the ring comment of the Appendix A pseudocode).
  fp8        -- the fp8 (OCP E4M3, per-tensor scale) draft KV cache: code
                values, quantization on append, attention over the
                dequantized rows (Section 7, KV-cache quantization).
  spec       -- speculative draft rows in the ring: chain rollback and
                tree-width rings (Section 7, tree speculation; Appendix A
                ring comment).
  paged      -- the paged token pool (page size 1): the draft's index list
                req_to_token[r, keep] and attention over the listed rows
                (Section 4 "Mechanism", Appendix A pseudocode).

Every function states the passage it follows.  Readings of points where the
paper is silent are listed in the module docstrings.  No function here is
"parity unpinned": each is pinned by the CPU tests in tests/test_oracle_*.py
against closed forms, brute force, invariants, a library routine
(torch scaled_dot_product_attention in float64) and the facts the paper prints
(tests/golden/).
"""

from . import attention, fp8, paged, ring, spec  # noqa: F401
