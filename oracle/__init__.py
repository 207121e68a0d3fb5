"""CPU oracle for the chunk-scheduled GEMMs.

TEST INFRASTRUCTURE ONLY: only ``tests/``, ``__graft_entry__.smoke()`` and the
CPU-baseline leg of ``bench.py`` may import, call, link or execute anything in
this package. The product library (``paper_2601_20595_amd``) never does, and
the two share no code; they meet only in the seeded inputs of
``seeded_inputs.py``.

Contents (each function cites the paper passage it follows):
  schedule.py  one rank's chunk list and arrival/emission order
               (Section 5.1, communication schedule abstraction and templates)
  depmap.py    chunk-tile dependence map and chunk-ordered tile list
               (Section 5.2, dependency parsing and tile-scheduler swizzling)
  gemm.py      chunk-by-chunk plain GEMMs in fp64 (Overview: numerical meaning
               of the local kernel is preserved), the tiny fsum reference and
               the error metric
  ref_gemm.c   the plain C loops gemm.py calls

Every function is pinned by ``tests/test_oracle_*.py`` to values fixed by the
mathematics (brute force, closed forms, invariants, hand-worked examples).
The paper prints no numeric worked example, so no stored value comes from it.
"""
from .schedule import (Chunk, ScheduleError, uniform_chunks, uniform_schedule, grouped_schedule,
                       order_ring, order_swizzle1d, order_rs_ring, order_permutation, validate)
from .depmap import dep_map, tile_grid, DepMap
from .attention import attention, attention_chunked, attention_fsum
from .gemm import (ag_gemm, gemm_rs, gemm_ar, grouped_gemm, gemm_rows, gemm_elems, exact_dot_fsum,
                   max_rel_error, num_threads)
