"""CPU oracle for the multi-bitwidth additive-codebook linear layer (Drop-by-Drop).

TEST INFRASTRUCTURE ONLY. This package is imported by ``tests/``, by the smoke
check in ``__graft_entry__.smoke()`` and by the ``cpu_baseline`` leg of
``bench.py``; nothing on the product path imports, calls or links it, and it
imports nothing from the product package. It is plain, slow and written to be
checked against the paper by eye:

* ``formats``   - exact decoding of fp16/bf16 bit patterns and round-to-nearest-
                  even encodings (own bit manipulation for bf16, numpy for fp16,
                  plus a format-generic rounding used to pin both);
* ``aq``        - the partial reconstruction, the linear layer, the canonical
                  rounded dequantization, the GEMM reference, the weighted MSE,
                  the distortion of every prefix level and the average-bits formula;
* ``search``    - residual k-means encoding, exhaustive / beam code search on tiny
                  groups (plain or data-weighted error), and the beam searches with
                  decisions taken in binary32 (the references of the GPU searches).

Every function cites the passage of the paper it follows. Pins live in
``tests/test_oracle_*.py``; functions without a pin say "parity unpinned".
"""
from . import formats, aq, search  # noqa: F401
from .aq import (reconstruct, linear, dequant_canonical, gemm_reference, wmse_frobenius,
                 wmse_trace, prefix_distortions, bits_per_weight, code_bits_per_weight)  # noqa: F401
from .search import (encode_residual_kmeans, brute_force_codes, beam_search_codes, beam_search_codes_f32,  # noqa: F401
                     beam_search_codes_weighted_f32, group_hessian_blocks)
