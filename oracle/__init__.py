"""fp64 CPU oracle for the KV-block splice path (test infrastructure only).

Imported by ``tests/``, ``__graft_entry__.smoke()`` and ``bench.py``'s ``cpu_baseline`` leg.
Never imported by the GPU library or its binding.
"""
from .nexus_oracle import *  # noqa: F401,F403
from .nexus_oracle import (NEOX, INTERLEAVED, ROWMAJOR, TRANSPOSED, rope_frequencies,  # noqa: F401
                           rotate_pairs, rope, rephase, bf16_bits_to_f64, f64_to_bf16_bits,
                           round_to_storage, storage_to_f64, splice_paged, gather_logical,
                           rephase_paged, rephase_paged_bits, suffix_attention, recompute_fraction, redecode_len)
