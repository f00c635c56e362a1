"""MI355X (gfx950) KV-block splice path of Nexus (arXiv 2608.20397).

Re-anchoring of rotary keys, splice into a paged KV cache and suffix-redecode causal GQA
attention, as hand-written HIP kernels behind the C ABI of ``include/nexus.h``
(``libnexus.so``); ``paper_2608_20397_amd.nexus`` is the thin Python binding.
"""
from . import nexus  # noqa: F401
from .nexus import (Block, PagedKVCache, NexusError, splice_pages, rephase_k,  # noqa: F401
                    rephase_k_paged, suffix_attn, suffix_attn_varlen, redecode_len,
                    check_page_table, lib)
