"""MI355X-native per-token LDA topic draw with butterfly-patterned partial
sums (Steele and Tristan, arXiv 1505.03851).

``draw_naive``, ``draw_butterfly``, ``draw_transposed``, ``draw_docs``,
``route_build`` / ``draw_routed`` / ``draw_routed_philox``, ``butterfly_table`` and
``count_topics`` (the topic counts of the draws; with ``word_index_build`` and
``count_topics_indexed``, counted word by word) call the HIP
library through its C ABI (``include/lda_draw.h``).  The binding is imported
on first use, so ``paper_1505_03851_amd.inputs`` can be used without it.
"""

_BINDING = ("draw_naive", "draw_butterfly", "draw_transposed", "draw_docs", "draw_doc_lanes",
            "draw_philox", "philox_uniforms",
            "draw_variant", "VARIANTS",
            "butterfly_table", "count_topics", "count_topics_docs",
            "word_index_build", "word_index_bytes", "count_topics_indexed", "WordIndex",
            "route_build", "draw_routed", "draw_routed_philox", "route_workspace_bytes", "Route",
            "draw_routed_scratch", "ROUTED_SCRATCH_BYTES",
            "butterfly_width", "status_string", "version", "LdaError",
            "load", "MAX_K", "MAX_TABLE_BYTES", "MAX_COUNT_TABLE_BYTES", "STATUS")

__all__ = list(_BINDING)


def __getattr__(name):
    if name in _BINDING:
        from . import _lib
        return getattr(_lib, name)
    raise AttributeError(name)
