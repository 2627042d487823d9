"""Eviction-masked attention for MI355X (gfx950): the training-side hot path of
KV-streams (one masked pass over a continuous agent trace, Section 2).

``paper_2609_35750_amd.kvs`` is the binding of the HIP library ``libkvs.so``
(importing it fails loudly if the library is not built);
``paper_2609_35750_amd.inputs`` builds seeded synthetic traces.
"""

_BINDING = ("evict_attn", "kvs_evict_attn_fwd", "kvs_evict_attn_bwd", "kvs_classify_tiles", "kvs_check_evict_at",
            "kvs_prof_enable", "kvs_prof_reset", "kvs_prof_read", "KvsError")


def __getattr__(name):
    if name in _BINDING:
        from . import kvs

        return getattr(kvs, name)
    raise AttributeError(name)
