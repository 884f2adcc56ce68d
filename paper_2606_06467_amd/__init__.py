"""CLSA shared-routing sparse attention on MI355X (gfx950).

The compute path is the C-ABI library ``libclsa.so`` (``include/clsa.h``),
built from the HIP sources in ``csrc/``.  ``binding`` is its thin Python
binding (same names as the C entry points, torch tensors in); ``inputs`` holds
the seeded synthetic workloads.  The binding is imported lazily so that the
generator can be used without torch or a GPU.
"""

_BINDING_NAMES = (
    "clsa_index_scores", "clsa_topk", "clsa_sparse_attn", "clsa_decode_step",
    "clsa_workspace_bytes", "clsa_status_string", "clsa_set_phase_events",
    "ClsaShape", "ClsaError", "make_shape", "workspace", "HipEvents",
    "CLSA_OP_INDEX", "CLSA_OP_TOPK", "CLSA_OP_ATTN", "CLSA_OP_DECODE",
)


def __getattr__(name):
    if name in _BINDING_NAMES:
        from . import binding
        return getattr(binding, name)
    raise AttributeError(name)
