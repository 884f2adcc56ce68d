"""CLSA shared-routing sparse attention on MI355X (gfx950).

The compute path is the C-ABI library ``libclsa.so`` (``include/clsa.h``),
built from the HIP sources in ``csrc/``.  ``binding`` is its thin Python
binding (same names as the C entry points, torch tensors in); ``inputs`` holds
the seeded synthetic workloads.  The binding is imported lazily so that the
generator can be used without torch or a GPU.
"""

_BINDING_NAMES = (
    "clsa_index_scores", "clsa_topk", "clsa_sparse_attn", "clsa_decode_step",
    "clsa_decode_step_grouped", "clsa_decode_step_noalloc", "clsa_dense_attn", "clsa_project_append", "clsa_kd_target",
    "clsa_kd_loss", "clsa_workspace_bytes", "clsa_status_string", "clsa_set_phase_events",
    "clsa_get_device_error",
    "ClsaShape", "ClsaError", "make_shape", "workspace", "HipEvents", "lib",
    "CLSA_OP_INDEX", "CLSA_OP_TOPK", "CLSA_OP_ATTN", "CLSA_OP_DECODE", "CLSA_OP_DENSE",
    "CLSA_OP_KD_TARGET", "CLSA_OP_KD_LOSS", "CLSA_DEVERR_SEQ_LEN", "CLSA_DEVERR_N_SEL",
)


def __getattr__(name):
    if name in _BINDING_NAMES:
        from . import binding
        return getattr(binding, name)
    raise AttributeError(name)
