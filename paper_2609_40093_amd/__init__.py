"""MI355X-native expert-parallel MoE token dispatch and combine (one rank's share).

The work happens in libep.so (HIP kernels for gfx950 plus SDMA host legs; C ABI in
include/ep.h).  ``paper_2609_40093_amd.api`` is its Python binding; the names below are
re-exported lazily so that ``paper_2609_40093_amd.synth`` (input generation only) can be
imported without torch or a GPU.
"""

_API = ("EPError", "Layout", "Staging", "SimPeers", "dispatch_layout", "layout_validate", "dispatch", "dispatch_fused",
        "combine", "trace_enable", "trace_read", "trace_reset", "copy_probe", "stream_probe", "workspace_bytes",
        "pcie_probe",
        "MODE_PER_SENDER", "MODE_DUPLEX", "MODE_REMOTE_ONLY", "MODE_ACCUMULATE", "LocalLayout", "dispatch_layout_local", "pack",
        "combine_rows", "Dense", "allgather", "reducescatter", "round_advance", "round_read", "dispatch_graph",
        "combine_graph", "graph_legs_sdma")

__all__ = list(_API)


def __getattr__(name):
    if name in _API:
        from . import api
        value = getattr(api, name)
        globals()[name] = value  # later lookups skip this function
        return value
    raise AttributeError(name)
