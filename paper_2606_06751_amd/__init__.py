"""libstagefrontier: StageFrontier frontier accounting on AMD MI355X (gfx950).

The library is a C ABI (``include/stagefrontier.h``) over hand-written HIP
kernels; ``paper_2606_06751_amd.stagefrontier`` is its Python binding.  The
binding is imported on first attribute access so that ``import
paper_2606_06751_amd`` alone loads nothing.
"""
__version__ = "0.1.0"

_BINDING_NAMES = ("sf_frontier", "sf_frontier_checked", "sf_frontier_evidence", "sf_frontier_lag", "sf_rank_spread",
                  "sf_window_median", "sf_window_summary", "sf_frontier_summary", "sf_window_lead_exposed", "sf_window_leader_switches", "sf_ingest", "sf_route",
                  "sf_exposure_gain", "sf_read_xor", "sf_read_xor_pieces", "sf_num_windows", "sf_strerror", "sf_version",
                  "StageFrontierError", "SF_OK", "SF_EINVAL", "SF_ERANGE", "SF_EHIP", "SF_MAX_R",
                  "SF_MAX_PREFIX_NS", "SF_XOR_PIECE_BYTES")


def __getattr__(name):
    if name in _BINDING_NAMES:
        from . import stagefrontier
        return getattr(stagefrontier, name)
    raise AttributeError(name)
