"""MI355X (gfx950) permutohedral-lattice filter of the Permutohedral
Attention Module (Joutard et al., 2019): a HIP library behind a C ABI
(include/pam_lattice.h, include/pam_probe.h) and its thin Python binding."""
from .binding import (  # noqa: F401
    PAM_EGRAD_AUGMENTED,
    PAM_NORMALIZE,
    BlockDesc,
    Lattice,
    block_desc,
    pam_block_bwd,
    pam_block_bwd_noalloc,
    pam_block_fwd,
    PamError,
    pam_filter_bwd,
    pam_filter_bwd_asym,
    pam_filter_fwd,
    pam_filter_fwd_asym,
    pam_kernel_names,
    pam_lattice_build,
    pam_lattice_destroy,
    pam_lattice_export,
    pam_lattice_export_groups,
    pam_lattice_set_capacity,
    pam_lattice_stats,
    pam_probe_copy_rows,
    pam_timing_enable,
    pam_timing_read,
)
