"""Row-typed associative-algebra projections (Y = X *_q W) on MI355X.

The computation lives in ``libstarq.so`` (hand-written gfx950 HIP kernels
behind the C ABI of ``include/star_proj.h``); this package is its thin
ctypes binding.  Importing it fails if the library has not been built
(``python -m paper_2609_32814_amd.build``).
"""

from .binding import (  # noqa: F401
    LIB_PATH,
    Algebra,
    StarError,
    star_count_macs,
    star_count_products,
    star_decode,
    star_ffn_bwd,
    star_ffn_fwd,
    star_proj_bwd_data,
    star_proj_bwd_weight,
    star_proj_fwd,
    star_status_string,
    star_validate_types,
    star_workspace_bytes,
)
