"""MI355X (gfx950) implementation of the data-parallel hot path of TSID matrix
completion (arXiv 2608.00977): the template fit of Stage I and the chunked
extension of Stage II, as hand-written HIP behind the C ABI of
``include/tsid.h``.  ``binding`` is the thin Python layer over that ABI."""
from .binding import (  # noqa: F401
    Tsid,
    TsidError,
    make_opts,
    make_adam_opts,
    tsid_chunk_plan,
    lib,
    LIB_PATH,
)
