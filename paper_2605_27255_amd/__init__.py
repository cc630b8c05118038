"""MI355X (gfx950) implementation of the PIPO pair-in/pair-out decode step and
compressed-prompt prefill, behind the C ABI in ``include/pipo.h``."""
from .pipo import (  # noqa: F401
    PipoModel, PipoError, load_library, make_config, unpack_pairs, LIB_PATH, EXPORTED, opd_teacher_rows, opd_targets,
    calibrate_stream, calibrate_mfma,
    PIPO_OK, PIPO_EINVAL, PIPO_ENOMEM, PIPO_EHIP, PIPO_ECAPACITY, PIPO_ESTATE,
)
