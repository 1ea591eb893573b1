"""CPU oracle (test infrastructure only; see oracle.oracle for the rules)."""

from .oracle import *  # noqa: F401,F403
from .oracle import (  # noqa: F401
    BY_BUCKET, BY_COLUMN, REORDER_COLUMNS, REORDER_ELEMENTS, FormatError, Params,
    TileCOO, bf16_rne_bits, bf16_to_f64, codes, coo_sorted, csr_bytes, dense_part,
    dequant, f16_to_f64, matmul, matmul_tile_coo, outlier_part, pack_tile_coo,
    storage_bytes, unpack_tile_coo, zero_points,
)
from . import quant  # noqa: F401,E402
