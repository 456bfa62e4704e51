"""CPU oracle for the Q4NX projection path and its next steps (the quantizer
into Q4NX, FlowKV decode attention, the MXFP4 block variant) -- TEST
INFRASTRUCTURE ONLY.

A plain, slow, obviously correct NumPy implementation of what the GPU path
computes: the Q4NX block format, the block-wise asymmetric dequantization
(Eq. 3) and the projection as a matrix-vector (Eq. 14/15) or matrix-matrix
product (Sec. 3.1.2), accumulated in float64.

Only ``tests/``, ``__graft_entry__.smoke()`` and the ``cpu_baseline`` leg of
``bench.py`` may import this package.  It shares no code with the HIP path
(``paper_2602_06063_amd``) and never imports it.

Pins (checked by ``tests/test_oracle_*.py`` against facts fixed outside the
oracle): the block geometry and byte count the paper prints, the closed form
of Eq. 3 on exactly representable operands, special cases that reduce to an
integer mat-vec / column extraction / row sums, a pure-Python brute-force
re-implementation with exact rational arithmetic on tiny shapes, and the
float32->bfloat16 rounding against torch's conversion.  The byte layout inside
a block is a reading (the paper does not fix it); it is pinned by a
hand-written fixture of expected bytes, not by the paper.
"""
from .q4nx import (  # noqa: F401
    BLOCK_ROWS, BLOCK_COLS, GROUP, CODE_BYTES, SCALE_BYTES, OFFSET_BYTES, BLOCK_BYTES,
    GROUPS_PER_BLOCK_ROW, bf16_to_f32, f32_to_bf16, packed_size, pack, unpack,
    dequant_f32, dequant_bf16, dequant_blob_f32, gemv_f64, gemm_f64, abs_bound,
    tolerance, check_close,
)
from .quantize import quantize, clamp_weights, group_scale_offset  # noqa: F401,E402
from .attention import attended_range, decode_attention, decode_attention_chunked  # noqa: F401,E402
from .mxfp4 import (  # noqa: F401,E402
    MX_BLOCK_BYTES, fp4_value, e8m0_value, mx_packed_size, mx_pack, mx_unpack, mx_dequant_f32, mx_quantize,
)
