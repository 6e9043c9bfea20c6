"""CPU oracle for the convolution hot path and the vision operators.

TEST INFRASTRUCTURE ONLY: the tests, the smoke check and the bench's CPU
baseline may import this package; the product library never does.  It shares
no code with the HIP path.  See ``ref_conv.c`` for the operator definition it
writes out, ``ref.py`` for the numpy-facing wrapper and ``vision.py`` for
segmented argsort, prefix sum and box_nms.
"""
from .ref import (  # noqa: F401
    build,
    lib_path,
    num_threads,
    out_dims,
    conv2d,
    conv2d_bf16,
    dwconv2d,
    maxpool2d,
    add_act,
    f32_to_bf16,
    bf16_to_f32,
    conv2d_bf16_cl,
    maxpool2d_bf16_cl,
)
from .vision import (  # noqa: F401
    segmented_argsort,
    scan_inclusive_i32,
    scan_exclusive_i32,
    scan_inclusive_f32,
    box_nms,
)
