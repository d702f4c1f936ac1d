"""Symmetry-aware Taylor attention on MI355X (gfx950).

Hand-written HIP kernels behind a C ABI (include/sata.h, built into
libsata.so); this package is the thin Python binding over it.

    from paper_2602_00294_amd import prefill, decode_step, feature_map
    y, S = prefill(q, k, v, P=4, chunk=64)      # q, k, v: [B, H, n, d] on the GPU
    y_t = decode_step(S, q_t, k_t, v_t, P=4)     # S updated in place
"""
from ._binding import (SataError, backward, decode_step, decode_step_compensated, decode_step_grouped, feature_count, feature_index, feature_map, load_library,
                       prefill, prefill_grouped, prefill_operands, prefill_parts, release, residual_elems, state_elems)

__all__ = ["SataError", "backward", "decode_step", "decode_step_compensated", "decode_step_grouped", "feature_count", "feature_index", "feature_map", "load_library",
           "prefill", "prefill_grouped", "prefill_operands", "prefill_parts", "release", "residual_elems", "state_elems"]
