"""CPU oracle for the DynamicPTQ quantized linear layer.

TEST INFRASTRUCTURE ONLY.  This package is the plain, slow, obviously-correct
definition of what the HIP path computes.  Only the test suite, the smoke check
in ``__graft_entry__`` and the ``cpu_baseline`` leg of ``bench.py`` may import
or run it; the product library never does, and it shares no code, tables or
constants with the HIP sources.

Every floating-point step is written out in fp32 in a pinned order (the paper
fixes no precision or summation order for the rotation; the readings chosen
here are listed in the module docstrings).  Integer work (codes, packing,
accumulators) is exact.

Modules
  hadamard  Sylvester / Paley Hadamard matrices and the block rotation x.B_h
            (Section 2, Eq. 4 "rotation_activation" and Eq. 5 "rotation_equiv").
  quant     per-token / per-channel symmetric quantizer and nibble packing
            (Section 2, Eq. 1-3; Section 4.2 quantizer facts), and the
            weight byte order of the W4A8 GEMM.
  gemm      exact integer GEMM and the per-token x per-channel dequant epilogue
            (Section 2, Y = X W^T).
  policy    phase-aware activation bit policy (Eq. 21, Algorithm 1 step 2).
  residual  Jump Ratio, Historical Feature SNR and the sensitive-layer rule
            (Section 3.1 Eq. 8-11, Section 3.3 Eq. 20).
  kv        group-wise 4-bit KV-cache quantizer and its reconstruction
            (Section 4.2, Eq. 1-2).
  variants  the randomized-sign (QuaRot-style) rotation of Section 4.2 and
            its weight absorption (Eq. 4-5).
  range_quant  the range-based quantizer of Eq. 1 with an integer zero point,
            and the zero-point correction of the integer GEMM.
"""

from .hadamard import (sylvester, paley28, hadamard, split_had_size,
                       rotate_rows)
from .quant import (qmax_for_bits, quantize_rows, pack_int4, unpack_int4,
                    pack_int4_a8order, unpack_int4_a8order,
                    rotate_quant_ref, prepare_weights_ref, dequant_rows)
from .gemm import qlinear_acc_ref, qlinear_acc_entries, epilogue_ref, qlinear_ref
from .policy import layer_policy_ref
from .residual import (jump_ratio_tokens_ref, inverse_rotate_f64, reconstructed_history_ref,
                       hist_snr_tokens_ref, residual_dynamics_ref, select_sensitive_layers_ref)
from .kv import kv_quant_ref, kv_dequant_ref, pack_u4, unpack_u4
from .variants import (signs_from_bits, apply_signs, rotate_quant_signed_ref,
                       prepare_weights_signed_ref)
from .range_quant import (range_levels, quantize_rows_range, rotate_quant_range_ref,
                          dequant_rows_range, weight_sums_ref, zero_point_acc_ref,
                          qlinear_range_ref)

__all__ = [
    "sylvester", "paley28", "hadamard", "split_had_size", "rotate_rows",
    "qmax_for_bits", "quantize_rows", "pack_int4", "unpack_int4",
    "pack_int4_a8order", "unpack_int4_a8order",
    "rotate_quant_ref", "prepare_weights_ref", "dequant_rows",
    "qlinear_acc_ref", "qlinear_acc_entries", "epilogue_ref", "qlinear_ref",
    "layer_policy_ref",
    "jump_ratio_tokens_ref", "inverse_rotate_f64", "reconstructed_history_ref",
    "hist_snr_tokens_ref", "residual_dynamics_ref", "select_sensitive_layers_ref",
    "kv_quant_ref", "kv_dequant_ref", "pack_u4", "unpack_u4",
    "signs_from_bits", "apply_signs", "rotate_quant_signed_ref", "prepare_weights_signed_ref",
    "range_levels", "quantize_rows_range", "rotate_quant_range_ref", "dequant_rows_range",
    "weight_sums_ref", "zero_point_acc_ref", "qlinear_range_ref",
]
