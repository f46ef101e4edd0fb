"""CPU oracle for the 1.5-SPSA probe regenerate-and-apply sweep.

TEST INFRASTRUCTURE, NOT PRODUCT CODE. This package is a plain, slow, obviously correct
restatement of what the GPU library computes, written from the paper ("Probe-Space
Preconditioning for Fast and Stable Zero-Order Training") and from the published
definition of the Philox generator. Only the tests, the package smoke check and the
benchmark's CPU-baseline leg may import it; the library never does, and this package
imports nothing from the library.

Modules:
  philox   -- Philox-4xW (Salmon et al., SC'11), generic in word width and rounds
  probes   -- Rademacher probes from (seed, step, k, element index), 8 probes per byte
  numerics -- bf16 storage format and single-step rounding
  sweep    -- perturb (theta + e z_k), the fused update (theta - lr sum_k c_k z_k), and the
              fused transitions perturb2 / update_restore
  coeffs   -- curvature, alpha-saturated weight and per-probe coefficients
  step     -- one single-device step composed from the above

Every function is pinned by CPU tests against values the paper or mathematics fixes;
see tests/test_oracle_*.py. Floating point is float64 except where the storage format
fixes it.
"""

from .coeffs import DEFAULT_ALPHA, DEFAULT_LAMBDA_REG, probe_coeffs
from .numerics import bf16_to_f32, bf16_to_f64, f32_to_bf16, f64_to_bf16, f64_to_f32
from .philox import philox4
from .probes import (DEFAULT_ROUNDS, PROBES_PER_GROUP, TILE, element_bytes, materialize_Z,
                     signs, tile_bytes, tile_words)
from .step import full_step, full_step_fused
from .sweep import perturb, perturb2, perturb_schedule, probe_sum, update, update_restore
