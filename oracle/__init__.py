"""fp64 CPU oracle of the LionMuon step (test infrastructure only; see
``oracle.lionmuon_oracle``)."""
from .lionmuon_oracle import (CUBIC, adamw_update, adaptive_uses_muon,
                              lionmuon_adaptive_step, NS_EPS, NS_STEPS, QUINTIC, SCALE_NONE,
                              SCALE_RMS02, coefficient_schedule,
                              elementwise_sign, is_muon_step,
                              lionmuon_step, lionmuon_update, newton_schulz,
                              ns_output_scale, stable_rank_estimate)

__all__ = [
    "adamw_update", "adaptive_uses_muon", "lionmuon_adaptive_step", "CUBIC", "NS_EPS", "coefficient_schedule", "NS_STEPS", "QUINTIC", "SCALE_NONE", "SCALE_RMS02",
    "elementwise_sign", "is_muon_step", "lionmuon_step", "lionmuon_update",
    "newton_schulz", "ns_output_scale", "stable_rank_estimate",
]
