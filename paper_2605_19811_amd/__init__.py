"""MI355X-native LionMuon optimizer step (arXiv 2605.19811, Algorithm 1).

The step runs as hand-written gfx950 HIP kernels behind the C ABI of
``include/lionmuon.h``; this package holds their sources (``csrc/``), the
in-tree build (``build.py``) and a thin ctypes binding (``lionmuon.py``).
"""
from .lionmuon import (LM_NS_BF16, LM_NS_FP32, LM_NS_SCALE_NONE, LM_NS_SCALE_RMS02,
                       LM_TENSOR_ADAMW, LM_TENSOR_LION_ONLY, LionMuonError, TensorList, config,
                       library, lionmuon_abi_version, lionmuon_ns, lionmuon_plan_info,
                       lionmuon_profiling_enable, lionmuon_profiling_read,
                       lionmuon_profiling_reset, lionmuon_release, lionmuon_step,
                       lionmuon_step_adaptive, lionmuon_step_ex, lionmuon_workspace_bytes)

__all__ = [
    "LM_NS_BF16", "LM_NS_FP32", "LM_NS_SCALE_NONE", "LM_NS_SCALE_RMS02",
    "LM_TENSOR_ADAMW", "LM_TENSOR_LION_ONLY", "LionMuonError", "TensorList", "config", "library",
    "lionmuon_abi_version", "lionmuon_ns", "lionmuon_plan_info",
    "lionmuon_profiling_enable", "lionmuon_profiling_read", "lionmuon_profiling_reset",
    "lionmuon_release", "lionmuon_step", "lionmuon_step_adaptive", "lionmuon_step_ex",
    "lionmuon_workspace_bytes",
]
