"""MI355X-native batched sliding-window anomaly scorer (ENOVA performance detection, arXiv 2407.09486).

The compute path is ``libenova_detect.so`` (HIP kernels for gfx950 behind the C ABI of
``include/enova_detect.h``); ``binding`` marshals torch/numpy arguments to it and
``workloads`` draws seeded synthetic monitoring streams and detector weights.
"""
__all__ = ["binding", "workloads", "build"]
