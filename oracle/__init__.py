"""Oracle: a plain, slow, float64 CPU implementation of the segmented
training hot path of Visual Context Segmentation (ScaleCUA, Sec. 3.3,
App. D, Eq. loss).

TEST INFRASTRUCTURE ONLY.  Nothing in the product path may import, call or
execute this package; only the tests, the smoke check and the CPU-baseline
leg of the benchmark do.  It shares no code with the HIP library: it builds
the full dense visibility mask of every segment and computes everything from
that mask with NumPy in float64.

Modules
-------
layout     segmentation, packing, visibility mask, tile map, loss rows
attention  masked GQA softmax attention forward and backward
loss       action-token log-prob, clipped policy-ratio loss, gradients
layer      decoder layer (RMSNorm, rotary GQA attention, SwiGLU) around the
           segmented attention, forward and backward
"""
from . import layout, attention, loss, layer  # noqa: F401
