"""Fused Convolutional Modules (depthwise + pointwise) for AMD MI355X (gfx950).

`paper_2404_19331_amd.fcm` is the ctypes binding of libfcm.so (HIP kernels + planner);
`paper_2404_19331_amd.workloads` draws the seeded synthetic inputs.
"""
