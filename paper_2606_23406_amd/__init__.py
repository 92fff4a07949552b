"""MI355X-native HyperQuant codec: HIP kernels for gfx950 behind a C ABI.

The binding (``paper_2606_23406_amd.hq``) loads ``libhq.so`` on first use;
importing this package loads nothing.
"""
