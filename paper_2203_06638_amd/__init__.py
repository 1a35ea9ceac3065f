"""MI355X (gfx950) implementation of the LPP-SGD per-node step.

Submodules: lpp (ctypes binding of liblpp.so), models (layer lists of the
workloads), build (hipcc build of the library).
"""
