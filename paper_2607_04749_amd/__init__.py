"""MI355X-native resharding of model states between (TP, PP) configurations.

The work happens in libetc.so (C ABI, include/etc.h): a host planner and
gfx950 kernels for the cost matrix, pack and unpack.  `etc` is its Python
binding; `workloads` describes the model shapes and migrations.
"""
