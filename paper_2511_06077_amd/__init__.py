"""MI355X-native STCA (stacked target-to-history cross attention) under
request level batching: a C-ABI HIP library and its thin Python binding.

The binding lives in :mod:`paper_2511_06077_amd.stca`; seeded synthetic inputs
in :mod:`paper_2511_06077_amd.workload`.  Importing the package itself loads
nothing native.
"""
