"""MI355X-native routed-attention path of Hierarchical Global Attention.

The compute path lives in the HIP library ``libhga.so`` (built from
``csrc/``); ``hga`` is its thin ctypes binding and ``workloads`` the seeded
input generator.
"""
