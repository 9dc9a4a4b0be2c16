"""MI355X-native discrete HMM/POMDP belief updates (FPI, VMP, MMP).

The compute path lives in the HIP library ``libbi.so`` behind a C-ABI
(``include/bi.h``); :mod:`paper_2607_17855_amd.bi` is its thin ctypes binding
and :mod:`paper_2607_17855_amd.synth` draws seeded synthetic workloads.
"""
