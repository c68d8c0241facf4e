"""WiSP paged MoE layer for AMD MI355X (gfx950).

Submodules:
  ``wisp``      ctypes binding of the C-ABI library ``libwisp.so`` (HIP kernels + expert pager).
  ``datagen``   seeded synthetic inputs (weights, router weights, hidden states).
  ``workloads`` workload shapes and VRAM budgets.

Importing the package loads nothing native; ``wisp`` loads the HIP library on first use and
raises if it is missing.
"""
