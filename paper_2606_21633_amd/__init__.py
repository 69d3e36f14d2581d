"""MI355X-native hot path of HERALD's sparse block-dLLM decode.

``paper_2606_21633_amd.herald`` is the thin ctypes binding of the C-ABI
library ``libherald.so`` (HIP kernels for gfx950, built from ``csrc/``);
``paper_2606_21633_amd.synth`` holds the seeded synthetic workloads.
Importing this package loads nothing; the binding loads the library on first
use and raises if it has not been built.
"""
