"""GRPO rollout, scoring and loss hot path on one MI355X (gfx950).

The compute runs in hand-written HIP kernels behind the C-ABI declared in
``include/grpo_hip.h`` (``libgrpo_hip.so``); ``paper_2510_17158_amd.api`` is the
thin ctypes binding over it.  Importing the package does not load the library.
"""
