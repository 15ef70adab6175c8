"""CHAOS per-sample back-propagation hot path for AMD MI355X (gfx950).

Controlled Hogwild with Arbitrary Order of Synchronization (Viebke & Pllana,
"The Potential of the Intel Xeon Phi for Supervised Deep Learning", HPCC 2015),
Section III-A: many workers, each owning one sample, back-propagate through a
small CNN and push lock-free updates to one shared weight vector.

Submodules:
  workloads  seeded synthetic inputs, layer lists of the evaluated nets and
             initial weights (no forward/backward arithmetic)
  chaos      ctypes binding of the C-ABI library libchaos.so (HIP kernels)

Nothing is imported eagerly so that the input generators can be used
without loading the GPU library.
"""
__all__ = ["workloads", "chaos"]
