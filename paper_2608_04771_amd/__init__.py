"""MI355X (gfx950) hot path of reward-coordinated KV-cache compression and decoding.

The kernels live in ``libreco.so`` (HIP, built by ``paper_2608_04771_amd.build``)
behind the C ABI of ``include/reco.h``; ``paper_2608_04771_amd.binding`` is the
Python binding with the same function names,
``paper_2608_04771_amd.controller`` drives the kernels through the method's
step loop, and ``paper_2608_04771_amd.inputs`` draws the seeded synthetic
workloads.
Importing this package loads nothing; importing ``binding`` functions loads the
library and fails if it has not been built."""

__all__ = ["binding", "controller", "inputs", "build"]
