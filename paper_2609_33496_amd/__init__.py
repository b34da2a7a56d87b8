"""MI355X-native (gfx950) hot path of Chameleon's format-adaptive post-training quantization:
per-channel weight-format search, activation statistics / LUT / quantization, and the
mixed-format linear layer.  The compute lives in a HIP shared library behind a C ABI
(``include/chameleon.h``); ``paper_2609_33496_amd.cham`` is its thin Python binding and
``paper_2609_33496_amd.synth`` the seeded synthetic workloads."""
