"""MI355X-native hot path of convolutional spiking networks (Spyker, arXiv 2301.13659).

``paper_2301_13659_amd.spk`` is the Python binding of libspk (C ABI in
``include/spk.h``); ``paper_2301_13659_amd.pipeline`` chains the calls into
one training/readout step per workload; ``paper_2301_13659_amd.workloads``
holds the seeded synthetic inputs.
"""
