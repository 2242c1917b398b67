"""MI355X-native paged mixed-bitwidth MoE expert forward (PagedWeight, arXiv 2607.16184).

Importing the package loads nothing. ``paper_2607_16184_amd.pw`` binds the HIP
library ``libpagedweight.so`` (and fails loudly if it is missing);
``paper_2607_16184_amd.synth`` draws the seeded synthetic workloads.
"""
__all__ = ["pw", "synth"]
