"""MI355X-native clairvoyant access planner (NoPFS planning path).

Import ``paper_2101_08734_amd.nopfs`` for the GPU binding (needs the built
``libnopfs.so``) and ``paper_2101_08734_amd.workloads`` for the seeded
synthetic workloads.
"""
__all__ = ["nopfs", "workloads", "build"]
