"""MI355X-native modality-aware permutation sparse attention (MMInference hot path).

libmmi.so (built from csrc/ by build.py) holds the HIP kernels and the C-ABI
declared in include/mmi.h; mmi.py is the ctypes binding.
"""
