"""ctypes binding of ``libmoeq_peaks.so`` (include/moeq_peaks.h): the
benchmark's measured roofline denominators, a streaming read of device memory
and a register-only binary16 MFMA loop.  Argument marshalling only."""
import ctypes
import os

LIB_PATH = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))), "libmoeq_peaks.so")
HEADER_PATH = os.path.join(os.path.dirname(os.path.dirname(os.path.dirname(os.path.abspath(__file__)))),
                           "include", "moeq_peaks.h")


def load():
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"{LIB_PATH} is not built; run __graft_entry__.build()")
    try:
        import torch  # noqa: F401  (bind to torch's HIP runtime, as the layer library does)
    except ImportError:
        pass
    lib = ctypes.CDLL(LIB_PATH)
    P, I32, SZ = ctypes.c_void_p, ctypes.c_int, ctypes.c_size_t
    lib.moeq_peaks_stream_read.argtypes = [P, SZ, P, P]
    lib.moeq_peaks_stream_read.restype = I32
    lib.moeq_peaks_read_workgroups.argtypes = [SZ]
    lib.moeq_peaks_read_workgroups.restype = I32
    lib.moeq_peaks_mfma.argtypes = [I32, I32, P, P]
    lib.moeq_peaks_mfma.restype = I32
    lib.moeq_peaks_mfma_flops.argtypes = [I32, I32]
    lib.moeq_peaks_mfma_flops.restype = ctypes.c_double
    return lib


def header_functions():
    import re
    with open(HEADER_PATH) as f:
        text = f.read()
    return sorted(set(re.findall(r"^\s*(?:int|double)\s+(moeq_peaks_\w+)\s*\(", text, re.M)))
