"""MI355X-native WFST Viterbi decoder with exact lattice generation.

The decoder itself is the HIP library libwfstdec.so (C ABI in
include/wfstdec.h); `wfstdec` is its ctypes binding.  Importing the package
does not load the library; the first call does, and raises if it is missing.
"""
from . import wfstdec  # noqa: F401
from .wfstdec import Graph, WdError, decode, decode_batch  # noqa: F401
