"""MI355X-native self-speculative decode step of KnapSpec (arXiv 2602.20217).

The compute lives in libknapspec.so (HIP for gfx950, C ABI in
include/knapspec.h); ``_lib`` is its ctypes binding and ``engine`` the
device-memory helpers built on PyTorch.  Importing ``_lib`` fails if the
library has not been built (``python -m paper_2602_20217_amd.build``).
"""
import os

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libknapspec.so")
HEADER_PATH = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))),
                           "include", "knapspec.h")
