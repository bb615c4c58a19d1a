"""MI355X-native flow-matching action-expert denoiser (libjpi).

The compute path is the HIP library ``libjpi.so`` built from ``csrc/``;
``jpi`` is its ctypes binding and ``expert`` a convenience wrapper that uses
PyTorch only for device memory and streams.
"""
import os

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libjpi.so")
