"""GSRQ hot path (arXiv 2607.01065) on AMD MI355X: HIP kernels behind a C ABI.

The library (libgsrq.so, built from csrc/gsrq.hip) does all the work; this
package only binds it (see gsrq.py).
"""
from .gsrq import (  # noqa: F401
    GSRQ_F16, GSRQ_F32, GsrqError, LIB_PATH, TrainResult, bits_per_element, code_words,
    decode, encode, encode_workspace_bytes, load_library, status_string, train_stage,
    train_workspace_bytes,
)
