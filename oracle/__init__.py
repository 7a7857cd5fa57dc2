"""CPU oracle for the LS-SVM reduced-system solve (test infrastructure only).

Only tests/, the smoke check and the benchmark's CPU-baseline leg may import
this package. It shares no code with the HIP path or the native file IO. See
lssvm_oracle.py for the passages of the paper each function follows, and
libsvm_format.py for the plain reader of the data and model file formats.
"""
from .lssvm_oracle import *  # noqa: F401,F403
from .lssvm_oracle import __all__  # noqa: F401
from . import libsvm_format  # noqa: F401
