"""MI355X-native detect-and-aggregate step of Aspis (MLSys 2022).

The product is libaspis.so (include/aspis.h): HIP kernels for gfx950 plus
the host steps of the method.  This package only binds it (aspis.py) and
builds it (build.py).
"""
from . import aspis  # noqa: F401
from .aspis import (AspisError, DetectBuffers, aggregate, assign, clique,  # noqa: F401
                    detect, detect_aggregate, num_files, read_probe)
