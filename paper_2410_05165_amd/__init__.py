"""MI355X (gfx950) speculative-decoding verify path of AtSpeed (arXiv 2410.05165).

The product is the HIP library ``libatspeed.so`` (C ABI in include/atspeed.h);
``binding`` is its ctypes binding.  Importing ``binding`` fails loudly when the
library is not built: there is no fallback path.
"""
from .build import LIB, build  # noqa: F401
