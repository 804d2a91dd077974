"""HeadWiseKV grouped-cache runtime for MI355X (gfx950).

``paper_2609_02029_amd.hwkv`` is the ctypes binding of ``libhwkv.so`` (the
C ABI in ``include/hwkv.h``); ``paper_2609_02029_amd.build`` compiles it.
The binding is not imported here so that the build step can run before the
library exists.
"""
