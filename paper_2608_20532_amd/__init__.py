"""MI355X-native GF(2) affine-map learner (fit by streaming elimination, encode with span check).

The product is the C-ABI library ``libf2gpu.so`` (``include/f2gpu.h``); ``f2gpu`` is
its thin Python binding.
"""
__all__ = ["f2gpu"]
