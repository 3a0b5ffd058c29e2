"""Parser-stack-classification masks for grammar-constrained decoding on MI355X.

``psc`` is the binding of libpsc.so (C ABI in include/psc.h); ``build``
compiles it.  Importing the package has no side effects.
"""
