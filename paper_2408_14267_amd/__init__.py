"""MI355X-native 1-bit FQT layer backward (AGP + SCQ + binary products).

The computation lives in the HIP library ``libfqt.so`` (built from ``csrc/``
for gfx950); ``fqt`` is a thin ctypes binding over its C ABI.  Importing the
binding raises if the library has not been built -- there is no fallback.
"""
