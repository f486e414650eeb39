"""MI355X-native rotated, key-centered INT2 KV cache and decode attention (HIP, gfx950).

The compute path is ``libint2kv.so`` (see include/int2kv.h); ``int2kv`` is its thin ctypes
binding. Importing the package does not load the library; the first call does, and raises if
it has not been built.
"""
