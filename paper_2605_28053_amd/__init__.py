"""MI355X-native owner-scoped fast-weight READ/WRITE path of RW-TTT serving.

The compute lives in ``librwttt.so`` (HIP kernels for gfx950 plus the host
planner and owner table behind ``include/rwttt.h``).  ``_rwttt`` is its ctypes
binding and raises ImportError when the library has not been built;
``serving`` is the serving loop (Algorithm 1) that calls it.  Importing the
package itself loads nothing, so ``build`` works before the first build.
"""
