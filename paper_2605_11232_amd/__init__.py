"""MI355X-native prefix-cached paged attention.

The compute path lives in the HIP/C++ library ``libpa.so`` (sources under
``csrc/``, C ABI in ``include/pa.h``); ``binding`` is its thin ctypes
wrapper.  ``synth`` draws the seeded synthetic workloads.  Importing this
package loads nothing; the library is loaded on first use of ``binding``.
"""
