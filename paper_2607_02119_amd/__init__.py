"""MI355X-native multi-codebook audio decode head (arXiv 2607.02119).

The hot path lives in the HIP library ``libmcd.so`` (sources in ``csrc/``,
C ABI in ``include/mcd.h``); ``mcd`` is its thin ctypes binding.  Importing the
package loads nothing: ``from paper_2607_02119_amd import mcd`` loads the
library and raises if it has not been built.
"""
