"""MI355X (gfx950) contrastive-decoding tree verification.

The product is ``libdcd.so`` (HIP kernels behind the C ABI declared in
``include/dcd.h``); :mod:`paper_2608_12913_amd.dcd` is its thin ctypes binding and
:mod:`paper_2608_12913_amd.synth` the seeded input generator.  Importing the
package loads nothing; the library is opened on first use and a missing build is
an error, never a fallback.
"""
