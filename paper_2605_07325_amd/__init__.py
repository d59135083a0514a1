"""MI355X (gfx950) cached-prefix extend attention for Cached State Representations.

The compute path is the C-ABI library ``libcsr.so`` (hand-written HIP kernels);
``paper_2605_07325_amd.csr`` is its thin ctypes binding and
``paper_2605_07325_amd.datagen`` builds seeded synthetic inputs.  Importing the
package loads nothing; the binding loads the library on first use and fails
loudly if it has not been built.
"""
__all__ = ["csr", "datagen"]
