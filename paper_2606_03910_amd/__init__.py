"""NetKV decode-instance selection on MI355X (gfx950).

The compute path is the C-ABI library ``libnetkv.so`` built from ``csrc/``;
``netkv`` is its thin ctypes binding.  ``workload`` draws seeded synthetic
inputs.  Importing the package loads nothing; the binding loads the library
on first use and raises if it has not been built.
"""
