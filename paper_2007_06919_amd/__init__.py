"""MI355X-native integer low-bit convolution path of AQD (arXiv 2007.06919).

Submodules:
  workloads  seeded synthetic inputs and network wiring (no method arithmetic)
  aqd        ctypes binding of the C-ABI library ``libaqd.so``
  runner     stream-ordered whole-network runner on top of the binding

Importing the package loads nothing native; ``aqd`` loads the library on
first use and raises if it is missing.
"""
