"""CPU oracle of AQD's integer-only convolution path (arXiv 2007.06919).

TEST INFRASTRUCTURE: only the test suite, the smoke check and the CPU
baseline leg of the benchmark may import anything here. The GPU path never
does, and this package imports nothing from the GPU path.
"""
