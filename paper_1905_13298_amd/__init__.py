"""DeepShift shift operators (LinearShift, ConvShift) for AMD Instinct MI355X.

The compute path is the HIP library ``libdeepshift.so`` behind the C ABI in
``include/deepshift.h``; ``ops`` wraps it for PyTorch tensors and
``workloads`` generates seeded synthetic inputs.
"""
