"""M+Adam optimizer step for AMD Instinct MI355X (gfx950).

The product is the HIP library ``libmadd.so`` built from ``csrc/madd.hip``
with the C ABI of ``include/madd.h``; ``binding`` is its ctypes binding,
``optim`` a torch.optim front end over it, and ``workloads`` builds seeded
synthetic inputs (shapes and distributions of the benchmark parameter
lists).  Importing the package loads nothing.
"""
