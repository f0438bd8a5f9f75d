"""MI355X (gfx950) Coverage-Aware Grid Query.

The compute path is the HIP library ``libcagq.so`` (sources in ``csrc/``,
C ABI in ``include/cagq.h``); ``cagq`` is its Python binding and
``workloads`` the seeded synthetic inputs. Importing the package loads
nothing: ``from paper_1912_02984_amd import cagq`` needs torch, the
workload generators need only numpy.
"""
