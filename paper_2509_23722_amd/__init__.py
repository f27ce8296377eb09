"""MI355X-native batched pipeline-schedule simulation (OctoPipe, arXiv 2509.23722).

The compute path is the HIP library ``libocto.so`` behind the C ABI in ``include/octo.h``;
``paper_2509_23722_amd._lib`` is its ctypes binding. Importing the package loads nothing.
"""
