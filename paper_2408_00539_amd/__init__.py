"""MI355X-native ISM attention (arXiv 2408.00539).

Importing the package is cheap: the HIP library is loaded only when an op of
:mod:`paper_2408_00539_amd.ops` is first called. The seeded input generators
live in :mod:`paper_2408_00539_amd.workloads`.
"""
