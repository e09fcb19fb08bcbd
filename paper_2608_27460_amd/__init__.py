"""MI355X-native vector-index output head: dense top-k, HNSW search, scatter.

Importing the package is cheap; the HIP library is loaded on first use of
:mod:`paper_2608_27460_amd.vie`.
"""
