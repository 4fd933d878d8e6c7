"""MI355X-native pipelined CNN training with stale weights (arXiv 1912.12675).

The package is deliberately light at import: the HIP library is loaded by
``paper_1912_12675_amd.psw`` on first use.
"""
