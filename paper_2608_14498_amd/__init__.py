"""MI355X-native prefix/suffix backbone path of Rollplex (arXiv 2608.14498).

Importing the package is light: the HIP library is loaded by
``paper_2608_14498_amd.binding`` on first use and fails loudly when missing.
"""
__all__ = ["configs", "inputs"]
