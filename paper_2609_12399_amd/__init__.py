"""MI355X-native large-beam Gated DeltaNet decode (OneLA, arXiv 2609.12399).

The compute path is the HIP library ``libonela.so`` (see ``onela.py`` for the
Python binding); this package import does not load it.
"""
