"""MI355X-native batched, ragged Llama-2 greedy decode (the hot path of Sprout, arXiv 2403.12900).

Importing the package loads nothing native; ``paper_2403_12900_amd.binding``
loads the HIP library and fails loudly when it is missing.
"""
