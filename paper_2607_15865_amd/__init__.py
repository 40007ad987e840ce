"""MI355X-native three-stage W4A16 decoder layer (prefill, prefill_kv, decode).

Importing the package loads nothing native; ``paper_2607_15865_amd.binding``
loads the HIP library and fails loudly when it is missing.
"""
