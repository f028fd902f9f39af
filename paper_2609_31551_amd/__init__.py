"""MI355X-native Encode-stage encoder: packed micro-batch -> modality embeddings.

The compute path is the HIP library ``libeas.so`` (built from ``csrc/``);
``eas`` is its thin ctypes binding.  Importing the package loads nothing;
``paper_2609_31551_amd.eas`` loads the library and raises if it is missing.
"""
