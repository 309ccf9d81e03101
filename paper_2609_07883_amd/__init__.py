"""MI355X-native mixed prefill+decode iteration for deadline-aware chunking (SLOWeave).

The compute path lives in the HIP library ``libsloweave.so`` (built from
``csrc/``); ``api`` is its thin ctypes binding.  Importing this package loads
nothing: the library is opened on first use and a missing library raises.
"""
