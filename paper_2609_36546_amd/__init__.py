"""MI355X-native verifier-side window scoring for Interactive-Policy Distillation.

The compute path lives in the HIP library ``libipdv.so`` (built from
``csrc/``); ``ops`` is its thin ctypes binding.  Importing the package loads
nothing: the library is opened on the first call.
"""
