"""KVarN quantize + decode-attention hot path for AMD Instinct MI355X (gfx950).

The compute path lives in the HIP library ``libkvarn.so`` (``csrc/``); ``kvarn.py`` is its thin
ctypes binding.  ``datagen`` draws the seeded synthetic workloads.
"""
