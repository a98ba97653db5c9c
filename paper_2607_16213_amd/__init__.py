"""SelKV one-shot KV-cache compression and biased decode on MI355X (gfx950).

The compute lives in the HIP library ``libselkv.so`` (C ABI, include/selkv.h);
``selkv`` is its thin ctypes binding and ``synth`` draws seeded inputs.
"""
