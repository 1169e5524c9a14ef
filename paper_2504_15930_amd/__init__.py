"""Paged GQA decode attention for MI355X (gfx950).

The compute path is the HIP library ``libsl`` (C ABI: ``include/sl.h``,
``include/sl_engine.h``, ``include/sl_dispatch.h``); this package only marshals
into it: ``sl`` (decode attention with a bf16 or E4M3 cache, its prefix-shared
and allocation-free variants, the KV append), ``engine`` (the multi-step decode
loop), ``dispatch`` (skewness-aware dispatching), and ``inputs`` draws seeded
synthetic batches.
"""
