"""Paged GQA decode attention for MI355X (gfx950).

The compute path is the HIP library ``libsl`` (C ABI, ``include/sl.h``); this
package only marshals torch tensors into it (``decode_attn``,
``decode_attn_fp8``) and draws seeded synthetic batches (``inputs``).
"""
