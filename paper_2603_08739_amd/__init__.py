"""Batched KV-cache tier-configuration evaluation on MI355X (HIP, gfx950).

The public interface is the C ABI in include/kvcfg.h; :mod:`.kvcfg` binds it
with the same names and :mod:`.host` adds array marshalling helpers.
"""
