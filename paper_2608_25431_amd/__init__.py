"""Segmented per-user AES-256-GCM seal/open and owner-label check on MI355X.

The compute path is the HIP library libgift.so (include/gift.h); `gift` is its
ctypes binding and `workloads` builds the seeded benchmark inputs.
"""
from . import gift, workloads  # noqa: F401
from .gift import GiftError, KeyTable, check_owner, key_table_create, open, seal  # noqa: F401
