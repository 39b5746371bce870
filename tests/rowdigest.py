"""Per-row digests of Opt and choice tables, for comparing a full-size table with
stored oracle results without storing the table itself.

A row is the M+1 budgets of one span (s,t), spans in upper-triangle row-major order
(the order both the oracle's rows() and the solver binding's rows() use).  Opt rows
are hashed as little-endian int32 (infinity as INT32_MAX), choice rows as
little-endian int16.  The digest is CRC-32 (zlib): a row that differs in any entry
changes its digest except with probability about 2^-32.
"""
from __future__ import annotations

import zlib

import numpy as np


def row_digests(table: np.ndarray, dtype) -> np.ndarray:
    """[n_rows] uint32 CRC-32 of each row of a [n_rows, W] table, as `dtype` bytes."""
    t = np.ascontiguousarray(table, dtype=np.dtype(dtype).newbyteorder("<"))
    return np.fromiter((zlib.crc32(t[k].tobytes()) for k in range(t.shape[0])),
                       dtype=np.uint32, count=t.shape[0])


def opt_digests(opt: np.ndarray) -> np.ndarray:
    return row_digests(opt, np.int32)


def arg_digests(arg: np.ndarray) -> np.ndarray:
    return row_digests(arg, np.int16)
