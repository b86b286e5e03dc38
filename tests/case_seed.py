"""Stable per-case seeds: the same test id draws the same inputs in every process."""

import zlib


def case_seed(case):
    """CRC-32 of the case id (its fields joined by '-'), independent of PYTHONHASHSEED."""
    return zlib.crc32("-".join(map(str, case)).encode())
