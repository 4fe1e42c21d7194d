"""The paged-cache record layout of isoq_kv_append / isoq_kv_scores, written
out from its definition in include/isoquant.h: a cache of shape
[n_blocks, n_heads, block_size, R] bytes holds, per (block, head), the
block_size records of R bytes piece-major -- each record cut into pieces of
P bytes (16 if 16 divides R, else 8 if 8 divides R, else P = R: records
stored whole), piece j of position s at byte (j * block_size + s) * P of the
(block, head) region.  to_cache turns record-major records into that byte
order, from_cache back."""
import numpy as np


def piece_bytes(R):
    return 16 if R % 16 == 0 else 8 if R % 8 == 0 else R


def to_cache(records):
    """records [..., block_size, R] uint8, one record per row -> the same
    shape in the cache's byte order (numpy or torch)."""
    *lead, bs, R = records.shape
    P = piece_bytes(R)
    x = records.reshape(*lead, bs, R // P, P)
    if isinstance(x, np.ndarray):
        return np.ascontiguousarray(np.swapaxes(x, -3, -2)).reshape(*lead, bs, R)
    return x.transpose(-3, -2).contiguous().reshape(*lead, bs, R)


def from_cache(cache):
    """The inverse of to_cache: [..., block_size, R] in the cache's byte order
    -> one record per row."""
    *lead, bs, R = cache.shape
    P = piece_bytes(R)
    x = cache.reshape(*lead, R // P, bs, P)
    if isinstance(x, np.ndarray):
        return np.ascontiguousarray(np.swapaxes(x, -3, -2)).reshape(*lead, bs, R)
    return x.transpose(-3, -2).contiguous().reshape(*lead, bs, R)
