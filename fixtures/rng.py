"""Counter-based SplitMix64 -> uniform(0,1) -> Box-Muller normals."""
import os
from concurrent.futures import ThreadPoolExecutor

import numpy as np

BASE_SEED = 2605
_GOLDEN = np.uint64(0x9E3779B97F4A7C15)
_M1 = np.uint64(0xBF58476D1CE4E5B9)
_M2 = np.uint64(0x94D049BB133111EB)
_CHUNK = 1 << 18


def _mix(z):
    """SplitMix64 finaliser on a uint64 array (wrapping arithmetic)."""
    z = (z ^ (z >> np.uint64(30))) * _M1
    z = (z ^ (z >> np.uint64(27))) * _M2
    return z ^ (z >> np.uint64(31))


def _mix_int(x):
    with np.errstate(over="ignore"):
        return int(_mix(np.array([x & 0xFFFFFFFFFFFFFFFF], dtype=np.uint64))[0])


def _fnv1a(s):
    h = 0xCBF29CE484222325
    for ch in s.encode():
        h ^= ch
        h = (h * 0x100000001B3) & 0xFFFFFFFFFFFFFFFF
    return h


def stream_key(workload, stream_id, name=""):
    k = _mix_int(BASE_SEED)
    k = _mix_int(k ^ _fnv1a(workload))
    k = _mix_int(k ^ (stream_id * 0x9E3779B97F4A7C15))
    k = _mix_int(k ^ _fnv1a(name))
    return k


def _pool():
    n = min(16, os.cpu_count() or 1)
    return ThreadPoolExecutor(max_workers=n)


class Stream:
    """One independent counter-based stream. Element i uses counter i."""

    def __init__(self, workload, stream_id, name=""):
        self.key = np.uint64(stream_key(workload, stream_id, name))

    def bits(self, start, n):
        with np.errstate(over="ignore"):
            c = np.arange(start + 1, start + n + 1, dtype=np.uint64)
            return _mix(self.key + c * _GOLDEN)

    def uniform(self, n, start=0):
        """Uniforms in the open interval (0, 1): ((z >> 11) + 0.5) * 2^-53."""
        z = self.bits(start, n)
        return ((z >> np.uint64(11)).astype(np.float64) + 0.5) * (2.0 ** -53)

    def _normal_chunk(self, start_pair, npairs):
        u = self.uniform(2 * npairs, start=2 * start_pair)
        u1, u2 = u[0::2], u[1::2]
        r = np.sqrt(-2.0 * np.log(u1))
        out = np.empty(2 * npairs, dtype=np.float64)
        out[0::2] = r * np.cos(2.0 * np.pi * u2)
        out[1::2] = r * np.sin(2.0 * np.pi * u2)
        return out

    def normal_pairs_into(self, out, start_pair, npairs, post=None):
        """Write normals 2*start_pair .. 2*(start_pair+npairs) into out,
        passed through the element-wise function `post` when given."""
        v = self._normal_chunk(start_pair, npairs)
        out[2 * start_pair:2 * (start_pair + npairs)] = v if post is None else post(v)

    def normal(self, n, dtype=np.float32):
        """n standard normals; element 2j and 2j+1 share one Box-Muller pair."""
        npairs = (n + 1) // 2
        out = np.empty(2 * npairs, dtype=dtype)
        if npairs <= _CHUNK:
            out[:] = self._normal_chunk(0, npairs)
        else:
            starts = list(range(0, npairs, _CHUNK))

            def work(s):
                m = min(_CHUNK, npairs - s)
                out[2 * s:2 * (s + m)] = self._normal_chunk(s, m)

            with _pool() as ex:
                list(ex.map(work, starts))
        return out[:n]

    def integers(self, lo, hi, n):
        """Integers uniform on [lo, hi) via floor(u * (hi - lo))."""
        return (lo + np.floor(self.uniform(n) * (hi - lo))).astype(np.int64)


def bf16_round(x):
    """Round float32 values to the nearest bfloat16 (ties to even), as float32.
    Finite inputs only."""
    x = np.ascontiguousarray(x, dtype=np.float32)
    b = x.view(np.uint32)
    b = (b + np.uint32(0x7FFF) + ((b >> np.uint32(16)) & np.uint32(1))) & np.uint32(0xFFFF0000)
    return b.view(np.float32).reshape(x.shape)


def normal_many(items, dtype=np.float32):
    """Fill several streams at once: items is a list of (Stream, n, post)
    with `post` an element-wise function (or None) applied to the float64
    normals; returns a list of arrays.  Work is split into chunks over a
    thread pool (NumPy releases the GIL inside its element-wise loops)."""
    outs, jobs = [], []
    for st, n, post in items:
        npairs = (n + 1) // 2
        buf = np.empty(2 * npairs, dtype=dtype)
        outs.append((buf, n))
        for s0 in range(0, npairs, _CHUNK):
            jobs.append((st, buf, s0, min(_CHUNK, npairs - s0), post))
    with _pool() as ex:
        list(ex.map(lambda j: j[0].normal_pairs_into(j[1], j[2], j[3], j[4]), jobs))
    return [b[:n] for b, n in outs]
