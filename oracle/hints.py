"""Reference of the reuse-hint machinery: chained block hashes, the counted hint index, and the
prefix probes, in plain Python.

TEST INFRASTRUCTURE ONLY (see the package docstring).

What is computed, with the passages it follows (Design of WavePP, "Fast Reuse Hints"):

* Chained prefix hash (Eq. 5): for each full token block B_i, H_{-1} = 0 and
  H_i = hash(B_i, extraKeys_i, salt, H_{i-1}); the parent hash makes each key depend on the whole
  prefix.  Only full blocks are hashed.
* The hint index holds no blocks: per (cache window, H_i) a counter, incremented when a block
  enters the cache tree and decremented when it is detached, the entry disappearing at zero.
  Offloading a block leaves it unchanged.
* Dense attention prefixes: the reusable endpoint is the longest prefix of the request's block
  hashes that are all in the index.  Its definition is the plain scan from the first block to the
  first miss; the native probe reaches it with O(log N) probes (depths at growing powers of two
  until the first miss, then bisection), which agrees whenever the indexed set is prefix-closed,
  as a cache tree's is.
* Recurrent snapshots are sparse: from the attention-limited endpoint the scan goes backwards to
  the nearest boundary that has a snapshot (boundary 0, the empty prefix, always qualifies).

Readings (the paper does not fix them):
* hash = SHA-256 (FIPS 180-4) of the byte string
      salt || H_{i-1} (32 bytes) || extraKeys_i (int64, little endian, each) || B_i (int32 tokens,
      little endian)
  with H_{-1} = 32 zero bytes; H_i is the full 32-byte digest.
* Index key of a block = (window, first 8 bytes of H_i as a little-endian unsigned 64-bit integer).
* A snapshot "at boundary j" (j blocks of prefix) is indexed under the key of block j - 1.
"""
from __future__ import annotations

import hashlib
import struct


def chained_hashes(tokens, block: int, extra_keys=None, salt: bytes = b"") -> list[bytes]:
    """Eq. 5 over the full blocks of `tokens`; extra_keys[i] is a sequence of ints for block i (or None)."""
    n_full = len(tokens) // block
    out, parent = [], bytes(32)
    for i in range(n_full):
        msg = bytes(salt) + parent
        if extra_keys is not None and extra_keys[i] is not None:
            msg += b"".join(struct.pack("<q", int(x)) for x in extra_keys[i])
        msg += b"".join(struct.pack("<i", int(t)) for t in tokens[i * block:(i + 1) * block])
        parent = hashlib.sha256(msg).digest()
        out.append(parent)
    return out


def key64(digest: bytes) -> int:
    return struct.unpack("<Q", digest[:8])[0]


class HintIndex:
    """Counted keys (window, key64)."""

    def __init__(self):
        self.count = {}

    def add(self, window: int, keys):
        for k in keys:
            self.count[(window, k)] = self.count.get((window, k), 0) + 1

    def detach(self, window: int, keys):
        for k in keys:
            c = self.count.get((window, k), 0)
            if c <= 0:
                raise KeyError("detach of a key that is not indexed")
            if c == 1:
                del self.count[(window, k)]
            else:
                self.count[(window, k)] = c - 1

    def contains(self, window: int, k: int) -> bool:
        return (window, k) in self.count


def prefix_endpoint(index: HintIndex, window: int, keys) -> int:
    """Number of leading blocks whose keys are all indexed (the plain scan)."""
    n = 0
    for k in keys:
        if not index.contains(window, k):
            break
        n += 1
    return n


def recurrent_endpoint(snapshots: HintIndex, window: int, keys, limit: int) -> int:
    """Largest boundary j <= limit with a snapshot (j = 0 always qualifies), scanning backwards."""
    for j in range(limit, 0, -1):
        if snapshots.contains(window, keys[j - 1]):
            return j
    return 0
