"""Block-granular prefix identification — TEST INFRASTRUCTURE ONLY (CPU, pure Python integers).

Only ``tests/``, ``__graft_entry__.smoke()`` and ``bench.py``'s ``cpu_baseline`` leg may import this
module; the product path (the HIP library and its binding) never does and shares no code with it.

Sec. 4.4 of the paper: the inference engine's prefix cache keys every full prompt block by a hash; a
request's reusable prefix H (the H of the prefill cost of Eq. 1) is the longest run of its leading full
blocks whose hashes the cache holds.  The paper does not say which hash.  The library's definition, restated
here independently in big-integer Python (all arithmetic mod 2^64):

  mix(z)   = the SplitMix64 output function (Steele, Lea and Flood, OOPSLA 2014):
             z += 0x9E3779B97F4A7C15;  z = (z ^ z>>30) * 0xBF58476D1CE4E5B9;
             z = (z ^ z>>27) * 0x94D049BB133111EB;  return z ^ z>>31
  local(k) = x after x = mix(x ^ (t[16k+2j] | t[16k+2j+1] << 32)) for j = 0..7, from x = 0
  h(-1) = seed;  h(k) = h(k-1) * 0x9E3779B97F4A7C15 + local(k);  hash(k) = mix(h(k))

Only full 16-token pages are hashed (sharing is block-granular).  Parity of the hash *values* is the
library's own convention ("parity unpinned" beyond the SplitMix64 reference outputs); what the hashes are
used for — a group's shared whole pages and a request's reusable prefix — is pinned by brute force over
the token ids in the CPU tests.
"""
from __future__ import annotations

M64 = (1 << 64) - 1
GAMMA = 0x9E3779B97F4A7C15
PAGE = 16


def mix(z: int) -> int:
    """SplitMix64 output function of a 64-bit value."""
    z = (z + GAMMA) & M64
    z = ((z ^ (z >> 30)) * 0xBF58476D1CE4E5B9) & M64
    z = ((z ^ (z >> 27)) * 0x94D049BB133111EB) & M64
    return z ^ (z >> 31)


def local_hash(tokens16) -> int:
    """Hash of one page's 16 token ids, folded pair by pair."""
    x = 0
    for j in range(8):
        a = int(tokens16[2 * j]) & 0xFFFFFFFF
        b = int(tokens16[2 * j + 1]) & 0xFFFFFFFF
        x = mix(x ^ (a | (b << 32)))
    return x


def block_hashes(tokens, seed: int = 0) -> list:
    """hash(k) for every full page k of one sequence's token ids."""
    out, h = [], seed & M64
    for k in range(len(tokens) // PAGE):
        h = (h * GAMMA + local_hash(tokens[PAGE * k:PAGE * (k + 1)])) & M64
        out.append(mix(h))
    return out


def group_shared_pages(member_hashes) -> int:
    """Leading pages on which every member's hash equals the first member's (0 without members)."""
    if not member_hashes:
        return 0
    n = min(len(h) for h in member_hashes)
    for k in range(n):
        if any(h[k] != member_hashes[0][k] for h in member_hashes[1:]):
            return k
    return n


class PrefixTable:
    """Block hash -> pool page; a hash's page is the largest inserted, None after that page is erased."""

    def __init__(self):
        self.d = {}

    @staticmethod
    def key(h: int) -> int:
        return h if h else 1

    def insert(self, hashes, pages):
        for h, p in zip(hashes, pages):
            k = self.key(int(h))
            cur = self.d.get(k)
            self.d[k] = int(p) if cur is None else max(cur, int(p))

    def erase(self, hashes, pages):
        for h, p in zip(hashes, pages):
            k = self.key(int(h))
            if self.d.get(k) == int(p):
                self.d[k] = -1

    def lookup(self, hashes):
        """(matched leading pages, their pages followed by -1 for the rest)."""
        pages = []
        for h in hashes:
            p = self.d.get(self.key(int(h)), -1)
            if p is None or p < 0:
                break
            pages.append(p)
        return len(pages), pages + [-1] * (len(hashes) - len(pages))
