"""Reference model of the window-safe prefix cache (the oracle).

TEST INFRASTRUCTURE ONLY: only tests, the smoke check and the benchmark's CPU
baseline may use this module.

Source in the paper: "SWA-Aware Prefix Cache Tree". Token equality alone no
longer implies reusable KV under SWA; a hit additionally needs the tail W
tokens to hold valid SWA slots and the match length is clipped to that
boundary (window-safe length); nodes carry dual indices (the Full Attention
segment and the SWA segment); out-of-window SWA segments can be evicted on
their own while the Full Attention segments stay, or whole segments go.

The model stores, for every cached token prefix (a tuple of token ids), the
FULL slot and the SWA slot of its last token. No tree structure is modelled.

Readings where the paper is silent:
  * A prefix of length P can be reused when all its FULL slots are held and
    the W - 1 positions before P (the keys the first new query at position P
    reads from the SWA pool, W counting the query itself) hold SWA slots.
  * Re-inserting a cached position replaces its slots.
  * Evicting at position k removes that position of the path and every cached
    continuation of it.
"""

from __future__ import annotations


class PrefixModel:
    def __init__(self, window):
        self.w = int(window)
        self.d = {}  # tuple(tokens[:i + 1]) -> [full_slot, swa_slot]

    def insert(self, tokens, full, swa):
        tokens = [int(t) for t in tokens]
        for i in range(len(tokens)):
            self.d[tuple(tokens[:i + 1])] = [int(full[i]), int(swa[i])]

    def match(self, tokens):
        tokens = [int(t) for t in tokens]
        n = 0
        while n < len(tokens) and tuple(tokens[:n + 1]) in self.d and self.d[tuple(tokens[:n + 1])][0] >= 0:
            n += 1
        slots = [self.d[tuple(tokens[:i + 1])] for i in range(n)]
        swa_ok = [s[1] >= 0 for s in slots]
        safe = 0
        for p in range(n, 0, -1):
            if all(swa_ok[j] for j in range(max(0, p - self.w + 1), p)):
                safe = p
                break
        return n, safe, [s[0] for s in slots], [s[1] for s in slots]

    def release_swa(self, tokens, upto):
        tokens = [int(t) for t in tokens]
        cnt = 0
        for i in range(min(int(upto), len(tokens))):
            key = tuple(tokens[:i + 1])
            if key not in self.d:
                break
            if self.d[key][1] >= 0:
                self.d[key][1] = -1
                cnt += 1
        return cnt

    def evict(self, tokens, keep):
        tokens = [int(t) for t in tokens]
        if keep >= len(tokens):
            return 0
        head = tuple(tokens[:keep + 1])
        gone = [k for k in self.d if len(k) > keep and k[:keep + 1] == head]
        for k in gone:
            del self.d[k]
        return len(gone)

    def stats(self):
        return len(self.d), sum(1 for v in self.d.values() if v[1] >= 0)
