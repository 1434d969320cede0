"""Reference model of the explicit-release dual-pool allocator (the oracle).

TEST INFRASTRUCTURE ONLY: only tests, the smoke check and the benchmark's CPU
baseline may use this module.

Sources in the paper: "KVCache Dual-Pool Design" (separate FULL and SWA
pools; the SWA pool is sized for the window and evicts by window; admission
validates both capacities; the FULL index is authoritative with a FULL -> SWA
mapping) and "SWA-Aware Prefix Cache Tree" (out-of-window SWA release at chunk
completion, at request termination and every N generated tokens; SWA usage
stays at window or chunk magnitude).

The model tracks positions, not physical page ids: which positions of each
sequence the SWA pool stores, and below which position everything has been
released. A page is held while it contains a stored position that has not
been released. Physical ids are not modelled: any assignment is correct as
long as no page is held twice (the tests check that separately).

Readings where the paper is silent:
  * Logical page i of a sequence covers positions i*PG .. i*PG+PG-1 in both
    pools (the FULL index is the mapping key).
  * Growing a sequence from L to L' stores in the SWA pool only the new
    positions that a query still reads from the pool: the query at L' - 1 (a
    decode step appends its token and reads it back) needs keys from L' - W
    on and the next query (at L') from L' - W + 1, so [max(L, L' - W), L') is
    stored; a prefill chunk reads its own earlier keys from its inputs.
  * A release frees every SWA page that lies wholly before L - W + 1 (the
    first key of the next query's window). Prefill chunk ends always release;
    decode steps release on every N-th step.
  * Admission needs ceil(L / PG) free FULL pages and ceil(min(L, W+C) / PG)
    + 1 free SWA pages (the window plus one chunk of C tokens) and reserves
    nothing.
"""

from __future__ import annotations

OK, INVALID, CAPACITY = 0, -1, -3


def _ceil(a, b):
    return -(-a // b)


class DualPoolModel:
    def __init__(self, page_size, window, full_pages, swa_pages, max_seqs, table_stride, release_every):
        self.pg, self.w = int(page_size), int(window)
        self.full_cap, self.swa_cap = int(full_pages), int(swa_pages)
        self.max_seqs, self.stride, self.n = int(max_seqs), int(table_stride), int(release_every)
        self.seqs = {}

    # -- derived quantities -------------------------------------------------
    def full_pages_of(self, seq):
        return _ceil(self.seqs[seq]["len"], self.pg)

    def swa_pages_of(self, seq):
        """Logical pages held in the SWA pool by one sequence."""
        s = self.seqs[seq]
        return {pos // self.pg for pos in s["stored"] if pos >= s["released_below"]}

    def full_free(self):
        return self.full_cap - sum(self.full_pages_of(b) for b in self.seqs)

    def swa_free(self):
        return self.swa_cap - sum(len(self.swa_pages_of(b)) for b in self.seqs)

    # -- operations -------------------------------------------------------------
    def admit(self, seq, length, chunk):
        if not (0 <= seq < self.max_seqs) or length < 0 or chunk < 1 or seq in self.seqs:
            return INVALID
        full_need = _ceil(length, self.pg)
        swa_need = 0 if length == 0 else _ceil(min(length, self.w + chunk), self.pg) + 1
        if full_need > self.stride or full_need > self.full_free() or swa_need > self.swa_free():
            return CAPACITY
        self.seqs[seq] = {"len": 0, "stored": set(), "released_below": 0, "steps": 0}
        return OK

    def extend(self, seq, new_len):
        if seq not in self.seqs:
            return INVALID
        s = self.seqs[seq]
        if new_len < s["len"]:
            return INVALID
        if new_len == s["len"]:
            return OK
        if _ceil(new_len, self.pg) > self.stride:
            return CAPACITY
        new_stored = set(range(max(s["len"], new_len - self.w), new_len))
        held = self.swa_pages_of(seq)
        extra_swa = {p // self.pg for p in new_stored} - held
        extra_full = _ceil(new_len, self.pg) - self.full_pages_of(seq)
        if extra_full > self.full_free() or len(extra_swa) > self.swa_free():
            return CAPACITY
        s["stored"] |= new_stored
        s["len"] = new_len
        return OK

    def step_end(self, seq, decode_step):
        if seq not in self.seqs:
            return INVALID, 0
        s = self.seqs[seq]
        if decode_step:
            s["steps"] += 1
            if s["steps"] < self.n:
                return OK, 0
        s["steps"] = 0
        before = len(self.swa_pages_of(seq))
        bound = s["len"] - self.w + 1
        # everything wholly before the next query's window goes back
        whole_pages_below = max(bound, 0) // self.pg * self.pg
        s["released_below"] = max(s["released_below"], whole_pages_below)
        s["stored"] = {p for p in s["stored"] if p >= s["released_below"]}
        return OK, before - len(self.swa_pages_of(seq))

    def free(self, seq):
        if seq not in self.seqs:
            return INVALID
        del self.seqs[seq]
        return OK
