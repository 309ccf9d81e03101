"""Oracle for the paged-KV block manager (Table 1, "KV manager").

Test infrastructure only (see ``oracle/__init__``).

The paper keeps the runtime's paged KV layout unchanged and allocates
blocks as each chunk is processed (Table 1).  It does not spell out an
allocation order, so this takes the following reading:

* blocks hold ``block_size`` (16) consecutive positions of one sequence;
* a sequence grows by whole blocks, always taking the lowest-numbered free
  block first;
* a reservation that the free pool cannot cover fails and changes nothing;
  a group of reservations made for one iteration is all-or-nothing, taken
  in the order given (the prefill sequences first, in the order their rows
  come, then the decodes in batch order);
* freeing a sequence returns all its blocks to the pool.

The slot of position p of a sequence is bt[p // bs] * bs + p % bs.
"""
from __future__ import annotations

import heapq


class OutOfBlocks(Exception):
    """The free pool cannot cover a reservation (state is unchanged)."""


class BlockManager:
    def __init__(self, num_blocks: int, block_size: int = 16):
        if num_blocks < 0 or block_size <= 0:
            raise ValueError("bad pool size")
        self.block_size = block_size
        self.num_blocks = num_blocks
        self._free = list(range(num_blocks))
        heapq.heapify(self._free)
        self._tables: dict[int, list[int]] = {}
        self._reserved: dict[int, int] = {}

    # -- sequences -----------------------------------------------------------
    def create(self, sid: int) -> None:
        if sid in self._tables:
            raise KeyError(f"sequence {sid} exists")
        self._tables[sid] = []
        self._reserved[sid] = 0

    def free(self, sid: int) -> None:
        for b in self._tables.pop(sid):
            heapq.heappush(self._free, b)
        del self._reserved[sid]

    def blocks_needed(self, sid: int, new_len: int) -> int:
        want = -(-max(new_len, self._reserved[sid]) // self.block_size)
        return max(0, want - len(self._tables[sid]))

    def reserve_many(self, requests) -> None:
        """Grow each (sid, new_len) in order; all-or-nothing."""
        for sid, _ in requests:
            if sid not in self._tables:
                raise KeyError(f"sequence {sid} unknown")
        total = 0
        seen = {}
        for sid, new_len in requests:
            # a sequence listed twice grows to the larger length once
            seen[sid] = max(seen.get(sid, 0), new_len)
        for sid, new_len in seen.items():
            total += self.blocks_needed(sid, new_len)
        if total > len(self._free):
            raise OutOfBlocks(f"need {total} blocks, {len(self._free)} free")
        done = set()
        for sid, _ in requests:
            if sid in done:
                continue
            done.add(sid)
            new_len = seen[sid]
            for _ in range(self.blocks_needed(sid, new_len)):
                self._tables[sid].append(heapq.heappop(self._free))
            self._reserved[sid] = max(self._reserved[sid], new_len)

    def reserve(self, sid: int, new_len: int) -> None:
        self.reserve_many([(sid, new_len)])

    # -- queries -------------------------------------------------------------
    def block_table(self, sid: int) -> list[int]:
        return list(self._tables[sid])

    def reserved(self, sid: int) -> int:
        return self._reserved[sid]

    def free_count(self) -> int:
        return len(self._free)

    def slot(self, sid: int, pos: int) -> int:
        bt = self._tables[sid]
        return bt[pos // self.block_size] * self.block_size + pos % self.block_size


def iteration_metadata(mgr: BlockManager, chunk: int, prefill_seq: int, prefix_len: int,
                       decode_seqs, context_lens, prefills=None):
    """Reservations and slot mapping of one mixed iteration.

    Reserves the prefill sequence up to prefix_len + chunk (if chunk > 0), or
    with prefill batching each (sequence, prefix, chunk) of ``prefills`` in
    turn up to prefix + chunk, then each decode b up to context_lens[b] + 1;
    returns the slot of every row (chunk rows first, in prefill order) and
    each participating sequence's block table.
    """
    if prefills is None:
        prefills = [(prefill_seq, prefix_len, chunk)]
    prefills = [(s, p, c) for s, p, c in prefills if c > 0]
    req = [(s, p + c) for s, p, c in prefills]
    req += [(s, L + 1) for s, L in zip(decode_seqs, context_lens)]
    mgr.reserve_many(req)
    slots = []
    for s, p, c in prefills:
        slots += [mgr.slot(s, p + j) for j in range(c)]
    slots += [mgr.slot(s, L) for s, L in zip(decode_seqs, context_lens)]
    tables = {}
    for s, _, _ in prefills:
        tables[s] = mgr.block_table(s)
    for s in decode_seqs:
        tables[s] = mgr.block_table(s)
    return slots, tables
