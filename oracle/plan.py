"""Oracle: SuperBatch aggregation (Alg. 1) over partition-grouped texts.

TEST INFRASTRUCTURE ONLY (see the package docstring).

Alg. 1 streams (key, text) pairs ordered by key; each key change hands the
finished partition to AddPartition, which appends it to the buffer, adds its
size to the running total and flushes when the total reaches the upper
threshold (memory-safety trigger) or the lower threshold B_min (efficiency
trigger).  Flush concatenates the buffered partitions, records one
(start, end, key) bound per partition, encodes once and slices per bound.
The final partition is added and flushed at the end of the stream.

Here the stream is given in CSR form: ``part_offsets[p] .. part_offsets[p+1]``
are the global indices of partition p's texts, partitions in arrival order.
A partition with no texts never appears in a (key, text) stream, so it never
reaches AddPartition and produces no bound.  A flush of an empty buffer
encodes nothing and produces no SuperBatch.

The paper is not consistent about the upper threshold, so two readings are
provided:

* ``R1`` (literal Alg. 1): append, then flush if total >= B_max or
  total >= B_min.  With B_max >= B_min both branches flush, so only B_min
  matters; partitions are never split.
* ``R2`` (the prose of Sec. 3.2 and the operational note of Sec. 6): the
  upper threshold ``cap`` is a pre-append safety flush - if the buffer is not
  empty and adding the arriving partition would take the total past ``cap``,
  flush first; a partition larger than ``cap`` is split into cap-sized
  chunks, each its own SuperBatch, and its remainder is appended like any
  other partition; then flush if total >= B_min.  Every SuperBatch then holds
  at most ``cap`` texts.  ``cap <= 0`` means no cap (R2 then equals R1).

Each SuperBatch is reported as its global text range and its bounds
(segments): (first_text, count, partition, row_offset), where row_offset is
the row of ``first_text`` inside its partition (non-zero only for the later
chunks of a split partition).
"""
from __future__ import annotations

import dataclasses
from typing import List, Sequence, Tuple

R2 = 0
R1 = 1


@dataclasses.dataclass(frozen=True)
class Segment:
    first_text: int
    count: int
    partition: int
    row_offset: int


@dataclasses.dataclass
class SuperBatch:
    text_begin: int
    text_end: int
    segments: List[Segment]

    @property
    def n_texts(self) -> int:
        return self.text_end - self.text_begin


class _Aggregator:
    """Alg. 1's state: the buffered bounds and the running total."""

    def __init__(self):
        self.buffer: List[Segment] = []
        self.total = 0
        self.out: List[SuperBatch] = []

    def append(self, seg: Segment):
        self.buffer.append(seg)
        self.total += seg.count

    def flush(self):
        if not self.buffer:
            return
        begin = self.buffer[0].first_text
        end = self.buffer[-1].first_text + self.buffer[-1].count
        self.out.append(SuperBatch(begin, end, list(self.buffer)))
        self.buffer = []
        self.total = 0


def plan(part_offsets: Sequence[int], b_min: int, cap: int = 0,
         policy: int = R2) -> List[SuperBatch]:
    """SuperBatches of a partition-grouped input.

    ``b_min`` is the efficiency trigger (>= 1); ``cap`` is the upper threshold
    (B_max, or the per-SuperBatch text cap); ``cap <= 0`` disables it.
    """
    if b_min < 1:
        raise ValueError("b_min must be >= 1")
    agg = _Aggregator()
    n_parts = len(part_offsets) - 1
    for p in range(n_parts):
        start = int(part_offsets[p])
        n = int(part_offsets[p + 1]) - start
        if n < 0:
            raise ValueError("part_offsets must be non-decreasing")
        if n == 0:
            continue
        if policy == R1:
            agg.append(Segment(start, n, p, 0))
            if cap > 0 and agg.total >= cap:
                agg.flush()
            elif agg.total >= b_min:
                agg.flush()
        elif policy == R2:
            if cap > 0 and agg.total > 0 and agg.total + n > cap:
                agg.flush()
            row = 0
            while cap > 0 and n - row > cap:
                agg.append(Segment(start + row, cap, p, row))
                agg.flush()
                row += cap
            agg.append(Segment(start + row, n - row, p, row))
            if agg.total >= b_min:
                agg.flush()
        else:
            raise ValueError(f"unknown policy {policy}")
    agg.flush()
    return agg.out


def flatten(sbs: List[SuperBatch]) -> Tuple[List[Tuple[int, int, int, int]],
                                            List[Tuple[int, int, int, int]]]:
    """The plan as plain tuples: superbatches (text_begin, text_end, seg_begin,
    seg_end) and segments (first_text, count, partition, row_offset)."""
    sb_rows, seg_rows = [], []
    for sb in sbs:
        s0 = len(seg_rows)
        for s in sb.segments:
            seg_rows.append((s.first_text, s.count, s.partition, s.row_offset))
        sb_rows.append((sb.text_begin, sb.text_end, s0, len(seg_rows)))
    return sb_rows, seg_rows


# --- Cost model (Sec. 2.3 and Theorem 1) ---------------------------------
#
# A call that encodes n texts on G GPUs costs c_call + n c_enc / G: a fixed
# per-call overhead plus a per-text cost shared by the GPUs.  A plan with F
# calls over N texts therefore takes F c_call + N c_enc / G.

def call_time(n_texts: int, c_call: float, c_enc: float, n_gpus: int = 1) -> float:
    """Time of one encode call of n_texts texts (Sec. 2.3)."""
    return c_call + n_texts * c_enc / n_gpus


def plan_time(call_sizes: Sequence[int], c_call: float, c_enc: float, n_gpus: int = 1) -> float:
    """Sum of the call times of a plan."""
    return float(sum(call_time(n, c_call, c_enc, n_gpus) for n in call_sizes))


def ipc_alpha(n_parts: int, c_call: float, n_texts: int, c_enc: float, n_gpus: int = 1) -> float:
    """Theorem 1's IPC-to-compute ratio of one-call-per-partition processing."""
    return n_parts * c_call / (n_texts * c_enc / n_gpus)


def ipc_speedup(alpha: float, n_flushes: int, n_parts: int) -> float:
    """Theorem 1: T_PBP / T_SURGE when PBP makes n_parts calls and SURGE
    n_flushes calls over the same texts."""
    return (1.0 + alpha) / (1.0 + alpha * n_flushes / n_parts)


def ipc_threshold(c_call: float, c_enc: float, n_gpus: int = 1) -> float:
    """n*: partitions smaller than this spend more time on the fixed call
    overhead than on encoding (Sec. 2.3)."""
    return c_call * n_gpus / c_enc


# --- PB-PBP-LB baseline (Sec. 5.x "stronger baseline") --------------------
#
# Partition sizes are known up front; partitions are taken largest first
# (ties: lower index first) and each goes into the first open batch whose
# remaining capacity holds it, else into a new batch.  Partitions are never
# split, so a partition larger than the capacity forms a batch of its own.

def ffd_pack(part_sizes: Sequence[int], capacity: int) -> List[List[int]]:
    """First-Fit-Decreasing batches (lists of partition indices, in packing
    order) of the non-empty partitions."""
    if capacity < 1:
        raise ValueError("capacity must be >= 1")
    order = sorted((p for p, n in enumerate(part_sizes) if n > 0),
                   key=lambda p: (-part_sizes[p], p))
    bins: List[List[int]] = []
    load: List[int] = []
    for p in order:
        n = part_sizes[p]
        for b in range(len(bins)):
            if load[b] + n <= capacity:
                bins[b].append(p)
                load[b] += n
                break
        else:
            bins.append([p])
            load.append(n)
    return bins


def superbatch_memory(n_texts: int, mean_text_bytes: float, d: int) -> float:
    """Lemma 1 (Sec. 4.3, "SuperBatch memory"): the data-resident size of a
    SuperBatch of S texts of average size L bytes with fp32 embeddings of
    width d is M(S) = S L + 4 S d bytes (the raw texts plus the [S, d]
    embedding matrix)."""
    return n_texts * mean_text_bytes + 4 * n_texts * d


def device_superbatch_memory(n_texts: int, n_tokens: int, d: int) -> int:
    """Lemma 1's M(S) for a SuperBatch held on the device as packed int32
    token IDs: the text part is 4 bytes per token, i.e. L = 4 n_tokens / S."""
    return 4 * n_tokens + 4 * n_texts * d


def largest_superbatch_bound(b_min: int, n_big: int, cap: int = 0, policy: int = R2) -> int:
    """Lemma 1's bound on the texts of one SuperBatch: the buffer holds less
    than B_min texts before the arriving partition (at most n_max texts) is
    appended, so S <= B_min - 1 + n_max; with the pre-append cap of the R2
    reading every SuperBatch also holds at most ``cap`` texts."""
    bound = b_min - 1 + n_big
    if policy == R2 and cap > 0:
        bound = min(bound, cap)
    return bound
