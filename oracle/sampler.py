"""Worker shards and mini-batch sample indices.

The paper states only that each worker holds different training data
(Introduction, parameter-server description) and that a worker runs SGD with a
fixed mini-batch size (Related Works, Local SGD).  Reading used here:

* worker k owns the contiguous rows [off_k, off_{k+1}) with
  off_k = floor(k * N / K);
* a worker samples without replacement, epoch by epoch; the position in the
  epoch persists across rounds; a batch that crosses an epoch boundary takes
  the tail of epoch e and then the head of epoch e + 1;
* the epoch-e order of worker k is a Durstenfeld (Fisher-Yates) shuffle of
  0..n_k-1: for i = n_k-1 down to 1, j = r mod (i + 1), swap a[i], a[j], with
  r drawn from SplitMix64 (Steele, Lea and Flood, OOPSLA 2014) whose state
  starts at seed XOR (k << 32 | e).

Pinned by tests against the published SplitMix64 test vectors, the
permutation property of every epoch, the closed form of the n = 2 shuffle and
the uniformity of the n = 3 shuffle over many seeds.
"""
from __future__ import annotations

from typing import Dict, List, Sequence, Tuple

_MASK64 = (1 << 64) - 1
_GOLDEN_GAMMA = 0x9E3779B97F4A7C15


class SplitMix64:
    """SplitMix64: state advances by the golden gamma, output is the state
    passed through the variant-13 finaliser (shifts 30/27/31)."""

    def __init__(self, state: int):
        self.state = state & _MASK64

    def next(self) -> int:
        self.state = (self.state + _GOLDEN_GAMMA) & _MASK64
        z = self.state
        z = ((z ^ (z >> 30)) * 0xBF58476D1CE4E5B9) & _MASK64
        z = ((z ^ (z >> 27)) * 0x94D049BB133111EB) & _MASK64
        return z ^ (z >> 31)


def shard_offsets(n_rows: int, K: int) -> List[int]:
    """off_k = floor(k * n_rows / K), k = 0..K (exact integer arithmetic)."""
    if K < 1 or n_rows < 0:
        raise ValueError("K >= 1 and n_rows >= 0 required")
    return [k * n_rows // K for k in range(K + 1)]


def epoch_permutation(seed: int, k: int, e: int, n_k: int) -> List[int]:
    """Visiting order of worker k's shard in epoch e."""
    rng = SplitMix64((seed ^ ((k << 32) | e)) & _MASK64)
    a = list(range(n_k))
    for i in range(n_k - 1, 0, -1):
        j = rng.next() % (i + 1)
        a[i], a[j] = a[j], a[i]
    return a


def batch_rows(seed: int, offsets: Sequence[int], k: int, step: int, B: int,
               _cache: Dict[Tuple[int, int, int, int], List[int]] = None) -> List[int]:
    """Global dataset rows of worker k's mini-batch number ``step`` (counted
    from the worker's first step ever).  Position p = step * B + b of the
    worker's sample stream lies in epoch p // n_k at offset p mod n_k."""
    n_k = offsets[k + 1] - offsets[k]
    if n_k < 1:
        raise ValueError(f"worker {k} has an empty shard")
    rows = []
    for b in range(B):
        p = step * B + b
        e, o = divmod(p, n_k)
        key = (seed, k, e, n_k)
        if _cache is not None and key in _cache:
            perm = _cache[key]
        else:
            perm = epoch_permutation(seed, k, e, n_k)
            if _cache is not None:
                _cache[key] = perm
        rows.append(offsets[k] + perm[o])
    return rows
