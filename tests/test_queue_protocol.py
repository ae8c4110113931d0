"""The attention launch's two-queue work protocol, modelled on the host: G
persistent workgroups, two atomic counters (chunk items, decode items) and a
count of finished workgroups.  Workgroups below `first` start on the decode
queue, the others on the chunk queue; a workgroup whose queue is empty tries
the other one once, and leaves when both are.  Under random interleavings of
the atomic operations every item is taken exactly once, every workgroup
leaves, and the last one to leave finds every other workgroup's atomics done
and zeroes the counters (the kernel's loop in attention_kernel)."""
import numpy as np
import pytest


def run_protocol(G, n_chunk, n_dec, first, rng):
    work = [0, 0, 0]  # next chunk item, workgroups done, next decode item
    taken = []
    # each workgroup is a generator yielding before each atomic operation
    def wg(b):
        on_dec = b < first
        while True:
            it = -1
            for _ in range(2):
                yield
                if on_dec:
                    d = work[2]; work[2] += 1
                    if d < n_dec:
                        it = n_chunk + d
                else:
                    c = work[0]; work[0] += 1
                    if c < n_chunk:
                        it = c
                if it >= 0:
                    break
                on_dec = not on_dec
            if it < 0:
                break
            taken.append((b, it))
        yield
        done = work[1]; work[1] += 1
        if done == G - 1:
            work[0] = work[1] = work[2] = 0
    live = {b: wg(b) for b in range(G)}
    steps = 0
    while live:
        b = list(live)[rng.integers(len(live))]
        try:
            next(live[b])
        except StopIteration:
            del live[b]
        steps += 1
        assert steps < 100 * (G + n_chunk + n_dec) + 1000, "a workgroup never leaves"
    return taken, work


@pytest.mark.parametrize("seed", range(40))
def test_every_item_once_and_counters_zeroed(seed):
    rng = np.random.default_rng(seed)
    G = int(rng.integers(1, 12))
    n_chunk, n_dec = int(rng.integers(0, 30)), int(rng.integers(0, 30))
    first = int(rng.integers(0, G + 1))
    taken, work = run_protocol(G, n_chunk, n_dec, first, rng)
    items = sorted(it for _, it in taken)
    assert items == list(range(n_chunk + n_dec))
    assert work == [0, 0, 0]


def test_decode_first_workgroups_start_on_decode():
    # with items to spare, each decode-first workgroup's first item is a decode item
    rng = np.random.default_rng(5)
    taken, _ = run_protocol(6, 40, 40, 3, rng)
    first_item = {}
    for b, it in taken:
        first_item.setdefault(b, it)
    assert all((first_item[b] >= 40) == (b < 3) for b in first_item)
