"""The LDS ring schedule of the ping-pong attention kernel, checked on the CPU.

The kernel streams K and V~ tiles into LDS rings with direct-to-LDS loads and
synchronises its eight waves with a workgroup barrier at the end of every
fourth phase only.  This test replays the schedule for every tile count up to 24,
every per-wave tile count (causal waves see fewer tiles than their
workgroup) and both wave groups, with and without the K pre-read, and checks
the two properties the ring needs:

* a tile is read only after the barrier that follows its landing wait;
* a slot is refilled only after every read of its previous tile has been
  consumed, in an earlier barrier interval.

Barrier interval k holds phases 4k .. 4k+3 (the barrier ends phase 4k+3);
waves in the same interval are unordered.
"""
import os
import re

import pytest

SRC = os.path.join(os.path.dirname(__file__), "..", "paper_2609_09721_amd", "csrc", "efq_attn.hip")

P = 4            # tiles streamed ahead
KEEP = P - 3     # batches left in flight at odd phases (the K pre-read is compiled in)
KRING, VRING = P + 2, P + 3
BAR = 4          # phases per barrier interval


def test_constants_match_kernel_source():
    src = open(SRC).read()
    assert re.search(r"#define EFQ_KPRE 1\b", src)
    assert re.search(r"#define EFQ_PREFETCH \(3 \+ EFQ_KPRE\)", src)
    assert "constexpr int kPPK = kPP + 2;" in src
    assert "constexpr int kPPV = kPP + 3;" in src
    assert "constexpr int kBarPhases = 4;" in src
    assert "constexpr int kKeep = kPP - 2 - (kKPre ? 1 : 0);" in src
    # every wave issues the same loads in every even phase (past the last
    # tile, the last tile again), so the landing wait is one constant
    assert "constexpr int keep = kKeep * kLoads;" in src
    assert "const int xt = x < ntiles ? x : ntiles - 1;" in src
    # the phase end with t % 4 known at compile time: wait at odd phases,
    # the barrier at phase 3 (mod 4) only
    end = src[src.index("  auto end = [&](auto tm) {"):]
    end = end[:end.index("\n  };")]
    assert "if constexpr (TM == 1 || TM == 3) {" in end
    assert "wait_vmem_le(keep);" in end
    assert "if constexpr (TM == 3) wg_barrier();" in end
    assert end.count("wg_barrier") == 1
    # the loop's phases: M(j), V(j), M(j+1), V(j+1) of group G at t = 2j + G
    # (j odd) .. 2j + 3 + G
    assert "constexpr int TA = (2 + G) & 3, TB = (3 + G) & 3, TC = G, TD = (1 + G) & 3;" in src
    # the empty phases after the wave's last tile, with t at run time
    tail = src[src.index("  for (int t = 2 * T + 1 + G; t < 2 * ntiles + 2; ++t) {"):]
    tail = tail[:tail.index("\n  }\n")]
    assert "wait_vmem_le(keep);" in tail
    assert "if ((t & 3) == 3) wg_barrier();" in tail


def landing_phase(x):
    """Odd phase at whose end every wave's load of tile x has completed."""
    if x < 2:
        return -1                       # resident before phase 0
    # the fifo at odd phase 2k+1 holds tiles k+2 .. k+P; all but the last
    # KEEP have landed, so tile x lands at k = x - P + KEEP
    return 2 * (x - P + KEEP) + 1


def interval(phase):
    return phase // BAR


def wave_reads(T, G, pre):
    """(slot kind, tile, read phase, consume phase) for one wave with T tiles."""
    reads = []
    for j in range(T):
        m = 2 * j + G                   # M(j)
        v = 2 * j + 1 + G               # V(j)
        reads.append(("K", j, m, m))
        reads.append(("V", j, v, v + 1))          # consumed by M(j+1) or F
        if pre and j + 1 < T:
            reads.append(("K", j + 1, v, v + 1))  # first operands of M(j+1)
    return reads


@pytest.mark.parametrize("pre", [False, True])
def test_ring_schedule_is_safe(pre):
    cases = 0
    for ntiles in range(1, 25):
        reads = []
        for T in range(1, ntiles + 1):
            for G in (0, 1):
                reads += wave_reads(T, G, pre)
        # every read happens after its tile's landing barrier
        for kind, x, t, c in reads:
            assert x < ntiles
            assert interval(landing_phase(x)) < interval(t) or landing_phase(x) < 0, (kind, x, t)
            cases += 1
        # every refill comes after the consumption of the slot's previous
        # tile; the even phases 2 .. 2 ntiles stream tiles P+1 .. ntiles+P,
        # those past the end as copies of the last tile into their own slots
        for x in range(P + 1, ntiles + P + 1):
            issue = 2 * (x - P)
            for kind, ring in (("K", KRING), ("V", VRING)):
                old = x - ring
                if old < 0:
                    continue
                last = max((c for k, y, t, c in reads if k == kind and y == old), default=-1)
                assert interval(last) < interval(issue), (kind, x, old, last, issue)
        # every wave runs 2 ntiles + 2 phases, so all pass the same barriers
        phases = 2 * ntiles + 2
        assert sum(1 for t in range(phases) if t % BAR == BAR - 1) == phases // BAR
    assert cases > 1000
