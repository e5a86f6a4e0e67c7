"""Reads of the caller's code array by the tiled FC path's code re-layout
(fc_codes_kernel in csrc/fc_tiled.hip), modelled on the CPU.

The re-layout runs on a grid that rounds the subspace groups up to whole
phases (mgroups dwords per channel) and the channels up to whole channel
blocks (ct_pad), so some of its threads stand past the last code.  This test
copies the planner's candidate layouts (every (lanes per channel, subspaces
per phase) pair the planner may pick, whatever its cost model prefers) and
the kernel's address arithmetic for its three read paths (aligned byte codes,
unaligned byte codes, packed bit stream), enumerates every thread of the
grid, and checks that every dword read lies within the code stream: byte
codes C_t M bytes (a dword read may only be the one holding the last byte),
packed codes qcnn_packed_bytes = 4 ceil(C_t M b / 32) bytes.  The same model
with the guard on the group index removed must fail on the ragged shapes, so
the check would have caught that mistake.
"""
import math

import numpy as np
import pytest

WAVE, WAVES, NI, LDS_BYTES = 64, 16, 8, 160 * 1024


def code_bits(K):
    b = 0
    while (1 << b) < K:
        b += 1
    return b


def candidate_layouts(N, Cs, M, K, Csp, Ct):
    """(mgroups, ct_pad) of every layout the FC planner accepts."""
    if K > 64 or Csp > 8:
        return []
    out = []
    for LPC in (16, 32):
        for MC in (4, 8):
            NS = 4 * LPC
            if LPC == 32 and (K > 32 or N <= 64):
                continue
            KP = (K + 15) // 16 * 16
            nphases = math.ceil(M / MC)
            mgroups = nphases * (MC // 4)
            lds = 2 * MC * KP * NS * 4
            if lds > LDS_BYTES or (MC == 8 and (LPC != 16 or KP > 32)):
                continue
            tc = WAVES * NI * (WAVE // LPC)
            ct_pad = math.ceil(Ct / tc) * tc
            out.append((mgroups, ct_pad))
    return out


def dwords_read(Ct, M, bits, mgroups, ct_pad, guard=True):
    """Every dword index of the code stream one launch reads."""
    gq = np.arange(math.ceil(mgroups / 64) * 64, dtype=np.int64)[:, None]
    t = np.arange(math.ceil(ct_pad / 64) * 64, dtype=np.int64)[None, :]
    has = (gq < mgroups) & (t < Ct)
    if guard:
        has &= 4 * gq < M
    gq, t = np.broadcast_arrays(gq, t)
    gq, t = gq[has], t[has]
    if bits == 8 and M % 4 == 0:               # one dword per group
        return (t * M + 4 * gq) // 4
    if bits == 8:                              # code_at on each byte of the group
        reads = []
        for k in range(4):
            sel = 4 * gq + k < M
            reads.append((t[sel] * M + 4 * gq[sel] + k) >> 2)
        return np.concatenate(reads)
    if bits == 0:                              # K = 1: nothing is read
        return np.zeros(0, np.int64)
    n = np.minimum(4, M - 4 * gq)              # a 64-bit window over the group's bits
    n = np.maximum(n, 1)                       # (only the unguarded model reaches n <= 0)
    bit = (t * M + 4 * gq) * bits
    first = bit >> 5
    second = first[(bit & 31) + n * bits > 32] + 1
    return np.concatenate([first, second])


def stream_dwords(Ct, M, bits):
    if bits == 8:
        return math.ceil(Ct * M / 4)           # the dword holding the last byte ends the reads
    return math.ceil(Ct * M * bits / 32)       # qcnn_packed_bytes / 4


# (N, C_s, C_t, C'_s, K): the FC parity edge shapes and packed-code shapes,
# then M = 12 and M = 100 (K <= 32), where whole phases overshoot M.
SHAPES = [
    (1, 64, 10, 4, 32), (65, 96, 257, 4, 32), (130, 300, 1000, 3, 16), (64, 4096, 1000, 4, 32),
    (7, 48, 33, 1, 16), (3, 10, 5, 5, 1), (96, 640, 300, 8, 64), (200, 192, 70, 4, 48), (128, 68, 40, 4, 32),
    (64, 9216 // 4, 512, 4, 32), (64, 4096, 1000, 1, 16), (5, 64, 33, 4, 1), (130, 512, 257, 8, 61),
    (64, 48, 70, 4, 32), (130, 96, 1000, 8, 32), (65, 36, 129, 3, 7),
    (64, 400, 33, 4, 16), (65, 100, 257, 1, 8), (200, 300, 64, 3, 32), (1, 800, 5, 8, 2),
]


@pytest.mark.parametrize("shape", SHAPES, ids=[str(s) for s in SHAPES])
def test_code_reads_stay_in_stream(shape):
    N, Cs, Ct, Csp, K = shape
    M = Cs // Csp
    layouts = candidate_layouts(N, Cs, M, K, Csp, Ct)
    assert layouts, shape
    for bits in sorted({8, code_bits(K)}):
        for mgroups, ct_pad in layouts:
            d = dwords_read(Ct, M, bits, mgroups, ct_pad)
            limit = stream_dwords(Ct, M, bits)
            assert d.size == 0 or (d.min() >= 0 and d.max() < limit), (shape, bits, mgroups, ct_pad, d.max(), limit)


@pytest.mark.parametrize("shape", [(64, 48, 70, 4, 32), (64, 400, 33, 4, 16), (130, 96, 1000, 8, 32)])
def test_unguarded_groups_would_read_past_the_stream(shape):
    # Without the guard on 4 gq < M, the groups that round M up to a whole
    # phase read past the end for the last channel.
    N, Cs, Ct, Csp, K = shape
    M = Cs // Csp
    over = False
    for bits in (8, code_bits(K)):
        for mgroups, ct_pad in candidate_layouts(N, Cs, M, K, Csp, Ct):
            if mgroups * 4 > M:
                d = dwords_read(Ct, M, bits, mgroups, ct_pad, guard=False)
                over |= bool(d.max() >= stream_dwords(Ct, M, bits))
    assert over, shape
