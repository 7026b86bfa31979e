"""CPU replay of the head-dimension-128 key/value staging of the FP8 attention kernel.

At D = 128 each key block (128 keys) is copied from global memory into LDS by
global_load_lds_dwordx4: lane l of wave instruction j writes LDS bytes
[1024 j + 16 l, +16), and the 16-byte chunk c of LDS row r holds logical chunk
c ^ swz(r) (swz(r) = (r >> 1) & 7 for 128-byte K rows, (r >> 2) & 3 for 64-byte
rows of the tile-transposed V).  This replays, for 4 and 8 waves, the index
math that assigns the copies (the piece j of wave w is w + W i) and checks that
every LDS byte of a stage is written exactly once, from inside the source
tensor, and that the operand reads (chunk c of row r at r * RB + ((c ^ swz(r))
<< 4)) return the bytes of logical chunk c.  Keys past N read row N - 1 and
64-key tiles past the end read the last tile (their scores are masked)."""
import numpy as np
import pytest

D, BKV = 128, 128
NP = BKV // 64


def swz(rb, r):
    return (r >> 1) & 7 if rb == 128 else (r >> 2) & 3


def replay(W, N, kb):
    kpieces, vpieces = BKV * D // 1024, NP * D * 64 // 1024
    assert kpieces % W == 0 and vpieces % W == 0
    ntiles64 = (N + 63) // 64
    kmem = np.arange(N * D) % 251
    vmem = np.arange(ntiles64 * D * 64) % 241
    klds = np.full(BKV * D, -1)
    vlds = np.full(NP * D * 64, -1)
    for wave in range(W):
        for lane in range(64):
            for i in range(kpieces // W):
                j = wave + W * i
                at = j * 1024 + lane * 16
                r, pos = at // D, (at % D) >> 4
                key = min(kb * BKV + r, N - 1)
                g = key * D + ((pos ^ swz(128, r)) << 4)
                assert 0 <= g and g + 16 <= N * D
                assert (klds[at:at + 16] == -1).all()
                klds[at:at + 16] = kmem[g:g + 16]
            for i in range(vpieces // W):
                j = wave + W * i
                at = j * 1024 + lane * 16
                r, pos = at // 64, (at % 64) >> 4
                t64 = min(kb * NP + r // D, ntiles64 - 1)
                g = t64 * D * 64 + (r % D) * 64 + ((pos ^ swz(64, r)) << 4)
                assert 0 <= g and g + 16 <= ntiles64 * D * 64
                assert (vlds[at:at + 16] == -1).all()
                vlds[at:at + 16] = vmem[g:g + 16]
    assert (klds >= 0).all() and (vlds >= 0).all()
    for r in range(BKV):
        key = min(kb * BKV + r, N - 1)
        for c in range(D // 16):
            off = r * D + ((c ^ swz(128, r)) << 4)
            assert (klds[off:off + 16] == kmem[key * D + c * 16:key * D + c * 16 + 16]).all()
    for r in range(NP * D):
        t64 = min(kb * NP + r // D, ntiles64 - 1)
        for c in range(4):
            off = r * 64 + ((c ^ swz(64, r)) << 4)
            src = t64 * D * 64 + (r % D) * 64 + c * 16
            assert (vlds[off:off + 16] == vmem[src:src + 16]).all()


@pytest.mark.parametrize("W", [4, 8])
@pytest.mark.parametrize("N,kb", [(65536, 0), (65536, 511), (300, 2), (129, 1), (1, 0)])
def test_staging_writes_every_lds_byte_once_and_reads_the_right_bytes(W, N, kb):
    replay(W, N, kb)
