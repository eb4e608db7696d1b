"""Bounds of the MFMA attention kernel's cache reads, replayed on the CPU (no GPU, no oracle).

The kernel reads a (sequence, KV head) region of ld x HD bf16 elements per cache (ld = max_len
rounded up to 64), in 1 KB blocks (512 elements, 8 per lane): the loop's step loads and the L2
prefetch that each query block issues before its walk.  This replays the index arithmetic of
both for every query block, wave and kv_end in [1, ld] and checks that each block lies inside the
region; a prefetch that addressed the next step's blocks once read past the end of the V cache.
"""
import pytest

K_ATTN_WAVES = 8
K_PRE = 4


def kernel_reads(HD, kv_end, qblocks, qb, wave):
    """(cache, first element) of every 1 KB block the kernel reads for one wave of query block qb."""
    KK, DB = HD // 32, HD // 16
    k_blk = 2 * KK + DB
    out = []
    n_steps_all = (kv_end + 31) // 32
    for i in range(K_PRE):  # prefetch
        j = wave + K_ATTN_WAVES * i
        st = qb + qblocks * (j // k_blk)
        bi = j % k_blk
        stc = st if st < n_steps_all else 0
        if bi < 2 * KK:
            out.append(("K", stc * 32 * HD + bi * 512))
        else:
            out.append(("V", stc * 32 * HD + (bi - 2 * KK) * 512))
    k_stride = 32 * K_ATTN_WAVES
    p_last = (kv_end - 1) // 32 * 32
    n_steps = (kv_end - 32 * wave + k_stride - 1) // k_stride if kv_end > 32 * wave else 0
    t_end = n_steps
    p = 32 * wave - 2 * k_stride
    t = -2
    while t < t_end:  # loop loads (two steps per iteration)
        for pp in (min(p + 2 * k_stride, p_last), min(p + 3 * k_stride, p_last)):
            so = (pp // 32) * 32 * HD
            out += [("K", so + b * 512) for b in range(2 * KK)]
            out += [("V", so + db * 512) for db in range(DB)]
        t += 2
        p += 2 * k_stride
    return out


@pytest.mark.parametrize("HD,max_len,rows,grp", [(128, 50, 9, 4), (64, 64, 13, 4), (128, 64, 33, 8),
                                                  (128, 1100, 33, 8), (64, 200, 33, 4), (128, 4160, 33, 8)])
def test_attention_reads_stay_in_the_head_region(HD, max_len, rows, grp):
    ld = (max_len + 63) // 64 * 64
    extent = ld * HD
    qblocks = (rows * grp + 15) // 16
    ends = range(1, ld + 1) if ld <= 256 else list(range(1, 70)) + list(range(ld - 300, ld + 1))
    for kv_end in ends:
        for qb in range(qblocks):
            for wave in range(K_ATTN_WAVES):
                for cache, off in kernel_reads(HD, kv_end, qblocks, qb, wave):
                    assert 0 <= off and off + 512 <= extent, (cache, off, extent, kv_end, qb, wave)
