"""Host model of the decode kernel's buffer windows (no GPU).

The decode kernel reads each tile's cache rows through a raw buffer resource
whose base is the tile's first row and whose record count ends at the key
range's last row; the lane's whole offset is the vector operand, which is what
the hardware compares with the record count (the scalar offset is not part of
that check, so the kernel passes 0 there). A load whose offset is at or past
the count returns zeros and touches no memory.

This model replays, for every split, wave and tile (including the prefetch of
the next tile, clamped to the last), the offsets each lane uses for every
stream, and checks at ragged T = t_cap (the tightest legal cache) that:
* every performed access lies inside the sequence's rows [0, t_cap);
* a multi-byte load is either wholly in range or wholly out;
* every key below the range's end is read (none is dropped by the window).
The formulas mirror those of decode_kernel.hpp (load_keys_buf, load_values_buf).
"""
import pytest

TILE = 256          # keys per workgroup tile
WTILE = 64          # keys per wave tile
WAVES = 4


def plan(T, S):
    tiles = (T + TILE - 1) // TILE
    S = max(1, min(S, tiles))
    split_len = (tiles + S - 1) // S * TILE
    return (T + split_len - 1) // split_len, split_len


def streams(mant_bits, v8):
    """(name, row bytes, limit kind, [(offset(lane), size)])."""
    K = mant_bits
    out = [("codes", 32, "t", [(lambda l: l * 32, 16), (lambda l: l * 32 + 16, 16)]),
           ("scales", 4, "t", [(lambda l: l * 4, 4)])]
    if K:
        out.append(("planes", 8 * K, "t",
                    [(lambda l, b=b: l * 8 * K + 8 * b, 8) for b in range(K)]))
    gb = 8 * 64 if v8 else 16 * 64           # bytes of one 8-token group
    frag = 8 if v8 else 16
    vl = []
    for kb in range(2):
        for nb in range(4):
            vl.append((lambda l, kb=kb, nb=nb: (l >> 4) * gb + (l & 15) * frag
                       + kb * 4 * gb + nb * 16 * frag, frag))
    out.append(("values", gb // 8, "v", vl))
    if v8:
        out.append(("exps", 1, "v", [(lambda l: 32 * ((l & 15) >> 3) + 8 * (l >> 4), 8)]))
    return out


def check(T, t_cap, S, mant_bits, v8):
    n_splits, split_len = plan(T, S)
    for split in range(n_splits):
        t_begin = split * split_len
        t_end = min(T, t_begin + split_len)
        v_end = ((t_end - 1) & ~7) + 8
        assert v_end <= t_cap                 # t_cap is a multiple of 8
        n_tiles = (t_end - t_begin + WTILE - 1) // WTILE
        for name, rb, kind, loads in streams(mant_bits, v8):
            lim = t_end if kind == "t" else v_end
            covered = set()
            for wave in range(WAVES):
                js = list(range(wave, n_tiles, WAVES))
                js += [min(j + WAVES, n_tiles - 1) for j in js]      # prefetches
                for j in js:
                    t0 = t_begin + WTILE * j
                    assert t0 < lim
                    base, n_rec = t0 * rb, (lim - t0) * rb
                    for lane in range(64):
                        for off, size in loads:
                            o = off(lane)
                            if o >= n_rec:
                                continue              # returns zeros, no access
                            assert o + size <= n_rec, (name, lane, o, size, n_rec)
                            lo, hi = base + o, base + o + size
                            assert 0 <= lo and hi <= t_cap * rb, (name, lo, hi)
                            covered.update(range(lo // rb, (hi - 1) // rb + 1))
            want = set(range(t_begin, t_end))
            assert want <= covered, (name, sorted(want - covered)[:4])


@pytest.mark.parametrize("T,S", [(4104, 1), (4104, 3), (4104, 16), (64, 1), (65, 1),
                                 (1000, 2), (8, 1), (32768, 4), (33024 - 8, 5), (257, 2)])
@pytest.mark.parametrize("mant_bits,v8", [(0, False), (4, False), (0, True), (1, True)])
def test_buffer_windows_stay_inside_the_sequence(T, S, mant_bits, v8):
    t_cap = (T + 7) // 8 * 8                    # the tightest legal capacity
    check(T, t_cap, S, mant_bits, v8)
