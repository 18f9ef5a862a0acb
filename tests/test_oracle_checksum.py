"""Pins of the oracle's parameter-set checksum (ChecksumMatch, Algorithm 1:
replicas compare a hash of theta with a random peer). The paper fixes no
hash; what the checksum must do is fixed here and checked independently of the
oracle's code: the mixer is a bijection (inverted below from its structure),
it avalanches, and the set checksum is additive and order-free over tensors
while detecting any single bit flip, element swap or tensor-id change."""
import numpy as np
import pytest

M64 = (1 << 64) - 1


def unshift_xor(y: int, s: int) -> int:
    """Inverse of x -> x ^ (x >> s) on 64 bits."""
    x = y
    for _ in range(64 // s + 1):
        x = y ^ (x >> s)
    return x & M64


def fmix64_inverse(y: int) -> int:
    c1, c2 = 0xFF51AFD7ED558CCD, 0xC4CEB9FE1A85EC53
    y = unshift_xor(y, 33)
    y = (y * pow(c2, -1, 1 << 64)) & M64
    y = unshift_xor(y, 33)
    y = (y * pow(c1, -1, 1 << 64)) & M64
    return unshift_xor(y, 33)


def test_fmix64_is_a_bijection_with_the_stated_structure(orc):
    rng = np.random.Generator(np.random.PCG64(41))
    xs = [0, 1, M64, 1 << 63] + [int(v) for v in rng.integers(0, 2**63, size=2000)] + \
         [int(v) * 2 + 1 for v in rng.integers(0, 2**62, size=100)]
    for x in xs:
        assert fmix64_inverse(orc.fmix64(x)) == x
    assert orc.fmix64(0) == 0


def test_fmix64_avalanche(orc):
    rng = np.random.Generator(np.random.PCG64(42))
    flips = []
    for x in (int(v) for v in rng.integers(0, 2**63, size=300)):
        y = orc.fmix64(x)
        for bit in range(0, 64, 7):
            flips.append(bin(y ^ orc.fmix64(x ^ (1 << bit))).count("1"))
    assert 30 < np.mean(flips) < 34 and min(flips) >= 8


def set_(seed, sizes=(1, 5, 8, 1001, 4096), dtype=np.float32):
    rng = np.random.Generator(np.random.PCG64(seed))
    if dtype == np.float32:
        return [rng.standard_normal(n).astype(np.float32) * 0.02 for n in sizes]
    return [rng.integers(0, 1 << 16, size=n, dtype=np.uint64).astype(np.uint16) for n in sizes]


def test_set_checksum_is_additive_and_order_free(orc):
    ts = set_(1)
    ids = [3, 9, 0, 77, 1 << 31]
    total = orc.checksum(ts, ids)
    parts = (orc.checksum(ts[:2], ids[:2]) + orc.checksum(ts[2:], ids[2:])) & M64
    assert total == parts
    perm = [4, 0, 3, 1, 2]
    assert orc.checksum([ts[i] for i in perm], [ids[i] for i in perm]) == total


@pytest.mark.parametrize("dtype", [np.float32, np.uint16])
def test_every_single_bit_flip_changes_the_checksum(orc, dtype):
    t = set_(2, sizes=(37,), dtype=dtype)[0]
    base = orc.checksum_tensor(t, 5)
    raw = t.view(np.uint8).copy()
    seen = set()
    for byte in range(raw.size):
        for bit in range(8):
            r = raw.copy()
            r[byte] ^= 1 << bit
            c = orc.checksum_tensor(r.view(dtype), 5)
            assert c != base
            seen.add(c)
    assert len(seen) == raw.size * 8   # no two flips collide either


def test_position_and_tensor_id_matter(orc):
    t = set_(3, sizes=(64,))[0]
    swapped = t.copy()
    swapped[[2, 40]] = swapped[[40, 2]]
    assert orc.checksum_tensor(t, 0) != orc.checksum_tensor(swapped, 0)
    assert orc.checksum_tensor(t, 0) != orc.checksum_tensor(t, 1)
    # chunks are 8-byte aligned to the tensor start: moving data by one
    # element changes every chunk
    assert orc.checksum_tensor(t[1:], 0) != orc.checksum_tensor(t[:-1], 0)


def test_tail_chunk_is_zero_padded(orc):
    """The last chunk is padded with zero bytes: a tensor and the same tensor
    with zero bytes appended up to the chunk boundary hash the same; one more
    chunk (even of zeros) changes the sum."""
    t = set_(4, sizes=(5,))[0]                      # 20 bytes: chunks 0, 1, 2 (half)
    padded = np.concatenate([t, np.zeros(1, np.float32)])   # 24 bytes: same 3 chunks
    assert orc.checksum_tensor(t, 7) == orc.checksum_tensor(padded, 7)
    longer = np.concatenate([t, np.zeros(3, np.float32)])    # 32 bytes: 4 chunks
    assert orc.checksum_tensor(longer, 7) != orc.checksum_tensor(t, 7)
    b = set_(5, sizes=(5,), dtype=np.uint16)[0]     # 10 bytes: chunks 0, 1 (quarter)
    assert orc.checksum_tensor(b, 2) == orc.checksum_tensor(
        np.concatenate([b, np.zeros(3, np.uint16)]), 2)
    assert orc.checksum_tensor(np.zeros(0, np.float32), 1) == 0
