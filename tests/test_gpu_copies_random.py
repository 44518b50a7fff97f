"""Seeded random Ulysses copies through the C ABI, bit for bit against the
oracle: head dimensions that are any multiple of 8 (powers of two and not,
so both index paths of the copy kernels run), ragged token counts, and
random head maps -- dummy (-1) slots anywhere and repeated heads for the
pack, a random injective slot -> head assignment for the unpack, repeated
and unnamed heads for the summing unpack."""
import numpy as np
import pytest

import oracle
from tests.helpers import bits_from_dev, to_dev
from workloads import randn_bf16_bits

pytestmark = pytest.mark.gpu
SEEDS = list(range(24))


@pytest.fixture(scope="module")
def sp():
    import torch
    assert torch.cuda.is_available()
    import paper_2505_22296_amd as m
    m.load()
    return m


def _case(seed):
    rng = np.random.default_rng(5300 + seed)
    D = int(rng.choice([8, 24, 64, 96, 128, 136, 256]))
    T = int(rng.integers(1, 3000))
    spn = int(rng.integers(1, 9))
    hl = int(rng.integers(1, 9))
    return rng, D, T, spn, hl


@pytest.mark.parametrize("seed", SEEDS)
def test_random_pack(sp, seed):
    rng, D, T, spn, hl = _case(seed)
    hs = int(rng.integers(1, 20))
    hm = np.where(rng.random(spn * hl) < 0.2, -1, rng.integers(0, hs, spn * hl)).astype(np.int32)
    print(f"pack seed={seed} T={T} hs={hs} sp={spn} H_dst_loc={hl} D={D}", flush=True)
    bits = randn_bf16_bits((T, hs, D), seed=6000 + seed)
    got = bits_from_dev(sp.sp_ulysses_pack(to_dev(bits), spn, hl, hm))
    assert np.array_equal(got, oracle.ulysses_pack(bits, spn, hl, hm))


@pytest.mark.parametrize("seed", SEEDS)
def test_random_unpack(sp, seed):
    rng, D, T, spn, hl = _case(seed)
    slots = spn * hl
    H_dst = int(rng.integers(1, slots + 1))
    hm = np.full(slots, -1, np.int32)
    hm[rng.choice(slots, H_dst, replace=False)] = rng.permutation(H_dst)
    print(f"unpack seed={seed} T={T} sp={spn} H_src_loc={hl} H_dst={H_dst} D={D}", flush=True)
    bits = randn_bf16_bits((spn, T, hl, D), seed=6100 + seed)
    got = bits_from_dev(sp.sp_ulysses_unpack(to_dev(bits), hm, H_dst))
    assert np.array_equal(got, oracle.ulysses_unpack(bits, hm, H_dst))


@pytest.mark.parametrize("seed", SEEDS)
def test_random_unpack_add(sp, seed):
    rng, D, T, spn, hl = _case(seed)
    slots = spn * hl
    H_dst = int(rng.integers(1, 12))
    hm = np.where(rng.random(slots) < 0.2, -1, rng.integers(0, H_dst, slots)).astype(np.int32)
    print(f"unpack_add seed={seed} T={T} sp={spn} H_src_loc={hl} H_dst={H_dst} D={D}", flush=True)
    bits = randn_bf16_bits((spn, T, hl, D), seed=6200 + seed)
    got = bits_from_dev(sp.sp_ulysses_unpack_add(to_dev(bits), hm, H_dst))
    assert np.array_equal(got, oracle.ulysses_unpack_add_bf16(bits, hm, H_dst))
