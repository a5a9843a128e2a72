"""Pins of the oracle's shard layout (ZeRO Sec. 5.1: N_d equal partitions, rank i
owns partition i; tail padding when N_d does not divide Psi).

The shard sizes below are those of the five synthetic workloads (one rank of
GPT-2 1.5B, 13B, 100B at MP 16, 1T at MP 16 and N_d 1024); brute force checks
cover, order and disjointness for every small case.
"""
import pytest

import oracle


@pytest.mark.parametrize("psi,nd,rank,S,off,valid,padded", [
    (4_194_304, 4, 1, 1_048_576, 1_048_576, 1_048_576, 4_194_304),
    (1_500_000_000, 16, 0, 93_750_000, 0, 93_750_000, 1_500_000_000),
    (13_000_000_000, 64, 0, 203_125_000, 0, 203_125_000, 13_000_000_000),
    (6_250_000_000, 25, 0, 250_000_000, 0, 250_000_000, 6_250_000_000),
    # 1T / MP 16 = 62.5e9 over 1024 ranks: 61,035,157-element shards, last rank padded by 768.
    (62_500_000_000, 1024, 1023, 61_035_157, 62_438_965_611, 61_034_389, 62_500_000_768),
    (62_500_000_000, 1024, 0, 61_035_157, 0, 61_035_157, 62_500_000_768),
])
def test_workload_shards(psi, nd, rank, S, off, valid, padded):
    assert oracle.layout(psi, nd, rank) == (S, off, valid, padded)


def test_brute_force_cover():
    for psi in range(0, 65):
        for nd in range(1, 17):
            shards = [oracle.layout(psi, nd, r) for r in range(nd)]
            S = shards[0][0]
            assert all(s[0] == S and s[3] == nd * S for s in shards)
            covered = []
            for r, (_S, off, valid, _pad) in enumerate(shards):
                assert off == r * S
                assert 0 <= valid <= S
                covered.extend(range(off, off + valid))
            assert covered == list(range(psi))        # in rank order, disjoint, complete
            assert 0 <= nd * S - psi < nd               # padding is minimal
            if psi > 0:
                assert (S - 1) * nd < psi               # S = ceil(psi / nd)
            # only trailing ranks are short
            valids = [s[2] for s in shards]
            assert valids == sorted(valids, reverse=True)


def test_many_empty_tail_ranks():
    # 5 elements over 4 ranks: S = 2, ranks 0..2 hold 2, 2, 1 and rank 3 holds nothing.
    assert [oracle.layout(5, 4, r)[2] for r in range(4)] == [2, 2, 1, 0]


@pytest.mark.parametrize("psi,nd,rank", [(-1, 4, 0), (10, 0, 0), (10, 4, 4), (10, 4, -1), ((1 << 62) + 1, 2, 0)])
def test_invalid(psi, nd, rank):
    with pytest.raises((ValueError, OverflowError)):
        oracle.layout(psi, nd, rank)
