"""Pins of the scheduling closed forms: Eq. (3) footprint and Eq. (4) quota,
against hand-computed values."""
import oracle


def test_x_moe_eq3():
    # ceil(1/128) + ceil(128/128) + ceil(129/128) + ceil(300/128), empty experts skipped
    assert oracle.x_moe([0, 1, 128, 129, 300], 128) == 1 + 1 + 2 + 3
    assert oracle.x_moe([0, 0], 64) == 0
    assert oracle.x_moe([5] * 32, 32) == 32
    assert oracle.count_tiles([0, 1, 128, 129, 300], 128, 3072, 256) == 7 * 12
    assert oracle.count_tiles([10], 16, 100, 64) == 1 * 2


def test_quota_eq4():
    # fixed quota: 25% of 256 workgroups, cluster multiple 8
    assert oracle.decode_quota(64, 50, 0, 128, 8) == 64
    assert oracle.decode_quota(60, 7, -1, 128, 8) == 64          # 60 rounds up to 64
    # footprint equal to the expectation keeps q
    assert oracle.decode_quota(64, 50, 50, 128, 8) == 64
    # 64 * 51 / 50 = 65.28 -> next multiple of 8 is 72
    assert oracle.decode_quota(64, 51, 50, 128, 8) == 72
    # 64 * 25 / 50 = 32 exactly (no spurious round-up)
    assert oracle.decode_quota(64, 25, 50, 128, 8) == 32
    # 64 * 26 / 50 = 33.28 -> 40
    assert oracle.decode_quota(64, 26, 50, 128, 8) == 40
    # capped by Q_max
    assert oracle.decode_quota(64, 200, 50, 128, 8) == 128
    # no decode footprint, no decode workgroups
    assert oracle.decode_quota(64, 0, 50, 128, 8) == 0
    # c = 1 is a plain ceiling
    assert oracle.decode_quota(10, 3, 4, 100, 1) == 8            # 7.5 -> 8
