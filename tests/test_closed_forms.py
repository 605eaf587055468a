"""Closed forms from the paper's work model (Sec. 3 example) and the AlexNet conv work, as unit tests of
the benchmark's work-model helper."""
import pytest

from paper_1404_1869_amd import workmodel


def test_paper_example_regions_and_speedup():
    # N = 1000, M = 200, stride 16: about 2.5K regions and a 100x speedup (Sec. 3)
    assert workmodel.region_count(1000, 200) == 2500
    assert workmodel.dense_speedup(1000, 200) == 100


def test_alexnet_conv_work():
    # 227 x 227: the five conv layers of AlexNet hold about 666M multiply-adds
    f = workmodel.conv_flops(227, 227)
    assert [x // 2 for x in f] == [105415200, 223948800, 149520384, 112140288, 74760192]
    assert sum(f) == pytest.approx(1.3316e9, rel=1e-4)
    assert workmodel.sides(227) == (55, 27, 27, 13, 13, 13, 13, 6)
    assert workmodel.sides(1200) == (298, 149, 149, 74, 74, 74, 74, 37)
    assert sum(workmodel.conv_flops(1200, 1200)) == pytest.approx(41.63e9, rel=1e-3)
