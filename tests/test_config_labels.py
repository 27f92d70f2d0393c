"""Configuration labels (no GPU): Config.label and Config.parse, the library's
own form and the paper's SDQ names of its evaluated configurations."""
import pytest

import synth

sdq = pytest.importorskip("paper_2406_13868_amd")


@pytest.mark.parametrize("wid", sorted(synth.WORKLOADS))
def test_workload_formats_round_trip(wid):
    for f in synth.WORKLOADS[wid].formats:
        c = sdq.Config.of(f)
        assert c.label == f.label
        assert sdq.Config.parse(c.label) == c


@pytest.mark.parametrize("name,n_o,n_i", [("SDQ-W7:8-1:8int8-6:8fp4", 1, 6), ("SDQ-W6:8-2:8int8-4:8fp4", 2, 4),
                                           ("SDQ-W8:8-1:8int8-7:8fp4", 1, 7)])
def test_paper_names(name, n_o, n_i):
    c = sdq.Config.parse(name)
    assert c == sdq.Config.dual_family(n_o, n_i, metric="product")
    sdq.check(c, 4096, 4096)  # the kernels take all three


def test_paper_name_int_inliers():
    c = sdq.Config.parse("SDQ-W4:8-1:8int8-3:8int4")
    assert c == sdq.Config.int_family(1, 8, "int8", 3, metric="product")


@pytest.mark.parametrize("bad", ["SDQ-S7:8-1:8int8-6:8fp4", "SDQ-W7:8-1:8int8-5:8fp4", "SDQ-W7:8-1:8fp8-6:8fp4",
                                 "SDQ-W7:16-1:8int8-6:8fp4", "int-1:8e4m3-3:8int4", "mx-1:8e4m3-2:8e2m1-Afp8", "",
                                 "dual-1:8int8-6:8e2m1-Aint8 "])
def test_malformed_or_unbuilt_labels(bad):
    with pytest.raises(ValueError):
        sdq.Config.parse(bad)


def test_parse_is_syntax_check_is_support():
    c = sdq.Config.parse("int-2:8e4m3-3:8int4-Aint8")  # well formed, two outliers per 8 not built for INT
    with pytest.raises(sdq.SDQError) as e:
        sdq.check(c, 128, 128)
    assert e.value.status == -6
