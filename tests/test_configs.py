"""The workload records (paper_1611_06172_amd/configs.py): JSON round trip,
unknown fields refused, and the values the paper states (Sec. 2: dim 300,
negative 5, window 5, sample 1e-4, alpha 0.025) in the throughput workload."""
import pytest

from paper_1611_06172_amd import configs


@pytest.mark.parametrize("name", sorted(configs.ALL))
def test_json_round_trip(name):
    cfg = configs.ALL[name]()
    assert configs.from_json(configs.to_json(cfg)) == cfg


def test_unknown_field_refused():
    text = configs.to_json(configs.Tiny()).replace('"K"', '"negatives_k"')
    with pytest.raises(ValueError):
        configs.from_json(text)


def test_throughput_workload_uses_the_papers_hyper_parameters():
    lv = configs.LargeVocab()
    assert (lv.D, lv.K, lv.window, lv.sample, lv.alpha0) == (300, 5, 5, 1e-4, 0.025)
    assert (lv.V, lv.T) == (1_000_000, 10**9)
    kt = configs.KernelTest()
    assert (kt.B, kt.N, kt.K, kt.V, kt.D) == (65_536, 10, 5, 100_000, 300)
