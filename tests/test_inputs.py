"""The seeded input generators (no arithmetic of the method): the
counter-based Zipf stream that the throughput benchmark draws on the GPU and
the oracle's stored results draw on the host."""
import numpy as np
import torch

from paper_1611_06172_amd import inputs


def test_splitmix64_known_value_and_numpy_agreement():
    # SplitMix64's first output for state 0 (its increment added once, then
    # the finaliser), as published with the generator
    assert int(inputs.splitmix64_numpy(np.array([0], np.uint64))[0]) == 0xE220A8397B1DCDAF
    x = np.arange((6 << 40), (6 << 40) + 50_000, dtype=np.uint64)
    x[::7] = np.random.default_rng(0).integers(0, 2**63, x[::7].shape, dtype=np.uint64)
    t = inputs._splitmix64_torch(torch.from_numpy(x.view(np.int64)))
    assert np.array_equal(t.numpy().view(np.uint64), inputs.splitmix64_numpy(x))


def test_hashed_corpus_prefixes_and_law():
    V, s = 1000, 1.07
    a = inputs.zipf_corpus_hashed(200_000, V, s, 6)
    b = inputs.zipf_corpus_hashed(5_000, V, s, 6, begin=123_456)
    assert a.dtype == torch.int32 and int(a.min()) >= 0 and int(a.max()) < V
    assert torch.equal(a[123_456:128_456], b)
    # chunking does not change the stream
    c = inputs.zipf_corpus_hashed(200_000, V, s, 6, chunk=4096)
    assert torch.equal(a, c)
    # another seed gives another stream
    assert not torch.equal(a, inputs.zipf_corpus_hashed(200_000, V, s, 7))
    # frequencies follow the Zipf law (chi-square over the 50 head words)
    pmf = inputs.zipf_pmf(V, s)
    hist = np.bincount(a.numpy(), minlength=V)
    exp = pmf * len(a)
    head = slice(0, 50)
    rest_obs, rest_exp = hist[50:].sum(), exp[50:].sum()
    chi2 = (((hist[head] - exp[head]) ** 2) / exp[head]).sum() + (rest_obs - rest_exp) ** 2 / rest_exp
    assert chi2 < 95.6  # 50 dof, p = 1e-4
