"""The value draw gives the same bits on the GPU as on the host: the inputs of
every GPU test are the ones the CPU tests and the oracle would draw from the
same seed."""
import numpy as np
import pytest
import torch

import workloads as W

pytestmark = pytest.mark.gpu


def _bits(t):
    return t.detach().cpu().contiguous().view(torch.int16 if t.element_size() == 2 else torch.int32)


@pytest.mark.parametrize("name", ["tiny", "long_cot"])
def test_values_identical_on_host_and_device(name):
    st = W.make_structure(name)
    if name == "long_cot":  # a slice of the pool keeps the host draw short
        st = W.custom_structure(8, st.Hq, st.Hkv, st.D, [1024, 1, 17, 300, 2048, 5000, 16, 4097], seed=st.seed)
        st.k_offset_std = 0.5
    host = W.fill_values(st, "cpu", fill="nan")
    dev = W.fill_values(st, "cuda", fill="nan")
    for a, b in zip(host, dev):
        assert torch.equal(_bits(a), _bits(b))
    assert torch.equal(_bits(W.fill_multi_q(st, 5, "cpu")), _bits(W.fill_multi_q(st, 5, "cuda")))
    for a, b in zip(W.fill_new_kv(st, 3, "cpu"), W.fill_new_kv(st, 3, "cuda")):
        assert torch.equal(_bits(a), _bits(b))
    print(f"{name}: q/K/V, multi-token q and new K/V rows bit-identical on host and device", flush=True)


@pytest.mark.parametrize("dtype", [torch.bfloat16, torch.float32])
def test_logits_identical_on_host_and_device(dtype):
    xh, th = W.make_logits(6, 5000, seed=70, device="cpu", dtype=dtype)
    xd, td = W.make_logits(6, 5000, seed=70, device="cuda", dtype=dtype)
    assert np.array_equal(th, td)
    assert torch.equal(_bits(xh), _bits(xd))
