"""The device build of the input generator produces the host build's bits."""
import numpy as np
import pytest

import synth
from tests.gpu_helpers import say

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("name,t_idx,role", [("tiny", 0, 0), ("tiny", 0, 2), ("layer", 4, 1), ("1.5b", 2, 3),
                                             ("7b", 5, 4)])
def test_device_generator_matches_host(name, t_idx, role):
    import torch
    say(f"synth {name} t{t_idx} r{role}")
    wl = synth.workload(name)
    n = min(wl.tensors[t_idx].numel, 1 << 20)
    first = 12345 if n == 1 << 20 else 0
    host = synth.fill_host(wl, t_idx, role, first=first, n=n)
    dt = torch.int16 if wl.dtype == "bf16" else torch.int32
    dev = torch.empty(n, dtype=dt, device="cuda")
    synth.fill_device(dev.data_ptr(), n, wl, t_idx, role, stream=torch.cuda.current_stream().cuda_stream, first=first)
    torch.cuda.synchronize()
    got = dev.cpu().numpy().view(host.dtype)
    assert np.array_equal(got.view(np.uint8), host.view(np.uint8))
