"""The device-side input generator draws exactly the numpy generator's values."""
import numpy as np
import pytest
import torch

import gcn_synth as gs

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("p,binary", [(0.1, False), (0.5, False), (0.013, True), (0.001, False), (1.0, False)])
def test_device_bernoulli_matches_numpy(p, binary):
    from gcn_synth import device
    n, f = 700, 4096
    X = torch.full((n, f + 4), float("nan"), device="cuda")
    device.bernoulli_into(X[:, :f], p, seed=0, stream=3, binary=binary)
    ref = gs.features_bernoulli(n, f, p, seed=0, stream=3, binary=binary)
    got = X[:, :f].cpu().numpy()
    np.testing.assert_array_equal(got.view(np.int32), ref.view(np.int32))
    assert torch.isnan(X[:, f:]).all()
    # a row range drawn alone equals the same rows of the whole matrix
    Y = torch.empty((50, f), device="cuda")
    device.bernoulli_into(Y, p, seed=0, stream=3, row0=333, binary=binary)
    np.testing.assert_array_equal(Y.cpu().numpy().view(np.int32), ref[333:383].view(np.int32))
