"""The predictor entry point that allocates nothing (sae_predict_sessions_noalloc),
called through the C ABI, against the entry point with a caller workspace:
the same kernels on the same inputs, so the logits and predictions must be
bit-identical.  Two calls in a row, the second with fewer rows (the library's
buffer keeps the first call's contents), then the size limit."""
import numpy as np
import pytest
import torch

pytestmark = pytest.mark.gpu

from harness import say  # noqa: E402
from paper_2605_18825_amd import api  # noqa: E402
from synth import predictor as S  # noqa: E402


def dev(a, dt):
    return torch.as_tensor(np.ascontiguousarray(a)).to(device="cuda", dtype=dt)


def weights(d, seed):
    w = S.weights(d, seed)
    return dict(w1=dev(w["w1"].view(np.int16), torch.int16), b1=dev(w["b1"], torch.float32),
                w2=dev(w["w2"], torch.float32), b2=dev(w["b2"], torch.float32), w3=dev(w["w3"], torch.float32),
                b3=dev(w["b3"], torch.float32))


def both(n, d, wd, seed):
    h = dev(S.hidden_states(n, d, seed).view(np.int16), torch.int16).reshape(n, d)
    work = torch.full((4, n, 256), float("nan"), dtype=torch.float32, device="cuda")
    ly = torch.full((n,), float("nan"), dtype=torch.float32, device="cuda")
    lp = torch.full((n,), 7, dtype=torch.uint8, device="cuda")
    ny = torch.full((n,), float("nan"), dtype=torch.float32, device="cuda")
    np_ = torch.full((n,), 7, dtype=torch.uint8, device="cuda")
    say("no-alloc predictor n %d d %d" % (n, d))
    api.sae_predict_sessions(h, wd, work, ly, lp)
    api.sae_predict_sessions_noalloc(h, wd, ny, np_)
    torch.cuda.synchronize()
    return ly.cpu().numpy(), lp.cpu().numpy(), ny.cpu().numpy(), np_.cpu().numpy()


def test_noalloc_predictor_matches_workspace_entry_point():
    d = 4096
    wd = weights(d, 4242)
    for n, seed in ((4096, 11), (1000, 12), (77, 13)):
        ly, lp, ny, np_ = both(n, d, wd, seed)
        assert np.all(np.isfinite(ly))
        assert np.array_equal(ly.view(np.uint32), ny.view(np.uint32)), "logits differ (n %d)" % n
        assert np.array_equal(lp, np_), "predictions differ (n %d)" % n


def test_noalloc_predictor_size_limit():
    d = 256
    wd = weights(d, 7)
    n = api.PRED_NOALLOC_MAX_N + 1
    h = torch.zeros((n, d), dtype=torch.int16, device="cuda")
    out = torch.zeros(n, dtype=torch.float32, device="cuda")
    with pytest.raises(api.SaeError, match="SAE_PRED_NOALLOC_MAX_N"):
        api.sae_predict_sessions_noalloc(h, wd, out)
    api.sae_predict_sessions_noalloc(h[:0], wd, out)  # n = 0: nothing to do
