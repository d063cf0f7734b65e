"""Helpers shared by the GPU tests (device transfer, tolerances)."""
import numpy as np
import torch

# fp32 logits: |z_gpu - z_ref| <= 1e-4 * max(1, |z_ref|)  (a pure relative bound
# is ill-posed near z = 0); bf16 scores: |s_gpu - s_ref| <= 2e-2.
FP32_LOGIT_RTOL = 1e-4
BF16_SCORE_ATOL = 2e-2


def dev(a, dtype=None):
    t = torch.as_tensor(np.ascontiguousarray(a))
    if dtype is not None:
        t = t.to(dtype)
    return t.cuda()


def assert_logits_close(got, ref, rtol=FP32_LOGIT_RTOL, what="logits"):
    got = np.asarray(got, np.float64)
    ref = np.asarray(ref, np.float64)
    err = np.abs(got - ref) / np.maximum(1.0, np.abs(ref))
    k = int(np.argmax(err)) if err.size else 0
    assert err.size == 0 or err.max() <= rtol, (
        f"{what}: max scaled error {err.max():.3e} at {k} (gpu {got[k]!r}, ref {ref[k]!r})")
    return float(err.max()) if err.size else 0.0


def run_model(G, w, dims, x, ei, logits=True):
    m = G.Model(w, dims)
    try:
        xd, eid = dev(x), dev(ei)
        out = m(xd, eid, logits=logits)
        torch.cuda.synchronize()
        return out.cpu().numpy()
    finally:
        m.close()
