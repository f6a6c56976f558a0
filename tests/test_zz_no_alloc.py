"""The allocation-free sampler (ldr_sample_noalloc) against ldr_sample with a
caller workspace: same logits, seed and step give the same tokens, lse and
log q bit for bit, on two calls in a row (the second smaller, so it runs on
the scratch the first left behind), with and without a top-k support, and a
request beyond the static scratch is refused before anything is enqueued."""
import numpy as np
import pytest
import torch

pytestmark = pytest.mark.gpu


def _logits(rows, V, seed):
    g = torch.Generator(device="cuda").manual_seed(seed)
    return torch.randn(rows, V, generator=g, device="cuda") * 3.0


@pytest.mark.parametrize("T,top_k", [(1.0, 0), (0.7, 40), (0.0, 0)])
def test_noalloc_matches_the_workspace_call(gpu_lib, T, top_k):
    for rows, V, seed, step in ((256, 151936, 1, 7), (37, 5003, 2, 8)):
        z = _logits(rows, V, seed)
        ref = gpu_lib.sample(z, T, top_k, seed=seed, step=step)
        out = gpu_lib.sample_noalloc(z, T, top_k, seed=seed, step=step)
        torch.cuda.synchronize()
        for a, b in zip(ref, out):
            assert torch.equal(a, b) or np.array_equal(a.cpu().numpy().view(np.uint32),
                                                       b.cpu().numpy().view(np.uint32))
        assert torch.equal(ref[0], out[0])


def test_noalloc_refuses_requests_beyond_the_scratch(gpu_lib):
    rows, V = 600000, 16
    assert gpu_lib.sample_workspace_bytes(rows, V) > gpu_lib.NOALLOC_SCRATCH_BYTES
    z = torch.zeros(rows, V, device="cuda")
    with pytest.raises(gpu_lib.LdrError) as e:
        gpu_lib.sample_noalloc(z, 1.0, 0, seed=0, step=0)
    assert e.value.code == gpu_lib.LDR_ESCRATCH
    # a fitting request on the same GPU still works after the refusal
    tok, _, _ = gpu_lib.sample_noalloc(z[:64], 0.0, 0, seed=0, step=0)
    torch.cuda.synchronize()
    assert torch.all(tok == 0)
