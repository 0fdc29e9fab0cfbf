"""The allocation-free sampler entry point against the allocating one.

sara_sample_logits_noalloc runs the stand-alone sampler's kernels over a
static device array instead of per-call allocations.  Its tokens must equal
sara_sample_logits's on the same inputs (integer results: bit-exact), on two
calls in a row with the second smaller than the first (the array keeps the
first call's contents), with and without the top-p passes; inputs beyond
its stated limits are refused before anything is enqueued."""
import numpy as np
import pytest

import workloads as W

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def torch_cuda():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a HIP device"
    import paper_2607_26253_amd  # noqa: F401  (fails loudly when libsara.so is missing)
    return torch


def _inputs(torch, n, V, seed):
    g = np.random.default_rng(seed)
    logits = (g.standard_normal((n, V)) * np.where(np.arange(n) % 2 == 0, 0.8, 5.0)[:, None]).astype(np.float32)
    logits[0, : V // 4] = logits[0, 0]       # a large tie group
    rid = (np.arange(n, dtype=np.int32) * 7 + 3).astype(np.int32)
    pos = ((np.arange(n, dtype=np.int32) * 13) % 2048).astype(np.int32)
    return (torch.from_numpy(logits).cuda(), torch.from_numpy(rid).cuda(), torch.from_numpy(pos).cuda())


@pytest.mark.parametrize("V,top_p,sizes", [(151936, 1.0, (300, 37)), (151936, 0.9, (64, 9)),
                                           (512, 0.5, (40, 3)), (509, 1.0, (4096, 1))])
def test_noalloc_sampler_equals_allocating_sampler(torch_cuda, V, top_p, sizes):
    import paper_2607_26253_amd as sara
    torch = torch_cuda
    seed, step = W.sampling_seed(W.get_config("qwen1p5b_shape")), 4
    eos, feos = V - 1, (1 << 32) // 64
    for call, n in enumerate(sizes):
        lg, rid, pos = _inputs(torch, n, V, 100 * call + n)
        want = torch.full((n,), -1, dtype=torch.int32, device="cuda")
        got = torch.full((n,), -2, dtype=torch.int32, device="cuda")
        sara.sara_sample_logits(lg, rid, pos, seed, step, 1.0, eos, feos, want, top_p=top_p)
        sara.sara_sample_logits_noalloc(lg, rid, pos, seed, step, 1.0, eos, feos, got, top_p=top_p)
        torch.cuda.synchronize()
        w, g = want.cpu().numpy(), got.cpu().numpy()
        print(f"[noalloc] V={V} top_p={top_p} call {call}: {n} rows, {int(np.sum(w == g))} equal", flush=True)
        assert np.array_equal(w, g)
        assert g.min() >= 0 and g.max() < V


def test_noalloc_sampler_refuses_inputs_beyond_its_limits(torch_cuda):
    import paper_2607_26253_amd as sara
    torch = torch_cuda
    lg, rid, pos = _inputs(torch, 2, 512, 1)
    tok = torch.zeros(2, dtype=torch.int32, device="cuda")
    L = sara._lib
    stream = torch.cuda.current_stream().cuda_stream
    args = (lg.data_ptr(), rid.data_ptr(), pos.data_ptr(), 1, 0, 1.0)
    big = sara.NOALLOC_MAX_ROWS + 1
    assert L.sara_sample_logits_noalloc(args[0], big, 512, args[1], args[2], 1, 0, 1.0, 1.0, -1, 0,
                                        tok.data_ptr(), stream) == sara.SARA_EINVAL
    assert L.sara_sample_logits_noalloc(args[0], sara.NOALLOC_MAX_TOPP_ROWS + 1, 512, args[1], args[2], 1, 0, 1.0,
                                        0.9, -1, 0, tok.data_ptr(), stream) == sara.SARA_EINVAL
    assert b"SARA_NOALLOC_MAX" in L.sara_last_error()
    assert L.sara_sample_logits_noalloc(args[0], 2, 512, args[1], args[2], 1, 0, 1.0, 0.0, -1, 0,
                                        tok.data_ptr(), stream) == sara.SARA_EINVAL
    torch.cuda.synchronize()
