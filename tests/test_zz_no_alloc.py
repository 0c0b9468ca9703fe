"""mz_q4_gemm_split_noalloc (the entry point that allocates nothing) against
mz_q4_gemm_split on the same inputs: the same kernels with the partials in the
library's fixed device array instead of a caller workspace, so the outputs are
the same bits.  Two calls in a row on one GPU, the second with a smaller input
(the array keeps the first call's partials; nothing of them may show), for the
store, residual-add and SwiGLU epilogues; then the size limit."""

import numpy as np
import pytest

from paper_2609_01338_amd import mz
from paper_2609_01338_amd import workloads as W
from gpu_util import report, stream, torch_cuda

pytestmark = pytest.mark.gpu


def _inputs(torch, M, N, K, epi, seed):
    rng = np.random.default_rng(seed)
    if epi == 2:
        g = W.encode_q4_0((rng.standard_normal((N, K)) * 0.02).astype(np.float32))
        u = W.encode_q4_0((rng.standard_normal((N, K)) * 0.02).astype(np.float32))
        packed = mz.mz_q4_gemm_pack(g, N, K, w_up=u)
        n_pad = 2 * ((N + 127) // 128 * 128)
    else:
        packed = mz.mz_q4_gemm_pack(W.encode_q4_0((rng.standard_normal((N, K)) * 0.02).astype(np.float32)), N, K)
        n_pad = (N + 255) // 256 * 256
    gen = torch.Generator(device="cuda").manual_seed(seed)
    x = torch.randn(M, K, device="cuda", generator=gen).to(torch.float16)
    w = torch.from_numpy(packed).cuda()
    if epi == 2:
        y0 = torch.zeros(M, n_pad // 2, device="cuda", dtype=torch.float16)
    elif epi == 1:
        y0 = torch.randn(M, n_pad, device="cuda", generator=gen)
    else:
        y0 = torch.zeros(M, n_pad, device="cuda")
    return x, w, n_pad, y0


@pytest.mark.parametrize("epi", [0, 1, 2])
def test_noalloc_matches_workspace_entry(epi):
    torch = torch_cuda()
    m = W.WORKLOADS["8b"].model
    N, K = {0: (2 * m.dkv, m.d_model), 1: (m.d_model, m.dq), 2: (m.d_ffn, m.d_model)}[epi]
    # first call larger than the second: 129 rows (a 128-token prompt and the
    # last context row), then a single decode row
    for call, (M, n_split) in enumerate([(129, 8), (1, 16)]):
        x, w, n_pad, y0 = _inputs(torch, M, N, K, epi, seed=10 * epi + call)
        # as many splits as the fixed array holds partials for (at most the one asked)
        n_split = min(n_split, mz.NOALLOC_SCRATCH_BYTES // (M * n_pad * 4))
        report("noalloc", epi=epi, call=call, M=M, N=N, K=K, n_pad=n_pad, n_split=n_split,
               partial_bytes=mz.mz_q4_gemm_split_workspace_bytes(M, n_pad, n_split))
        assert mz.mz_q4_gemm_split_workspace_bytes(M, n_pad, n_split) <= mz.NOALLOC_SCRATCH_BYTES
        ref = y0.clone()
        wsb = mz.mz_q4_gemm_split_workspace_bytes(M, n_pad, n_split)
        ws = torch.full((wsb // 4,), float("nan"), device="cuda")
        mz.mz_q4_gemm_split(x.data_ptr(), M, n_pad, K, w.data_ptr(), epi, ref.data_ptr(), n_split, ws.data_ptr(),
                            wsb, stream())
        got = y0.clone()
        mz.mz_q4_gemm_split_noalloc(x.data_ptr(), M, n_pad, K, w.data_ptr(), epi, got.data_ptr(), n_split, stream())
        torch.cuda.synchronize()
        assert torch.equal(got.view(torch.uint8), ref.view(torch.uint8)), (epi, call)
        assert bool(torch.isfinite(got.float()).all())


def test_noalloc_rejects_sizes_beyond_its_scratch():
    torch = torch_cuda()
    with pytest.raises(mz.MzError) as e:
        # 64 splits x 1024 rows x 4096 columns x 4 bytes = 1 GiB of partials
        mz.mz_q4_gemm_split_noalloc(1, 1024, 4096, 4096, 1, 0, 1, 64, stream())
    assert e.value.status == mz.MZ_EINVAL and "scratch" in str(e.value)
    torch.cuda.synchronize()
