"""HIP graph capture of the layer: rrs_linear and rrs_linear_reorder captured on
a stream and replayed several times, with other eager work and
synchronizations between the replays; every replay must equal the eager
result bit for bit (the kernels are deterministic and write every output, and
no call of the library records a memset)."""
import numpy as np
import pytest

import synth
from tests._gpu_util import to_gpu

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


@pytest.fixture(scope="module", autouse=True)
def _need_gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2409_20361_amd as rrs
    rrs.lib()


def _rrs():
    import paper_2409_20361_amd as rrs
    return rrs


@pytest.mark.parametrize("M,K,N,g,reorder", [
    (8, 8192, 256, 128, False),    # one-launch few-token quantizer, few-token GEMM
    (1, 4096, 4112, 128, False),   # the whole layer in one launch (one token)
    (2, 8192, 512, 256, False),    # the whole layer in one launch (two tokens)
    (40, 8192, 4112, 128, False),  # per-row quantizer (shared reads), few-token GEMM
    (300, 4096, 384, 128, False),  # two-launch quantizer, main GEMM
    (16, 2048, 128, 64, True),     # reorder: three quantizer launches, few-token gather
    (260, 1024, 256, 256, True),   # reorder: main-kernel gather
])
def test_graph_replay_matches_eager(M, K, N, g, reorder):
    rrs = _rrs()
    w = synth.custom("gr", M, K, N, g, 61 + M + K, n_chan=max(1, K // 100), n_spike=3,
                     spike_mag=(100, 500))
    print(f"[case] graph replay M={M} K={K} N={N} g={g} reorder={reorder}", flush=True)
    X = to_gpu(synth.activations(w))
    Wq, beta = rrs.prepare_weight(to_gpu(synth.weights(w)))
    if reorder:
        ws = torch.zeros((rrs.linear_reorder_workspace_bytes(M, K, g),), dtype=torch.uint8,
                         device=X.device)
        call = lambda out: rrs.linear_reorder(X, Wq, beta, g, workspace=ws, out=out)  # noqa: E731
    else:
        ws = torch.zeros((rrs.linear_workspace_bytes(M, K, g),), dtype=torch.uint8,
                         device=X.device)
        call = lambda out: rrs.linear(X, Wq, beta, g, workspace=ws, out=out)  # noqa: E731
    Y_eager = torch.empty((M, N), dtype=torch.float16, device=X.device)
    call(Y_eager)
    torch.cuda.synchronize()
    ref = Y_eager.clone()

    Y = torch.empty_like(Y_eager)
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):   # warm the allocator and the library off the capture
        call(Y)
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        call(Y)
    for rep in range(4):
        Y.fill_(0)
        scratch = torch.randn(1024, 1024, device=X.device)   # eager work between replays
        (scratch @ scratch).sum().item()
        graph.replay()
        torch.cuda.synchronize()
        assert torch.equal(Y, ref), f"replay {rep} differs from the eager result"
        # eager call between replays, on the same buffers
        call(Y)
        torch.cuda.synchronize()
        assert torch.equal(Y, ref)
    assert np.isfinite(ref.float().cpu().numpy()).all()
