"""rrs_linear_noalloc: the allocation-free variant of rrs_linear (for callers
that cannot allocate device memory) must give bit-identical outputs to
rrs_linear with a caller workspace, on consecutive calls that reuse the
library-held scratch (the second one smaller), and must reject calls whose
workspace would exceed the scratch without enqueuing anything."""
import numpy as np
import pytest

import synth
from tests._gpu_util import to_gpu

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")

WORKSPACE = -5


@pytest.fixture(scope="module", autouse=True)
def _need_gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2409_20361_amd as rrs
    rrs.lib()


def _rrs():
    import paper_2409_20361_amd as rrs
    return rrs


def _layer(M, K, N, g, seed, perm=False):
    rrs = _rrs()
    w = synth.custom("na", M, K, N, g, seed, n_chan=max(1, K // 100), chan_factor=(20, 100),
                     n_spike=max(1, M * K // 10000), spike_mag=(100, 500))
    X = to_gpu(synth.activations(w))
    p = to_gpu(synth.permutation(K, seed)) if perm else None
    Wq, beta = rrs.prepare_weight(to_gpu(synth.weights(w)), p)
    return X, Wq, beta, p


def _compare(M, K, N, g, seed, perm=False):
    rrs = _rrs()
    print(f"[case] no-alloc linear M={M} K={K} N={N} g={g} perm={perm}", flush=True)
    X, Wq, beta, p = _layer(M, K, N, g, seed, perm)
    ref = rrs.linear(X, Wq, beta, g, perm=p)
    got = rrs.linear_noalloc(X, Wq, beta, g, perm=p)
    torch.cuda.synchronize()
    assert torch.equal(got, ref), f"M={M} K={K} N={N} g={g}: outputs differ"


def test_no_alloc_matches_linear_on_consecutive_calls():
    # the first call fills the scratch, the second (smaller) reuses it
    _compare(300, 4096, 272, 128, 1)
    _compare(5, 4096, 48, 128, 2)


def test_no_alloc_decode_and_large_then_small():
    _compare(2048, 4096, 64, 128, 3)          # qkv's token count: a large workspace
    _compare(8, 8192, 112, 128, 4)            # decode shape, few-token kernels
    _compare(3, 1024, 32, 64, 5, perm=True)   # static reorder
    _compare(2, 8192, 64, 128, 6)             # the layer in one launch (two tokens)
    _compare(1, 4096, 48, 256, 7)             # the layer in one launch (one token)


def test_no_alloc_rejects_oversize_without_enqueuing():
    rrs = _rrs()
    M, K, N, g = 4100, 8192, 16, 128          # workspace just above 16 MiB
    assert rrs.linear_workspace_bytes(M, K, g) > (16 << 20)
    X = torch.zeros((M, K), dtype=torch.float16, device="cuda")
    Wq = torch.zeros((N, K // 2), dtype=torch.uint8, device="cuda")
    beta = torch.ones((N,), dtype=torch.float32, device="cuda")
    Y = torch.full((M, N), 7.0, dtype=torch.float16, device="cuda")
    code = rrs.lib().rrs_linear_noalloc(X.data_ptr(), Wq.data_ptr(), beta.data_ptr(), M, N, K,
                                        g, None, Y.data_ptr(),
                                        torch.cuda.current_stream().cuda_stream)
    assert code == WORKSPACE
    torch.cuda.synchronize()
    assert bool((Y == 7.0).all())
    # the largest accepted size at K = 8192 works and matches rrs_linear
    _compare(3995, 8192, 32, 128, 6)
