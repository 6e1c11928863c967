"""The allocation-free linear (dfssm_scaffold_lora_linear_noalloc) against
the linear with a caller workspace (dfssm_scaffold_lora_linear), through the
C ABI: two calls in a row on the library's scratch array, the second with a
smaller input, each bit-identical to the workspace entry point's y and
within the oracle's bar; a call too large for the scratch is refused."""
import ctypes

import numpy as np
import pytest

import dfssm_synth as S
import oracle
from gpu_util import assert_y, dev, dev_weights, host, say, torch_cuda

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def env():
    torch = torch_cuda()
    import paper_2606_10932_amd as D
    oracle.build()
    return torch, D, oracle.get()


def _noalloc(D, qd, sd, d, y, r):
    p = lambda t: None if t is None else t.data_ptr()
    M, K = qd.shape
    N = d["w_bits"].shape[0]
    return D.lib.dfssm_scaffold_lora_linear_noalloc(
        qd.data_ptr(), sd.data_ptr(), M, K, N, r, d["w_bits"].data_ptr(), d["alpha"].data_ptr(), p(d["A"]),
        p(d["B"]), p(d["beta"]), y.data_ptr(), D._stream(None))


def test_noalloc_two_calls_smaller_second(env):
    torch, D, o = env
    # the 1.3B out_proj at 130 tokens, then the 1.3B in_proj at 3 tokens
    for i, (M, K, N, r) in enumerate([(130, 4096, 2048, 64), (3, 2048, 8512, 64)]):
        say(f"no-alloc call {i}: M={M} K={K} N={N} r={r}")
        assert D.linear_workspace_bytes(M, K, N, r) <= D.lib.dfssm_noalloc_scratch_bytes()
        ws = S.weights(K, N, r, key=(180, i))
        q, s = o.quantize_act(S.activations(M, K, key=(181, i)))
        d = dev_weights(ws)
        qd, sd = dev(q), dev(s)
        y = torch.full((M, N), np.nan, dtype=torch.float32, device="cuda")
        assert _noalloc(D, qd, sd, d, y, r) == D.OK, D.last_error()
        y_ws = D.scaffold_lora_linear(qd, sd, d["w_bits"], d["alpha"], d["A"], d["B"], d["beta"])
        torch.cuda.synchronize()
        assert np.array_equal(host(y).view(np.uint32), host(y_ws).view(np.uint32)), f"call {i}: y differs"
        assert_y(host(y), o.linear(q, s, **ws), what=f"no-alloc call {i}")


def test_noalloc_refuses_oversize(env):
    torch, D, o = env
    M, K, N, r = 8192, 4096, 64, 64
    assert D.linear_workspace_bytes(M, K, N, r) > D.lib.dfssm_noalloc_scratch_bytes()
    q = torch.zeros((M, K), dtype=torch.int8, device="cuda")
    s = torch.zeros((M,), dtype=torch.float32, device="cuda")
    d = dev_weights(S.weights(K, N, r, key=(182,)))
    y = torch.zeros((M, N), dtype=torch.float32, device="cuda")
    assert _noalloc(D, q, s, d, y, r) == D.ERR_WORKSPACE
    assert "scratch" in D.last_error()
