"""GPU parity of the linear with int4 LoRA factors (dfssm_scaffold_lora_linear_i4)
against the oracle (the int8 linear on the unpacked factors) on the same
seeded bytes: acc_s, acc_a, acc_b bit-exact, y bit-exact against the
oracle's fp32 order and within 1e-3 of max|y| against fp64.  Every nibble
value -8..7 occurs (the factors are uniform random bytes).

Paths: the few-token kernel reading the packed bytes directly (M <= 512,
in 64-token blocks above 32, with and without its LoRA workgroups), and the
prefill MFMA and popcount
paths on factors expanded in the workspace.  Shapes: the 1.3B projections,
ragged K and N, r not a multiple of 16 (unaligned packed B rows), r = 2, 0."""
import numpy as np
import pytest

import dfssm_synth as S
import oracle
from gpu_util import assert_y, dev, forced_switch, host, say, torch_cuda

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def env():
    torch = torch_cuda()
    import paper_2606_10932_amd as D
    oracle.build()
    return torch, D, oracle.get()


def _run(env, M, K, N, r, path, key=(160,)):
    torch, D, o = env
    ws = S.weights_i4(K, N, r, key=key + (M, K, N, r))
    x = S.activations(M, K, key=key + (M, K))
    q, s = o.quantize_act(x)
    ref = o.linear_i4(q, s, **ws)
    d = {k: dev(v) for k, v in ws.items()}
    y, acc_s, acc_a, acc_b = D.scaffold_lora_linear_i4(
        dev(q), dev(s), d["w_bits"], d["alpha"], d["A4"] if r else None, d["B4"] if r else None,
        d["beta"] if r else None, path=path, acc=True)
    torch.cuda.synchronize()
    return ref, host(y), host(acc_s), host(acc_a), host(acc_b)


def _check(ref, y, acc_s, acc_a, acc_b, r, what):
    assert np.array_equal(acc_s, ref["acc_s"]), what + " acc_s"
    if r:
        assert np.array_equal(acc_a, ref["acc_a"]), what + " acc_a"
    assert np.array_equal(acc_b, ref["acc_b"]), what + " acc_b"
    assert_y(y, ref, what=what)


SHAPES = [
    # (M, K, N, r)
    (1, 2048, 8512, 64),     # Mamba-2-1.3B in_proj
    (1, 4096, 2048, 64),     # Mamba-2-1.3B out_proj
    (2, 4096, 2048, 64),     # the most tokens the copies' token-major polls take (int4)
    (4, 4096, 2048, 64),
    (7, 2048, 8512, 64),     # the copies polled by four waves together (2 tokens each)
    (16, 2048, 8512, 64),    # more tokens than the waves' group polls take: one copy
    (17, 4096, 2048, 64),    # two token tiles
    (32, 2048, 300, 64),
    (3, 160, 77, 6),         # r % 16 != 0: packed B rows of 3 bytes
    (2, 256, 31, 18),
    (5, 96, 33, 2),
    (2, 256, 40, 256),       # four 64-rank chunks
    (1, 768, 3352, 16),      # Mamba-2-130M in_proj
    (3, 64, 9, 0),
    (70, 2048, 300, 64),     # two 64-token blocks, the second ragged
    (200, 4096, 2048, 64),   # four blocks, out_proj shape
]


@pytest.mark.parametrize("M,K,N,r", SHAPES)
def test_int4_few_tokens(env, M, K, N, r):
    torch, D, o = env
    say(f"int4 linear few M={M} K={K} N={N} r={r}")
    _check(*_run(env, M, K, N, r, D.PATH_MFMA_FEW), r, f"int4 few {M}x{K}x{N} r{r}")


@pytest.mark.parametrize("M,K,N,r", [(3, 160, 77, 6), (17, 4096, 2048, 64), (2, 256, 40, 256)])
def test_int4_few_tokens_local_lora(env, M, K, N, r):
    # no LoRA workgroups: every output lane computes the down-projection
    # itself from the packed A rows
    torch, D, o = env
    say(f"int4 linear few, local LoRA M={M} K={K} N={N} r={r}")
    with forced_switch(D, D.TEST_LOCAL_LORA, 1):
        res = _run(env, M, K, N, r, D.PATH_MFMA_FEW)
    _check(*res, r, f"int4 few local {M}x{K}x{N} r{r}")


@pytest.mark.parametrize("M,K,N,r", [(33, 2048, 8512, 64), (130, 4096, 2048, 64), (40, 160, 77, 6),
                                     (64, 256, 40, 256)])
def test_int4_prefill(env, M, K, N, r):
    torch, D, o = env
    say(f"int4 linear prefill M={M} K={K} N={N} r={r}")
    _check(*_run(env, M, K, N, r, D.PATH_MFMA), r, f"int4 prefill {M}x{K}x{N} r{r}")


@pytest.mark.parametrize("M,K,N,r", [(1, 2048, 8512, 64), (3, 160, 77, 6), (2, 256, 31, 18)])
def test_int4_popcount(env, M, K, N, r):
    torch, D, o = env
    say(f"int4 linear popcount M={M} K={K} N={N} r={r}")
    _check(*_run(env, M, K, N, r, D.PATH_DECODE), r, f"int4 popcount {M}x{K}x{N} r{r}")


def test_int4_auto_matches_int8_on_unpacked(env):
    # the int4 entry point and the int8 one on the same factors, unpacked by
    # the oracle, give the same bits
    torch, D, o = env
    say("int4 auto vs int8 on unpacked factors")
    M, K, N, r = 2, 2048, 8512, 64
    ws = S.weights_i4(K, N, r, key=(161,))
    q, s = o.quantize_act(S.activations(M, K, key=(161,)))
    A = o.unpack_int4(ws["A4"], r * K).reshape(r, K)
    B = o.unpack_int4(ws["B4"], N * r).reshape(N, r)
    d = {k: dev(v) for k, v in ws.items()}
    y4 = D.scaffold_lora_linear_i4(dev(q), dev(s), d["w_bits"], d["alpha"], d["A4"], d["B4"], d["beta"])
    y8 = D.scaffold_lora_linear(dev(q), dev(s), d["w_bits"], d["alpha"], dev(A), dev(B), d["beta"])
    torch.cuda.synchronize()
    assert np.array_equal(host(y4).view(np.uint32), host(y8).view(np.uint32))
